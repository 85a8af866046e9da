// Stable LSD radix sort of (key, value) pairs and an exclusive prefix sum,
// hand-written for gfx950 (wave64).  Used to build per-feature occurrence
// lists (sort stored entries by feature) and to group examples by level.
//
// The key bits go in as few passes as 8-bit digits need, spread evenly over
// them (21 bits: three 7-bit digits).  One pass over d-bit digits (d <= 8):
//   1. histogram: each 4096-element tile counts its digits in LDS
//      (per-wave private counters), writes counts digit-major;
//   2. exclusive prefix sum over the digit-major table gives, for every
//      (digit, tile), the first output slot;
//   3. scatter: each tile ranks its elements stably inside the tile.  A wave
//      finds the lanes holding the same digit with one ballot per digit bit
//      (no LDS atomics, so a Zipf-hot digit costs nothing extra), counts per
//      (item slot, wave, digit) go to LDS, one thread per digit turns them
//      into running offsets, the tile is staged in LDS in digit order and
//      written out from there, consecutive lanes to consecutive slots.
#include "pdb_internal.h"

namespace pdbk {

namespace {

constexpr int kWavesPerBlock = kBlock / kWave;

__device__ uint32_t block_excl_scan_u32(uint32_t v, uint32_t *s_wave, uint32_t *total) {
    const int lane = lane_id(), wave = wave_in_block();
    const uint32_t incl = wave_incl_scan_u32(v);
    if (lane == kWave - 1) s_wave[wave] = incl;
    __syncthreads();
    uint32_t before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < kWavesPerBlock; ++w) {
        const uint32_t s = s_wave[w];
        if (w < wave) before += s;
        all += s;
    }
    __syncthreads();
    *total = all;
    return before + incl - v;
}

__global__ __launch_bounds__(kBlock) void k_scan_reduce(const uint32_t *__restrict__ in,
                                                        int64_t count,
                                                        uint32_t *__restrict__ partials) {
    __shared__ uint32_t s_wave[kWavesPerBlock];
    const int64_t base = (int64_t)blockIdx.x * kTile;
    uint32_t s = 0;
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        const int64_t idx = base + (int64_t)j * kBlock + threadIdx.x;
        if (idx < count) s += in[idx];
    }
    uint32_t total;
    block_excl_scan_u32(s, s_wave, &total);
    if (threadIdx.x == 0) partials[blockIdx.x] = total;
}

__global__ __launch_bounds__(kBlock) void k_scan_top(uint32_t *partials, int64_t nblk) {
    __shared__ uint32_t s_wave[kWavesPerBlock];
    uint32_t carry = 0;
    for (int64_t base = 0; base < nblk; base += kBlock) {
        const int64_t idx = base + threadIdx.x;
        const uint32_t v = idx < nblk ? partials[idx] : 0u;
        uint32_t total;
        const uint32_t ex = block_excl_scan_u32(v, s_wave, &total);
        if (idx < nblk) partials[idx] = carry + ex;
        carry += total;
    }
}

__global__ __launch_bounds__(kBlock) void k_scan_down(const uint32_t *in, uint32_t *out,
                                                      int64_t count,
                                                      const uint32_t *__restrict__ partials) {
    __shared__ uint32_t s_wave[kWavesPerBlock];
    const int64_t base = (int64_t)blockIdx.x * kTile + (int64_t)threadIdx.x * kItems;
    uint32_t v[kItems];
    uint32_t s = 0;
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        const int64_t idx = base + j;
        v[j] = idx < count ? in[idx] : 0u;
        s += v[j];
    }
    uint32_t total;
    uint32_t run = partials[blockIdx.x] + block_excl_scan_u32(s, s_wave, &total);
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        const int64_t idx = base + j;
        if (idx < count) out[idx] = run;
        run += v[j];
    }
}

__global__ __launch_bounds__(kBlock) void k_radix_hist(const uint32_t *__restrict__ keys,
                                                       int64_t count, int shift, int nb,
                                                       uint32_t *__restrict__ hist,
                                                       int64_t ntiles) {
    __shared__ uint32_t s_h[kWavesPerBlock][256];
    const int t = threadIdx.x, wave = wave_in_block();
    uint32_t *flat = &s_h[0][0];
    for (int i = t; i < kWavesPerBlock * 256; i += kBlock) flat[i] = 0;
    __syncthreads();
    const uint32_t mask = (1u << nb) - 1u;
    const int64_t base = (int64_t)blockIdx.x * kTile;
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        const int64_t idx = base + (int64_t)j * kBlock + t;
        if (idx < count) atomicAdd(&s_h[wave][(keys[idx] >> shift) & mask], 1u);
    }
    __syncthreads();
    if (t < (1 << nb)) {
        uint32_t s = 0;
#pragma unroll
        for (int w = 0; w < kWavesPerBlock; ++w) s += s_h[w][t];
        hist[(int64_t)t * ntiles + blockIdx.x] = s;
    }
}

__global__ __launch_bounds__(kBlock) void k_radix_scatter(
    const uint32_t *__restrict__ keys, const uint32_t *__restrict__ vals, int64_t count,
    int shift, int nb, const uint32_t *__restrict__ offsets, int64_t ntiles,
    uint32_t *__restrict__ kout, uint32_t *__restrict__ vout) {
    // the per-(item slot, wave, digit) counts, then (same LDS) the tile in
    // digit order
    __shared__ union {
        uint16_t cnt[kItems][kWavesPerBlock][256];
        struct {
            uint32_t k[kTile];
            uint32_t v[kTile];
        } st;
    } U;
    static_assert(sizeof(U.cnt) == sizeof(U.st), "the staged tile reuses the counts' LDS");
    __shared__ uint32_t s_goff[256];    // first output slot of each digit of this tile
    __shared__ uint32_t s_dstart[256];  // first position of each digit in the staged tile
    __shared__ uint32_t s_wave[kWavesPerBlock];
    const int t = threadIdx.x, wave = wave_in_block();
    const int radix = 1 << nb;
    const uint32_t mask = (uint32_t)radix - 1u;
    uint16_t *flat = &U.cnt[0][0][0];
    for (int i = t; i < kItems * kWavesPerBlock * 256; i += kBlock) flat[i] = 0;
    if (t < radix) s_goff[t] = offsets[(int64_t)t * ntiles + blockIdx.x];
    __syncthreads();

    const int64_t base = (int64_t)blockIdx.x * kTile;
    uint32_t k[kItems], v[kItems], rk[kItems];
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        const int64_t idx = base + (int64_t)j * kBlock + t;
        const bool valid = idx < count;
        k[j] = valid ? keys[idx] : 0u;
        v[j] = valid ? (vals ? vals[idx] : (uint32_t)idx) : 0u;
        const uint32_t dg = (k[j] >> shift) & mask;
        unsigned long long peers = __ballot(valid);
        for (int b = 0; b < nb; ++b) {
            const bool bit = (dg >> b) & 1u;
            const unsigned long long bb = __ballot(bit);
            peers &= bit ? bb : ~bb;
        }
        const unsigned r = lanes_below(peers);
        rk[j] = r;
        if (valid && r == 0) U.cnt[j][wave][dg] = (uint16_t)__popcll(peers);
    }
    __syncthreads();
    // per digit: the counts become running offsets inside the digit's run
    // (item slot, then wave: tile order), and the run's length is scanned
    // over the digits into its start in the staged tile
    uint32_t len = 0;
    if (t < radix) {
        for (int j = 0; j < kItems; ++j) {
#pragma unroll
            for (int w = 0; w < kWavesPerBlock; ++w) {
                const uint32_t c = U.cnt[j][w][t];
                U.cnt[j][w][t] = (uint16_t)len;
                len += c;
            }
        }
    }
    uint32_t all;
    const uint32_t start = block_excl_scan_u32(len, s_wave, &all);
    if (t < radix) s_dstart[t] = start;
    __syncthreads();
    uint32_t pos[kItems];
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        const uint32_t dg = (k[j] >> shift) & mask;
        pos[j] = s_dstart[dg] + (uint32_t)U.cnt[j][wave][dg] + rk[j];
    }
    __syncthreads();  // every count read before the staged tile overwrites them
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        if (base + (int64_t)j * kBlock + t < count) {
            U.st.k[pos[j]] = k[j];
            U.st.v[pos[j]] = v[j];
        }
    }
    __syncthreads();
    // the staged tile in order: consecutive lanes write consecutive slots of
    // a digit's run, so a wave's stores form a few contiguous segments
    const int nvalid = (int)min((int64_t)kTile, count - base);
    for (int i = t; i < nvalid; i += kBlock) {
        const uint32_t kk = U.st.k[i];
        const uint32_t dg = (kk >> shift) & mask;
        const uint32_t dst = s_goff[dg] + ((uint32_t)i - s_dstart[dg]);
        kout[dst] = kk;
        vout[dst] = U.st.v[i];
    }
}

}  // namespace

size_t scan_tmp_elems(int64_t count) { return (size_t)cdiv(count, kTile) + 1; }

hipError_t exclusive_scan_u32(const uint32_t *in, uint32_t *out, int64_t count, uint32_t *tmp,
                              hipStream_t s) {
    if (count <= 0) return hipSuccess;
    const int64_t nblk = cdiv(count, kTile);
    k_scan_reduce<<<(unsigned)nblk, kBlock, 0, s>>>(in, count, tmp);
    k_scan_top<<<1, kBlock, 0, s>>>(tmp, nblk);
    k_scan_down<<<(unsigned)nblk, kBlock, 0, s>>>(in, out, count, tmp);
    return hipGetLastError();
}

hipError_t radix_sort_pairs(const uint32_t *keys_in, const uint32_t *vals_in, int64_t count,
                            int bits, uint32_t *kA, uint32_t *vA, uint32_t *kB, uint32_t *vB,
                            uint32_t *hist, uint32_t *scan_tmp, uint32_t **keys_out,
                            uint32_t **vals_out, hipStream_t s, int lo_bit) {
    if (bits < 1) bits = 1;
    *keys_out = kA;
    *vals_out = vA;
    if (count <= 0) return hipSuccess;
    if (lo_bit >= bits) {  // nothing to sort: the input is the result
        *keys_out = const_cast<uint32_t *>(keys_in);
        *vals_out = const_cast<uint32_t *>(vals_in);
        return hipSuccess;
    }
    const int64_t ntiles = cdiv(count, kTile);
    const uint32_t *ck = keys_in, *cv = vals_in;
    uint32_t *dk = kA, *dv = vA;
    // as few passes as 8-bit digits need, with the bits spread evenly over
    // them: fewer digits per pass make each tile's runs of one digit longer,
    // so its writes cover whole cache lines more often
    const int passes = (bits - lo_bit + 7) / 8;
    const int step = (bits - lo_bit + passes - 1) / passes;
    for (int shift = lo_bit; shift < bits; shift += step) {
        const int nb = bits - shift < step ? bits - shift : step;
        k_radix_hist<<<(unsigned)ntiles, kBlock, 0, s>>>(ck, count, shift, nb, hist, ntiles);
        hipError_t e = exclusive_scan_u32(hist, hist, (int64_t)(1 << nb) * ntiles, scan_tmp, s);
        if (e != hipSuccess) return e;
        k_radix_scatter<<<(unsigned)ntiles, kBlock, 0, s>>>(ck, cv, count, shift, nb, hist,
                                                            ntiles, dk, dv);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        ck = dk;
        cv = dv;
        dk = (dk == kA) ? kB : kA;
        dv = (dv == vA) ? vB : vA;
    }
    *keys_out = const_cast<uint32_t *>(ck);
    *vals_out = const_cast<uint32_t *>(cv);
    return hipSuccess;
}

}  // namespace pdbk
