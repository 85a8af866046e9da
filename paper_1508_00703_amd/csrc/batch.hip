// Mini-batch gradient descent (gfx950, wave64): a batch of B consecutive
// examples is one iteration (Sec. 6.3 runs gradient descent with a fixed
// batch of examples per iteration).  Its parameter set is the union of its
// examples' features; within the iteration every read precedes every write
// (Definition 3), so all examples of a batch see the batch-start weights.
// Batches conflict when their unions share a feature; the read and write
// constraints of Sec. 4.4 at feature grain then order them, and Theorem 2
// lets batches of one conflict level run concurrently.
//
// Schedule: the union of each batch (features ascending) with, per union
// feature, the batch's entries on it in example order -- a stable sort of
// the entries by feature, then by batch -- is itself a CSR whose rows are the
// batches.  pdb_schedule on that CSR gives the batch levels.
//
// Epoch: one block per batch.  Phase 1: one wave per example, the dot
// product in the matched order (lane k holds entries k, k+64, ...), the step
// s_i = lr * g_i into LDS.  Phase 2: one thread per union feature applies the
// batch's contributions in example order, w = fma(-s_i, x, w), and writes the
// weight once.  Levels run one after another: a level wider than `thin` is
// spread over the grid followed by a device-wide barrier, runs of narrow
// levels go to block 0 with block barriers between batches.
#include <climits>

#include "pdb_math.h"
#include "pdb_words.h"

namespace pdbk {

namespace {

constexpr int kBB = 1024;                 // threads per batch block
constexpr int kBWaves = kBB / kWave;
constexpr int64_t kMaxBatch = 4096;       // examples per batch (LDS steps)
constexpr int kG = 8;                     // examples a wave loads together in phase 1
constexpr int kH = 8;                     // union features a thread takes in phase 2
constexpr int64_t kCap = kBB * kH;        // entries of a batch staged in LDS (8192)

// LDS of a batch block: steps by example; for staged batches the weights read
// in phase 1 by entry, and per occurrence its example (relative to the
// batch) and value
struct BatchShared {
    float s[kMaxBatch];
    float w[kCap];
    int32_t oi[kCap];
    float ox[kCap];
};

__device__ __forceinline__ int64_t readlane64(int64_t v, int lane) {
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, lane);
    const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)((uint64_t)v >> 32), lane);
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// row of every stored entry, one wave per row
__global__ __launch_bounds__(kBlock) void k_entry_row(const int64_t *__restrict__ row_ptr,
                                                      int64_t n, int32_t *__restrict__ row_idx) {
    const int lane = lane_id();
    const int64_t nw = (int64_t)gridDim.x * (kBlock / kWave);
    for (int64_t i = blockIdx.x * (int64_t)(kBlock / kWave) + wave_in_block(); i < n; i += nw) {
        const int64_t b = row_ptr[i], e = row_ptr[i + 1];
        for (int64_t p = b + lane; p < e; p += kWave) row_idx[p] = (int32_t)i;
    }
}

// keys of the second sort: the batch of each entry, in feature order
__global__ __launch_bounds__(kBlock) void k_batch_keys(const uint32_t *__restrict__ sv1,
                                                       int64_t nnz,
                                                       const int32_t *__restrict__ row_idx,
                                                       int64_t B, uint32_t *__restrict__ key2,
                                                       uint32_t *__restrict__ val2) {
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < nnz;
         q += (int64_t)gridDim.x * blockDim.x) {
        const uint32_t p = sv1[q];
        key2[q] = (uint32_t)((int64_t)row_idx[p] / B);
        val2[q] = p;
    }
}

// entries in (batch, feature, index) order: occurrence lists, and a 1 at the
// first entry of every (batch, feature) group
__global__ __launch_bounds__(kBlock) void k_union_flags(const uint32_t *__restrict__ sk2,
                                                        const uint32_t *__restrict__ sv2,
                                                        int64_t nnz, const int32_t *__restrict__ col,
                                                        const int32_t *__restrict__ row_idx,
                                                        uint32_t *__restrict__ flag,
                                                        int32_t *__restrict__ occ,
                                                        int32_t *__restrict__ occ_row) {
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < nnz;
         q += (int64_t)gridDim.x * blockDim.x) {
        const uint32_t p = sv2[q];
        occ[q] = (int32_t)p;
        occ_row[q] = row_idx[p];
        flag[q] = (q == 0 || sk2[q] != sk2[q - 1] || col[p] != col[sv2[q - 1]]) ? 1u : 0u;
    }
}

// union entries: feature, first occurrence, batch; the union size into
// *u_total (and uptr[U] = nnz)
__global__ __launch_bounds__(kBlock) void k_union_write(
    const uint32_t *__restrict__ sk2, const uint32_t *__restrict__ sv2, int64_t nnz,
    const int32_t *__restrict__ col, const uint32_t *__restrict__ uidx,
    int32_t *__restrict__ ucol, int64_t *__restrict__ uptr, uint32_t *__restrict__ ubatch,
    int32_t *__restrict__ occ_u, int64_t *__restrict__ u_total) {
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < nnz;
         q += (int64_t)gridDim.x * blockDim.x) {
        const uint32_t p = sv2[q];
        const bool head = q == 0 || sk2[q] != sk2[q - 1] || col[p] != col[sv2[q - 1]];
        const int64_t u = uidx[q];
        // uidx counts the heads before q: q's own union entry is uidx[q] at a
        // head, uidx[q] - 1 elsewhere
        occ_u[q] = (int32_t)(head ? u : u - 1);
        if (head) {
            ucol[u] = col[p];
            uptr[u] = q;
            ubatch[u] = sk2[q];
        }
        if (q == nnz - 1) {
            const int64_t U = u + (head ? 1 : 0);
            uptr[U] = nnz;
            *u_total = U;
        }
    }
}

// bptr[b] = first union entry of batch b (union entries are in batch order);
// bptr[nb] already holds U
__global__ __launch_bounds__(kBlock) void k_bptr(const uint32_t *__restrict__ ubatch, int64_t nb,
                                                 int64_t *__restrict__ bptr) {
    const int64_t U = bptr[nb];
    for (int64_t b = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; b < nb;
         b += (int64_t)gridDim.x * blockDim.x) {
        int64_t lo = 0, hi = U;
        while (lo < hi) {
            const int64_t mid = (lo + hi) >> 1;
            if ((int64_t)ubatch[mid] < b) lo = mid + 1; else hi = mid;
        }
        bptr[b] = lo;
    }
}

// next union entry on the same feature (the inverse of the previous-writer
// relation over union entries), -1 if none
__global__ __launch_bounds__(kBlock) void k_union_next(const int32_t *__restrict__ uprev,
                                                       int64_t U, int32_t *__restrict__ unext) {
    for (int64_t u = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; u < U;
         u += (int64_t)gridDim.x * blockDim.x)
        if (uprev[u] >= 0) unext[uprev[u]] = (int32_t)u;
}

__global__ void k_fill32(int32_t *p, int64_t count, int32_t v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

__global__ void k_fill64(int64_t *p, int64_t count, int64_t v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

// ---------------------------------------------------------------------------
// epoch

// oi[q] (an example relative to the batch) becomes that example's step,
// stored in place as the float's bits; count occurrences, the whole block
__device__ __forceinline__ void resolve_steps(int32_t *oi, const float *s, int64_t count) {
    for (int64_t q = threadIdx.x; q < count; q += kBB) oi[q] = __float_as_int(s[oi[q]]);
}

// w after the contributions of occurrences [q0, q1): w = fma(-step, x, w)
// in order; the loads of a group of 8 are issued before its fmas
template <bool VAL>
__device__ __forceinline__ float chain_apply(float w, const float *step, const float *x,
                                             int32_t q0, int32_t q1) {
    int32_t q = q0;
    for (; q + 8 <= q1; q += 8) {
        float sv[8], xv[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            sv[k] = step[q + k];
            xv[k] = VAL ? x[q + k] : 1.0f;
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) w = __builtin_fmaf(-sv[k], xv[k], w);
    }
    for (; q < q1; ++q) w = __builtin_fmaf(-step[q], VAL ? x[q] : 1.0f, w);
    return w;
}

template <int LOSS, bool VAL>
struct BatchOp {
    const int64_t *row_ptr;
    const int32_t *col;
    const float *val;
    const float *y;
    float *w;
    const int64_t *bptr;
    const int32_t *ucol;
    const int64_t *uptr;
    const int32_t *occ;
    const int32_t *occ_row;
    const int32_t *occ_u;
    const int32_t *unext;  // may be null
    int64_t n, B;
    float lr;

    // Batch b with the whole block.  Sh holds the batch's steps and, when the
    // batch has at most kCap entries, the weights phase 1 read (by entry) and
    // each occurrence's example and value, so that phase 2 reads LDS only.
    __device__ __forceinline__ void run(int64_t b, BatchShared &Sh) const {
        const int lane = lane_id();
        const int wave = (int)(threadIdx.x >> 6);
        const int64_t i0 = b * B, i1 = min(i0 + B, n);
        const int64_t pb = row_ptr[i0], pe = row_ptr[i1];   // the batch's entries
        const int64_t ub = bptr[b], ue = bptr[b + 1];       // its union features
        const bool staged = pe - pb <= kCap;
        // union features this thread updates, and (staged) the entry of each
        // one's first occurrence, whose weight phase 1 reads
        // (positions fit in 32 bits: nnz < 2^31)
        int32_t f[kH], q0[kH], q1[kH], pf[kH];
        const int64_t u0 = ub + threadIdx.x;
#pragma unroll
        for (int h = 0; h < kH; ++h) {
            const int64_t u = u0 + (int64_t)kBB * h;
            const bool live = u < ue;
            f[h] = live ? ucol[u] : 0;
            q0[h] = live ? (int32_t)uptr[u] : 0;
            q1[h] = live ? (int32_t)uptr[u + 1] : 0;
        }
        if (staged) {
#pragma unroll
            for (int h = 0; h < kH; ++h)
                pf[h] = (u0 + (int64_t)kBB * h < ue) ? occ[q0[h]] - (int32_t)pb : 0;
            // occurrences of the batch are its entries' positions [pb, pe)
            for (int64_t q = pb + threadIdx.x; q < pe; q += kBB) {
                Sh.oi[q - pb] = occ_row[q] - (int32_t)i0;
                if (VAL) Sh.ox[q - pb] = val[occ[q]];
            }
        }
        // phase 1: every example against the batch-start weights.  A wave
        // takes kG examples at a time; every load is unconditional (indices
        // clamped into the batch's entries), so all of them are in flight
        // before the first use: row bounds (lane j for example j), two chunks
        // of 64 columns per example, then the weights.
        if (pe > pb) {
            for (int64_t base = i0 + wave; base < i1; base += (int64_t)kBWaves * kG) {
                const int64_t my_i = base + (int64_t)kBWaves * lane;
                const bool has = lane < kG && my_i < i1;
                const int64_t rb = row_ptr[has ? my_i : i0];
                const int64_t re = has ? row_ptr[my_i + 1] : rb;
                const float yv = y[has ? my_i : i0];
                int64_t p[kG], m[kG];
#pragma unroll
                for (int j = 0; j < kG; ++j) {
                    p[j] = readlane64(rb, j);
                    m[j] = readlane64(re, j) - p[j];
                }
                int c[2 * kG];
                float x[2 * kG], wv[2 * kG], acc[kG];
#pragma unroll
                for (int t = 0; t < 2 * kG; ++t) {
                    const int64_t e = min(max(p[t >> 1] + (t & 1) * kWave + lane, pb), pe - 1);
                    c[t] = col[e];
                    x[t] = VAL ? val[e] : 1.0f;
                }
#pragma unroll
                for (int t = 0; t < 2 * kG; ++t) wv[t] = w[c[t]];
#pragma unroll
                for (int j = 0; j < kG; ++j) {
                    const int k0 = lane, k1 = kWave + lane;
                    // lanes without an entry hold +0, as in the summation order
                    acc[j] = k0 < m[j] ? __builtin_fmaf(wv[2 * j], x[2 * j], 0.0f) : 0.0f;
                    if (k1 < m[j]) acc[j] = __builtin_fmaf(wv[2 * j + 1], x[2 * j + 1], acc[j]);
                    if (staged) {
                        if (k0 < m[j]) Sh.w[p[j] + k0 - pb] = wv[2 * j];
                        if (k1 < m[j]) Sh.w[p[j] + k1 - pb] = wv[2 * j + 1];
                    }
                }
#pragma unroll
                for (int j = 0; j < kG; ++j) {
                    if (base + (int64_t)kBWaves * j >= i1) break;  // wave-uniform
                    for (int64_t k = 2 * kWave + lane; k < m[j]; k += kWave) {
                        const float wk = w[col[p[j] + k]];
                        acc[j] = __builtin_fmaf(wk, VAL ? val[p[j] + k] : 1.0f, acc[j]);
                        if (staged) Sh.w[p[j] + k - pb] = wk;
                    }
                    const float yj =
                        __int_as_float(__builtin_amdgcn_readlane(__float_as_int(yv), j));
                    const float sj = sgd_scale<LOSS>(wave_sum64(acc[j]), yj, lr);
                    if (lane == 0) Sh.s[base + (int64_t)kBWaves * j - i0] = sj;
                }
            }
        } else {
            // no entries: z = 0 for every example
            for (int64_t i = i0 + threadIdx.x; i < i1; i += kBB)
                Sh.s[i - i0] = sgd_scale<LOSS>(0.0f, y[i], lr);
        }
        __syncthreads();
        // phase 2: each union feature takes the batch's contributions in
        // example order; no other batch of the level touches it
        if (staged) {
            resolve_steps(Sh.oi, Sh.s, pe - pb);
            __syncthreads();
#pragma unroll
            for (int h = 0; h < kH; ++h) {
                if (u0 + (int64_t)kBB * h >= ue) break;
                w[f[h]] = chain_apply<VAL>(Sh.w[pf[h]], reinterpret_cast<const float *>(Sh.oi),
                                           Sh.ox, q0[h] - (int32_t)pb, q1[h] - (int32_t)pb);
            }
        } else {
            for (int64_t u = u0; u < ue; u += kBB) {
                const int32_t fu = ucol[u];
                const int64_t qe = uptr[u + 1];
                float v = w[fu];
                for (int64_t q = uptr[u]; q < qe; ++q)
                    v = __builtin_fmaf(-Sh.s[occ_row[q] - i0], VAL ? val[occ[q]] : 1.0f, v);
                w[fu] = v;
            }
        }
        __syncthreads();
    }
};

// first level >= l whose width exceeds thin (L if none); block-uniform
__device__ int64_t batch_run_end(int64_t l, int64_t L, const int64_t *level_ptr, int64_t thin) {
    __shared__ int64_t s_w[kBWaves];
    for (int64_t start = l; start < L; start += kBB) {
        const int64_t c = start + threadIdx.x;
        const bool wide = c < L && level_ptr[c + 1] - level_ptr[c] > thin;
        const unsigned long long bal = __ballot(wide);
        if (lane_id() == 0)
            s_w[threadIdx.x >> 6] = bal ? start + (threadIdx.x & ~63) + (__ffsll(bal) - 1)
                                        : INT64_MAX;
        __syncthreads();
        int64_t m = INT64_MAX;
#pragma unroll
        for (int v = 0; v < kBWaves; ++v) m = min(m, s_w[v]);
        __syncthreads();
        if (m != INT64_MAX) return m;
    }
    return L;
}

template <int LOSS, bool VAL>
__global__ __launch_bounds__(kBB) void k_batch_levels(BatchOp<LOSS, VAL> op,
                                                     const int32_t *__restrict__ perm,
                                                     const int64_t *__restrict__ level_ptr,
                                                     const int32_t *__restrict__ n_levels,
                                                     int64_t thin, Ctrl *ctrl, int64_t timeout) {
    __shared__ BatchShared Sh;
    const int64_t L = *n_levels;
    if (gridDim.x == 1) {
        // one block: every batch in level order, one after another
        const int64_t nb = level_ptr[L];
        for (int64_t e = 0; e < nb; ++e) op.run(perm[e], Sh);
        return;
    }
    int64_t l = 0;
    while (l < L) {
        const int64_t beg = level_ptr[l], end = level_ptr[l + 1];
        if (end - beg <= thin) {
            const int64_t l2 = batch_run_end(l, L, level_ptr, thin);
            if (blockIdx.x == 0)
                for (int64_t e = beg; e < level_ptr[l2]; ++e) op.run(perm[e], Sh);
            l = l2;
        } else {
            for (int64_t e = beg + blockIdx.x; e < end; e += gridDim.x) op.run(perm[e], Sh);
            ++l;
        }
        if (l < L && !grid_barrier(ctrl, timeout)) return;
    }
}

// ---------------------------------------------------------------------------
// Sync-free mini-batch epoch (the Read Protocol of Sec. 5 at feature grain,
// with a batch as the iteration): no batch levels, no barriers.  Each
// feature's weight and the union entry that last wrote it share one 64-bit
// word.  Blocks take batches in index order; a batch waits until each of its
// union features' words carries that feature's previous union entry (the
// schedule's prev_nz over the union CSR, -1 for none), runs both phases on
// those values and publishes (new weight, its union entry).  The earliest
// unfinished batch never waits for a later one, so the grid always makes
// progress; batches that share no feature run concurrently on different CUs.

__global__ void k_bw_in(const float *__restrict__ w, unsigned long long *__restrict__ bw,
                        int64_t d) {
    for (int64_t f = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; f < d;
         f += (int64_t)gridDim.x * blockDim.x)
        bw[f] = word_pack(w[f], -1);
}

__global__ void k_bw_out(const unsigned long long *__restrict__ bw, float *__restrict__ w,
                         int64_t d) {
    for (int64_t f = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; f < d;
         f += (int64_t)gridDim.x * blockDim.x)
        w[f] = word_value(bw[f]);
}

// Polls the words f[h] of the slots not yet ready until each carries tag[h];
// every round reloads all of them at once, so a wave confirms several
// arrivals in one round trip.  False on timeout or abort.
template <int H>
__device__ __forceinline__ bool bw_wait_slots(unsigned long long *base, const int32_t *f,
                                              const int32_t *tag, bool *ready,
                                              unsigned long long *v, Ctrl *ctrl,
                                              int64_t timeout) {
    int64_t t0 = 0;
    for (int round = 0;; ++round) {
        bool all = true;
#pragma unroll
        for (int h = 0; h < H; ++h) all = all && ready[h];
        if (__ballot(!all) == 0ull) return true;
        if (round == 0) {
            t0 = now_ticks();
        } else {
            if (aborted(ctrl)) return false;
            if (now_ticks() - t0 > timeout) {
                record_error(ctrl, DERR_WAIT_TIMEOUT);
                return false;
            }
        }
        word_backoff(round);
        __asm__ __volatile__("" ::: "memory");  // the loads below are issued again
#pragma unroll
        for (int h = 0; h < H; ++h) {
            if (!ready[h]) {
                v[h] = word_get(base, f[h]);
                ready[h] = (int)(unsigned)(v[h] >> 32) == tag[h];
            }
        }
    }
}

// A value every thread of the block reads from the same LDS word after a
// barrier, made wave-uniform for the compiler: the ticket loop's exits and
// the block barriers inside it then compile to scalar branches, so every
// wave runs the same sequence of barriers by construction.
__device__ __forceinline__ int block_uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ int64_t block_uniform64(int64_t v) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)v >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// LDS of a sync-free batch block: steps; for staged batches the weights of
// the union features, each entry's union feature, and per occurrence its
// example and value
struct SfShared {
    float s[kMaxBatch];
    float uw[kCap];
    int32_t eu[kCap];
    int32_t oi[kCap];
    float ox[kCap];
    int64_t ticket;
    int ok;
};

// A batch of any size: wait for every union feature's previous writer, then
// both phases on the words themselves (staged in LDS when they fit).  False
// when a wait gave up; every thread of the block returns the same.
template <int LOSS, bool VAL>
__device__ bool general_batch(const BatchOp<LOSS, VAL> &op, const int32_t *uprev,
                              unsigned long long *bw, SfShared &Sh, int64_t i0, int64_t i1,
                              int64_t pb, int64_t pe, int64_t ub, int64_t ue, Ctrl *ctrl,
                              int64_t timeout) {
    const int lane = lane_id();
    const int wave = (int)(threadIdx.x >> 6);
    const bool staged = pe - pb <= kCap;  // (ue - ub <= pe - pb)
    bool ok = true;
    for (int64_t u0 = ub + wave * kWave; u0 < ue; u0 += kBB) {
        const int64_t u = u0 + lane;
        const bool live = u < ue;
        const int32_t f = live ? op.ucol[u] : 0;
        const int tag = live ? uprev[u] : -1;
        unsigned long long v = 0;
        if (!word_wait_wave(bw, live, f, tag, &v, ctrl, timeout)) {
            ok = false;
            break;
        }
        if (staged && live) {
            Sh.uw[u - ub] = word_value(v);
            const int64_t q1 = op.uptr[u + 1];
            for (int64_t q = op.uptr[u]; q < q1; ++q) {
                const int32_t p = op.occ[q];
                Sh.eu[p - pb] = (int32_t)(u - ub);
                Sh.oi[q - pb] = op.occ_row[q] - (int32_t)i0;
                if (VAL) Sh.ox[q - pb] = op.val[p];
            }
        }
    }
    if (!ok && lane == 0) Sh.ok = 0;
    __syncthreads();
    if (block_uniform(Sh.ok) == 0) return false;
    // phase 1: every example against the weights the batch read
    for (int64_t i = i0 + wave; i < i1; i += kBWaves) {
        const int64_t p0 = op.row_ptr[i], m = op.row_ptr[i + 1] - p0;
        float acc = 0.0f;
        for (int64_t k = lane; k < m; k += kWave) {
            const int64_t p = p0 + k;
            const float wk = staged ? Sh.uw[Sh.eu[p - pb]] : word_value(word_get(bw, op.col[p]));
            acc = __builtin_fmaf(wk, VAL ? op.val[p] : 1.0f, acc);
        }
        const float s = sgd_scale<LOSS>(wave_sum64(acc), op.y[i], op.lr);
        if (lane == 0) Sh.s[i - i0] = s;
    }
    __syncthreads();
    if (staged) {
        resolve_steps(Sh.oi, Sh.s, pe - pb);
        __syncthreads();
    }
    // phase 2: contributions in example order, then publish
    for (int64_t u = ub + threadIdx.x; u < ue; u += kBB) {
        const int32_t f = op.ucol[u];
        const int64_t qa = op.uptr[u], qe = op.uptr[u + 1];
        float v = staged ? Sh.uw[u - ub] : word_value(word_get(bw, f));
        if (staged) {
            v = chain_apply<VAL>(v, reinterpret_cast<const float *>(Sh.oi), Sh.ox,
                                 (int32_t)(qa - pb), (int32_t)(qe - pb));
        } else {
            for (int64_t q = qa; q < qe; ++q)
                v = __builtin_fmaf(-Sh.s[op.occ_row[q] - i0], VAL ? op.val[op.occ[q]] : 1.0f, v);
        }
        word_put(bw, f, word_pack(v, (int)u));
    }
    __syncthreads();
    return true;
}

// A batch of at most kBWaves * kG examples and kCap entries.  Everything
// that does not depend on other batches comes first -- each wave's example
// bounds, labels and values in registers, every occurrence's example, value
// and union feature in LDS, each thread's union features in registers --
// then the words are read once and only those not yet written by their
// previous writer are polled; after that both phases read LDS only.
template <int LOSS, bool VAL>
__device__ bool fast_batch(const BatchOp<LOSS, VAL> &op, const int32_t *uprev,
                           unsigned long long *bw, SfShared &Sh, int64_t b, int64_t nb,
                           int64_t i0, int64_t i1, int64_t pb, int64_t pe, int64_t ub,
                           int64_t ue, Ctrl *ctrl, int64_t timeout) {
    const int lane = lane_id();
    const int wave = (int)(threadIdx.x >> 6);
    // this wave's examples i0 + wave + kBWaves * j, j < kG
    const int64_t my_i = i0 + wave + (int64_t)kBWaves * lane;
    const bool has = lane < kG && my_i < i1;
    const int64_t rb = op.row_ptr[has ? my_i : i0];
    const int64_t re = has ? op.row_ptr[my_i + 1] : rb;
    const float yv = op.y[has ? my_i : i0];
    int32_t p[kG], m[kG];  // first entry relative to pb, entry count
#pragma unroll
    for (int j = 0; j < kG; ++j) {
        const int64_t r0 = readlane64(rb, j);
        p[j] = (int32_t)(r0 - pb);
        m[j] = (int32_t)(readlane64(re, j) - r0);
    }
    float x[2 * kG];
#pragma unroll
    for (int t = 0; t < 2 * kG; ++t) {
        x[t] = 1.0f;
        if (VAL && pe > pb)
            x[t] = op.val[min(max(pb + p[t >> 1] + (t & 1) * kWave + lane, pb), pe - 1)];
    }
    for (int64_t q = pb + threadIdx.x; q < pe; q += kBB) {
        const int32_t pq = op.occ[q];
        Sh.oi[q - pb] = op.occ_row[q] - (int32_t)i0;
        if (VAL) Sh.ox[q - pb] = op.val[pq];
        Sh.eu[pq - pb] = op.occ_u[q] - (int32_t)ub;
    }
    int32_t f[kH], tag[kH], q0[kH], q1[kH];
    bool urgent[kH];  // the next batch writes this feature too: publish it first
    // union entries of the batches up to the next one end at soon_end
    const int64_t soon_end = op.unext ? op.bptr[min(b + 2, nb)] : 0;
#pragma unroll
    for (int h = 0; h < kH; ++h) {
        const int64_t u = ub + threadIdx.x + (int64_t)kBB * h;
        const bool live = u < ue;
        f[h] = live ? op.ucol[u] : 0;
        tag[h] = live ? uprev[u] : -1;
        q0[h] = live ? (int32_t)(op.uptr[u] - pb) : 0;
        q1[h] = live ? (int32_t)(op.uptr[u + 1] - pb) : 0;
        const int32_t nx = (live && op.unext) ? op.unext[u] : -1;
        urgent[h] = nx >= 0 && nx < soon_end;
    }
    // reads: every word once, then a wait for those not yet written
    unsigned long long v[kH];
    bool ready[kH];
#pragma unroll
    for (int h = 0; h < kH; ++h) {
        const bool live = ub + threadIdx.x + (int64_t)kBB * h < ue;
        v[h] = live ? word_get(bw, f[h]) : 0ull;
        ready[h] = !live || (int)(unsigned)(v[h] >> 32) == tag[h];
    }
    const bool ok = bw_wait_slots<kH>(bw, f, tag, ready, v, ctrl, timeout);
#pragma unroll
    for (int h = 0; h < kH; ++h)
        if (ub + threadIdx.x + (int64_t)kBB * h < ue) Sh.uw[threadIdx.x + kBB * h] = word_value(v[h]);
    if (!ok && lane == 0) Sh.ok = 0;
    __syncthreads();
    if (block_uniform(Sh.ok) == 0) return false;
    // phase 1 from LDS
#pragma unroll
    for (int j = 0; j < kG; ++j) {
        if (i0 + wave + (int64_t)kBWaves * j >= i1) break;  // wave-uniform
        const int k0 = lane, k1 = kWave + lane;
        float acc = k0 < m[j] ? __builtin_fmaf(Sh.uw[Sh.eu[p[j] + k0]], x[2 * j], 0.0f) : 0.0f;
        if (k1 < m[j]) acc = __builtin_fmaf(Sh.uw[Sh.eu[p[j] + k1]], x[2 * j + 1], acc);
        for (int k = 2 * kWave + lane; k < m[j]; k += kWave)
            acc = __builtin_fmaf(Sh.uw[Sh.eu[p[j] + k]], VAL ? op.val[pb + p[j] + k] : 1.0f, acc);
        const float yj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(yv), j));
        const float sj = sgd_scale<LOSS>(wave_sum64(acc), yj, op.lr);
        if (lane == 0) Sh.s[wave + kBWaves * j] = sj;
    }
    __syncthreads();
    // every occurrence's step, in parallel: the chains below then read one
    // LDS word per fma, none of which depends on the chain
    resolve_steps(Sh.oi, Sh.s, pe - pb);
    __syncthreads();
    // phase 2 from LDS; the features the next batch waits for are published
    // before the others (one CU issues a batch's thousands of scattered
    // stores, and the waiting batch needs only a few of them)
    float val[kH];
#pragma unroll
    for (int h = 0; h < kH; ++h) {
        val[h] = 0.0f;
        if (ub + threadIdx.x + (int64_t)kBB * h < ue)
            val[h] = chain_apply<VAL>(Sh.uw[threadIdx.x + kBB * h],
                                      reinterpret_cast<const float *>(Sh.oi), Sh.ox, q0[h], q1[h]);
    }
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
        for (int h = 0; h < kH; ++h) {
            const int64_t u = ub + threadIdx.x + (int64_t)kBB * h;
            if (u < ue && urgent[h] == (pass == 0)) word_put(bw, f[h], word_pack(val[h], (int)u));
        }
    }
    __syncthreads();
    return true;
}

template <int LOSS, bool VAL>
__global__ __launch_bounds__(kBB) void k_batch_syncfree(BatchOp<LOSS, VAL> op,
                                                       const int32_t *__restrict__ uprev,
                                                       unsigned long long *bw, int64_t nb,
                                                       Ctrl *ctrl, int64_t timeout) {
    __shared__ SfShared Sh;
    for (;;) {
        if (threadIdx.x == 0) {
            Sh.ticket = (int64_t)atomicAdd(&ctrl->ticket, 1ull);
            Sh.ok = 1;
        }
        __syncthreads();
        const int64_t b = block_uniform64(Sh.ticket);
        if (b >= nb) return;
        const int64_t i0 = b * op.B, i1 = min(i0 + op.B, op.n);
        const int64_t pb = op.row_ptr[i0], pe = op.row_ptr[i1];
        const int64_t ub = op.bptr[b], ue = op.bptr[b + 1];
        if (pe - pb <= kCap && i1 - i0 <= (int64_t)kBWaves * kG) {
            if (!fast_batch(op, uprev, bw, Sh, b, nb, i0, i1, pb, pe, ub, ue, ctrl, timeout))
                return;
        } else {
            if (!general_batch(op, uprev, bw, Sh, i0, i1, pb, pe, ub, ue, ctrl, timeout)) return;
        }
    }
}

__global__ void k_batch_ctrl_zero(Ctrl *c) {
    int *w = reinterpret_cast<int *>(c);
    for (int i = threadIdx.x; i < (int)(sizeof(Ctrl) / sizeof(int)); i += blockDim.x) w[i] = 0;
}

template <int LOSS, bool VAL>
int launch_batch(const BatchOp<LOSS, VAL> &op, const pdb_levels *lv, Ctrl *ctrl, const Opts &opt,
                 hipStream_t s) {
    const int64_t thin = opt.batch_thin_max;
    const int64_t timeout = opt.timeout;
    k_batch_ctrl_zero<<<1, 64, 0, s>>>(ctrl);
    PDB_LAUNCHED();
    const void *fn = reinterpret_cast<const void *>(&k_batch_levels<LOSS, VAL>);
    int grid = 1;
    if (lv->max_width_host > thin) {
        // the level barrier needs every block of the grid resident at once:
        // one block per CU at most (a 1024-thread block always fits one CU)
        int dev = 0, cus = 0, per_cu = 0;
        PDB_HIP(hipGetDevice(&dev));
        PDB_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
        PDB_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kBB, 0));
        if (per_cu < 1) return PDB_ERR_HIP;
        grid = (int)std::max<int64_t>(1, std::min<int64_t>(cus, lv->max_width_host));
    }
    BatchOp<LOSS, VAL> o = op;
    const int32_t *perm = lv->perm;
    const int64_t *level_ptr = lv->level_ptr;
    const int32_t *n_levels = lv->n_levels;
    if (grid == 1) {
        k_batch_levels<LOSS, VAL><<<1, kBB, 0, s>>>(o, perm, level_ptr, n_levels, thin, ctrl,
                                                    timeout);
        PDB_LAUNCHED();
    } else {
        int64_t thin_arg = thin, to = timeout;
        void *args[] = {&o, &perm, &level_ptr, &n_levels, &thin_arg, &ctrl, &to};
        PDB_HIP(hipLaunchCooperativeKernel(fn, dim3(grid), dim3(kBB), args, 0, s));
    }
    return PDB_OK;
}

int64_t batch_sf_ws_bytes(int64_t d) { return (int64_t)sizeof(Ctrl) + align_up(8 * d); }

template <int LOSS, bool VAL>
int launch_batch_syncfree(const BatchOp<LOSS, VAL> &op, const pdb_levels *lv, int64_t d,
                          int64_t nb, void *ws, const Opts &opt, hipStream_t s) {
    Ctrl *ctrl = static_cast<Ctrl *>(ws);
    unsigned long long *bw =
        reinterpret_cast<unsigned long long *>(static_cast<char *>(ws) + sizeof(Ctrl));
    const int64_t timeout = opt.timeout;
    k_batch_ctrl_zero<<<1, 64, 0, s>>>(ctrl);
    PDB_LAUNCHED();
    if (d > 0) {
        k_bw_in<<<grid_for(d, kBlock, 8192), kBlock, 0, s>>>(op.w, bw, d);
        PDB_LAUNCHED();
    }
    // one block per CU (the LDS of a block fills most of a CU); blocks need
    // not be co-resident: the earliest unfinished batch is always running
    int dev = 0, cus = 0;
    PDB_HIP(hipGetDevice(&dev));
    PDB_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
    // at most 32 blocks by default: more batches in flight only add polls
    // that slow the frontier's memory accesses
    const int64_t cap = opt.batch_sf_blocks;
    const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(std::min<int64_t>(cus, cap), nb));
    k_batch_syncfree<LOSS, VAL><<<grid, kBB, 0, s>>>(op, lv->prev_nz, bw, nb, ctrl, timeout);
    PDB_LAUNCHED();
    if (d > 0) {
        k_bw_out<<<grid_for(d, kBlock, 8192), kBlock, 0, s>>>(bw, op.w, d);
        PDB_LAUNCHED();
    }
    return PDB_OK;
}

int check_batch_sizes(int64_t n, int64_t d, int64_t nnz, int64_t B) {
    if (n < 0 || d < 0 || nnz < 0 || B < 1) return PDB_ERR_INVALID_ARG;
    if (B > kMaxBatch) return PDB_ERR_INVALID_ARG;
    if (n >= INT32_MAX || d >= INT32_MAX || nnz >= INT32_MAX) return PDB_ERR_UNSUPPORTED;
    return PDB_OK;
}

int bits_for(uint64_t maxval) {
    int b = 0;
    while (maxval) {
        ++b;
        maxval >>= 1;
    }
    return b > 0 ? b : 1;
}

}  // namespace
}  // namespace pdbk

using namespace pdbk;

extern "C" int pdb_batch_schedule(const pdb_csr *csr, int64_t n, int64_t d, int64_t batch,
                                  pdb_batches *bt, pdb_levels *lv, int method,
                                  pdb_schedule_info *info, void *ws, size_t ws_bytes,
                                  const pdb_options *opt, hipStream_t s) {
    if (!csr || !bt || !lv || !ws || (n > 0 && !csr->row_ptr) || (csr->nnz > 0 && !csr->col))
        return PDB_ERR_INVALID_ARG;
    const int64_t nnz = csr->nnz;
    int rc = check_batch_sizes(n, d, nnz, batch);
    if (rc != PDB_OK) return rc;
    {
        Opts o;
        rc = resolve_opts(opt, &o);  // checked here, applied by pdb_schedule
        if (rc != PDB_OK) return rc;
    }
    if (d == 0 && nnz > 0) return PDB_ERR_BAD_CSR;
    if (!bt->bptr || !bt->uptr ||
        (nnz > 0 && (!bt->ucol || !bt->occ || !bt->occ_row || !bt->occ_u)))
        return PDB_ERR_INVALID_ARG;
    SchedWs w = sched_ws_layout(ws, n, d, nnz);
    if (ws_bytes < w.total) return PDB_ERR_WORKSPACE;
    const int64_t nb = cdiv(n, batch);
    if (nnz == 0) {
        k_fill64<<<grid_for(nb + 1, kBlock, 4096), kBlock, 0, s>>>(bt->bptr, nb + 1, 0);
        k_fill64<<<1, 64, 0, s>>>(bt->uptr, 1, 0);
        PDB_LAUNCHED();
        bt->U_host = 0;
    } else {
        k_entry_row<<<grid_for(n, kBlock / kWave, 65536), kBlock, 0, s>>>(csr->row_ptr, n,
                                                                          w.row_idx);
        PDB_LAUNCHED();
        // entries by feature (stable), then by batch (stable): (batch, feature, index)
        uint32_t *sk1, *sv1, *sk2, *sv2;
        PDB_HIP(radix_sort_pairs(reinterpret_cast<const uint32_t *>(csr->col), nullptr, nnz,
                                 bits_for((uint64_t)(d > 1 ? d - 1 : 1)), w.kA, w.vA, w.kB, w.vB,
                                 w.hist, w.scan_tmp, &sk1, &sv1, s));
        // the second sort reads its input from the occurrence arrays, which
        // are rewritten below
        uint32_t *key2 = reinterpret_cast<uint32_t *>(bt->occ);
        uint32_t *val2 = reinterpret_cast<uint32_t *>(bt->occ_row);
        k_batch_keys<<<grid_for(nnz, kBlock, 1 << 16), kBlock, 0, s>>>(sv1, nnz, w.row_idx, batch,
                                                                      key2, val2);
        PDB_LAUNCHED();
        PDB_HIP(radix_sort_pairs(key2, val2, nnz, bits_for((uint64_t)(nb > 1 ? nb - 1 : 1)), w.kA,
                                 w.vA, w.kB, w.vB, w.hist, w.scan_tmp, &sk2, &sv2, s));
        uint32_t *flag = (sk2 == w.kA) ? w.kB : w.kA;   // the pair not holding the result
        uint32_t *ubatch = (sk2 == w.kA) ? w.vB : w.vA;
        k_union_flags<<<grid_for(nnz, kBlock, 1 << 16), kBlock, 0, s>>>(
            sk2, sv2, nnz, csr->col, w.row_idx, flag, bt->occ, bt->occ_row);
        PDB_LAUNCHED();
        PDB_HIP(exclusive_scan_u32(flag, flag, nnz, w.scan_tmp, s));
        k_union_write<<<grid_for(nnz, kBlock, 1 << 16), kBlock, 0, s>>>(
            sk2, sv2, nnz, csr->col, flag, bt->ucol, bt->uptr, ubatch, bt->occ_u, bt->bptr + nb);
        PDB_LAUNCHED();
        if (nb > 0) {
            k_bptr<<<grid_for(nb, kBlock, 65536), kBlock, 0, s>>>(ubatch, nb, bt->bptr);
            PDB_LAUNCHED();
        }
        int64_t U = 0;
        PDB_HIP(hipMemcpyAsync(&U, bt->bptr + nb, sizeof(U), hipMemcpyDeviceToHost, s));
        PDB_HIP(hipStreamSynchronize(s));
        bt->U_host = U;
    }
    // the batch levels: conflict levels of the union CSR, whose rows are the batches
    const pdb_csr ucsr{bt->bptr, bt->ucol, nullptr, bt->U_host};
    rc = pdb_schedule(&ucsr, nullptr, nb, d, lv, method, info, ws, ws_bytes, opt, s);
    if (rc != PDB_OK) return rc;
    // each union entry's next writer, when asked for and known
    if (bt->unext && bt->U_host > 0) {
        k_fill32<<<grid_for(bt->U_host, kBlock, 65536), kBlock, 0, s>>>(bt->unext, bt->U_host, -1);
        PDB_LAUNCHED();
        if (lv->prev_nz) {
            k_union_next<<<grid_for(bt->U_host, kBlock, 65536), kBlock, 0, s>>>(
                lv->prev_nz, bt->U_host, bt->unext);
            PDB_LAUNCHED();
        }
        PDB_HIP(hipStreamSynchronize(s));
    }
    return PDB_OK;
}

extern "C" int pdb_batch_epoch(const pdb_csr *csr, const float *labels, int64_t n, int64_t d,
                               int64_t batch, float *w, float lr, int loss,
                               const pdb_batches *bt, const pdb_levels *lv, void *ws,
                               size_t ws_bytes, const pdb_options *opt, hipStream_t s) {
    if (!csr || !labels || !w || !bt || !lv || !ws || !lv->perm || !lv->level_ptr ||
        !lv->n_levels)
        return PDB_ERR_INVALID_ARG;
    const int64_t nnz = csr->nnz;
    int rc = check_batch_sizes(n, d, nnz, batch);
    if (rc != PDB_OK) return rc;
    if (loss != PDB_LOGISTIC && loss != PDB_SQUARED) return PDB_ERR_INVALID_ARG;
    if (ws_bytes < sizeof(Ctrl)) return PDB_ERR_WORKSPACE;
    if (n == 0) return PDB_OK;
    if (!bt->bptr || !bt->uptr ||
        (nnz > 0 && (!bt->ucol || !bt->occ || !bt->occ_row || !bt->occ_u)))
        return PDB_ERR_INVALID_ARG;
    Ctrl *ctrl = static_cast<Ctrl *>(ws);
    Opts o;
    rc = resolve_opts(opt, &o);
    if (rc != PDB_OK) return rc;
    // sync-free when the previous writers over the union CSR are known and the
    // workspace holds a word per feature, unless the epoch mode option asks
    // for batch levels
    const bool sf_ok = lv->prev_nz != nullptr && (int64_t)ws_bytes >= batch_sf_ws_bytes(d);
    const bool syncfree = sf_ok && o.epoch_mode != PDB_EPOCH_LEVELS;
    const int64_t nb = cdiv(n, batch);
#define PDB_BATCH(LOSS, VAL)                                                                     \
    (syncfree ? launch_batch_syncfree<LOSS, VAL>(                                              \
                    BatchOp<LOSS, VAL>{csr->row_ptr, csr->col, csr->val, labels, w, bt->bptr,   \
                                       bt->ucol, bt->uptr, bt->occ, bt->occ_row, bt->occ_u,         \
                                       bt->unext, n, batch, lr}, \
                    lv, d, nb, ws, o, s)                                                        \
              : launch_batch<LOSS, VAL>(                                                       \
                    BatchOp<LOSS, VAL>{csr->row_ptr, csr->col, csr->val, labels, w, bt->bptr,   \
                                       bt->ucol, bt->uptr, bt->occ, bt->occ_row, bt->occ_u,         \
                                       bt->unext, n, batch, lr}, \
                    lv, ctrl, o, s))
    if (loss == PDB_LOGISTIC) return csr->val ? PDB_BATCH(PDB_LOGISTIC, true) : PDB_BATCH(PDB_LOGISTIC, false);
    return csr->val ? PDB_BATCH(PDB_SQUARED, true) : PDB_BATCH(PDB_SQUARED, false);
#undef PDB_BATCH
}
