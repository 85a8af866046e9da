// Internal header of the HIP library (gfx950, wave64).  Not installed.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "../../include/pdb.h"

namespace pdbk {

constexpr int kWave = 64;
constexpr int kBlock = 256;              // threads per block for streaming kernels
constexpr int kItems = 16;               // items per thread in tiled kernels
constexpr int kTile = kBlock * kItems;   // 4096 elements per tile
constexpr int64_t kAlign = 256;

// ----------------------------------------------------------------------------
// host-side error plumbing
void set_hip_error(hipError_t e);
#define PDB_HIP(call)                                   \
    do {                                                \
        hipError_t _e = (call);                         \
        if (_e != hipSuccess) {                         \
            ::pdbk::set_hip_error(_e);                  \
            return PDB_ERR_HIP;                         \
        }                                               \
    } while (0)
#define PDB_LAUNCHED()                                  \
    do {                                                \
        hipError_t _e = hipGetLastError();              \
        if (_e != hipSuccess) {                         \
            ::pdbk::set_hip_error(_e);                  \
            return PDB_ERR_HIP;                         \
        }                                               \
    } while (0)

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t align_up(int64_t x) { return cdiv(x, kAlign) * kAlign; }
inline int grid_for(int64_t work, int64_t per_block, int64_t cap = 1 << 20) {
    int64_t g = cdiv(work, per_block);
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (int)g;
}

// ----------------------------------------------------------------------------
// control block at the start of the epoch workspace and at the end of the
// schedule workspace: barrier counters, device error word, work tickets.
struct Ctrl {
    unsigned bar_count;
    unsigned bar_gen;
    int err;        // first device-side error code recorded (0 = none)
    int abort;      // set when any wave gives up; every spin loop watches it
    int changed;    // chain-scan: some level increased in this round
    int bad;        // validation failure flag
    int max_level;  // reductions read back by the host
    int pad0;
    unsigned long long ticket;  // work ticket for dataflow kernels
    long long max_width;
    // width-1 pipeline counters (clock cycles of the consumer wave): total,
    // waiting for staged examples, examples run, runs started
    long long stat_cycles, stat_wait, stat_rows, stat_runs;
    // spine levels: (count << 32) | (2^32 - 1 - feature) of the most frequent
    // feature; exceptional rows found; the solver's outcome
    unsigned long long top_feature;
    int spine_n_e;
    int spine_status;  // 0 solved, 1 too many exceptional rows or entries
    int spine_rounds;
    int chain_breaks;  // rows that do not conflict with the row before them
    // width-1 pipeline: the exactness check of its select-free step
    unsigned pipe_wmax;  // bits of max |w0|
    unsigned pipe_xmax;  // bits of max |x|
    int pipe_bad;        // some w0 is not finite or is -0, or some x is not finite
    int pipe_fast;       // the select-free step is exact for this epoch
    int pad[34];
    float sink[64];  // target of stores from lanes with nothing to store
};
static_assert(sizeof(Ctrl) == 512, "Ctrl is two 256-byte lines");

enum DeviceErr { DERR_NONE = 0, DERR_BARRIER_TIMEOUT = 1, DERR_WAIT_TIMEOUT = 2 };

// The caller's pdb_options, checked, with the watchdog converted to ticks of
// the constant clock the kernels read (s_memrealtime) on the current device.
struct Opts {
    int epoch_mode;          // pdb_epoch_mode
    bool pipeline;           // runs of narrow levels through the one-block pipeline
    int64_t pipeline_width;  // widest level a pipeline run may include
    int64_t thin_max;        // widest level run by one block alone
    int64_t hot_cap;         // cap on weights cached in LDS, -1 none
    int64_t timeout;         // watchdog of device-side waits, in clock ticks
    int64_t batch_thin_max;
    int64_t batch_sf_blocks;
    int stale_mode;          // pdb_stale_mode
    bool dense_stream;
    int mf_one_cu;           // -1 auto, 0 device-wide, 1 one compute unit
};
// PDB_ERR_INVALID_ARG for out-of-range fields; NULL gives the defaults.
int resolve_opts(const pdb_options *o, Opts *out);

// ----------------------------------------------------------------------------
// schedule workspace layout
struct SchedWs {
    int32_t *row_idx;   // [nnz]
    uint32_t *kA, *vA, *kB, *vB;  // [M] radix double buffers, M = max(nnz, n, 1)
    uint32_t *hist;     // [256 * tiles(M)]
    uint32_t *scan_tmp; // [scan partials]
    int32_t *pn;        // [nnz] previous-writer entries when the caller passes no prev_nz
    int32_t *cand;      // [nnz] chain-scan candidates, or previous-writer rows for dataflow
    void *spine;        // spine solver state (fixed size)
    int2 *seg_agg;      // [tiles(nnz)]
    int2 *seg_carry;    // [tiles(nnz)]
    int64_t *col_ptr;   // [d+1]
    Ctrl *ctrl;
    size_t total;
};
SchedWs sched_ws_layout(void *base, int64_t n, int64_t d, int64_t nnz);

// ----------------------------------------------------------------------------
// radix sort and scans (radix.hip)
size_t scan_tmp_elems(int64_t count);
hipError_t exclusive_scan_u32(const uint32_t *in, uint32_t *out, int64_t count, uint32_t *tmp,
                              hipStream_t s);
// Stable LSD sort of (key, value) pairs on bits [lo_bit, bits) of the key.
// vals_in == NULL means value = position.  Result in (*keys_out, *vals_out),
// which is one of the two buffer pairs (the inputs themselves when
// lo_bit >= bits; vals_in must then not be NULL).
hipError_t radix_sort_pairs(const uint32_t *keys_in, const uint32_t *vals_in, int64_t count,
                            int bits, uint32_t *kA, uint32_t *vA, uint32_t *kB, uint32_t *vB,
                            uint32_t *hist, uint32_t *scan_tmp, uint32_t **keys_out,
                            uint32_t **vals_out, hipStream_t s, int lo_bit = 0);

// ----------------------------------------------------------------------------
// device helpers

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & (kWave - 1)); }
__device__ __forceinline__ int wave_in_block() { return (int)(threadIdx.x >> 6); }

__device__ __forceinline__ unsigned lanes_below(unsigned long long mask) {
    return __builtin_amdgcn_mbcnt_hi((unsigned)(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo((unsigned)mask, 0u));
}

__device__ __forceinline__ int wave_max_i32(int v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v = max(v, __shfl_xor(v, off));
    return v;
}

__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
    return v;
}

// inclusive prefix sum across the wave
__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t v) {
    const int l = lane_id();
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        uint32_t t = __shfl_up(v, off);
        if (l >= off) v += t;
    }
    return v;
}

// max over the wave, every lane gets it: DPP within rows of 16, then the
// row and half swaps (max is idempotent, so any covering pattern works)
template <int CTRL>
__device__ __forceinline__ int dpp_max_i32(int v) {
    return max(v, __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, true));
}
__device__ __forceinline__ int wave_max_dpp(int v) {
    v = dpp_max_i32<0xB1>(v);   // quad_perm [1,0,3,2]
    v = dpp_max_i32<0x4E>(v);   // quad_perm [2,3,0,1]
    v = dpp_max_i32<0x141>(v);  // row_half_mirror
    v = dpp_max_i32<0x140>(v);  // row_mirror
    const auto r = __builtin_amdgcn_permlane16_swap((unsigned)v, (unsigned)v, false, false);
    v = max((int)r[0], (int)r[1]);
    const auto h = __builtin_amdgcn_permlane32_swap((unsigned)v, (unsigned)v, false, false);
    return max((int)h[0], (int)h[1]);
}

__device__ __forceinline__ int64_t now_ticks() { return (int64_t)wall_clock64(); }

__device__ __forceinline__ void record_error(Ctrl *c, int code) {
    atomicCAS(&c->err, 0, code);
    __hip_atomic_store(&c->abort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ bool aborted(Ctrl *c) {
    return __hip_atomic_load(&c->abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
}

// Grid-wide barrier for a co-resident (cooperatively launched) grid.
// Returns false if it gave up (watchdog or abort); the caller must then exit.
__device__ __forceinline__ bool grid_barrier(Ctrl *c, int64_t timeout) {
    __shared__ int ok_s;
    // every wave makes its own stores visible device-wide before arriving
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    __syncthreads();
    if (threadIdx.x == 0) {
        int ok = 1;
        const unsigned gen = __hip_atomic_load(&c->bar_gen, __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");  // publish this block's writes
        const unsigned arrived = __hip_atomic_fetch_add(&c->bar_count, 1u, __ATOMIC_ACQ_REL,
                                                        __HIP_MEMORY_SCOPE_AGENT);
        if (arrived == gridDim.x - 1) {
            __hip_atomic_store(&c->bar_count, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_fetch_add(&c->bar_gen, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        } else {
            const int64_t t0 = now_ticks();
            while (__hip_atomic_load(&c->bar_gen, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) ==
                   gen) {
                if (aborted(c)) { ok = 0; break; }
                if (now_ticks() - t0 > timeout) {
                    record_error(c, DERR_BARRIER_TIMEOUT);
                    ok = 0;
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        ok_s = ok;
    }
    __syncthreads();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    return ok_s != 0;
}

}  // namespace pdbk
