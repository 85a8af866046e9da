// Conflict levels on gfx950: which examples may run together without
// changing the sequential result.
//
// The read and write constraints (Sec. 4.4; Theorem 2) only order accesses to
// the same parameter partition.  With one feature per partition, example i
// must come after the latest earlier example touching each of its features
// (its "previous writers", the per-chunk iteration number the Read Protocol
// of Sec. 5 waits for).  level(i) = 1 + max level of its previous writers,
// 1 when it has none.
//
// Steps (all HIP kernels, launched on the caller's stream):
//   K0  row index of every stored entry;
//   K1  stable radix sort of the entries by feature -> per-feature occurrence
//       lists in example order;
//   K2  previous writer of every entry = its predecessor in its feature's list;
//   K3  levels, by one of
//         chain-scan relaxation: along every feature's list the level grows
//         by at least one per step, so a segmented max-scan of
//         (level - position) per feature followed by a max per example
//         raises every lower bound along whole chains in one round; start
//         from 1 and repeat until nothing changes (the least fixed point is
//         the exact level).  Rounds = 1 + chain switches on the critical
//         path: few when one feature dominates every example;
//         dataflow: every example waits for its previous writers' levels
//         (published with device-scope atomics) and publishes its own; waves
//         take batches of consecutive examples by ticket, so the smallest
//         unfinished example always runs.  Time ~ critical path length;
//   K4  stable radix sort of examples by level -> perm, level_ptr.
#include <climits>
#include <cstdlib>
#include <cstring>

#include "pdb_internal.h"

namespace pdbk {

namespace {

constexpr int kNone = INT_MIN;

struct Seg {
    int f;  // segment head seen
    int v;  // max since the last head
};

__device__ __forceinline__ Seg seg_comb(Seg a, Seg b) {
    return Seg{a.f | b.f, b.f ? b.v : max(a.v, b.v)};
}

__device__ __forceinline__ Seg seg_shfl_up(Seg x, int off) {
    return Seg{__shfl_up(x.f, off), __shfl_up(x.v, off)};
}

// Exclusive block scan of Seg in thread order; *agg = combination of all.
__device__ Seg block_excl_scan_seg(Seg x, Seg *s_wave, Seg *agg) {
    const int lane = lane_id(), wave = wave_in_block();
    const Seg ident{0, kNone};
    Seg incl = x;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const Seg y = seg_shfl_up(incl, off);
        if (lane >= off) incl = seg_comb(y, incl);
    }
    Seg excl = seg_shfl_up(incl, 1);
    if (lane == 0) excl = ident;
    if (lane == kWave - 1) s_wave[wave] = incl;
    __syncthreads();
    Seg before = ident, all = ident;
#pragma unroll
    for (int w = 0; w < kBlock / kWave; ++w) {
        const Seg s = s_wave[w];
        if (w < wave) before = seg_comb(before, s);
        all = seg_comb(all, s);
    }
    __syncthreads();
    *agg = all;
    return seg_comb(before, excl);
}

__global__ void k_fill_i32(int32_t *p, int64_t count, int32_t v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

__global__ void k_fill_i64(int64_t *p, int64_t count, int64_t v) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

__global__ void k_ctrl_init(Ctrl *c) {
    int *w = reinterpret_cast<int *>(c);
    for (int i = threadIdx.x; i < (int)(sizeof(Ctrl) / sizeof(int)); i += blockDim.x) w[i] = 0;
}

// K0: row of every stored entry.  One wave per row keeps stores contiguous.
__global__ __launch_bounds__(kBlock) void k_row_index(const int64_t *__restrict__ row_ptr,
                                                      int64_t n, int32_t *__restrict__ row_idx) {
    const int lane = lane_id();
    const int64_t nw = (int64_t)gridDim.x * (kBlock / kWave);
    for (int64_t i = blockIdx.x * (int64_t)(kBlock / kWave) + wave_in_block(); i < n; i += nw) {
        const int64_t b = row_ptr[i], e = row_ptr[i + 1];
        for (int64_t p = b + lane; p < e; p += kWave) row_idx[p] = (int32_t)i;
    }
}

// K2: previous writer of every entry from the feature-sorted order.
__global__ __launch_bounds__(kBlock) void k_prev_writer(
    const uint32_t *__restrict__ skeys, const uint32_t *__restrict__ svals, int64_t nnz,
    int64_t d, const int32_t *__restrict__ row_idx, int32_t *__restrict__ prev_row,
    int32_t *__restrict__ prev_nz, int64_t *__restrict__ col_ptr, int32_t *__restrict__ csc_row) {
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < nnz;
         q += (int64_t)gridDim.x * blockDim.x) {
        const uint32_t f = skeys[q];
        const uint32_t p = svals[q];
        const bool head = (q == 0) || skeys[q - 1] != f;
        if (head) {
            prev_row[p] = -1;
            if (prev_nz) prev_nz[p] = -1;
            const int64_t lo = (q == 0) ? 0 : (int64_t)skeys[q - 1] + 1;
            const int64_t hi = min((int64_t)f, d - 1);  // columns >= d: malformed input
            for (int64_t g = lo; g <= hi; ++g) col_ptr[g] = q;
        } else {
            const uint32_t pp = svals[q - 1];
            prev_row[p] = row_idx[pp];
            if (prev_nz) prev_nz[p] = (int32_t)pp;
        }
        if (q == nnz - 1)
            for (int64_t g = (int64_t)f + 1; g <= d; ++g) col_ptr[g] = nnz;
        if (csc_row) csc_row[q] = row_idx[p];
    }
}

__global__ __launch_bounds__(kBlock) void k_csc_row(const uint32_t *__restrict__ svals,
                                                    int64_t nnz, const int32_t *__restrict__ row_idx,
                                                    int32_t *__restrict__ csc_row) {
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < nnz;
         q += (int64_t)gridDim.x * blockDim.x)
        csc_row[q] = row_idx[svals[q]];
}

__global__ __launch_bounds__(kBlock) void k_max_diff(const int64_t *__restrict__ ptr,
                                                     int64_t count, Ctrl *ctrl) {
    long long m = 0;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * blockDim.x)
        m = max(m, (long long)(ptr[i + 1] - ptr[i]));
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = max(m, (long long)__shfl_xor(m, off));
    if (lane_id() == 0 && m > 0) atomicMax(&ctrl->max_width, m);
}

// ---- K3 chain-scan -------------------------------------------------------
// element q of the feature-sorted order: head = first entry of its feature,
// a_q = level(row of q) - q.  cand_q = q + max over earlier entries of the
// same feature of a = the bound that entry's chain imposes on q's example.

__device__ __forceinline__ Seg cs_elem(const uint32_t *skeys, const int32_t *csc_row,
                                       const int32_t *level, int64_t q) {
    const bool head = (q == 0) || skeys[q] != skeys[q - 1];
    return Seg{head ? 1 : 0, level[csc_row[q]] - (int)q};
}

__global__ __launch_bounds__(kBlock) void k_cs_reduce(const uint32_t *__restrict__ skeys,
                                                      const int32_t *__restrict__ csc_row,
                                                      const int32_t *__restrict__ level,
                                                      int64_t nnz, Seg *__restrict__ agg) {
    __shared__ Seg s_wave[kBlock / kWave];
    const int64_t base = (int64_t)blockIdx.x * kTile + (int64_t)threadIdx.x * kItems;
    Seg acc{0, kNone};
    for (int j = 0; j < kItems; ++j) {
        const int64_t q = base + j;
        if (q < nnz) acc = seg_comb(acc, cs_elem(skeys, csc_row, level, q));
    }
    Seg all;
    block_excl_scan_seg(acc, s_wave, &all);
    if (threadIdx.x == 0) agg[blockIdx.x] = all;
}

__global__ __launch_bounds__(kBlock) void k_cs_carry(const Seg *__restrict__ agg,
                                                     Seg *__restrict__ carry, int64_t ntiles) {
    __shared__ Seg s_wave[kBlock / kWave];
    Seg run{0, kNone};
    for (int64_t base = 0; base < ntiles; base += kBlock) {
        const int64_t i = base + threadIdx.x;
        const Seg x = i < ntiles ? agg[i] : Seg{0, kNone};
        Seg all;
        const Seg ex = block_excl_scan_seg(x, s_wave, &all);
        if (i < ntiles) carry[i] = seg_comb(run, ex);
        run = seg_comb(run, all);
    }
}

__global__ __launch_bounds__(kBlock) void k_cs_down(const uint32_t *__restrict__ skeys,
                                                    const int32_t *__restrict__ csc_row,
                                                    const uint32_t *__restrict__ svals,
                                                    const int32_t *__restrict__ level,
                                                    int64_t nnz, const Seg *__restrict__ carry,
                                                    int32_t *__restrict__ cand) {
    __shared__ Seg s_wave[kBlock / kWave];
    const int64_t base = (int64_t)blockIdx.x * kTile + (int64_t)threadIdx.x * kItems;
    Seg e[kItems];
    Seg acc{0, kNone};
    for (int j = 0; j < kItems; ++j) {
        const int64_t q = base + j;
        e[j] = q < nnz ? cs_elem(skeys, csc_row, level, q) : Seg{0, kNone};
        acc = seg_comb(acc, e[j]);
    }
    Seg all;
    Seg run = seg_comb(carry[blockIdx.x], block_excl_scan_seg(acc, s_wave, &all));
    for (int j = 0; j < kItems; ++j) {
        const int64_t q = base + j;
        if (q < nnz) {
            const int c = (e[j].f || run.v == kNone) ? kNone : run.v + (int)q;
            cand[svals[q]] = c;
        }
        run = seg_comb(run, e[j]);
    }
}

__global__ __launch_bounds__(kBlock) void k_cs_rows(const int64_t *__restrict__ row_ptr,
                                                    int64_t n, const int32_t *__restrict__ cand,
                                                    int32_t *__restrict__ level, Ctrl *ctrl) {
    int changed = 0;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        int c = kNone;
        for (int64_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) c = max(c, cand[p]);
        if (c > level[i]) {
            level[i] = c;
            changed = 1;
        }
    }
    if (__ballot(changed) != 0ull && lane_id() == 0)
        __hip_atomic_store(&ctrl->changed, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---- K3 dataflow ---------------------------------------------------------
constexpr int kFlowBatch = 32;

__global__ __launch_bounds__(kBlock) void k_levels_dataflow(const int64_t *__restrict__ row_ptr,
                                                            const int32_t *__restrict__ prev_row,
                                                            int64_t n, int32_t *level, Ctrl *ctrl,
                                                            int64_t timeout) {
    __shared__ int32_t s_lv[kBlock / kWave][kFlowBatch];
    const int lane = lane_id(), wave = wave_in_block();
    volatile int32_t *my = s_lv[wave];
    for (;;) {
        long long tk = 0;
        if (lane == 0) tk = (long long)atomicAdd(&ctrl->ticket, (unsigned long long)kFlowBatch);
        tk = __shfl(tk, 0);
        if (tk >= n) return;
        const int base = (int)tk;
        const int64_t end = min((int64_t)base + kFlowBatch, n);
        for (int64_t i = base; i < end; ++i) {
            int mx = 0;
            int bad = 0;
            for (int64_t p = row_ptr[i] + lane; p < row_ptr[i + 1]; p += kWave) {
                const int pr = prev_row[p];
                if (pr < 0) continue;
                int v;
                if (pr >= base) {
                    v = my[pr - base];
                } else {
                    v = __hip_atomic_load(&level[pr], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (v == 0) {
                        const int64_t t0 = now_ticks();
                        while (v == 0) {
                            if (aborted(ctrl)) { bad = 1; break; }
                            if (now_ticks() - t0 > timeout) {
                                record_error(ctrl, DERR_WAIT_TIMEOUT);
                                bad = 1;
                                break;
                            }
                            __builtin_amdgcn_s_sleep(1);
                            v = __hip_atomic_load(&level[pr], __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
                        }
                    }
                }
                mx = max(mx, v);
            }
            if (__ballot(bad) != 0ull) return;
            const int lv = wave_max_i32(mx) + 1;
            if (lane == 0) {
                my[i - base] = lv;
                __hip_atomic_store(&level[i], lv, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
        }
    }
}

__global__ __launch_bounds__(kBlock) void k_max_level(const int32_t *__restrict__ level,
                                                      int64_t n, Ctrl *ctrl) {
    int m = 0;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        m = max(m, level[i]);
    m = wave_max_i32(m);
    if (lane_id() == 0 && m > 0) atomicMax(&ctrl->max_level, m);
}

// ---- K4 ------------------------------------------------------------------
__global__ void k_level_keys(const int32_t *__restrict__ level, int64_t n,
                             uint32_t *__restrict__ keys) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        keys[i] = (uint32_t)(level[i] - 1);
}

__global__ void k_level_ptr(const uint32_t *__restrict__ skeys, const uint32_t *__restrict__ svals,
                            int64_t n, int64_t L, int64_t *__restrict__ level_ptr,
                            int32_t *__restrict__ perm, int32_t *__restrict__ n_levels) {
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < n;
         q += (int64_t)gridDim.x * blockDim.x) {
        const int64_t lv = skeys[q];
        perm[q] = (int32_t)svals[q];
        if (lv >= L) continue;  // cannot happen for levels in [1, L]
        if (q == 0 || skeys[q - 1] != skeys[q]) {
            const int64_t lo = (q == 0) ? 0 : (int64_t)skeys[q - 1] + 1;
            for (int64_t l = lo; l <= lv; ++l) level_ptr[l] = q;
        }
        if (q == n - 1) {
            for (int64_t l = lv + 1; l <= L; ++l) level_ptr[l] = n;
            *n_levels = (int32_t)L;
        }
    }
}

int bit_length(uint64_t x) {
    int b = 0;
    while (x) {
        ++b;
        x >>= 1;
    }
    return b;
}

int device_cus() {
    static int cus = 0;
    if (cus == 0) {
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus <= 0)
            cus = 256;
    }
    return cus;
}

int read_ctrl(Ctrl *dev, Ctrl *host, hipStream_t s) {
    PDB_HIP(hipMemcpyAsync(host, dev, sizeof(Ctrl), hipMemcpyDeviceToHost, s));
    PDB_HIP(hipStreamSynchronize(s));
    return PDB_OK;
}

int check_sizes(int64_t n, int64_t d, int64_t nnz) {
    if (n < 0 || d < 0 || nnz < 0) return PDB_ERR_INVALID_ARG;
    if (n >= INT32_MAX || d >= INT32_MAX || nnz >= INT32_MAX) return PDB_ERR_UNSUPPORTED;
    return PDB_OK;
}

// K0 + K1 + K2 into the workspace.  col_ptr, csc_row, prev_nz optional.
int build_conflicts(const pdb_csr *csr, int64_t n, int64_t d, SchedWs &w, int32_t *prev_nz,
                    int64_t *col_ptr, int32_t *csc_row, const uint32_t **skeys_out,
                    const uint32_t **svals_out, hipStream_t s) {
    const int64_t nnz = csr->nnz;
    if (n > 0) {
        k_row_index<<<grid_for(n, kBlock / kWave, 65536), kBlock, 0, s>>>(csr->row_ptr, n,
                                                                          w.row_idx);
        PDB_LAUNCHED();
    }
    uint32_t *sk = nullptr, *sv = nullptr;
    const int bits = bit_length(d > 1 ? (uint64_t)(d - 1) : 1);
    PDB_HIP(radix_sort_pairs(reinterpret_cast<const uint32_t *>(csr->col), nullptr, nnz, bits,
                             w.kA, w.vA, w.kB, w.vB, w.hist, w.scan_tmp, &sk, &sv, s));
    if (nnz > 0) {
        k_prev_writer<<<grid_for(nnz, kBlock, 1 << 16), kBlock, 0, s>>>(
            sk, sv, nnz, d, w.row_idx, w.prev_row, prev_nz, col_ptr, csc_row);
        PDB_LAUNCHED();
    } else {
        k_fill_i64<<<grid_for(d + 1, kBlock, 4096), kBlock, 0, s>>>(col_ptr, d + 1, 0);
        PDB_LAUNCHED();
    }
    *skeys_out = sk;
    *svals_out = sv;
    return PDB_OK;
}

}  // namespace

SchedWs sched_ws_layout(void *base, int64_t n, int64_t d, int64_t nnz) {
    SchedWs w{};
    const int64_t M = std::max<int64_t>(std::max<int64_t>(nnz, n), 1);
    const int64_t tilesM = cdiv(M, kTile);
    const int64_t tilesZ = cdiv(std::max<int64_t>(nnz, 1), kTile);
    char *p = static_cast<char *>(base);
    size_t off = 0;
    auto take = [&](int64_t bytes) {
        char *r = p ? p + off : nullptr;
        off += (size_t)align_up(bytes);
        return r;
    };
    w.ctrl = reinterpret_cast<Ctrl *>(take(sizeof(Ctrl)));
    w.row_idx = reinterpret_cast<int32_t *>(take(std::max<int64_t>(nnz, 1) * 4));
    w.kA = reinterpret_cast<uint32_t *>(take(M * 4));
    w.vA = reinterpret_cast<uint32_t *>(take(M * 4));
    w.kB = reinterpret_cast<uint32_t *>(take(M * 4));
    w.vB = reinterpret_cast<uint32_t *>(take(M * 4));
    w.hist = reinterpret_cast<uint32_t *>(take(256 * tilesM * 4));
    w.scan_tmp = reinterpret_cast<uint32_t *>(take((int64_t)scan_tmp_elems(256 * tilesM) * 4));
    w.prev_row = reinterpret_cast<int32_t *>(take(std::max<int64_t>(nnz, 1) * 4));
    w.cand = reinterpret_cast<int32_t *>(take(std::max<int64_t>(nnz, 1) * 4));
    w.seg_agg = reinterpret_cast<int2 *>(take(tilesZ * 8));
    w.seg_carry = reinterpret_cast<int2 *>(take(tilesZ * 8));
    w.col_ptr = reinterpret_cast<int64_t *>(take((d + 1) * 8));
    w.total = off;
    (void)n;
    return w;
}

}  // namespace pdbk

using namespace pdbk;

extern "C" int pdb_schedule_workspace_bytes(int64_t n, int64_t d, int64_t nnz, size_t *bytes) {
    if (!bytes) return PDB_ERR_INVALID_ARG;
    const int rc = check_sizes(n, d, nnz);
    if (rc != PDB_OK) return rc;
    *bytes = sched_ws_layout(nullptr, n, d, nnz).total;
    return PDB_OK;
}

static int sched_common_checks(const pdb_csr *csr, int64_t n, int64_t d, void *ws,
                               size_t ws_bytes, SchedWs *w) {
    if (!csr || !ws || (n > 0 && !csr->row_ptr) || (csr->nnz > 0 && !csr->col))
        return PDB_ERR_INVALID_ARG;
    const int rc = check_sizes(n, d, csr->nnz);
    if (rc != PDB_OK) return rc;
    if (d == 0 && csr->nnz > 0) return PDB_ERR_BAD_CSR;
    *w = sched_ws_layout(ws, n, d, csr->nnz);
    if (ws_bytes < w->total) return PDB_ERR_WORKSPACE;
    return PDB_OK;
}

extern "C" int pdb_transpose(const pdb_csr *csr, int64_t n, int64_t d, int64_t *col_ptr,
                             int32_t *csc_row, void *ws, size_t ws_bytes, hipStream_t stream) {
    SchedWs w;
    int rc = sched_common_checks(csr, n, d, ws, ws_bytes, &w);
    if (rc != PDB_OK) return rc;
    if (!col_ptr || (csr->nnz > 0 && !csc_row)) return PDB_ERR_INVALID_ARG;
    const uint32_t *sk, *sv;
    rc = build_conflicts(csr, n, d, w, nullptr, col_ptr, csc_row, &sk, &sv, stream);
    if (rc != PDB_OK) return rc;
    PDB_HIP(hipStreamSynchronize(stream));
    return PDB_OK;
}

extern "C" int pdb_prev_writer(const pdb_csr *csr, int64_t n, int64_t d, int32_t *prev_row,
                               int32_t *prev_nz, void *ws, size_t ws_bytes, hipStream_t stream) {
    SchedWs w;
    int rc = sched_common_checks(csr, n, d, ws, ws_bytes, &w);
    if (rc != PDB_OK) return rc;
    if (csr->nnz > 0 && !prev_row) return PDB_ERR_INVALID_ARG;
    const uint32_t *sk, *sv;
    rc = build_conflicts(csr, n, d, w, prev_nz, w.col_ptr, nullptr, &sk, &sv, stream);
    if (rc != PDB_OK) return rc;
    if (csr->nnz > 0)
        PDB_HIP(hipMemcpyAsync(prev_row, w.prev_row, csr->nnz * 4, hipMemcpyDeviceToDevice,
                               stream));
    PDB_HIP(hipStreamSynchronize(stream));
    return PDB_OK;
}

extern "C" int pdb_schedule(const pdb_csr *csr, const float *labels, int64_t n, int64_t d,
                            pdb_levels *lv, int method, pdb_schedule_info *info, void *ws,
                            size_t ws_bytes, hipStream_t s) {
    (void)labels;
    SchedWs w;
    int rc = sched_common_checks(csr, n, d, ws, ws_bytes, &w);
    if (rc != PDB_OK) return rc;
    if (!lv || !lv->level_ptr || !lv->n_levels || (n > 0 && (!lv->level || !lv->perm)))
        return PDB_ERR_INVALID_ARG;
    if (method < PDB_SCHED_AUTO || method > PDB_SCHED_DATAFLOW) return PDB_ERR_INVALID_ARG;
    const int64_t nnz = csr->nnz;
    Ctrl host{};
    k_ctrl_init<<<1, 64, 0, s>>>(w.ctrl);
    PDB_LAUNCHED();
    if (n == 0) {
        k_fill_i64<<<1, 64, 0, s>>>(lv->level_ptr, 1, 0);
        k_fill_i32<<<1, 64, 0, s>>>(lv->n_levels, 1, 0);
        PDB_LAUNCHED();
        PDB_HIP(hipStreamSynchronize(s));
        lv->L_host = 0;
        lv->max_width_host = 0;
        if (info) *info = pdb_schedule_info{method, 0, 0, 0};
        return PDB_OK;
    }

    // K0-K2
    const uint32_t *sk, *sv;
    rc = build_conflicts(csr, n, d, w, lv->prev_nz, w.col_ptr, nullptr, &sk, &sv, s);
    if (rc != PDB_OK) return rc;

    // which method: chain-scan converges in about (examples not holding the
    // most frequent feature) + 1 rounds; use it only when that is small.
    int use = method;
    int rounds = 0;
    if (method == PDB_SCHED_AUTO) {
        k_max_diff<<<grid_for(d, kBlock, 4096), kBlock, 0, s>>>(w.col_ptr, d, w.ctrl);
        PDB_LAUNCHED();
        rc = read_ctrl(w.ctrl, &host, s);
        if (rc != PDB_OK) return rc;
        use = (n - host.max_width <= 64) ? PDB_SCHED_CHAINSCAN : PDB_SCHED_DATAFLOW;
    }
    const int64_t timeout = spin_timeout_ticks();

    if (use == PDB_SCHED_CHAINSCAN) {
        // csc_row[q] = row of the q-th entry in feature order; the free radix
        // key buffer holds it (the sorted pair lives in the other pair)
        uint32_t *free_k = (sk == w.kA) ? w.kB : w.kA;
        int32_t *crow = reinterpret_cast<int32_t *>(free_k);
        if (nnz > 0)
            k_csc_row<<<grid_for(nnz, kBlock, 1 << 16), kBlock, 0, s>>>(sv, nnz, w.row_idx, crow);
        k_fill_i32<<<grid_for(n, kBlock, 65536), kBlock, 0, s>>>(lv->level, n, 1);
        PDB_LAUNCHED();
        const int64_t tiles = cdiv(std::max<int64_t>(nnz, 1), kTile);
        const int64_t max_rounds = (method == PDB_SCHED_AUTO) ? 256 : n + 1;
        bool converged = false;
        while (rounds < max_rounds) {
            k_fill_i32<<<1, 64, 0, s>>>(&w.ctrl->changed, 1, 0);
            if (nnz > 0) {
                k_cs_reduce<<<(unsigned)tiles, kBlock, 0, s>>>(sk, crow, lv->level, nnz,
                                                               reinterpret_cast<Seg *>(w.seg_agg));
                k_cs_carry<<<1, kBlock, 0, s>>>(reinterpret_cast<Seg *>(w.seg_agg),
                                                reinterpret_cast<Seg *>(w.seg_carry), tiles);
                k_cs_down<<<(unsigned)tiles, kBlock, 0, s>>>(
                    sk, crow, sv, lv->level, nnz, reinterpret_cast<Seg *>(w.seg_carry), w.cand);
                k_cs_rows<<<grid_for(n, kBlock, 65536), kBlock, 0, s>>>(csr->row_ptr, n, w.cand,
                                                                        lv->level, w.ctrl);
            }
            PDB_LAUNCHED();
            ++rounds;
            rc = read_ctrl(w.ctrl, &host, s);
            if (rc != PDB_OK) return rc;
            if (!host.changed) {
                converged = true;
                break;
            }
        }
        if (!converged) use = PDB_SCHED_DATAFLOW;
    }
    if (use == PDB_SCHED_DATAFLOW) {
        k_fill_i32<<<grid_for(n, kBlock, 65536), kBlock, 0, s>>>(lv->level, n, 0);
        k_fill_i32<<<1, 64, 0, s>>>(reinterpret_cast<int32_t *>(&w.ctrl->ticket), 2, 0);
        PDB_LAUNCHED();
        k_levels_dataflow<<<device_cus() * 4, kBlock, 0, s>>>(csr->row_ptr, w.prev_row, n,
                                                              lv->level, w.ctrl, timeout);
        PDB_LAUNCHED();
        rc = read_ctrl(w.ctrl, &host, s);
        if (rc != PDB_OK) return rc;
        if (host.err) return PDB_ERR_DEVICE;
    }

    // L, then K4
    k_max_level<<<grid_for(n, kBlock, 4096), kBlock, 0, s>>>(lv->level, n, w.ctrl);
    PDB_LAUNCHED();
    rc = read_ctrl(w.ctrl, &host, s);
    if (rc != PDB_OK) return rc;
    const int64_t L = host.max_level;
    if (L < 1 || L > n) return PDB_ERR_DEVICE;
    k_level_keys<<<grid_for(n, kBlock, 65536), kBlock, 0, s>>>(lv->level, n, w.kB);
    PDB_LAUNCHED();
    uint32_t *lk, *lvals;
    PDB_HIP(radix_sort_pairs(w.kB, nullptr, n, bit_length((uint64_t)(L - 1)), w.kA, w.vA, w.kB,
                             w.vB, w.hist, w.scan_tmp, &lk, &lvals, s));
    k_level_ptr<<<grid_for(n, kBlock, 65536), kBlock, 0, s>>>(lk, lvals, n, L, lv->level_ptr,
                                                              lv->perm, lv->n_levels);
    k_fill_i32<<<1, 64, 0, s>>>(reinterpret_cast<int32_t *>(&w.ctrl->max_width), 2, 0);
    PDB_LAUNCHED();
    k_max_diff<<<grid_for(L, kBlock, 4096), kBlock, 0, s>>>(lv->level_ptr, L, w.ctrl);
    PDB_LAUNCHED();
    rc = read_ctrl(w.ctrl, &host, s);
    if (rc != PDB_OK) return rc;
    lv->L_host = L;
    lv->max_width_host = host.max_width;
    if (info) *info = pdb_schedule_info{use, rounds, L, (int64_t)host.max_width};
    return PDB_OK;
}
