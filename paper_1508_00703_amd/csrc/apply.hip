// One SGD epoch level by level (gfx950, wave64).
//
// Sequential semantics (Algorithm 1, Definition 4): example i reads the
// parameters it touches, computes its gradient step (Sec. 2), writes them.
// Examples of one conflict level touch pairwise disjoint features, so by
// Theorem 2 running a level's examples concurrently, levels in increasing
// order, gives bitwise the sequential result: each example sees exactly the
// values the sequential run would show it, and its own arithmetic is fixed.
//
// One wavefront per example: lane k holds entries k, k+64, ... (coalesced
// loads of col/val, gather of w), fma into a per-lane partial sum, butterfly
// over the 64 lanes (every lane ends with the same z), sigmoid or residual,
// then each lane writes its own features -- no atomics, since no other
// example of the level touches them.  Matrix completion: one rating per
// 32-lane half, lane j holds component j of the user and item rows.
//
// Level driver (a persistent grid): a level wider than `thin_max` is spread
// over every wave of the grid, followed by a device-wide barrier.  A run of
// narrow levels is handled by block 0 alone, with block barriers between
// levels (none at all between levels of width 1, which its first wave runs
// back to back), while the other blocks wait at the next device barrier.
#include <cstdlib>

#include "pdb_internal.h"

namespace pdbk {

namespace {

constexpr int kWavesPerBlock = kBlock / kWave;

// e^x: k = rint(x log2 e), r = x - k ln 2 with ln 2 in two binary32 pieces,
// e^r from its Taylor series through r^7 (Horner), times 2^k built from the
// exponent field (two factors near the ends of the range).
__device__ __forceinline__ float dev_exp(float x) {
    if (!(x == x)) return x;
    if (x > 89.0f) return __builtin_huge_valf();
    if (x < -104.0f) return 0.0f;
    const float kf = __builtin_rintf(x * 0x1.715476p+0f);
    float r = __builtin_fmaf(-kf, 0x1.62e430p-1f, x);
    r = __builtin_fmaf(-kf, -0x1.05c610p-29f, r);
    float q = 0x1.a01a02p-13f;               // 1/5040
    q = __builtin_fmaf(q, r, 0x1.6c16c2p-10f);  // 1/720
    q = __builtin_fmaf(q, r, 0x1.111112p-7f);   // 1/120
    q = __builtin_fmaf(q, r, 0x1.555556p-5f);   // 1/24
    q = __builtin_fmaf(q, r, 0x1.555556p-3f);   // 1/6
    q = __builtin_fmaf(q, r, 0.5f);
    q = __builtin_fmaf(q, r, 1.0f);
    q = __builtin_fmaf(q, r, 1.0f);
    const int k = (int)kf;
    if (k > 127) return (q * __int_as_float(254 << 23)) * __int_as_float(k << 23);
    if (k < -126) return (q * __int_as_float((k + 253) << 23)) * __int_as_float(1 << 23);
    return q * __int_as_float((k + 127) << 23);
}

__device__ __forceinline__ float butterfly64(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v = v + __shfl_xor(v, off);
    return v;
}

__device__ __forceinline__ float butterfly32(float v) {
#pragma unroll
    for (int off = 16; off >= 1; off >>= 1) v = v + __shfl_xor(v, off);
    return v;
}

template <int LOSS>
__device__ __forceinline__ float sgd_scale(float z, float y, float lr) {
    float g;
    if (LOSS == PDB_LOGISTIC) {
        const float e = dev_exp(-z);
        const float sig = 1.0f / (1.0f + e);
        g = sig - (y > 0.0f ? 1.0f : 0.0f);
    } else {
        g = z - y;
    }
    return lr * g;
}

template <int LOSS, bool VAL>
struct SgdOp {
    const int64_t *row_ptr;
    const int32_t *col;
    const float *val;
    const float *y;
    float *w;
    const int32_t *perm;
    float lr;
    static constexpr int kUnits = 1;  // examples per wave per step

    __device__ __forceinline__ void operator()(int64_t e, int64_t end) const {
        (void)end;
        const int lane = lane_id();
        const int64_t i = perm[e];
        const int64_t b = row_ptr[i];
        const int m = (int)(row_ptr[i + 1] - b);
        const float yi = y[i];
        if (m <= kWave) {
            int c = 0;
            float x = 1.0f, wv = 0.0f, acc = 0.0f;
            if (lane < m) {
                c = col[b + lane];
                if (VAL) x = val[b + lane];
                wv = w[c];
                acc = __builtin_fmaf(wv, x, 0.0f);
            }
            const float s = sgd_scale<LOSS>(butterfly64(acc), yi, lr);
            if (lane < m) w[c] = __builtin_fmaf(-s, x, wv);
        } else {
            float acc = 0.0f;
            for (int k = lane; k < m; k += kWave) {
                const int c = col[b + k];
                acc = __builtin_fmaf(w[c], VAL ? val[b + k] : 1.0f, acc);
            }
            const float s = sgd_scale<LOSS>(butterfly64(acc), yi, lr);
            // no other example of this level touches these features and this
            // one has not written yet: w[c] still holds the value read above
            for (int k = lane; k < m; k += kWave) {
                const int c = col[b + k];
                w[c] = __builtin_fmaf(-s, VAL ? val[b + k] : 1.0f, w[c]);
            }
        }
    }
};

struct MfOp {
    const int32_t *user;
    const int32_t *item;
    const float *rating;
    float *U;
    float *V;
    const int32_t *perm;
    float lr, reg;
    static constexpr int kUnits = 2;  // two ratings per wave, one per 32-lane half

    __device__ __forceinline__ void operator()(int64_t e, int64_t end) const {
        const int lane = lane_id();
        const int h = lane >> 5, j = lane & 31;
        const int64_t ee = e + h;
        const bool valid = ee < end;
        float uj = 0.0f, vj = 0.0f, r = 0.0f;
        int64_t uo = 0, vo = 0;
        if (valid) {
            const int64_t t = perm[ee];
            uo = (int64_t)user[t] * 32 + j;
            vo = (int64_t)item[t] * 32 + j;
            uj = U[uo];
            vj = V[vo];
            r = rating[t];
        }
        const float err = r - butterfly32(__builtin_fmaf(uj, vj, 0.0f));
        if (valid) {
            const float a = err * vj, b = reg * uj;
            const float a2 = err * uj, b2 = reg * vj;
            U[uo] = __builtin_fmaf(lr, a - b, uj);
            V[vo] = __builtin_fmaf(lr, a2 - b2, vj);
        }
    }
};

// first level >= l whose width exceeds thin_max (L if none); block-uniform
__device__ int64_t find_run_end(int64_t l, int64_t L, const int64_t *level_ptr,
                                int64_t thin_max) {
    __shared__ int64_t s_w[kWavesPerBlock];
    for (int64_t start = l; start < L; start += kBlock) {
        const int64_t c = start + threadIdx.x;
        const bool wide = c < L && level_ptr[c + 1] - level_ptr[c] > thin_max;
        const unsigned long long bal = __ballot(wide);
        if (lane_id() == 0)
            s_w[wave_in_block()] = bal ? start + wave_in_block() * kWave + (__ffsll(bal) - 1)
                                       : INT64_MAX;
        __syncthreads();
        int64_t m = INT64_MAX;
#pragma unroll
        for (int w = 0; w < kWavesPerBlock; ++w) m = min(m, s_w[w]);
        __syncthreads();
        if (m != INT64_MAX) return m;
    }
    return L;
}

template <class Op>
__global__ __launch_bounds__(kBlock) void k_levels_apply(Op op, const int64_t *level_ptr,
                                                         const int32_t *n_levels,
                                                         int64_t thin_max, Ctrl *ctrl,
                                                         int64_t timeout) {
    constexpr int U = Op::kUnits;
    const int64_t L = *n_levels;
    const int wave = wave_in_block();
    const bool single = gridDim.x == 1;
    const int64_t gw = (int64_t)blockIdx.x * kWavesPerBlock + wave;
    const int64_t nw = (int64_t)gridDim.x * kWavesPerBlock;
    int64_t l = 0;
    while (l < L) {
        int64_t beg = level_ptr[l], end = level_ptr[l + 1];
        if (single || end - beg <= thin_max) {
            int64_t l2 = l;
            if (blockIdx.x == 0) {
                for (; l2 < L; ++l2) {
                    beg = level_ptr[l2];
                    end = level_ptr[l2 + 1];
                    if (!single && end - beg > thin_max) break;
                    if (end - beg <= U) {
                        if (wave == 0) op(beg, end);
                    } else {
                        __syncthreads();
                        for (int64_t e = beg + (int64_t)wave * U; e < end; e += kWavesPerBlock * U)
                            op(e, end);
                        __syncthreads();
                    }
                }
            } else {
                l2 = find_run_end(l, L, level_ptr, thin_max);
            }
            l = l2;
        } else {
            for (int64_t e = beg + gw * U; e < end; e += nw * U) op(e, end);
            ++l;
        }
        if (!single && l < L && !grid_barrier(ctrl, timeout)) return;
    }
}

__global__ void k_ctrl_zero(Ctrl *c) {
    int *w = reinterpret_cast<int *>(c);
    for (int i = threadIdx.x; i < (int)(sizeof(Ctrl) / sizeof(int)); i += blockDim.x) w[i] = 0;
}

int64_t thin_max_setting() {
    static int64_t v = -1;
    if (v < 0) {
        const char *s = getenv("PDB_THIN_MAX");
        v = s ? atoll(s) : 16;
        if (v < 1) v = 1;
    }
    return v;
}

template <class Op>
int launch_levels(const Op &op, const pdb_levels *lv, Ctrl *ctrl, hipStream_t s) {
    const int64_t thin = thin_max_setting();
    const int64_t timeout = spin_timeout_ticks();
    k_ctrl_zero<<<1, 64, 0, s>>>(ctrl);
    PDB_LAUNCHED();
    const void *fn = reinterpret_cast<const void *>(&k_levels_apply<Op>);
    int grid = 1;
    const int64_t widest = lv->max_width_host;
    if (widest <= 0 || widest > thin) {
        int dev = 0, cus = 0, per_cu = 0;
        PDB_HIP(hipGetDevice(&dev));
        PDB_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
        PDB_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kBlock, 0));
        // one block per CU at most: more blocks only lengthen every barrier
        int64_t g = (int64_t)cus * std::min(per_cu > 0 ? per_cu : 1, 1);
        if (widest > 0) g = std::min<int64_t>(g, cdiv(widest, (int64_t)kWavesPerBlock * Op::kUnits));
        grid = (int)std::max<int64_t>(g, 1);
    }
    Op o = op;
    const int64_t *level_ptr = lv->level_ptr;
    const int32_t *n_levels = lv->n_levels;
    if (grid == 1) {
        k_levels_apply<Op><<<1, kBlock, 0, s>>>(o, level_ptr, n_levels, thin, ctrl, timeout);
        PDB_LAUNCHED();
    } else {
        int64_t thin_arg = thin, to = timeout;
        void *args[] = {&o, &level_ptr, &n_levels, &thin_arg, &ctrl, &to};
        PDB_HIP(hipLaunchCooperativeKernel(fn, dim3(grid), dim3(kBlock), args, 0, s));
    }
    return PDB_OK;
}

int epoch_checks(const pdb_levels *lv, int64_t n, void *ws, size_t ws_bytes) {
    if (!lv || !ws) return PDB_ERR_INVALID_ARG;
    if (n > 0 && (!lv->perm || !lv->level_ptr || !lv->n_levels)) return PDB_ERR_INVALID_ARG;
    if (ws_bytes < sizeof(Ctrl)) return PDB_ERR_WORKSPACE;
    if (n < 0) return PDB_ERR_INVALID_ARG;
    if (n >= INT32_MAX) return PDB_ERR_UNSUPPORTED;
    return PDB_OK;
}

}  // namespace
}  // namespace pdbk

using namespace pdbk;

extern "C" int pdb_epoch_workspace_bytes(size_t *bytes) {
    if (!bytes) return PDB_ERR_INVALID_ARG;
    *bytes = sizeof(Ctrl);
    return PDB_OK;
}

extern "C" int pdb_sgd_epoch(const pdb_csr *csr, const float *labels, int64_t n, int64_t d,
                             float *w, float lr, int loss, const pdb_levels *lv, void *ws,
                             size_t ws_bytes, hipStream_t s) {
    int rc = epoch_checks(lv, n, ws, ws_bytes);
    if (rc != PDB_OK) return rc;
    if (!csr || (n > 0 && (!csr->row_ptr || !labels || !w)) || (csr->nnz > 0 && !csr->col))
        return PDB_ERR_INVALID_ARG;
    if (loss != PDB_LOGISTIC && loss != PDB_SQUARED) return PDB_ERR_INVALID_ARG;
    if (d < 0 || csr->nnz < 0) return PDB_ERR_INVALID_ARG;
    if (d >= INT32_MAX || csr->nnz >= INT32_MAX) return PDB_ERR_UNSUPPORTED;
    if (n == 0) return PDB_OK;
    Ctrl *ctrl = static_cast<Ctrl *>(ws);
    const bool has_val = csr->val != nullptr;
#define PDB_SGD_CASE(LS, HV)                                                                 \
    if (loss == LS && has_val == HV) {                                                       \
        SgdOp<LS, HV> op{csr->row_ptr, csr->col, csr->val, labels, w, lv->perm, lr};         \
        return launch_levels(op, lv, ctrl, s);                                               \
    }
    PDB_SGD_CASE(PDB_LOGISTIC, true)
    PDB_SGD_CASE(PDB_LOGISTIC, false)
    PDB_SGD_CASE(PDB_SQUARED, true)
    PDB_SGD_CASE(PDB_SQUARED, false)
#undef PDB_SGD_CASE
    return PDB_ERR_INVALID_ARG;
}

extern "C" int pdb_mf_epoch(const int32_t *user, const int32_t *item, const float *rating,
                            int64_t n, float *U, int64_t n_users, float *V, int64_t n_items,
                            int32_t rank, float lr, float reg, const pdb_levels *lv, void *ws,
                            size_t ws_bytes, hipStream_t s) {
    int rc = epoch_checks(lv, n, ws, ws_bytes);
    if (rc != PDB_OK) return rc;
    if (rank != 32) return PDB_ERR_INVALID_ARG;
    if (n_users < 0 || n_items < 0) return PDB_ERR_INVALID_ARG;
    if (n > 0 && (!user || !item || !rating || !U || !V)) return PDB_ERR_INVALID_ARG;
    if (n == 0) return PDB_OK;
    MfOp op{user, item, rating, U, V, lv->perm, lr, reg};
    return launch_levels(op, lv, static_cast<Ctrl *>(ws), s);
}
