// Dense full-batch gradient descent (gfx950, wave64): the update of Sec. 2
// with every example in every iteration, on a dense n x d example matrix X
// (the linear-regression workloads of Sec. 6.1-6.2).  One iteration:
//   z_i = <X_i, w>,  s_i = lr * g(z_i, y_i),  G_j = sum_i s_i X_ij,
//   w_j <- w_j - G_j,
// every z_i from the weights before the iteration.
//
// Workers and data-centric synchronisation.  The grid is an R x C array of
// workers, one block per CU, all resident.  Worker (r, c) owns the tile of
// rows [r Rb, (r+1) Rb) and columns [c Cb, (c+1) Cb) of X, and keeps its own
// copy of the column block w_c.  Per iteration it
//   1. publishes the partial dot products of its rows over its columns,
//   2. waits for the partials of the C workers of its row group, adds them in
//      column-block order and forms s_i for its rows,
//   3. publishes the partial gradients G_j over its rows for its columns,
//   4. waits for the partials of the R workers of its column group, adds them
//      in row-block order and steps its copy of w_c.
// Every worker of a row group forms the same s, and every worker of a column
// group the same w_c, bit for bit.  A worker waits only for the partitions it
// reads (Sec. 4.4's read constraint per partition), never on a grid barrier.
// Partials travel as (value, iteration) words in two buffers selected by the
// iteration's parity: a worker can run at most one iteration ahead of any
// worker that reads its partials, so a word is never overwritten before it
// is read (the write constraint).
//
// Summation order (reproduced by the oracle's matched mode): a partial dot
// product has 64 running sums, column k of the block (k from 0) in sum
// (k / 4) mod 64 -- lane k / 4 mod 64 takes four consecutive columns -- then
// the wave sum; z_i adds the column blocks' partials in block order.  A row
// block's partial gradient adds, in order, the partials of its chunks of 32
// rows, each an fma chain over the chunk's rows in order; G_j adds the row
// blocks' partials in block order.
//
// Waiting: a worker loads all the partial words it needs at once, many per
// thread, into LDS, and re-polls only those not yet written; the ordered sums
// then run from LDS.  The tile stays in LDS across iterations when it fits
// (resident variant); otherwise both passes stream it from memory every
// iteration.
#include <cmath>

#include "pdb_math.h"
#include "pdb_words.h"

namespace pdbk {

namespace {

constexpr int kDThreads = 1024;
constexpr int kDWaves = kDThreads / kWave;
constexpr int kZRowsRes = 8;            // rows per wave step of the dot-product pass (LDS tile)
constexpr int kGRows = 4;               // rows per step of the gradient pass (streaming)
constexpr int kGUnroll = 4;             // groups per lane in flight in the dot-product pass (streaming)
constexpr int kWaitBatch = 8;           // partial words per thread loaded before checking tags
constexpr int kRowChunk = 32;           // rows per fma chain of a partial gradient
constexpr int kLaneStride = kWave + 4;  // LDS floats per row of lane sums (b128 reads spread over the banks)
constexpr int64_t kMaxRowBlock = 4096;
constexpr int64_t kMaxColBlock = 16384;
constexpr int kLdsFloats = 36864;       // 144 KB: w_c, s and (resident) the tile

struct DenseWs {
    Ctrl *ctrl;
    unsigned long long *zw;  // [2][C][n] partial dot products
    unsigned long long *gw;  // [2][R][d] partial gradients
    size_t total;
};

DenseWs dense_layout(void *base, int64_t n, int64_t d, int64_t R, int64_t C) {
    DenseWs w{};
    char *p = static_cast<char *>(base);
    size_t off = 0;
    auto take = [&](int64_t bytes) {
        char *r = p ? p + off : nullptr;
        off += (size_t)align_up(bytes);
        return r;
    };
    w.ctrl = reinterpret_cast<Ctrl *>(take(sizeof(Ctrl)));
    w.zw = reinterpret_cast<unsigned long long *>(take(8 * std::max<int64_t>(2 * C * n, 1)));
    w.gw = reinterpret_cast<unsigned long long *>(take(8 * std::max<int64_t>(2 * R * d, 1)));
    w.total = off;
    return w;
}

struct DenseArgs {
    const float *X;
    int64_t ldx;
    const float *y;
    float *w;
    int64_t n, d, iters;
    float lr;
    int rb, cb, R, C;
    unsigned long long *zw, *gw;
    Ctrl *ctrl;
    int64_t timeout;
};

// floats of LDS a worker needs: w_c, s, and the tile when resident; the
// rest stages partial words and chunk partials
__host__ __device__ inline int64_t lds_floats(int64_t rb, int64_t cb, bool resident) {
    return cb + ((rb + 3) & ~int64_t(3)) + (resident ? rb * cb : 0);
}

// the resident variant also needs room to stage one row's or one column's
// partials and the chunk partials of its gradient pass
inline bool fits_resident(int64_t rb, int64_t cb, int64_t R, int64_t C) {
    const int64_t stage = std::max({R, C, cb * cdiv(rb, kRowChunk), (int64_t)kLaneStride});
    return lds_floats(rb, cb, true) + stage <= kLdsFloats;
}

__global__ void k_dense_clear(unsigned long long *__restrict__ a, int64_t count, Ctrl *ctrl) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < count; q += stride)
        a[q] = word_pack(0.0f, -1);
    if (ctrl && blockIdx.x == 0) {
        int *c = reinterpret_cast<int *>(ctrl);
        for (int i = threadIdx.x; i < (int)(sizeof(Ctrl) / sizeof(int)); i += blockDim.x) c[i] = 0;
    }
}

// Loads count words into stage[0..count), word e from base[idx(e)], once
// each carries tag.  Thread tid takes e = tid + m kDThreads, kWaitBatch words
// at a time; the words not yet written are polled again together, all their
// loads in flight at once.  False on timeout or abort.
template <class Idx>
__device__ __forceinline__ bool gather_words(unsigned long long *base, Idx idx, int count, int tag,
                                             float *stage, Ctrl *ctrl, int64_t timeout) {
    for (int e0 = threadIdx.x; e0 < count; e0 += kDThreads * kWaitBatch) {
        unsigned long long v[kWaitBatch];
        unsigned pending = 0;
#pragma unroll
        for (int u = 0; u < kWaitBatch; ++u) {
            const int e = e0 + u * kDThreads;
            if (e < count) v[u] = word_get(base, idx(e));
        }
#pragma unroll
        for (int u = 0; u < kWaitBatch; ++u) {
            const int e = e0 + u * kDThreads;
            if (e < count && word_tag(v[u]) != tag) pending |= 1u << u;
        }
        int64_t t0 = 0;
        for (int round = 0; pending != 0; ++round) {
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
            __asm__ __volatile__("" ::: "memory");
#pragma unroll
            for (int u = 0; u < kWaitBatch; ++u)
                if (pending & (1u << u)) v[u] = word_get(base, idx(e0 + u * kDThreads));
#pragma unroll
            for (int u = 0; u < kWaitBatch; ++u)
                if ((pending & (1u << u)) && word_tag(v[u]) == tag) pending &= ~(1u << u);
        }
#pragma unroll
        for (int u = 0; u < kWaitBatch; ++u) {
            const int e = e0 + u * kDThreads;
            if (e < count) stage[e] = word_value(v[u]);
        }
    }
    return true;
}

template <bool VEC>
__device__ __forceinline__ float4 load4(const float *p) {
    if (VEC) return *reinterpret_cast<const float4 *>(p);
    return make_float4(p[0], p[1], p[2], p[3]);
}

template <int LOSS, bool VEC, bool RES>
__global__ __launch_bounds__(kDThreads) void k_dense_gd(DenseArgs a) {
    __shared__ __align__(16) float lds[kLdsFloats];
    const int tid = threadIdx.x, lane = lane_id(), wave = wave_in_block();
    const int r = blockIdx.x / a.C, c = blockIdx.x % a.C;
    const int64_t row0 = (int64_t)r * a.rb, col0 = (int64_t)c * a.cb;
    const int rows = (int)std::min<int64_t>(a.rb, a.n - row0);
    const int cols = (int)std::min<int64_t>(a.cb, a.d - col0);
    const int groups = (cols + 3) >> 2;  // four consecutive columns per group
    float *sw = lds;                     // [cb] this worker's copy of w_c
    float *ss = lds + a.cb;              // [rb] steps s_i of the row block
    float *tile = ss + ((a.rb + 3) & ~3);  // [rb][cb] resident tile
    const int used = (int)lds_floats(a.rb, a.cb, RES);
    float *stage = lds + used;              // staged partials
    const int cap = kLdsFloats - used;
    const float *xt = a.X + row0 * a.ldx + col0;

    for (int k = tid; k < cols; k += kDThreads) sw[k] = a.w[col0 + k];
    if (RES) {
        for (int e = tid; e < rows * groups; e += kDThreads) {
            const int i = e / groups, g = e - i * groups;
            const float *src = xt + (int64_t)i * a.ldx + 4 * g;
            float *dst = tile + i * a.cb + 4 * g;
            if (4 * g + 3 < cols) {
                *reinterpret_cast<float4 *>(dst) = load4<VEC>(src);
            } else {
                for (int k = 0; k < 4; ++k)
                    if (4 * g + k < cols) dst[k] = src[k];
            }
        }
    }
    __syncthreads();

    // Partial dot products of this worker's rows over its columns, tag t.
    // Each lane keeps the running sums of its four-column groups.  Streamed:
    // a wave takes a row, kGUnroll groups per lane in flight, and sums the
    // lanes across the wave.  Resident: a wave takes kZRowsRes rows at once
    // and writes its lanes' sums to LDS; then a thread per row adds the 64 in
    // the butterfly's pairing (adjacent pairs, then pairs of pairs, ...) --
    // the value every lane of the butterfly ends with.  Rows past the end are
    // clamped (computed, not published) and columns past the end masked by a
    // select, so the loads of a step issue together.
    auto dot_pass = [&](int t) {
        unsigned long long *zw = a.zw + ((int64_t)(t & 1) * a.C + c) * a.n + row0;
        if constexpr (RES) {
            const int chunk = std::min(rows, std::max(1, cap / kLaneStride));
            for (int h0 = 0; h0 < rows; h0 += chunk) {
                const int nr = std::min(chunk, rows - h0);
                for (int i0 = wave * kZRowsRes; i0 < nr; i0 += kDWaves * kZRowsRes) {
                    float acc[kZRowsRes];
#pragma unroll
                    for (int u = 0; u < kZRowsRes; ++u) acc[u] = 0.0f;
                    for (int g = lane; g < groups; g += kWave) {
                        const int kk = 4 * g;
                        // w_c and the tile rows are padded to cb: in bounds
                        const float4 wv = *reinterpret_cast<const float4 *>(sw + kk);
                        float4 x[kZRowsRes];
#pragma unroll
                        for (int u = 0; u < kZRowsRes; ++u) {
                            const int i = h0 + std::min(i0 + u, nr - 1);
                            x[u] = *reinterpret_cast<const float4 *>(tile + i * a.cb + kk);
                        }
                        const bool c1 = kk + 1 < cols, c2 = kk + 2 < cols, c3 = kk + 3 < cols;
#pragma unroll
                        for (int u = 0; u < kZRowsRes; ++u) {
                            float v = __builtin_fmaf(x[u].x, wv.x, acc[u]);
                            const float v1 = __builtin_fmaf(x[u].y, wv.y, v);
                            v = c1 ? v1 : v;
                            const float v2 = __builtin_fmaf(x[u].z, wv.z, v);
                            v = c2 ? v2 : v;
                            const float v3 = __builtin_fmaf(x[u].w, wv.w, v);
                            acc[u] = c3 ? v3 : v;
                        }
                    }
#pragma unroll
                    for (int u = 0; u < kZRowsRes; ++u)
                        if (i0 + u < nr) stage[(i0 + u) * kLaneStride + lane] = acc[u];
                }
                __syncthreads();
                for (int i = tid; i < nr; i += kDThreads) {
                    float v[kWave];
#pragma unroll
                    for (int q = 0; q < kWave; q += 4) {
                        const float4 p4 = *reinterpret_cast<const float4 *>(stage + i * kLaneStride + q);
                        v[q] = p4.x;
                        v[q + 1] = p4.y;
                        v[q + 2] = p4.z;
                        v[q + 3] = p4.w;
                    }
#pragma unroll
                    for (int span = 1; span < kWave; span *= 2)
#pragma unroll
                        for (int q = 0; q < kWave; q += 2 * span) v[q] = v[q] + v[q + span];
                    word_put(zw, h0 + i, word_pack(v[0], t));
                }
                __syncthreads();
            }
        } else {
            for (int i = wave; i < rows; i += kDWaves) {
                const float *row = xt + (int64_t)i * a.ldx;
                float acc = 0.0f;
                for (int g0 = lane; g0 < groups; g0 += kWave * kGUnroll) {
                    float4 x[kGUnroll], wv[kGUnroll];
#pragma unroll
                    for (int q = 0; q < kGUnroll; ++q) {
                        const int kk = 4 * (g0 + q * kWave);
                        if (kk < cols) {
                            wv[q] = *reinterpret_cast<const float4 *>(sw + kk);
                            if (kk + 3 < cols) {
                                x[q] = load4<VEC>(row + kk);
                            } else {
                                x[q] = make_float4(row[kk], row[std::min(kk + 1, cols - 1)],
                                                   row[std::min(kk + 2, cols - 1)],
                                                   row[std::min(kk + 3, cols - 1)]);
                            }
                        }
                    }
#pragma unroll
                    for (int q = 0; q < kGUnroll; ++q) {
                        const int kk = 4 * (g0 + q * kWave);
                        if (kk < cols) {
                            const bool c1 = kk + 1 < cols, c2 = kk + 2 < cols, c3 = kk + 3 < cols;
                            float v = __builtin_fmaf(x[q].x, wv[q].x, acc);
                            const float v1 = __builtin_fmaf(x[q].y, wv[q].y, v);
                            v = c1 ? v1 : v;
                            const float v2 = __builtin_fmaf(x[q].z, wv[q].z, v);
                            v = c2 ? v2 : v;
                            const float v3 = __builtin_fmaf(x[q].w, wv[q].w, v);
                            acc = c3 ? v3 : v;
                        }
                    }
                }
                const float z = wave_sum64(acc);
                if (lane == 0) word_put(zw, i, word_pack(z, t));
            }
        }
    };

    // in-order sum p = 0..count-1 of stage[p * stride + j], loads in batches
    auto ordered_sum = [&](int j, int count, int stride) {
        float acc = stage[j];
        int p = 1;
        for (; p + 8 <= count; p += 8) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = stage[(p + u) * stride + j];
#pragma unroll
            for (int u = 0; u < 8; ++u) acc = acc + v[u];
        }
        for (; p < count; ++p) acc = acc + stage[p * stride + j];
        return acc;
    };

    dot_pass(0);
    for (int t = 0; t < a.iters; ++t) {
        // steps of this row block: the C column blocks' partials in order,
        // rows in chunks whose C partials fit the stage
        {
            const int chunk = std::max(1, std::min(rows, cap / a.C));
            for (int i0 = 0; i0 < rows; i0 += chunk) {
                const int nr = std::min(chunk, rows - i0);
                const int64_t base = (int64_t)(t & 1) * a.C * a.n + row0 + i0;
                const int64_t n = a.n;
                const bool ok = gather_words(
                    a.zw, [=](int e) { const int p = e / nr; return base + p * n + (e - p * nr); },
                    nr * a.C, t, stage, a.ctrl, a.timeout);
                if (__syncthreads_or(!ok)) return;
                for (int i = tid; i < nr; i += kDThreads)
                    ss[i0 + i] = sgd_scale<LOSS>(ordered_sum(i, a.C, nr), a.y[row0 + i0 + i], a.lr);
                __syncthreads();
            }
        }

        // partial gradients of this worker's columns over its rows
        unsigned long long *gw = a.gw + ((int64_t)(t & 1) * a.R + r) * a.d + col0;
        if (RES) {
            // one thread per (chunk, column), then the chunks added in order
            const int nch = (rows + kRowChunk - 1) / kRowChunk;
            for (int e = tid; e < nch * cols; e += kDThreads) {
                const int h = e / cols, k = e - h * cols;
                const int i1 = std::min(rows, (h + 1) * kRowChunk);
                const float *xc = tile + k;
                float acc = 0.0f;
                int i = h * kRowChunk;
                for (; i + 8 <= i1; i += 8) {
                    float x[8], sv[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        x[u] = xc[(i + u) * a.cb];
                        sv[u] = ss[i + u];
                    }
#pragma unroll
                    for (int u = 0; u < 8; ++u) acc = __builtin_fmaf(sv[u], x[u], acc);
                }
                for (; i < i1; ++i) acc = __builtin_fmaf(ss[i], xc[i * a.cb], acc);
                stage[e] = acc;
            }
            __syncthreads();
            for (int k = tid; k < cols; k += kDThreads)
                word_put(gw, k, word_pack(ordered_sum(k, nch, cols), t));
            __syncthreads();
        } else {
            for (int g = tid; g < groups; g += kDThreads) {
                float tot[4] = {0.0f, 0.0f, 0.0f, 0.0f};
                const float *xg = xt + 4 * g;
                const bool full = 4 * g + 3 < cols;
                for (int h0 = 0; h0 < rows; h0 += kRowChunk) {
                    const int h1 = std::min(rows, h0 + kRowChunk);
                    float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
                    if (full) {
                        int i = h0;
                        for (; i + kGRows <= h1; i += kGRows) {
                            float4 x[kGRows];
#pragma unroll
                            for (int u = 0; u < kGRows; ++u)
                                x[u] = load4<VEC>(xg + (int64_t)(i + u) * a.ldx);
#pragma unroll
                            for (int u = 0; u < kGRows; ++u) {
                                const float s = ss[i + u];
                                acc[0] = __builtin_fmaf(s, x[u].x, acc[0]);
                                acc[1] = __builtin_fmaf(s, x[u].y, acc[1]);
                                acc[2] = __builtin_fmaf(s, x[u].z, acc[2]);
                                acc[3] = __builtin_fmaf(s, x[u].w, acc[3]);
                            }
                        }
                        for (; i < h1; ++i) {
                            const float4 x = load4<VEC>(xg + (int64_t)i * a.ldx);
                            const float s = ss[i];
                            acc[0] = __builtin_fmaf(s, x.x, acc[0]);
                            acc[1] = __builtin_fmaf(s, x.y, acc[1]);
                            acc[2] = __builtin_fmaf(s, x.z, acc[2]);
                            acc[3] = __builtin_fmaf(s, x.w, acc[3]);
                        }
                    } else {
                        for (int i = h0; i < h1; ++i)
                            for (int k = 0; k < 4; ++k)
                                if (4 * g + k < cols)
                                    acc[k] = __builtin_fmaf(ss[i], xg[(int64_t)i * a.ldx + k], acc[k]);
                    }
#pragma unroll
                    for (int k = 0; k < 4; ++k) tot[k] = (h0 == 0) ? acc[k] : tot[k] + acc[k];
                }
                for (int k = 0; k < 4; ++k)
                    if (4 * g + k < cols) word_put(gw, 4 * g + k, word_pack(tot[k], t));
            }
        }

        // the step of w_c: the R row blocks' partials in order, columns in
        // chunks whose R partials fit the stage
        {
            const int chunk = std::max(1, std::min(cols, cap / a.R));
            for (int k0 = 0; k0 < cols; k0 += chunk) {
                const int nc = std::min(chunk, cols - k0);
                const int64_t base = (int64_t)(t & 1) * a.R * a.d + col0 + k0;
                const int64_t d = a.d;
                const bool ok = gather_words(
                    a.gw, [=](int e) { const int p = e / nc; return base + p * d + (e - p * nc); },
                    nc * a.R, t, stage, a.ctrl, a.timeout);
                if (__syncthreads_or(!ok)) return;
                for (int k = tid; k < nc; k += kDThreads)
                    sw[k0 + k] = sw[k0 + k] - ordered_sum(k, a.R, nc);
                __syncthreads();
            }
        }
        if (t + 1 < a.iters) dot_pass(t + 1);
    }
    if (r == 0)
        for (int k = tid; k < cols; k += kDThreads) a.w[col0 + k] = sw[k];
}

struct Plan {
    int64_t rb, cb, R, C;
};

int make_plan(int64_t n, int64_t d, int64_t workers, Plan *p) {
    if (workers < 1) return PDB_ERR_INVALID_ARG;
    const int64_t nn = std::max<int64_t>(n, 1), dd = std::max<int64_t>(d, 1);
    // C / R near sqrt(d / n) balances the two partial exchanges (n C^2 and
    // d R^2 words per iteration)
    const double ratio = std::sqrt((double)dd / (double)nn);
    int64_t R = (int64_t)std::llround(std::sqrt((double)workers / ratio));
    R = std::max<int64_t>(1, std::min<int64_t>({R, workers, nn}));
    int64_t C = std::max<int64_t>(1, std::min<int64_t>(workers / R, cdiv(dd, 4)));
    p->rb = cdiv(nn, R);
    p->cb = cdiv(cdiv(dd, C), 4) * 4;
    p->R = cdiv(nn, p->rb);
    p->C = cdiv(dd, p->cb);
    return PDB_OK;
}

int device_cus(int *cus) {
    int dev = 0;
    PDB_HIP(hipGetDevice(&dev));
    PDB_HIP(hipDeviceGetAttribute(cus, hipDeviceAttributeMultiprocessorCount, dev));
    return PDB_OK;
}

int check_blocks(int64_t n, int64_t d, int64_t rb, int64_t cb, Plan *p) {
    if (rb < 1 || cb < 4 || cb % 4 != 0) return PDB_ERR_INVALID_ARG;
    if (rb > kMaxRowBlock || cb > kMaxColBlock) return PDB_ERR_UNSUPPORTED;
    p->rb = rb;
    p->cb = cb;
    p->R = cdiv(std::max<int64_t>(n, 1), rb);
    p->C = cdiv(std::max<int64_t>(d, 1), cb);
    return PDB_OK;
}

template <int LOSS, bool VEC, bool RES>
int launch_dense(DenseArgs &a, hipStream_t s) {
    const void *fn = reinterpret_cast<const void *>(&k_dense_gd<LOSS, VEC, RES>);
    int cus = 0, per_cu = 0;
    const int rc = device_cus(&cus);
    if (rc != PDB_OK) return rc;
    PDB_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kDThreads, 0));
    // every worker waits on others: the whole grid must be resident
    if ((int64_t)a.R * a.C > (int64_t)cus * std::max(per_cu, 0)) return PDB_ERR_UNSUPPORTED;
    void *args[] = {&a};
    PDB_HIP(hipLaunchCooperativeKernel(fn, dim3((unsigned)(a.R * a.C)), dim3(kDThreads), args, 0, s));
    return PDB_OK;
}

template <int LOSS>
int dispatch_dense(DenseArgs &a, bool vec, bool res, hipStream_t s) {
    if (res) return vec ? launch_dense<LOSS, true, true>(a, s) : launch_dense<LOSS, false, true>(a, s);
    return vec ? launch_dense<LOSS, true, false>(a, s) : launch_dense<LOSS, false, false>(a, s);
}

}  // namespace
}  // namespace pdbk

using namespace pdbk;

extern "C" int pdb_dense_plan(int64_t n, int64_t d, int workers, int64_t *row_block,
                              int64_t *col_block) {
    if (!row_block || !col_block || n < 0 || d < 0) return PDB_ERR_INVALID_ARG;
    if (workers <= 0) {
        const int rc = device_cus(&workers);
        if (rc != PDB_OK) return rc;
    }
    Plan p{};
    const int rc = make_plan(n, d, workers, &p);
    if (rc != PDB_OK) return rc;
    if (p.rb > kMaxRowBlock || p.cb > kMaxColBlock) return PDB_ERR_UNSUPPORTED;
    *row_block = p.rb;
    *col_block = p.cb;
    return PDB_OK;
}

extern "C" int pdb_dense_workspace_bytes(int64_t n, int64_t d, int64_t row_block,
                                         int64_t col_block, size_t *bytes) {
    if (!bytes || n < 0 || d < 0) return PDB_ERR_INVALID_ARG;
    Plan p{};
    const int rc = check_blocks(n, d, row_block, col_block, &p);
    if (rc != PDB_OK) return rc;
    *bytes = dense_layout(nullptr, n, d, p.R, p.C).total;
    return PDB_OK;
}

extern "C" int pdb_dense_gd(const float *X, int64_t ldx, const float *labels, int64_t n,
                            int64_t d, float *w, float lr, int loss, int64_t iters,
                            int64_t row_block, int64_t col_block, void *ws, size_t ws_bytes,
                            const pdb_options *opt, hipStream_t s) {
    if (!ws || n < 0 || d < 0 || iters < 0 || ldx < d) return PDB_ERR_INVALID_ARG;
    Opts o;
    const int orc = resolve_opts(opt, &o);
    if (orc != PDB_OK) return orc;
    if (loss != PDB_LOGISTIC && loss != PDB_SQUARED) return PDB_ERR_INVALID_ARG;
    if (n >= INT32_MAX || d >= INT32_MAX || iters >= INT32_MAX) return PDB_ERR_UNSUPPORTED;
    if (n > 0 && d > 0 && (!X || !labels)) return PDB_ERR_INVALID_ARG;
    if (d > 0 && !w) return PDB_ERR_INVALID_ARG;
    Plan p{};
    int rc = check_blocks(n, d, row_block, col_block, &p);
    if (rc != PDB_OK) return rc;
    DenseWs lay = dense_layout(ws, n, d, p.R, p.C);
    if (ws_bytes < lay.total) return PDB_ERR_WORKSPACE;
    // nothing moves without examples, weights or iterations (the control
    // block is still cleared, so the workspace status reads OK)
    const bool idle = n == 0 || d == 0 || iters == 0;
    const int64_t words = idle ? 0 : (int64_t)((lay.total - align_up(sizeof(Ctrl))) / 8);
    k_dense_clear<<<grid_for(words, 256, 4096), 256, 0, s>>>(lay.zw, words, lay.ctrl);
    PDB_LAUNCHED();
    if (idle) return PDB_OK;
    const bool res = !o.dense_stream && fits_resident(p.rb, p.cb, p.R, p.C);
    const bool vec = (reinterpret_cast<uintptr_t>(X) % 16 == 0) && (ldx % 4 == 0);
    DenseArgs a{X, ldx, labels, w, n, d, iters, lr, (int)p.rb, (int)p.cb, (int)p.R, (int)p.C,
                lay.zw, lay.gw, lay.ctrl, o.timeout};
    return loss == PDB_LOGISTIC ? dispatch_dense<PDB_LOGISTIC>(a, vec, res, s)
                                : dispatch_dense<PDB_SQUARED>(a, vec, res, s);
}
