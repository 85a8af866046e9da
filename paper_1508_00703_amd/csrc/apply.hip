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
// loads of col/val, gather of w), fma into a per-lane partial sum, a
// butterfly over the 64 lanes (every lane ends with the same z), sigmoid or
// residual, then each lane writes its own features -- no atomics, since no
// other example of the level touches them.  Matrix completion: one rating per
// 32-lane half, lane j holds component j of the user and item rows.
//
// Level driver (a persistent grid): a level wider than `thin_max` is spread
// over every wave of the grid, followed by a device-wide barrier.  A run of
// narrow levels is handled by block 0 alone, with block barriers between
// levels, while the other blocks wait at the next device barrier.
//
// Runs of width-1 levels are a dependent chain: example t+1 reads what
// example t wrote.  There one wave runs the chain and the three other waves
// of the block stage upcoming examples (columns, values, and the CSR index
// of each entry's previous writer) into LDS.  Weights of features below
// `hot` live in LDS for the whole run; a feature that example t just wrote is
// not re-read at all: example t+1 takes the old value and x from example t's
// lane (a cross-lane permute issued before example t's step is known) and
// applies example t's step itself with the same fma -- so the only work
// between two steps is arithmetic.  Features written a few examples back come
// from a small LDS ring; all other cold features are prefetched from global
// memory kD examples ahead (their last writer finished before the prefetch).
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
    float q = 0x1.a01a02p-13f;                  // 1/5040
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

// v + v[partner] with the partner chosen by a DPP lane pattern
template <int CTRL>
__device__ __forceinline__ float dpp_add(float v) {
    return v + __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, false));
}

__device__ __forceinline__ float lane_value(float v, int l) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

// Butterfly p_l <- p_l + p_{l xor o} for o = 1, 2, 4, 8, 16, 32; returns the
// common result.  o = 1, 2: quad permutations.  o = 4: mirror within each
// group of 8 lanes -- once the quads hold equal values the mirrored partner
// holds the same value as lane l xor 4.  o = 8: mirror within each row of 16,
// likewise.  o = 16, 32: the four row values r0..r3 combine as
// (r0 + r1) + (r2 + r3).  Bitwise the same as the xor butterfly.
__device__ __forceinline__ float butterfly64(float v) {
    v = dpp_add<0xB1>(v);   // quad_perm [1,0,3,2]
    v = dpp_add<0x4E>(v);   // quad_perm [2,3,0,1]
    v = dpp_add<0x141>(v);  // row_half_mirror
    v = dpp_add<0x140>(v);  // row_mirror
    const float r0 = lane_value(v, 0), r1 = lane_value(v, 16);
    const float r2 = lane_value(v, 32), r3 = lane_value(v, 48);
    return (r0 + r1) + (r2 + r3);
}

// The same over each 32-lane half (o = 1..16); lanes of half h get half h's sum.
__device__ __forceinline__ float butterfly32(float v) {
    v = dpp_add<0xB1>(v);
    v = dpp_add<0x4E>(v);
    v = dpp_add<0x141>(v);
    v = dpp_add<0x140>(v);
    const float r0 = lane_value(v, 0), r1 = lane_value(v, 16);
    const float r2 = lane_value(v, 32), r3 = lane_value(v, 48);
    return lane_id() < 32 ? r0 + r1 : r2 + r3;
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
    const int32_t *prev_nz;  // may be null: no width-1 pipeline then
    float lr;
    static constexpr int kUnits = 1;  // examples per wave per step
    static constexpr bool kChain = true;

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
    static constexpr bool kChain = false;

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

// ---------------------------------------------------------------------------
// width-1 chain pipeline

constexpr int kD = 8;     // examples of look-ahead for cold prefetch; ring depth
constexpr int kRB = 32;   // staged examples (power of two)
constexpr int kPB = 8;    // examples per producer batch
constexpr int kChainMin = 32;  // shorter runs take the plain path

struct ChainLds {
    float *wcache;  // [hot]
    float *ring;    // [kD][64]
    int *st_col;    // [kRB][64]
    float *st_val;  // [kRB][64]
    int *st_pn;     // [kRB][64]
    int *mt_b;      // [kRB] first entry (CSR index) of the staged example
    int *mt_m;      // [kRB] its number of entries
    float *mt_y;    // [kRB] its label
    int *seq;       // [kRB] position staged in the slot (-1 none)
    int *ctl;       // [0] examples the consumer no longer needs staged, [1] stop
};

constexpr size_t kChainFixedLds =
    sizeof(float) * kD * 64 + (sizeof(int) * 2 + sizeof(float)) * kRB * 64 +
    (sizeof(int) * 3 + sizeof(float)) * kRB + sizeof(int) * 4;

__device__ __forceinline__ ChainLds chain_lds(unsigned char *base, int hot) {
    ChainLds S;
    S.ring = reinterpret_cast<float *>(base);
    S.st_col = reinterpret_cast<int *>(S.ring + kD * 64);
    S.st_val = reinterpret_cast<float *>(S.st_col + kRB * 64);
    S.st_pn = reinterpret_cast<int *>(S.st_val + kRB * 64);
    S.mt_b = S.st_pn + kRB * 64;
    S.mt_m = S.mt_b + kRB;
    S.mt_y = reinterpret_cast<float *>(S.mt_m + kRB);
    S.seq = reinterpret_cast<int *>(S.mt_y + kRB);
    S.ctl = S.seq + kRB;
    S.wcache = reinterpret_cast<float *>(S.ctl + 4);
    (void)hot;
    return S;
}

__device__ __forceinline__ void compiler_fence() { __asm__ __volatile__("" ::: "memory"); }

// Producer wave pid (0..2): stages examples perm[e_beg + t] for t in its
// batches, in order, never more than kRB ahead of the consumer.
template <int LOSS, bool VAL>
__device__ void chain_producer(const SgdOp<LOSS, VAL> &op, int pid, int64_t e_beg, int64_t len,
                               const ChainLds &S) {
    const int lane = lane_id();
    volatile int *ctl = S.ctl;
    volatile int *seq = S.seq;
    for (int64_t t0 = (int64_t)pid * kPB; t0 < len; t0 += 3 * kPB) {
        while (t0 + kPB - 1 >= (int64_t)ctl[0] + kRB) {
            if (ctl[1]) return;
            __builtin_amdgcn_s_sleep(1);
        }
        if (ctl[1]) return;
        int b = 0, e = 0;
        float yv = 0.0f;
        if (lane < kPB && t0 + lane < len) {
            const int64_t r = op.perm[e_beg + t0 + lane];
            b = (int)op.row_ptr[r];
            e = (int)op.row_ptr[r + 1];
            yv = op.y[r];
        }
        int c[kPB], p[kPB];
        float x[kPB];
#pragma unroll
        for (int i = 0; i < kPB; ++i) {
            const int bi = __builtin_amdgcn_readlane(b, i);
            const int mi = __builtin_amdgcn_readlane(e, i) - bi;
            c[i] = 0;
            p[i] = -1;
            x[i] = 1.0f;
            if (lane < mi && lane < kWave) {
                c[i] = op.col[bi + lane];
                p[i] = op.prev_nz[bi + lane];
                if (VAL) x[i] = op.val[bi + lane];
            }
        }
#pragma unroll
        for (int i = 0; i < kPB; ++i) {
            const int slot = (int)((t0 + i) & (kRB - 1));
            S.st_col[slot * 64 + lane] = c[i];
            S.st_pn[slot * 64 + lane] = p[i];
            if (VAL) S.st_val[slot * 64 + lane] = x[i];
        }
        if (lane < kPB) {
            const int slot = (int)((t0 + lane) & (kRB - 1));
            S.mt_b[slot] = b;
            S.mt_m[slot] = e - b;
            S.mt_y[slot] = yv;
        }
        compiler_fence();  // LDS executes one wave's operations in order
        if (lane < kPB && t0 + lane < len) seq[(t0 + lane) & (kRB - 1)] = (int)(t0 + lane);
        compiler_fence();
    }
}

struct Staged {
    int c, pn, b, m;
    float x, y;
};

// Waits until examples lo .. hi-1 (hi - lo <= kRB) are staged.
__device__ __forceinline__ void wait_staged(const ChainLds &S, int64_t lo, int64_t hi) {
    volatile int *seq = S.seq;
    const int64_t t = lo + lane_id();
    for (;;) {
        const bool ok = t >= hi || seq[t & (kRB - 1)] == (int)t;
        if (__ballot(!ok) == 0ull) break;
        __builtin_amdgcn_s_sleep(0);
    }
    compiler_fence();
}

template <bool VAL>
__device__ __forceinline__ Staged read_staged(const ChainLds &S, int64_t t) {
    const int slot = (int)(t & (kRB - 1)), lane = lane_id();
    Staged r;
    r.c = S.st_col[slot * 64 + lane];
    r.pn = S.st_pn[slot * 64 + lane];
    r.x = VAL ? S.st_val[slot * 64 + lane] : 1.0f;
    r.b = __builtin_amdgcn_readfirstlane(S.mt_b[slot]);
    r.m = __builtin_amdgcn_readfirstlane(S.mt_m[slot]);
    r.y = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(S.mt_y[slot])));
    return r;
}

// Consumer: runs examples t = 0.. of the run in order.  Returns the number
// processed: len, or the position of the first example with more than 64
// entries (the caller runs that one on the plain path).
template <int LOSS, bool VAL>
__device__ int64_t chain_consumer(const SgdOp<LOSS, VAL> &op, int64_t len, int hot,
                                  const ChainLds &S) {
    const int lane = lane_id();
    volatile int *ctl = S.ctl;
    float *__restrict__ w = op.w;
    int64_t stop = len;
    int wb[kD], wm[kD];   // window: first entry and count of the example at t mod kD
    float gv[kD];         // cold values prefetched for the example at t mod kD
#pragma unroll
    for (int j = 0; j < kD; ++j) {
        wb[j] = 0;
        wm[j] = 0;
        gv[j] = 0.0f;
    }
    // prefetch cold values for the first kD examples (nothing written yet)
    wait_staged(S, 0, std::min<int64_t>(kD, stop));
#pragma unroll
    for (int j = 0; j < kD; ++j) {
        if (j < stop) {
            const Staged r = read_staged<VAL>(S, j);
            if (r.m > kWave) stop = j;
            else if (lane < r.m && r.c >= hot) gv[j] = w[r.c];
        }
    }
    // example 0: no earlier example of the run wrote anything
    Staged cur = {0, -1, 0, 0, 1.0f, 0.0f};
    float cur_v = 0.0f, cur_fw = 0.0f, cur_fx = 0.0f;
    bool cur_fwd = false;
    if (stop > 0) {
        cur = read_staged<VAL>(S, 0);
        cur_v = (lane < cur.m) ? (cur.c < hot ? S.wcache[cur.c] : gv[0]) : 0.0f;
    }
    Staged nxt = {0, -1, 0, 0, 1.0f, 0.0f};
    if (stop > 1) nxt = read_staged<VAL>(S, 1);
    float s_prev = 0.0f;

    for (int64_t t0 = 0; t0 < stop; t0 += kD) {
        // examples read in this block: t+2 and t+kD for t in [t0, t0+kD)
        wait_staged(S, t0 + 2, std::min<int64_t>(t0 + 2 * kD, stop));
#pragma unroll
        for (int s = 0; s < kD; ++s) {
            const int64_t t = t0 + s;
            if (t < stop) {
                // (a) this example's weights: forwarded ones get the previous step now
                const float w_old = cur_fwd ? __builtin_fmaf(-s_prev, cur_fx, cur_fw) : cur_v;
                const bool live = lane < cur.m;
                const float acc = live ? __builtin_fmaf(w_old, cur.x, 0.0f) : 0.0f;
                wb[s] = cur.b;
                wm[s] = cur.m;
                // (b) resolve example t+1 against the window t+1-kD .. t
                float n_v = 0.0f, n_fw = 0.0f, n_fx = 0.0f;
                bool n_fwd = false;
                if (t + 1 < stop) {
                    int src = -1, off = 0;
#pragma unroll
                    for (int j = 0; j < kD; ++j) {
                        const unsigned o = (unsigned)(nxt.pn - wb[j]);
                        if (nxt.pn >= 0 && o < (unsigned)wm[j]) {
                            src = j;
                            off = (int)o;
                        }
                    }
                    n_fwd = (src == s);
                    const int addr = (n_fwd ? off : lane) << 2;
                    n_fw = __int_as_float(__builtin_amdgcn_ds_bpermute(addr, __float_as_int(w_old)));
                    n_fx = __int_as_float(__builtin_amdgcn_ds_bpermute(addr, __float_as_int(cur.x)));
                    if (lane < nxt.m && !n_fwd) {
                        if (nxt.c < hot) n_v = S.wcache[nxt.c];
                        else if (src >= 0) n_v = S.ring[src * 64 + off];
                        else n_v = gv[(s + 1) % kD];
                    }
                }
                Staged nxt2 = {0, -1, 0, 0, 1.0f, 0.0f};
                if (t + 2 < stop) nxt2 = read_staged<VAL>(S, t + 2);
                // (c) the step of example t
                const float st = sgd_scale<LOSS>(butterfly64(acc), cur.y, op.lr);
                const float w_new = __builtin_fmaf(-st, cur.x, w_old);
                if (live) {
                    if (cur.c < hot) S.wcache[cur.c] = w_new;
                    else w[cur.c] = w_new;
                    S.ring[s * 64 + lane] = w_new;
                }
                // (d) prefetch cold values of example t+kD (writes up to t are issued)
                if (t + kD < stop) {
                    const Staged r = read_staged<VAL>(S, t + kD);
                    if (r.m > kWave) {
                        stop = t + kD;  // producers keep staging until the run ends
                    } else {
                        gv[s] = (lane < r.m && r.c >= hot) ? w[r.c] : 0.0f;
                    }
                }
                ctl[0] = (int)(t + 3);
                // (e) rotate
                s_prev = st;
                cur = nxt;
                cur_v = n_v;
                cur_fw = n_fw;
                cur_fx = n_fx;
                cur_fwd = n_fwd;
                nxt = nxt2;
            }
        }
    }
    ctl[1] = 1;
    return stop;
}

// Runs perm[e_beg .. e_end) (consecutive width-1 levels) with the whole block.
template <int LOSS, bool VAL>
__device__ void chain_run(const SgdOp<LOSS, VAL> &op, int64_t e_beg, int64_t e_end, int hot,
                          unsigned char *lds) {
    const ChainLds S = chain_lds(lds, hot);
    const int wave = wave_in_block(), lane = lane_id();
    int64_t pos = e_beg;
    while (pos < e_end) {
        for (int i = threadIdx.x; i < hot; i += kBlock) S.wcache[i] = op.w[i];
        for (int i = threadIdx.x; i < kRB; i += kBlock) S.seq[i] = -1;
        if (threadIdx.x < 4) S.ctl[threadIdx.x] = 0;
        __syncthreads();
        int64_t done = e_end - pos;
        if (wave == 0) done = chain_consumer(op, e_end - pos, hot, S);
        else chain_producer(op, wave - 1, pos, e_end - pos, S);
        __syncthreads();
        __shared__ int64_t s_done;
        if (threadIdx.x == 0) s_done = done;
        for (int i = threadIdx.x; i < hot; i += kBlock) op.w[i] = S.wcache[i];
        __syncthreads();
        done = s_done;
        pos += done;
        if (pos < e_end) {
            // an example with more than 64 entries: plain path, then resume
            if (wave == 0) op(pos, pos + 1);
            __syncthreads();
            ++pos;
        }
    }
    (void)lane;
}

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

extern __shared__ __align__(16) unsigned char g_dyn_lds[];

template <class Op>
__global__ __launch_bounds__(kBlock) void k_levels_apply(Op op, const int64_t *level_ptr,
                                                         const int32_t *n_levels,
                                                         int64_t thin_max, int hot, Ctrl *ctrl,
                                                         int64_t timeout) {
    constexpr int U = Op::kUnits;
    const int64_t L = *n_levels;
    const int wave = wave_in_block();
    const bool single = gridDim.x == 1;
    const int64_t gw = (int64_t)blockIdx.x * kWavesPerBlock + wave;
    const int64_t nw = (int64_t)gridDim.x * kWavesPerBlock;
    int64_t l = 0;
    int64_t no_chain_before = 0;  // levels below this were found not to start a long run
    while (l < L) {
        int64_t beg = level_ptr[l], end = level_ptr[l + 1];
        if (single || end - beg <= thin_max) {
            int64_t l2 = l;
            if (blockIdx.x == 0) {
                while (l2 < L) {
                    beg = level_ptr[l2];
                    end = level_ptr[l2 + 1];
                    if (!single && end - beg > thin_max) break;
                    if constexpr (Op::kChain) {
                        if (hot >= 0 && end - beg == 1 && l2 >= no_chain_before) {
                            const int64_t l3 = find_run_end(l2, L, level_ptr, 1);
                            if (l3 - l2 >= kChainMin) {
                                chain_run(op, beg, level_ptr[l3], hot, g_dyn_lds);
                                l2 = l3;
                                continue;
                            }
                            no_chain_before = l3;
                        }
                    }
                    if (end - beg <= U) {
                        if (wave == 0) op(beg, end);
                    } else {
                        __syncthreads();
                        for (int64_t e = beg + (int64_t)wave * U; e < end; e += kWavesPerBlock * U)
                            op(e, end);
                        __syncthreads();
                    }
                    ++l2;
                }
                __syncthreads();
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

int64_t env_setting(const char *name, int64_t dflt) {
    const char *s = getenv(name);
    return s ? atoll(s) : dflt;
}

template <class Op>
int launch_levels(const Op &op, const pdb_levels *lv, int64_t d, bool chain_ok, Ctrl *ctrl,
                  hipStream_t s) {
    // tuning knobs, read per call: widest level run by block 0 alone, and a
    // cap on the number of weights cached in LDS by the width-1 pipeline
    const int64_t thin = std::max<int64_t>(env_setting("PDB_THIN_MAX", 16), 1);
    const int64_t hot_cap = env_setting("PDB_HOT_FEATURES", -1);
    const int64_t timeout = spin_timeout_ticks();
    k_ctrl_zero<<<1, 64, 0, s>>>(ctrl);
    PDB_LAUNCHED();
    const void *fn = reinterpret_cast<const void *>(&k_levels_apply<Op>);
    int dev = 0, cus = 0, max_lds = 0;
    PDB_HIP(hipGetDevice(&dev));
    PDB_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
    PDB_HIP(hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev));
    // LDS: the width-1 pipeline's fixed part plus as many cached weights as fit
    int hot = -1;
    size_t lds = 0;
    if (Op::kChain && chain_ok) {
        const int64_t room = (int64_t)max_lds - (int64_t)kChainFixedLds - 1024;
        int64_t h = std::min<int64_t>(room / 4, d);
        if (hot_cap >= 0) h = std::min<int64_t>(h, hot_cap);
        h = std::max<int64_t>(h, 0);
        hot = (int)h;
        lds = kChainFixedLds + (size_t)h * 4;
        PDB_HIP(hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
    }
    int grid = 1;
    const int64_t widest = lv->max_width_host;
    if (widest <= 0 || widest > thin) {
        int per_cu = 0;
        PDB_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kBlock, lds));
        // one block per CU at most: more blocks only lengthen every barrier
        int64_t g = (int64_t)cus * std::min(per_cu > 0 ? per_cu : 1, 1);
        if (widest > 0) g = std::min<int64_t>(g, cdiv(widest, (int64_t)kWavesPerBlock * Op::kUnits));
        grid = (int)std::max<int64_t>(g, 1);
    }
    Op o = op;
    const int64_t *level_ptr = lv->level_ptr;
    const int32_t *n_levels = lv->n_levels;
    if (grid == 1) {
        k_levels_apply<Op><<<1, kBlock, lds, s>>>(o, level_ptr, n_levels, thin, hot, ctrl, timeout);
        PDB_LAUNCHED();
    } else {
        int64_t thin_arg = thin, to = timeout;
        int hot_arg = hot;
        void *args[] = {&o, &level_ptr, &n_levels, &thin_arg, &hot_arg, &ctrl, &to};
        PDB_HIP(hipLaunchCooperativeKernel(fn, dim3(grid), dim3(kBlock), args, lds, s));
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
    const bool chain_env = env_setting("PDB_CHAIN", 1) != 0;
    const bool chain_ok = chain_env && lv->prev_nz != nullptr;
#define PDB_SGD_CASE(LS, HV)                                                                 \
    if (loss == LS && has_val == HV) {                                                       \
        SgdOp<LS, HV> op{csr->row_ptr, csr->col, csr->val, labels, w, lv->perm, lv->prev_nz, lr}; \
        return launch_levels(op, lv, d, chain_ok, ctrl, s);                                  \
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
    return launch_levels(op, lv, n_users + n_items, false, static_cast<Ctrl *>(ws), s);
}
