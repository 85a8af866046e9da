// Bounded-delay SGD (gfx950, wave64), the relaxation of Sec. 7: an
// iteration may read a partition once the write of iteration alpha - 1 -
// delay to it is done (Asynchronous Read Constraint), instead of waiting for
// every earlier writer.  The execution computed here reads as early as that
// allows: example alpha reads, for each of its features, the value written
// by the latest earlier example before alpha - delay (the initial weight if
// there is none), and every example's update is applied in example order to
// each of its features, w = fma(-s, x, w), so no update is lost.  delay = 0
// is the sequential computation.
//
// A first pass finds each stored entry's read source -- the previous entry
// on its feature, followed back past the entries of the last `delay`
// examples -- and its next writer.  Two executions follow.
//
// Windowed (one block): examples in windows of W = delay + 1.  Every read
// of window k has its source in window k - 1 or earlier, so the block holds
// the values written by window k - 1 in LDS and the state before it in w:
// it loads window k's reads, commits window k - 1's last writes to w, forms
// the W steps (a wave per example), then runs each feature's writes through
// the window in example order from its first entry.  Chosen when a window's
// entries fit the block's LDS.
//
// Sync-free (otherwise): every stored entry owns a 64-bit word (the value it
// wrote, its own index as the tag); waves take examples in index order; an
// example waits for its read sources' words, computes its step, then waits
// for each entry's previous writer and publishes its own words.  The
// earliest unfinished example never waits on a later one.  A last pass
// copies each feature's final value (the entry nothing overwrites) into w.
#include <climits>

#include "pdb_math.h"
#include "pdb_words.h"

namespace pdbk {

namespace {

constexpr int kSWaves = kBlock / kWave;
constexpr int kWinCap = 2048;          // entries (and examples) of a window held in LDS
constexpr int kWinThreads = 1024;
constexpr int kWinWaves = kWinThreads / kWave;
constexpr int kWinPer = kWinCap / kWinThreads;  // entries per thread

struct StaleWs {
    Ctrl *ctrl;
    unsigned long long *words;  // [nnz]
    int32_t *rd;                // [nnz] read source, -1 = the initial weight
    int32_t *overwritten;       // [nnz] 1 when a later entry writes the same feature
    int32_t *next;              // [nnz] next entry on the same feature, -1 = none
    size_t total;
};

__device__ __forceinline__ int64_t cdiv_dev(int64_t a, int64_t b) { return (a + b - 1) / b; }

StaleWs stale_layout(void *base, int64_t nnz) {
    StaleWs w{};
    char *p = static_cast<char *>(base);
    size_t off = 0;
    auto take = [&](int64_t bytes) {
        char *r = p ? p + off : nullptr;
        off += (size_t)align_up(bytes);
        return r;
    };
    const int64_t z = std::max<int64_t>(nnz, 1);
    w.ctrl = reinterpret_cast<Ctrl *>(take(sizeof(Ctrl)));
    w.words = reinterpret_cast<unsigned long long *>(take(8 * z));
    w.rd = reinterpret_cast<int32_t *>(take(4 * z));
    w.overwritten = reinterpret_cast<int32_t *>(take(4 * z));
    w.next = reinterpret_cast<int32_t *>(take(4 * z));
    w.total = off;
    return w;
}

__global__ void k_stale_clear(unsigned long long *__restrict__ words,
                              int32_t *__restrict__ overwritten, int32_t *__restrict__ next,
                              int64_t nnz) {
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < nnz;
         q += (int64_t)gridDim.x * blockDim.x) {
        words[q] = word_pack(0.0f, -1);
        overwritten[q] = 0;
        next[q] = -1;
    }
}

// next writer: the entry whose previous entry on the feature is q
__global__ void k_stale_next(const int32_t *__restrict__ prev, int64_t nnz,
                             int32_t *__restrict__ next) {
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < nnz;
         q += (int64_t)gridDim.x * blockDim.x) {
        const int32_t p = prev[q];
        if (p >= 0) next[p] = (int32_t)q;
    }
}

// examples (after the first) that share no feature with the example before
// them: few on chain-like inputs, where the windowed execution pays
__global__ __launch_bounds__(kBlock) void k_stale_breaks(const int64_t *__restrict__ row_ptr,
                                                         int64_t n, const int32_t *__restrict__ prev,
                                                         Ctrl *ctrl) {
    const int lane = lane_id();
    const int64_t nw = (int64_t)gridDim.x * kSWaves;
    int breaks = 0;
    for (int64_t i = 1 + blockIdx.x * (int64_t)kSWaves + wave_in_block(); i < n; i += nw) {
        const int64_t lo = row_ptr[i - 1], b = row_ptr[i], e = row_ptr[i + 1];
        bool found = false;
        for (int64_t p = b + lane; p < e && !found; p += kWave) found = prev[p] >= lo;
        if (__ballot(found) == 0ull) ++breaks;
    }
    if (lane == 0 && breaks) atomicAdd(&ctrl->chain_breaks, breaks);
}

// the largest number of entries in a window of W examples
__global__ void k_window_max(const int64_t *__restrict__ row_ptr, int64_t n, int64_t W,
                             Ctrl *ctrl) {
    const int64_t nwin = cdiv_dev(n, W);
    long long best = 0;
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < nwin;
         k += (int64_t)gridDim.x * blockDim.x)
        best = max(best, (long long)(row_ptr[min(n, (k + 1) * W)] - row_ptr[k * W]));
    if (best > 0) atomicMax(&ctrl->max_width, best);
}

__global__ void k_stale_ctrl_zero(Ctrl *c) {
    int *w = reinterpret_cast<int *>(c);
    for (int i = threadIdx.x; i < (int)(sizeof(Ctrl) / sizeof(int)); i += blockDim.x) w[i] = 0;
}

// Read sources, one wave per example a: the previous entry on the feature,
// then back while it belongs to one of the examples a - delay .. a - 1 (their
// entries are the CSR positions from row_ptr[a - delay] on).  Also marks
// every previous entry as overwritten.
__global__ __launch_bounds__(kBlock) void k_stale_sources(const int64_t *__restrict__ row_ptr,
                                                          int64_t n,
                                                          const int32_t *__restrict__ prev,
                                                          int64_t delay, int32_t *__restrict__ rd,
                                                          int32_t *__restrict__ overwritten) {
    const int lane = lane_id();
    const int64_t nw = (int64_t)gridDim.x * kSWaves;
    for (int64_t a = blockIdx.x * (int64_t)kSWaves + wave_in_block(); a < n; a += nw) {
        const int64_t b = row_ptr[a], e = row_ptr[a + 1];
        const bool all_in_window = a - delay <= 0;
        const int64_t lim = all_in_window ? 0 : row_ptr[a - delay];
        for (int64_t q = b + lane; q < e; q += kWave) {
            const int32_t pq = prev[q];
            if (pq >= 0) overwritten[pq] = 1;
            int32_t k = all_in_window ? -1 : pq;
            while (k >= 0 && (int64_t)k >= lim) k = prev[k];
            rd[q] = k;
        }
    }
}

// Examples are dealt to the waves in turn (wave k of W runs examples k,
// k + W, ...); the grid is launched cooperatively, so the earliest
// unfinished example is always being worked on.  A shared ticket counter
// would serve one request about every 200 ns.  An example of up to 2 x 64
// entries issues the loads and polls of both chunks together.
template <int LOSS, bool VAL>
__global__ __launch_bounds__(kBlock) void k_stale_epoch(
    const int64_t *__restrict__ row_ptr, const int32_t *__restrict__ col,
    const float *__restrict__ val, const float *__restrict__ y, const float *__restrict__ w0,
    const int32_t *__restrict__ prev, const int32_t *__restrict__ rd, unsigned long long *words,
    int64_t n, float lr, Ctrl *ctrl, int64_t timeout) {
    const int lane = lane_id();
    const int64_t nw = (int64_t)gridDim.x * kSWaves;
    for (int64_t a = (int64_t)blockIdx.x * kSWaves + wave_in_block(); a < n; a += nw) {
        const int64_t b = row_ptr[a];
        const int64_t m = row_ptr[a + 1] - b;
        if (m <= 2 * kWave) {
            const bool l0 = lane < m, l1 = kWave + lane < m;
            const int64_t q0 = b + lane, q1 = b + kWave + lane;
            const int32_t s0 = l0 ? rd[q0] : -1, s1 = l1 ? rd[q1] : -1;
            const int32_t p0 = l0 ? prev[q0] : -1, p1 = l1 ? prev[q1] : -1;
            const int32_t c0 = l0 ? col[q0] : 0, c1 = l1 ? col[q1] : 0;
            const float x0 = (VAL && l0) ? val[q0] : 1.0f, x1 = (VAL && l1) ? val[q1] : 1.0f;
            const float i0 = l0 ? w0[c0] : 0.0f, i1 = l1 ? w0[c1] : 0.0f;
            // reads: the value of each entry's read source (waits for it)
            unsigned long long v0 = 0, v1 = 0;
            if (!word_wait_wave2(words, s0 >= 0, s0, s0, &v0, s1 >= 0, s1, s1, &v1, ctrl, timeout))
                return;
            float acc = 0.0f;
            if (l0) acc = __builtin_fmaf(s0 >= 0 ? word_value(v0) : i0, x0, acc);
            if (l1) acc = __builtin_fmaf(s1 >= 0 ? word_value(v1) : i1, x1, acc);
            const float st = sgd_scale<LOSS>(wave_sum64(acc), y[a], lr);
            // writes: onto the value of each entry's previous writer
            if (!word_wait_wave2(words, p0 >= 0, p0, p0, &v0, p1 >= 0, p1, p1, &v1, ctrl, timeout))
                return;
            if (l0)
                word_put(words, q0,
                         word_pack(__builtin_fmaf(-st, x0, p0 >= 0 ? word_value(v0) : i0), (int)q0));
            if (l1)
                word_put(words, q1,
                         word_pack(__builtin_fmaf(-st, x1, p1 >= 0 ? word_value(v1) : i1), (int)q1));
            continue;
        }
        // reads: the value of each entry's read source (waits for it)
        float acc = 0.0f;
        for (int64_t k0 = 0; k0 < m; k0 += kWave) {
            const int64_t k = k0 + lane;
            const bool live = k < m;
            const int32_t src = live ? rd[b + k] : -1;
            unsigned long long v = 0;
            if (!word_wait_wave(words, src >= 0, src, src, &v, ctrl, timeout)) return;
            if (live) {
                const float r = src >= 0 ? word_value(v) : w0[col[b + k]];
                acc = __builtin_fmaf(r, VAL ? val[b + k] : 1.0f, acc);
            }
        }
        const float st = sgd_scale<LOSS>(wave_sum64(acc), y[a], lr);
        // writes: onto the value of each entry's previous writer
        for (int64_t k0 = 0; k0 < m; k0 += kWave) {
            const int64_t k = k0 + lane;
            const bool live = k < m;
            const int32_t pq = live ? prev[b + k] : -1;
            unsigned long long v = 0;
            if (!word_wait_wave(words, pq >= 0, pq, pq, &v, ctrl, timeout)) return;
            if (live) {
                const float cur = pq >= 0 ? word_value(v) : w0[col[b + k]];
                const float nv = __builtin_fmaf(-st, VAL ? val[b + k] : 1.0f, cur);
                word_put(words, b + k, word_pack(nv, (int)(b + k)));
            }
        }
    }
}

// The windowed execution, one block of kWinThreads threads.  Thread t
// handles entries t and t + kWinThreads of every window, and examples t and
// t + kWinThreads.  What a window reads from memory that earlier windows do
// not change (columns, values, read sources, previous and next writers, row
// bounds, labels) is loaded two windows ahead into registers; the weights it
// reads from w are loaded one window ahead, right after the commit that
// makes w the state they need.
struct WinBuf {
    int32_t col[kWinCap];
    float x[kWinCap];
    float rv[kWinCap];     // the value the entry reads
    float v[kWinCap];      // the value the entry writes
    int32_t nxt[kWinCap];  // next entry on the feature (CSR index), -1 = none
    int16_t ex[kWinCap];   // the entry's example within the window
    int32_t rp[kWinCap + 1];  // example bounds, relative to the window's first entry
    float y[kWinCap];
};

// a window's loads, per thread
struct WinMeta {
    int32_t col[kWinPer], rd[kWinPer], pv[kWinPer], nx[kWinPer];
    float x[kWinPer];
    int64_t rp[kWinPer + 1];  // row_ptr of examples t, t + kWinThreads (and the end)
    float y[kWinPer];
};

template <bool VAL>
__device__ __forceinline__ void win_load(WinMeta &m, int64_t k, int64_t nwin, int64_t W,
                                         int64_t n, int64_t nnz, int64_t q0,
                                         const int64_t *__restrict__ row_ptr,
                                         const int32_t *__restrict__ col,
                                         const float *__restrict__ val,
                                         const float *__restrict__ y,
                                         const int32_t *__restrict__ prev,
                                         const int32_t *__restrict__ rd,
                                         const int32_t *__restrict__ next) {
    if (k >= nwin) return;
    const int tid = threadIdx.x;
    const int64_t a0 = k * W, a1 = min(n, a0 + W);
#pragma unroll
    for (int u = 0; u < kWinPer; ++u) {
        // entries past the window's end are loaded (clamped) and ignored
        const int64_t q = min(q0 + tid + u * kWinThreads, nnz - 1);
        if (nnz > 0) {
            m.col[u] = col[q];
            m.rd[u] = rd[q];
            m.pv[u] = prev[q];
            m.nx[u] = next[q];
            m.x[u] = VAL ? val[q] : 1.0f;
        }
        const int64_t a = min(a0 + tid + u * kWinThreads, a1);
        m.rp[u] = row_ptr[a];
        m.y[u] = y[min(a, n - 1)];
    }
    m.rp[kWinPer] = row_ptr[min(a0 + tid + kWinPer * kWinThreads, a1)];
}

template <int LOSS, bool VAL>
__global__ __launch_bounds__(kWinThreads) void k_stale_window(
    const int64_t *__restrict__ row_ptr, const int32_t *__restrict__ col,
    const float *__restrict__ val, const float *__restrict__ y, float *w,
    const int32_t *__restrict__ prev, const int32_t *__restrict__ rd,
    const int32_t *__restrict__ next, int64_t n, int64_t nnz, int64_t W, float lr) {
    __shared__ WinBuf buf[2];
    __shared__ float S[kWinCap];
    const int tid = threadIdx.x, lane = lane_id(), wave = wave_in_block();
    const int64_t nwin = cdiv_dev(n, W);
    auto qstart = [&](int64_t k) { return row_ptr[min(n, k * W)]; };
    WinMeta m0, m1, m2;
    int64_t q0 = qstart(0), q1 = qstart(1), q2 = qstart(2);
    win_load<VAL>(m0, 0, nwin, W, n, nnz, q0, row_ptr, col, val, y, prev, rd, next);
    win_load<VAL>(m1, 1, nwin, W, n, nnz, q1, row_ptr, col, val, y, prev, rd, next);
    float wv[kWinPer];
#pragma unroll
    for (int u = 0; u < kWinPer; ++u) wv[u] = (nnz > 0) ? w[m0.col[u]] : 0.0f;
    int cur = 0;
    int64_t pq0 = 0;  // first entry of the previous window (its end is the current start)
    int pE = 0;       // entries of the previous window
    // One window.  mc, mn, mnn: the loads of windows k, k + 1, k + 2 (mnn is
    // issued here); qa, qb, qc: the first entries of windows k, k + 1, k + 2
    // (qa receives that of window k + 3).  The three calls per loop
    // iteration rotate the roles, so no register copy waits on a load still
    // in flight.
    auto window = [&](int64_t k, WinMeta &mc, WinMeta &mn, WinMeta &mnn, int64_t &qa,
                      int64_t qb, int64_t qc) {
        const int64_t a0 = k * W, a1 = min(n, a0 + W);
        const int64_t qs = qa;
        const int E = (int)(qb - qs), nex = (int)(a1 - a0);
        WinBuf &C = buf[cur];
        const WinBuf &P = buf[cur ^ 1];
        // window k into LDS; reads from window k - 1's writes, else from w
        // as it was before window k - 1
#pragma unroll
        for (int u = 0; u < kWinPer; ++u) {
            const int e = tid + u * kWinThreads;
            if (e < E) {
                const int32_t r = mc.rd[u];
                C.col[e] = mc.col[u];
                C.x[e] = mc.x[u];
                C.nxt[e] = mc.nx[u];
                C.rv[e] = (r >= pq0) ? P.v[r - pq0] : wv[u];
            }
            if (e <= nex) C.rp[e] = (int32_t)(mc.rp[u] - qs);
            if (e < nex) C.y[e] = mc.y[u];
        }
        if (tid + kWinPer * kWinThreads <= nex)
            C.rp[tid + kWinPer * kWinThreads] = (int32_t)(mc.rp[kWinPer] - qs);
        __syncthreads();
        // commit window k - 1: the last write of each feature it touched
        for (int e = tid; e < pE; e += kWinThreads) {
            const int32_t nx = P.nxt[e];
            if (nx < 0 || nx >= qs) w[P.col[e]] = P.v[e];
        }
        // window k + 2's loads, in flight while this window computes
        win_load<VAL>(mnn, k + 2, nwin, W, n, nnz, qc, row_ptr, col, val, y, prev, rd, next);
        qa = qstart(k + 3);
        // steps, a wave per example, dot products in the matched order
        for (int j = wave; j < nex; j += kWinWaves) {
            const int b = C.rp[j], mm = C.rp[j + 1] - b;
            float acc = 0.0f;
            for (int t = lane; t < mm; t += kWave) {
                acc = __builtin_fmaf(C.rv[b + t], C.x[b + t], acc);
                C.ex[b + t] = (int16_t)j;
            }
            const float z = wave_sum64(acc);
            if (lane == 0) S[j] = sgd_scale<LOSS>(z, C.y[j], lr);
        }
        __syncthreads();
        // window k + 1's reads of w: w is now the state before window k
        if (k + 1 < nwin && nnz > 0) {
#pragma unroll
            for (int u = 0; u < kWinPer; ++u) wv[u] = w[mn.col[u]];
        }
        // writes: each feature's entries of the window in example order,
        // from the value its previous writer left
#pragma unroll
        for (int u = 0; u < kWinPer; ++u) {
            const int e = tid + u * kWinThreads;
            const int32_t pv = mc.pv[u];
            if (e < E && pv < qs) {
                float v = (pv >= pq0) ? P.v[pv - pq0] : C.rv[e];
                int ee = e;
                for (;;) {
                    v = __builtin_fmaf(-S[C.ex[ee]], C.x[ee], v);
                    C.v[ee] = v;
                    const int32_t nx = C.nxt[ee];
                    if (nx < 0 || nx >= qb) break;
                    ee = (int)(nx - qs);
                }
            }
        }
        __syncthreads();
        pq0 = qs;
        pE = E;
        cur ^= 1;
    };
    for (int64_t k = 0; k < nwin; k += 3) {
        window(k, m0, m1, m2, q0, q1, q2);
        if (k + 1 >= nwin) break;
        window(k + 1, m1, m2, m0, q1, q2, q0);
        if (k + 2 >= nwin) break;
        window(k + 2, m2, m0, m1, q2, q0, q1);
    }
    const WinBuf &P = buf[cur ^ 1];
    for (int e = tid; e < pE; e += kWinThreads)
        if (P.nxt[e] < 0) w[P.col[e]] = P.v[e];
}

// each feature's final value: the entry no later entry overwrites
__global__ __launch_bounds__(kBlock) void k_stale_final(const int32_t *__restrict__ col,
                                                        const unsigned long long *__restrict__ words,
                                                        const int32_t *__restrict__ overwritten,
                                                        int64_t nnz, float *__restrict__ w) {
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < nnz;
         q += (int64_t)gridDim.x * blockDim.x)
        if (!overwritten[q]) w[col[q]] = word_value(words[q]);
}

template <int LOSS, bool VAL>
int launch_stale(const pdb_csr *csr, const float *labels, int64_t n, float *w, float lr,
                 int64_t delay, const int32_t *prev, StaleWs &ws, const Opts &opt, hipStream_t s) {
    const int64_t nnz = csr->nnz;
    const int64_t timeout = opt.timeout;
    k_stale_ctrl_zero<<<1, 64, 0, s>>>(ws.ctrl);
    PDB_LAUNCHED();
    if (nnz > 0) {
        k_stale_clear<<<grid_for(nnz, kBlock, 8192), kBlock, 0, s>>>(ws.words, ws.overwritten,
                                                                    ws.next, nnz);
        PDB_LAUNCHED();
        k_stale_sources<<<grid_for(n, kSWaves, 65536), kBlock, 0, s>>>(csr->row_ptr, n, prev,
                                                                       delay, ws.rd,
                                                                       ws.overwritten);
        PDB_LAUNCHED();
        k_stale_next<<<grid_for(nnz, kBlock, 8192), kBlock, 0, s>>>(prev, nnz, ws.next);
        PDB_LAUNCHED();
    }
    // windows of delay + 1 examples.  The windowed execution needs the
    // largest window to fit the block, and pays on chain-like inputs (most
    // examples share a feature with the one before: one block then beats a
    // device-scope hop per example); elsewhere the sync-free one runs many
    // examples at once.  Read back: this call synchronises the stream.
    const int mode = opt.stale_mode;
    const int64_t W = delay >= n ? std::max<int64_t>(n, 1) : delay + 1;  // no overflow at huge delays
    bool windowed = false;
    if (mode != PDB_STALE_SYNCFREE && W <= kWinCap) {
        k_window_max<<<grid_for(cdiv(n, W), kBlock, 4096), kBlock, 0, s>>>(csr->row_ptr, n, W,
                                                                           ws.ctrl);
        PDB_LAUNCHED();
        if (nnz > 0) {
            k_stale_breaks<<<grid_for(n, kSWaves, 65536), kBlock, 0, s>>>(csr->row_ptr, n, prev,
                                                                          ws.ctrl);
            PDB_LAUNCHED();
        }
        Ctrl host{};
        PDB_HIP(hipMemcpyAsync(&host, ws.ctrl, sizeof(Ctrl), hipMemcpyDeviceToHost, s));
        PDB_HIP(hipStreamSynchronize(s));
        const bool chain_like = 4 * (int64_t)host.chain_breaks <= n;
        windowed = host.max_width <= kWinCap && (mode == PDB_STALE_WINDOWED || chain_like);
    }
    if (windowed) {
        k_stale_window<LOSS, VAL><<<1, kWinThreads, 0, s>>>(csr->row_ptr, csr->col, csr->val,
                                                            labels, w, prev, ws.rd, ws.next, n,
                                                            nnz, W, lr);
        PDB_LAUNCHED();
        return PDB_OK;
    }
    // every block resident (a cooperative launch: the waves wait on each
    // other), at most one wave per example
    const void *fn = reinterpret_cast<const void *>(&k_stale_epoch<LOSS, VAL>);
    int dev = 0, cus = 0, per_cu = 0;
    PDB_HIP(hipGetDevice(&dev));
    PDB_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
    PDB_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kBlock, 0));
    const int64_t grid = std::max<int64_t>(
        1, std::min<int64_t>((int64_t)cus * std::max(per_cu, 1), cdiv(n, (int64_t)kSWaves)));
    {
        const int64_t *a_rp = csr->row_ptr;
        const int32_t *a_col = csr->col, *a_rd = ws.rd;
        const float *a_val = csr->val, *a_y = labels, *a_w0 = w;
        const int32_t *a_prev = prev;
        unsigned long long *a_words = ws.words;
        Ctrl *a_ctrl = ws.ctrl;
        int64_t a_n = n, a_timeout = timeout;
        float a_lr = lr;
        void *args[] = {&a_rp, &a_col, &a_val, &a_y, &a_w0, &a_prev, &a_rd, &a_words,
                        &a_n, &a_lr, &a_ctrl, &a_timeout};
        PDB_HIP(hipLaunchCooperativeKernel(fn, dim3((unsigned)grid), dim3(kBlock), args, 0, s));
    }
    if (nnz > 0) {
        k_stale_final<<<grid_for(nnz, kBlock, 8192), kBlock, 0, s>>>(csr->col, ws.words,
                                                                    ws.overwritten, nnz, w);
        PDB_LAUNCHED();
    }
    return PDB_OK;
}

}  // namespace
}  // namespace pdbk

using namespace pdbk;

extern "C" int pdb_stale_workspace_bytes(int64_t nnz, size_t *bytes) {
    if (!bytes || nnz < 0) return PDB_ERR_INVALID_ARG;
    if (nnz >= INT32_MAX) return PDB_ERR_UNSUPPORTED;
    *bytes = stale_layout(nullptr, nnz).total;
    return PDB_OK;
}

extern "C" int pdb_stale_epoch(const pdb_csr *csr, const float *labels, int64_t n, int64_t d,
                               float *w, float lr, int loss, int64_t delay,
                               const int32_t *prev_nz, void *ws, size_t ws_bytes,
                               const pdb_options *opt, hipStream_t s) {
    if (!csr || !ws || n < 0 || d < 0 || delay < 0) return PDB_ERR_INVALID_ARG;
    Opts o;
    const int orc = resolve_opts(opt, &o);
    if (orc != PDB_OK) return orc;
    if (n >= INT32_MAX || d >= INT32_MAX || csr->nnz >= INT32_MAX || csr->nnz < 0)
        return PDB_ERR_UNSUPPORTED;
    if (loss != PDB_LOGISTIC && loss != PDB_SQUARED) return PDB_ERR_INVALID_ARG;
    if (n > 0 && (!csr->row_ptr || !labels || !w)) return PDB_ERR_INVALID_ARG;
    if (csr->nnz > 0 && (!csr->col || !prev_nz)) return PDB_ERR_INVALID_ARG;
    StaleWs lay = stale_layout(ws, csr->nnz);
    if (ws_bytes < lay.total) return PDB_ERR_WORKSPACE;
    if (n == 0) return PDB_OK;
    const bool has_val = csr->val != nullptr;
    if (loss == PDB_LOGISTIC)
        return has_val ? launch_stale<PDB_LOGISTIC, true>(csr, labels, n, w, lr, delay, prev_nz, lay, o, s)
                       : launch_stale<PDB_LOGISTIC, false>(csr, labels, n, w, lr, delay, prev_nz, lay, o, s);
    return has_val ? launch_stale<PDB_SQUARED, true>(csr, labels, n, w, lr, delay, prev_nz, lay, o, s)
                   : launch_stale<PDB_SQUARED, false>(csr, labels, n, w, lr, delay, prev_nz, lay, o, s);
}
