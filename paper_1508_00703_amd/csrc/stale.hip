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
// Every stored entry owns a 64-bit word (the value it wrote, its own index
// as the tag).  A first pass finds each entry's read source -- the previous
// entry on its feature, followed back past the entries of the last `delay`
// examples -- and marks the entries that a later entry overwrites.  The
// epoch then runs sync-free: waves take examples in index order; an example
// waits for its read sources' words, computes its step, then waits for each
// entry's previous writer and publishes its own words.  The earliest
// unfinished example never waits on a later one.  A last pass copies each
// feature's final value (the entry nothing overwrites) into w.
#include <climits>

#include "pdb_math.h"
#include "pdb_words.h"

namespace pdbk {

namespace {

constexpr int kStaleB = 4;  // examples per ticket, run in order by one wave
constexpr int kSWaves = kBlock / kWave;

struct StaleWs {
    Ctrl *ctrl;
    unsigned long long *words;  // [nnz]
    int32_t *rd;                // [nnz] read source, -1 = the initial weight
    int32_t *overwritten;       // [nnz] 1 when a later entry writes the same feature
    size_t total;
};

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
    w.total = off;
    return w;
}

__global__ void k_stale_clear(unsigned long long *__restrict__ words,
                              int32_t *__restrict__ overwritten, int64_t nnz) {
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < nnz;
         q += (int64_t)gridDim.x * blockDim.x) {
        words[q] = word_pack(0.0f, -1);
        overwritten[q] = 0;
    }
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

template <int LOSS, bool VAL>
__global__ __launch_bounds__(kBlock) void k_stale_epoch(
    const int64_t *__restrict__ row_ptr, const int32_t *__restrict__ col,
    const float *__restrict__ val, const float *__restrict__ y, const float *__restrict__ w0,
    const int32_t *__restrict__ prev, const int32_t *__restrict__ rd, unsigned long long *words,
    int64_t n, float lr, Ctrl *ctrl, int64_t timeout) {
    const int lane = lane_id();
    for (;;) {
        long long tk = 0;
        if (lane == 0) tk = (long long)atomicAdd(&ctrl->ticket, (unsigned long long)kStaleB);
        tk = __shfl(tk, 0);
        if (tk >= n) return;
        const int64_t stop = min((int64_t)tk + kStaleB, n);
        for (int64_t a = tk; a < stop; ++a) {
            const int64_t b = row_ptr[a];
            const int64_t m = row_ptr[a + 1] - b;
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
            const float s = sgd_scale<LOSS>(wave_sum64(acc), y[a], lr);
            // writes: onto the value of each entry's previous writer
            for (int64_t k0 = 0; k0 < m; k0 += kWave) {
                const int64_t k = k0 + lane;
                const bool live = k < m;
                const int32_t pq = live ? prev[b + k] : -1;
                unsigned long long v = 0;
                if (!word_wait_wave(words, pq >= 0, pq, pq, &v, ctrl, timeout)) return;
                if (live) {
                    const float cur = pq >= 0 ? word_value(v) : w0[col[b + k]];
                    const float nv = __builtin_fmaf(-s, VAL ? val[b + k] : 1.0f, cur);
                    word_put(words, b + k, word_pack(nv, (int)(b + k)));
                }
            }
        }
    }
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
                 int64_t delay, const int32_t *prev, StaleWs &ws, hipStream_t s) {
    const int64_t nnz = csr->nnz;
    const int64_t timeout = spin_timeout_ticks();
    k_stale_ctrl_zero<<<1, 64, 0, s>>>(ws.ctrl);
    PDB_LAUNCHED();
    if (nnz > 0) {
        k_stale_clear<<<grid_for(nnz, kBlock, 8192), kBlock, 0, s>>>(ws.words, ws.overwritten, nnz);
        PDB_LAUNCHED();
        k_stale_sources<<<grid_for(n, kSWaves, 65536), kBlock, 0, s>>>(csr->row_ptr, n, prev,
                                                                       delay, ws.rd,
                                                                       ws.overwritten);
        PDB_LAUNCHED();
    }
    // every block resident; about as many waves as there are examples in
    // flight (tickets of kStaleB examples)
    const void *fn = reinterpret_cast<const void *>(&k_stale_epoch<LOSS, VAL>);
    int dev = 0, cus = 0, per_cu = 0;
    PDB_HIP(hipGetDevice(&dev));
    PDB_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
    PDB_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kBlock, 0));
    const int64_t grid = std::max<int64_t>(
        1, std::min<int64_t>((int64_t)cus * std::max(per_cu, 1), cdiv(n, (int64_t)kStaleB * kSWaves)));
    k_stale_epoch<LOSS, VAL><<<(unsigned)grid, kBlock, 0, s>>>(
        csr->row_ptr, csr->col, csr->val, labels, w, prev, ws.rd, ws.words, n, lr, ws.ctrl,
        timeout);
    PDB_LAUNCHED();
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
                               const int32_t *prev_nz, void *ws, size_t ws_bytes, hipStream_t s) {
    if (!csr || !ws || n < 0 || d < 0 || delay < 0) return PDB_ERR_INVALID_ARG;
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
        return has_val ? launch_stale<PDB_LOGISTIC, true>(csr, labels, n, w, lr, delay, prev_nz, lay, s)
                       : launch_stale<PDB_LOGISTIC, false>(csr, labels, n, w, lr, delay, prev_nz, lay, s);
    return has_val ? launch_stale<PDB_SQUARED, true>(csr, labels, n, w, lr, delay, prev_nz, lay, s)
                   : launch_stale<PDB_SQUARED, false>(csr, labels, n, w, lr, delay, prev_nz, lay, s);
}
