// C-ABI plumbing: error strings, HIP error capture, CSR validation, device
// status word, spin-wait budget.
#include <atomic>

#include "pdb_internal.h"

namespace pdbk {

namespace {
thread_local int g_last_hip_error = 0;

__global__ __launch_bounds__(kBlock) void k_validate_csr(const int64_t *__restrict__ row_ptr,
                                                         const int32_t *__restrict__ col,
                                                         int64_t n, int64_t d, int64_t nnz,
                                                         Ctrl *ctrl) {
    int bad = 0;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t b = row_ptr[i], e = row_ptr[i + 1];
        if (i == 0 && b != 0) bad = 1;
        if (i == n - 1 && e != nnz) bad = 1;
        // bounds first: never read columns through a malformed row range
        if (b < 0 || e < b || e > nnz) {
            bad = 1;
            continue;
        }
        int prev = -1;
        for (int64_t p = b; p < e; ++p) {
            const int c = col[p];
            if (c < 0 || (int64_t)c >= d || c <= prev) bad = 1;
            prev = c;
        }
    }
    if (__ballot(bad) != 0ull && lane_id() == 0)
        __hip_atomic_store(&ctrl->bad, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ void k_ctrl_clear(Ctrl *c) {
    int *w = reinterpret_cast<int *>(c);
    for (int i = threadIdx.x; i < (int)(sizeof(Ctrl) / sizeof(int)); i += blockDim.x) w[i] = 0;
}
}  // namespace

void set_hip_error(hipError_t e) { g_last_hip_error = (int)e; }

namespace {
// constant-clock rate (kHz) per device, queried once; 0 = not yet known.
// Concurrent first calls may both query: they store the same value.
constexpr int kMaxDevices = 64;
std::atomic<int> g_clock_khz[kMaxDevices];

int clock_khz() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 100000;
    std::atomic<int> *slot = dev < kMaxDevices ? &g_clock_khz[dev] : nullptr;
    int khz = slot ? slot->load(std::memory_order_relaxed) : 0;
    if (khz > 0) return khz;
    if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
        khz <= 0)
        khz = 100000;  // the gfx9 constant clock runs at 100 MHz
    if (slot) slot->store(khz, std::memory_order_relaxed);
    return khz;
}
}  // namespace

int resolve_opts(const pdb_options *o, Opts *out) {
    pdb_options d;
    pdb_options_init(&d);
    if (!o) o = &d;
    if (o->epoch_mode < PDB_EPOCH_AUTO || o->epoch_mode > PDB_EPOCH_SYNCFREE)
        return PDB_ERR_INVALID_ARG;
    if (o->stale_mode < PDB_STALE_AUTO || o->stale_mode > PDB_STALE_WINDOWED)
        return PDB_ERR_INVALID_ARG;
    if ((o->pipeline != 0 && o->pipeline != 1) || (o->dense_stream != 0 && o->dense_stream != 1))
        return PDB_ERR_INVALID_ARG;
    if (o->mf_one_cu < -1 || o->mf_one_cu > 1) return PDB_ERR_INVALID_ARG;
    if (o->pipeline_width < 1 || o->thin_max < 1 || o->batch_thin_max < 1 ||
        o->batch_syncfree_blocks < 1 || o->hot_features < -1 || o->spin_timeout_us < 0)
        return PDB_ERR_INVALID_ARG;
    // at most about 10^5 s, so the tick count stays far from overflow
    if (o->spin_timeout_us > (int64_t)100000 * 1000000) return PDB_ERR_INVALID_ARG;
    out->epoch_mode = o->epoch_mode;
    out->pipeline = o->pipeline != 0;
    out->pipeline_width = o->pipeline_width;
    out->thin_max = o->thin_max;
    out->hot_cap = o->hot_features;
    out->timeout = o->spin_timeout_us * (int64_t)clock_khz() / 1000;
    out->batch_thin_max = o->batch_thin_max;
    out->batch_sf_blocks = o->batch_syncfree_blocks;
    out->stale_mode = o->stale_mode;
    out->dense_stream = o->dense_stream != 0;
    out->mf_one_cu = o->mf_one_cu;
    return PDB_OK;
}

}  // namespace pdbk

using namespace pdbk;

extern "C" const char *pdb_strerror(int status) {
    switch (status) {
    case PDB_OK: return "ok";
    case PDB_ERR_INVALID_ARG: return "invalid argument (null pointer, negative size, bad enum or rank)";
    case PDB_ERR_BAD_CSR: return "malformed CSR (row_ptr not monotone / not ending at nnz, column out of range, columns not strictly increasing in a row)";
    case PDB_ERR_WORKSPACE: return "workspace missing or smaller than the size query returned";
    case PDB_ERR_HIP: return "a HIP runtime call failed (see pdb_last_hip_error)";
    case PDB_ERR_DEVICE: return "device-side failure (spin-wait watchdog expired, or the schedule check failed)";
    case PDB_ERR_UNSUPPORTED: return "size beyond 2^31-1 entries, or beyond the limit the entry point states";
    default: return "unknown pdb status";
    }
}

extern "C" int pdb_last_hip_error(void) { return g_last_hip_error; }

extern "C" int pdb_options_init(pdb_options *o) {
    if (!o) return PDB_ERR_INVALID_ARG;
    o->epoch_mode = PDB_EPOCH_AUTO;
    o->pipeline = 1;
    o->pipeline_width = 4;
    o->thin_max = 16;
    o->hot_features = -1;
    o->spin_timeout_us = 20000000;
    o->batch_thin_max = 2;
    o->batch_syncfree_blocks = 32;
    o->stale_mode = PDB_STALE_AUTO;
    o->dense_stream = 0;
    o->mf_one_cu = -1;
    return PDB_OK;
}

extern "C" int pdb_validate_csr(const pdb_csr *csr, int64_t n, int64_t d, void *ws,
                                size_t ws_bytes, hipStream_t s) {
    if (!csr || !ws || n < 0 || d < 0 || csr->nnz < 0) return PDB_ERR_INVALID_ARG;
    if (ws_bytes < sizeof(Ctrl)) return PDB_ERR_WORKSPACE;
    if (n > 0 && !csr->row_ptr) return PDB_ERR_INVALID_ARG;
    if (csr->nnz > 0 && !csr->col) return PDB_ERR_INVALID_ARG;
    if (n == 0) return csr->nnz == 0 ? PDB_OK : PDB_ERR_BAD_CSR;
    Ctrl *ctrl = static_cast<Ctrl *>(ws);
    k_ctrl_clear<<<1, 64, 0, s>>>(ctrl);
    k_validate_csr<<<grid_for(n, kBlock, 16384), kBlock, 0, s>>>(csr->row_ptr, csr->col, n, d,
                                                                 csr->nnz, ctrl);
    PDB_LAUNCHED();
    int bad = 0;
    PDB_HIP(hipMemcpyAsync(&bad, &ctrl->bad, sizeof(int), hipMemcpyDeviceToHost, s));
    PDB_HIP(hipStreamSynchronize(s));
    return bad ? PDB_ERR_BAD_CSR : PDB_OK;
}

extern "C" int pdb_workspace_status(void *ws, hipStream_t s) {
    if (!ws) return PDB_ERR_INVALID_ARG;
    Ctrl *ctrl = static_cast<Ctrl *>(ws);
    int err = 0;
    PDB_HIP(hipMemcpyAsync(&err, &ctrl->err, sizeof(int), hipMemcpyDeviceToHost, s));
    PDB_HIP(hipStreamSynchronize(s));
    if (err) {
        k_ctrl_clear<<<1, 64, 0, s>>>(ctrl);
        PDB_LAUNCHED();
        PDB_HIP(hipStreamSynchronize(s));
        return PDB_ERR_DEVICE;
    }
    return PDB_OK;
}
