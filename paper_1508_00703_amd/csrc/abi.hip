// C-ABI plumbing: error strings, HIP error capture, CSR validation, device
// status word, spin-wait budget.
#include <cstdlib>

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

int64_t spin_timeout_ticks() {
    static int64_t ticks = -1;
    if (ticks < 0) {
        const char *s = getenv("PDB_SPIN_TIMEOUT_MS");
        const int64_t ms = s ? atoll(s) : 20000;
        int dev = 0, khz = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
            khz <= 0)
            khz = 100000;
        ticks = (ms > 0 ? ms : 1) * (int64_t)khz;
    }
    return ticks;
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
    case PDB_ERR_DEVICE: return "device-side failure (spin-wait watchdog expired or inconsistent schedule)";
    case PDB_ERR_UNSUPPORTED: return "size beyond 2^31-1 entries";
    default: return "unknown pdb status";
    }
}

extern "C" int pdb_last_hip_error(void) { return g_last_hip_error; }

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
