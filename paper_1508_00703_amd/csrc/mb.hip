// Microbenchmarks (gfx950, wave64): streaming copy, device-scope hand-over
// latency between two compute units, grid-wide barrier cost.  They measure
// the costs that bound the epoch kernels and compute nothing of the method.
#include "../../include/pdb_mb.h"
#include "pdb_internal.h"

namespace pdbk {
namespace {

constexpr size_t kMbWs = 1024;  // control block + one 256-byte line for the hop word

// Four 16-byte chunks per thread per step, all loads issued before the
// stores; consecutive lanes take consecutive chunks (each wave moves 1 KiB
// per load instruction).
constexpr int kCopyUnroll = 4;
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
__global__ __launch_bounds__(kBlock) void k_mb_copy(const u32x4 *__restrict__ src,
                                                    u32x4 *__restrict__ dst, int64_t count) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    for (; i + (kCopyUnroll - 1) * stride < count; i += kCopyUnroll * stride) {
        u32x4 v[kCopyUnroll];
#pragma unroll
        for (int k = 0; k < kCopyUnroll; ++k) v[k] = __builtin_nontemporal_load(&src[i + k * stride]);
#pragma unroll
        for (int k = 0; k < kCopyUnroll; ++k) __builtin_nontemporal_store(v[k], &dst[i + k * stride]);
    }
    for (; i < count; i += stride) dst[i] = src[i];
}

__device__ __forceinline__ int xcd_id() {
    unsigned x;
    __asm__ volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
    return (int)(x & 0xF);
}

// Ctrl fields used: stat_cycles = constant-clock ticks of block 0 over all
// rounds, stat_rows = rounds completed, spine_n_e / spine_status = XCD of
// block 0 / of the partner.
__global__ void k_mb_hop(unsigned long long *word, int64_t rounds, int partner, Ctrl *ctrl,
                         int64_t timeout) {
    const bool a = blockIdx.x == 0, b = (int)blockIdx.x == partner;
    if ((!a && !b) || threadIdx.x != 0) return;
    if (a) ctrl->spine_n_e = xcd_id(); else ctrl->spine_status = xcd_id();
    const int64_t t_start = now_ticks();
    int64_t r = 0;
    for (; r < rounds; ++r) {
        const unsigned long long want = a ? 2ull * r : 2ull * r + 1;
        const int64_t t0 = now_ticks();
        bool ok = true;
        while (__hip_atomic_load(word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != want) {
            if (aborted(ctrl)) { ok = false; break; }
            if (now_ticks() - t0 > timeout) {
                record_error(ctrl, DERR_WAIT_TIMEOUT);
                ok = false;
                break;
            }
        }
        if (!ok) return;
        __hip_atomic_store(word, want + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (a) {
        const int64_t t0 = now_ticks();
        while (__hip_atomic_load(word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) !=
               2ull * rounds) {
            if (aborted(ctrl)) return;
            if (now_ticks() - t0 > timeout) {
                record_error(ctrl, DERR_WAIT_TIMEOUT);
                return;
            }
        }
        ctrl->stat_cycles = now_ticks() - t_start;
        ctrl->stat_rows = r;
    }
}

__global__ __launch_bounds__(kBlock) void k_mb_barrier(int64_t rounds, Ctrl *ctrl,
                                                       int64_t timeout) {
    const int64_t t_start = now_ticks();
    int64_t r = 0;
    for (; r < rounds; ++r)
        if (!grid_barrier(ctrl, timeout)) return;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        ctrl->stat_cycles = now_ticks() - t_start;
        ctrl->stat_rows = r;
    }
}

__global__ void k_mb_ctrl_zero(Ctrl *c, unsigned long long *word) {
    int *w = reinterpret_cast<int *>(c);
    for (int i = threadIdx.x; i < (int)(sizeof(Ctrl) / sizeof(int)); i += blockDim.x) w[i] = 0;
    if (threadIdx.x == 0) *word = 0;
}

int clock_khz_now() {
    int dev = 0, khz = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess || khz <= 0)
        khz = 100000;
    return khz;
}

}  // namespace
}  // namespace pdbk

using namespace pdbk;

extern "C" int pdb_mb_workspace_bytes(size_t *bytes) {
    if (!bytes) return PDB_ERR_INVALID_ARG;
    *bytes = kMbWs;
    return PDB_OK;
}

extern "C" int pdb_mb_copy(const void *src, void *dst, size_t bytes, hipStream_t s) {
    if (bytes % 16 != 0) return PDB_ERR_INVALID_ARG;
    if (bytes == 0) return PDB_OK;
    if (!src || !dst || (uintptr_t)src % 16 || (uintptr_t)dst % 16) return PDB_ERR_INVALID_ARG;
    const int64_t count = (int64_t)(bytes / 16);
    int dev = 0, cus = 0;
    PDB_HIP(hipGetDevice(&dev));
    PDB_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
    // eight blocks per compute unit, four chunks per thread in flight: enough
    // outstanding loads to cover HBM latency
    const int grid = grid_for(count, (int64_t)kBlock * kCopyUnroll, (int64_t)std::max(cus, 1) * 8);
    k_mb_copy<<<grid, kBlock, 0, s>>>(static_cast<const u32x4 *>(src), static_cast<u32x4 *>(dst),
                                      count);
    PDB_LAUNCHED();
    return PDB_OK;
}

extern "C" int pdb_mb_hop(int64_t rounds, int32_t partner, void *ws, size_t ws_bytes,
                          double *ns_per_round, int32_t *xcd_a, int32_t *xcd_b,
                          const pdb_options *opt, hipStream_t s) {
    if (!ws || !ns_per_round || !xcd_a || !xcd_b || rounds < 1 || partner < 1 || partner > 1023)
        return PDB_ERR_INVALID_ARG;
    if (ws_bytes < kMbWs) return PDB_ERR_WORKSPACE;
    Opts o;
    int rc = resolve_opts(opt, &o);
    if (rc != PDB_OK) return rc;
    Ctrl *ctrl = static_cast<Ctrl *>(ws);
    unsigned long long *word =
        reinterpret_cast<unsigned long long *>(static_cast<char *>(ws) + 512);
    k_mb_ctrl_zero<<<1, 64, 0, s>>>(ctrl, word);
    PDB_LAUNCHED();
    // cooperative: both players resident at once (each spins on the other)
    int64_t a_rounds = rounds, a_timeout = o.timeout;
    int a_partner = partner;
    void *args[] = {&word, &a_rounds, &a_partner, &ctrl, &a_timeout};
    PDB_HIP(hipLaunchCooperativeKernel(reinterpret_cast<const void *>(&k_mb_hop),
                                       dim3((unsigned)partner + 1), dim3(64), args, 0, s));
    Ctrl host;
    PDB_HIP(hipMemcpyAsync(&host, ctrl, sizeof(Ctrl), hipMemcpyDeviceToHost, s));
    PDB_HIP(hipStreamSynchronize(s));
    if (host.err || host.stat_rows != rounds) return PDB_ERR_DEVICE;
    *ns_per_round = (double)host.stat_cycles * 1e6 / clock_khz_now() / (double)rounds;
    *xcd_a = host.spine_n_e;
    *xcd_b = host.spine_status;
    return PDB_OK;
}

extern "C" int pdb_mb_barrier(int64_t rounds, int32_t blocks, void *ws, size_t ws_bytes,
                              double *ns_per_barrier, const pdb_options *opt, hipStream_t s) {
    if (!ws || !ns_per_barrier || rounds < 1 || blocks < 1) return PDB_ERR_INVALID_ARG;
    if (ws_bytes < kMbWs) return PDB_ERR_WORKSPACE;
    Opts o;
    int rc = resolve_opts(opt, &o);
    if (rc != PDB_OK) return rc;
    Ctrl *ctrl = static_cast<Ctrl *>(ws);
    unsigned long long *word =
        reinterpret_cast<unsigned long long *>(static_cast<char *>(ws) + 512);
    k_mb_ctrl_zero<<<1, 64, 0, s>>>(ctrl, word);
    PDB_LAUNCHED();
    int64_t a_rounds = rounds, a_timeout = o.timeout;
    void *args[] = {&a_rounds, &ctrl, &a_timeout};
    PDB_HIP(hipLaunchCooperativeKernel(reinterpret_cast<const void *>(&k_mb_barrier),
                                       dim3((unsigned)blocks), dim3(kBlock), args, 0, s));
    Ctrl host;
    PDB_HIP(hipMemcpyAsync(&host, ctrl, sizeof(Ctrl), hipMemcpyDeviceToHost, s));
    PDB_HIP(hipStreamSynchronize(s));
    if (host.err || host.stat_rows != rounds) return PDB_ERR_DEVICE;
    *ns_per_barrier = (double)host.stat_cycles * 1e6 / clock_khz_now() / (double)rounds;
    return PDB_OK;
}
