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
//         spine: when one feature is held by all rows but a few, levels
//         along that feature's rows follow from a prefix maximum over the
//         few side inputs from the other rows (see the spine kernels);
//         chain-scan relaxation: along every feature's list the level grows
//         by at least one per step, so a segmented max-scan of
//         (level - position) per feature followed by a max per example
//         raises every lower bound along whole chains in one round; start
//         from 1 and repeat until nothing changes (the least fixed point is
//         the exact level).  Rounds = 1 + chain switches on the critical
//         path: few when one feature dominates every example;
//         dataflow: every example waits for its previous writers' levels
//         (published with device-scope atomics) and publishes its own;
//         batches of consecutive examples are dealt to the resident waves
//         in turn, so the smallest unfinished example always runs.  Time ~
//         critical path length;
//         short-row walk (rows of at most four entries): one block settles
//         64-row sub-chunks in order, each by Jacobi rounds across a wave;
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

// K2: previous writer of every entry from the feature-sorted order: pn[p] =
// the entry just before p in p's feature list (its CSR index), -1 at a head.
// K2 in two streaming passes instead of a scatter.  Scattered 4-byte stores
// of prev_nz in entry order land one per 32-byte sector and wrote 8x the
// array (config 3: 16 GB for 2 GB, 21 ms).  Here:
//   1. k_prev_pairs: in feature order, each entry's previous entry on its
//      feature (the entry before it in the sorted order, when it has the same
//      feature) as an (entry, previous) pair, written in order; col_ptr and
//      csc_row as before;
//   2. the pairs sorted by entry index above its low kPlaceBits bits (the
//      stable radix sort's passes on the high digits only);
//   3. k_prev_place: entry indices are a permutation of 0 .. nnz-1, so block
//      b finds exactly the entries [b 2^kPlaceBits, (b+1) 2^kPlaceBits) at
//      those positions of the sorted pairs; it places their previous entries
//      in LDS and writes the range out in order.
constexpr int kPlaceBits = 13;  // 8192 entries, 32 KB of LDS per block

__global__ __launch_bounds__(kBlock) void k_prev_pairs(
    const uint32_t *__restrict__ skeys, const uint32_t *__restrict__ svals, int64_t nnz,
    int64_t d, const int32_t *__restrict__ row_idx, uint32_t *__restrict__ pk,
    uint32_t *__restrict__ pv, int64_t *__restrict__ col_ptr, int32_t *__restrict__ csc_row) {
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < nnz;
         q += (int64_t)gridDim.x * blockDim.x) {
        const uint32_t f = skeys[q];
        const uint32_t p = svals[q];
        const bool head = (q == 0) || skeys[q - 1] != f;
        pk[q] = p;
        pv[q] = head ? 0xFFFFFFFFu : svals[q - 1];
        if (head) {
            const int64_t lo = (q == 0) ? 0 : (int64_t)skeys[q - 1] + 1;
            const int64_t hi = min((int64_t)f, d - 1);  // columns >= d: malformed input
            for (int64_t g = lo; g <= hi; ++g) col_ptr[g] = q;
        }
        if (q == nnz - 1)
            for (int64_t g = (int64_t)f + 1; g <= d; ++g) col_ptr[g] = nnz;
        if (csc_row) csc_row[q] = row_idx[p];
    }
}

// pv may be pn itself: a block reads all of its range before writing it.
__global__ __launch_bounds__(kBlock) void k_prev_place(const uint32_t *__restrict__ pk,
                                                       const uint32_t *pv, int64_t nnz,
                                                       int32_t *pn) {
    __shared__ int32_t s_prev[1 << kPlaceBits];
    const int64_t base = (int64_t)blockIdx.x << kPlaceBits;
    const int cnt = (int)min((int64_t)1 << kPlaceBits, nnz - base);
    for (int i = threadIdx.x; i < cnt; i += kBlock) {
        const uint32_t off = pk[base + i] - (uint32_t)base;
        if (off < (uint32_t)cnt) s_prev[off] = (int32_t)pv[base + i];
    }
    __syncthreads();
    for (int i = threadIdx.x; i < cnt; i += kBlock) pn[base + i] = s_prev[i];
}

// Previous-writer row of every entry: prev_row[p] = row of pn[p], -1 if none.
__global__ __launch_bounds__(kBlock) void k_prev_row(const int32_t *__restrict__ pn, int64_t nnz,
                                                     const int32_t *__restrict__ row_idx,
                                                     int32_t *__restrict__ prev_row) {
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < nnz;
         p += (int64_t)gridDim.x * blockDim.x) {
        const int32_t q = pn[p];
        prev_row[p] = q < 0 ? -1 : row_idx[q];
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
// Every example waits for its previous writers' levels and publishes its own.
// Batches of kFlowB consecutive examples are dealt to the waves in turn
// (wave k of W runs batches k, k + W, ...), and the whole grid is resident,
// so the smallest unfinished example always runs.  Per batch:
//   1. the batch's row bounds and the previous-writer rows of all its
//      entries go to LDS, with the levels of previous writers outside the
//      batch loaded at the same time (device-scope loads, as levels are
//      published with device-scope stores: a level is written once, so a
//      load sees 0, re-polled later, or the final value);
//   2. lane j owns example j of the batch: it walks its entries from where
//      it stopped, taking known levels and the batch's own examples from
//      LDS, and publishes its level as soon as every writer is known.  No
//      example waits for more than its own writers.  Outside writers not
//      seen yet sit in a list that is re-polled as a whole (all loads in
//      flight at once) before each walk; past the list's capacity the walk
//      polls them itself.
constexpr int kFlowB = 64;             // examples per batch, one per lane
constexpr int kFlowEnt = 64 * 96;      // entries of a batch kept in LDS
constexpr int kFlowPend = 2048;        // outside writers tracked in a re-poll list
constexpr int kFlowWaveLds = kFlowEnt + kFlowB + kFlowPend;  // ints of LDS per wave
constexpr int kFlowUnroll = 8;         // entry chunks whose loads are in flight together
constexpr int kFlowShort = 4;          // longest row resolved by Jacobi rounds
// Entry codes: >= 0 a known level (0: no previous writer); -1 - j the
// batch's example j (j < 64); kPendBase + r an outside writer r whose level
// was not seen yet (r < n <= kFlowMaxN keeps the two ranges apart).
constexpr int kPendBase = INT_MIN;
constexpr int64_t kRowWaveMinAvg = 16;  // mean entries per row from which dataflow runs a wave per example
constexpr int64_t kFlowMaxN = (int64_t)INT_MAX - 128;

// Level of entry e's writer: known, an example of the batch (already
// resolved when this is called), or an outside writer polled until set.
__device__ __forceinline__ bool flow_entry(const int *src, int e, const int *lvb,
                                           const int32_t *level, int *v, Ctrl *ctrl,
                                           int64_t timeout) {
    const int c = src[e];
    if (c >= 0) {
        *v = c;
        return true;
    }
    if (c >= -kFlowB) {
        *v = lvb[-1 - c];
        return true;
    }
    const int64_t t0 = now_ticks();
    int idle = 0;
    while ((*v = __hip_atomic_load(&level[c - kPendBase], __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT)) == 0) {
        if (aborted(ctrl)) return false;
        if (now_ticks() - t0 > timeout) {
            record_error(ctrl, DERR_WAIT_TIMEOUT);
            return false;
        }
        if (++idle < 16) __builtin_amdgcn_s_sleep(1);
        else __builtin_amdgcn_s_sleep(8);
    }
    return true;
}

__global__ __launch_bounds__(kBlock) void k_levels_dataflow(const int64_t *__restrict__ row_ptr,
                                                            const int32_t *__restrict__ prev_row,
                                                            int64_t n, int32_t *level, Ctrl *ctrl,
                                                            int64_t timeout) {
    // per wave (dynamic LDS, kFlowWaveLds ints): entry codes, levels of the
    // batch, the list of entries whose outside writer was not seen yet
    extern __shared__ int g_flow[];
    const int lane = lane_id(), wave = wave_in_block();
    int *src = g_flow + wave * kFlowWaveLds;
    int *lvb = src + kFlowEnt;
    int *pend = lvb + kFlowB;
    // batches dealt to the waves in turn (the launch is cooperative)
    const int64_t fstride = (int64_t)gridDim.x * (kBlock / kWave) * kFlowB;
    int64_t fnext = ((int64_t)blockIdx.x * (kBlock / kWave) + wave) * kFlowB;
    for (;;) {
        const int64_t base = fnext;
        fnext += fstride;
        if (base >= n) return;
        const int cnt = (int)min((int64_t)kFlowB, n - base);
        const bool mine_ok = lane < cnt;
        const int64_t r0 = row_ptr[base + min(lane, cnt)];
        const int64_t r1 = row_ptr[base + min(lane + 1, cnt)];
        const int64_t b0 = __shfl(r0, 0);
        const int64_t E = row_ptr[base + cnt] - b0;
        lvb[lane] = 0;
        if (E > kFlowEnt) {
            // too many entries for LDS: one example at a time, direct reads
            for (int i = 0; i < cnt; ++i) {
                int mx = 0, bad = 0;
                const int64_t p0 = row_ptr[base + i], p1 = row_ptr[base + i + 1];
                for (int64_t p = p0 + lane; p < p1; p += kWave) {
                    const int pr = prev_row[p];
                    if (pr < 0) continue;
                    int v = 0;
                    if (pr >= base) {
                        v = lvb[pr - base];
                    } else {
                        const int64_t t0 = now_ticks();
                        while ((v = __hip_atomic_load(&level[pr], __ATOMIC_RELAXED,
                                                      __HIP_MEMORY_SCOPE_AGENT)) == 0) {
                            if (aborted(ctrl)) { bad = 1; break; }
                            if (now_ticks() - t0 > timeout) {
                                record_error(ctrl, DERR_WAIT_TIMEOUT);
                                bad = 1;
                                break;
                            }
                            __builtin_amdgcn_s_sleep(1);
                        }
                    }
                    mx = max(mx, v);
                }
                if (__ballot(bad) != 0ull) return;
                const int lv = wave_max_dpp(mx) + 1;
                if (lane == 0) {
                    lvb[i] = lv;
                    __hip_atomic_store(&level[base + i], lv, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
                }
            }
            continue;
        }
        // 1. codes of every entry, outside levels loaded with them
        int npend = 0;          // wave-uniform
        bool overflow = false;  // some unseen writer did not fit in the list
        int64_t ninner = 0;     // entries whose writer is in the batch
        for (int64_t e0 = 0; e0 < E; e0 += kWave * kFlowUnroll) {
            int pr[kFlowUnroll], v[kFlowUnroll];
#pragma unroll
            for (int u = 0; u < kFlowUnroll; ++u)
                pr[u] = prev_row[b0 + min(e0 + u * kWave + lane, E - 1)];
#pragma unroll
            for (int u = 0; u < kFlowUnroll; ++u)
                v[u] = __hip_atomic_load(&level[max(pr[u], 0)], __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
            for (int u = 0; u < kFlowUnroll; ++u) {
                const int64_t e = e0 + u * kWave + lane;
                const int code = pr[u] < 0       ? 0
                                 : pr[u] >= base ? -1 - (int)(pr[u] - base)
                                 : v[u] != 0     ? v[u]
                                                 : kPendBase + pr[u];
                if (e < E) src[e] = code;
                const unsigned long long pb = __ballot(e < E && code < -kFlowB);
                const int at = npend + (int)lanes_below(pb);
                if (e < E && code < -kFlowB && at < kFlowPend) pend[at] = (int)e;
                overflow |= npend + __popcll(pb) > kFlowPend;
                npend = min(npend + __popcll(pb), kFlowPend);
                ninner += __popcll(__ballot(e < E && code < 0 && code >= -kFlowB));
            }
        }
        // row bounds of this lane's example inside the batch's entries
        const int my0 = (int)(r0 - b0), my1 = (int)(r1 - b0);
        const int longest = wave_max_dpp(mine_ok ? my1 - my0 : 0);
        const bool chainlike = E >= 8 * (int64_t)cnt && 4 * ninner >= E;
        const bool shortrows = longest <= kFlowShort;
        int64_t t0 = now_ticks();  // last time anything moved
        int idle = 0;
        if (chainlike || shortrows) {
            // 2a. wait for every listed outside writer, re-polling the list as
            // a whole (all loads in flight at once)
            while (npend > 0) {
                int kept = 0;
                for (int k0 = 0; k0 < npend; k0 += kWave * kFlowUnroll) {
                    int ent[kFlowUnroll], v[kFlowUnroll];
#pragma unroll
                    for (int u = 0; u < kFlowUnroll; ++u) {
                        ent[u] = pend[min(k0 + u * kWave + lane, npend - 1)];
                        v[u] = __hip_atomic_load(&level[src[ent[u]] - kPendBase],
                                                 __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    }
#pragma unroll
                    for (int u = 0; u < kFlowUnroll; ++u) {
                        const bool live = k0 + u * kWave + lane < npend;
                        if (live && v[u] != 0) src[ent[u]] = v[u];
                        const unsigned long long kb = __ballot(live && v[u] == 0);
                        if (live && v[u] == 0) pend[kept + (int)lanes_below(kb)] = ent[u];
                        kept += __popcll(kb);
                    }
                }
                if (kept < npend) {
                    t0 = now_ticks();
                    idle = 0;
                } else {
                    if (aborted(ctrl)) return;
                    if (now_ticks() - t0 > timeout) {
                        record_error(ctrl, DERR_WAIT_TIMEOUT);
                        return;
                    }
                    if (++idle < 16) __builtin_amdgcn_s_sleep(1);
                    else __builtin_amdgcn_s_sleep(8);
                }
                npend = kept;
            }
            // outside writers that did not fit in the list: waited for in
            // place (flow_entry)
            if (chainlike) {
                // 2b. chain-like batch (long rows, many writers inside the
                // batch): one example at a time, the whole wave over its entries
                for (int i = 0; i < cnt; ++i) {
                    const int o0 = __builtin_amdgcn_readlane(my0, i);
                    const int o1 = __builtin_amdgcn_readlane(my1, i);
                    int mx = 0, bad = 0;
                    for (int e = o0 + lane; e < o1; e += kWave) {
                        int v = 0;
                        if (!flow_entry(src, e, lvb, level, &v, ctrl, timeout)) bad = 1;
                        mx = max(mx, v);
                    }
                    if (__ballot(bad) != 0ull) return;
                    const int lv = wave_max_dpp(mx) + 1;
                    if (lane == 0) {
                        lvb[i] = lv;
                        __hip_atomic_store(&level[base + i], lv, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
                    }
                }
            } else {
                // 2c. short rows (matrix completion): lane j holds example j;
                // Jacobi rounds from the outside bounds until nothing changes
                int known = 0, nin = 0, bad = 0;
                int pin[kFlowShort];
                for (int k = 0; k < kFlowShort; ++k) {
                    pin[k] = 0;
                    if (mine_ok && my0 + k < my1) {
                        const int c = src[my0 + k];
                        if (c < 0 && c >= -kFlowB) {
                            pin[nin++] = -1 - c;
                        } else {
                            int v = 0;
                            if (!flow_entry(src, my0 + k, lvb, level, &v, ctrl, timeout)) bad = 1;
                            known = max(known, v);
                        }
                    }
                }
                if (__ballot(bad) != 0ull) return;
                int lv = known + 1;
                lvb[lane] = mine_ok ? lv : 0;
                for (;;) {
                    int nl = known + 1;
                    for (int k = 0; k < kFlowShort; ++k)
                        if (k < nin) nl = max(nl, lvb[pin[k]] + 1);
                    const bool ch = mine_ok && nl != lv;
                    lv = nl;
                    if (mine_ok) lvb[lane] = lv;
                    if (__ballot(ch) == 0ull) break;
                }
                if (mine_ok)
                    __hip_atomic_store(&level[base + lane], lv, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
            }
            continue;
        }
        // 2d. otherwise (wide levels) lane j resolves example j and publishes
        // it as soon as its own writers are known.  First one pass over its
        // row: known levels fold into kmax, the other entries are compacted
        // to the front of the row's own range.
        int kmax = 0, nun = 0;
        for (int e = my0; e < my1; e += 4) {
            int c[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) c[u] = src[min(e + u, my1 - 1)];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                if (e + u >= my1) continue;
                if (c[u] >= 0) kmax = max(kmax, c[u]);
                else src[my0 + nun++] = c[u];
            }
        }
        bool done = !mine_ok;
        for (;;) {
            bool moved = false;
            if (!done) {
                // every remaining writer: batch examples from LDS, outside
                // ones polled, four requests in flight at a time
                int keep = 0;
                for (int k = 0; k < nun; k += 4) {
                    int c[4], v[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        c[u] = src[my0 + min(k + u, nun - 1)];
                        v[u] = c[u] >= -kFlowB ? lvb[-1 - c[u]]
                                               : __hip_atomic_load(&level[c[u] - kPendBase],
                                                                   __ATOMIC_RELAXED,
                                                                   __HIP_MEMORY_SCOPE_AGENT);
                    }
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        if (k + u >= nun) continue;
                        if (v[u] != 0) kmax = max(kmax, v[u]);
                        else src[my0 + keep++] = c[u];
                    }
                }
                moved = keep < nun;
                nun = keep;
                if (nun == 0) {
                    lvb[lane] = kmax + 1;
                    __hip_atomic_store(&level[base + lane], kmax + 1, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
                    done = true;
                    moved = true;
                }
            }
            if (__ballot(!done) == 0ull) break;
            if (__ballot(moved) == 0ull) {
                if (aborted(ctrl)) return;
                if (now_ticks() - t0 > timeout) {
                    record_error(ctrl, DERR_WAIT_TIMEOUT);
                    return;
                }
                if (++idle < 16) __builtin_amdgcn_s_sleep(1);
                else __builtin_amdgcn_s_sleep(8);
            } else {
                t0 = now_ticks();
                idle = 0;
            }
        }
    }
}

// Dataflow with a wave per example, for inputs with long rows and wide
// levels (not chain-like: many examples share nothing with the one before).
// Examples are dealt to the waves in turn (cooperative launch); a wave polls
// the published levels of all writer rows of up to 2 x 64 entries at once
// and publishes 1 + their maximum.  Beside the batch form it spends no time
// on batch-mates: an example waits only for its own writers.
// Writer rows are looked up here (row_idx of the previous-writer entry)
// rather than gathered by a pass of their own: an example's lookups happen
// while it waits for its turn, off the dependence chain.
__global__ __launch_bounds__(kBlock) void k_levels_rowwave(const int64_t *__restrict__ row_ptr,
                                                           const int32_t *__restrict__ prev_nz,
                                                           const int32_t *__restrict__ row_idx,
                                                           int64_t n, int32_t *level, Ctrl *ctrl,
                                                           int64_t timeout) {
    const int lane = lane_id();
    const int64_t nw = (int64_t)gridDim.x * (kBlock / kWave);
    for (int64_t a = (int64_t)blockIdx.x * (kBlock / kWave) + wave_in_block(); a < n; a += nw) {
        const int64_t b = row_ptr[a], m = row_ptr[a + 1] - b;
        int mx = 0;
        for (int64_t k0 = 0; k0 < m; k0 += 2 * kWave) {
            const bool l0 = k0 + lane < m, l1 = k0 + kWave + lane < m;
            const int e0 = l0 ? prev_nz[b + k0 + lane] : -1;
            const int e1 = l1 ? prev_nz[b + k0 + kWave + lane] : -1;
            const int p0 = e0 >= 0 ? row_idx[e0] : -1;
            const int p1 = e1 >= 0 ? row_idx[e1] : -1;
            int v0 = 0, v1 = 0;
            bool r0 = p0 < 0, r1 = p1 < 0;
            int64_t t0 = 0;
            for (int round = 0;; ++round) {
                if (!r0) v0 = __hip_atomic_load(&level[p0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (!r1) v1 = __hip_atomic_load(&level[p1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                r0 |= v0 != 0;
                r1 |= v1 != 0;
                if (__ballot(!(r0 && r1)) == 0ull) break;
                if (round == 0) t0 = now_ticks();
                // the abort flag (a device-scope load) and the watchdog
                // every 64 rounds (a waiter reading the flag when its
                // writer's level lands sees it a load later; every 8 rounds
                // cost config 4 0.5 ms), a short back-off every round
                if ((round & 63) == 63) {
                    if (aborted(ctrl)) return;
                    if (now_ticks() - t0 > timeout) {
                        record_error(ctrl, DERR_WAIT_TIMEOUT);
                        return;
                    }
                }
                __builtin_amdgcn_s_sleep(1);
            }
            mx = max(mx, max(v0, v1));
        }
        const int lv = wave_max_dpp(mx) + 1;
        if (lane == 0) __hip_atomic_store(&level[a], lv, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// ---- K3r short-row walk --------------------------------------------------
// One block walks the examples in sub-chunks of 64 consecutive rows, one row
// per lane, for inputs whose rows hold at most kShortR entries (matrix
// completion: a user and an item).  The sub-chunks are settled strictly in
// order, kShortPer consecutive ones per turn of a wave: turn t (sub-chunks
// kShortPer t ...) belongs to wave t mod kShortWaves, and the turns are
// handed on by an LDS counter (s_done = number of settled sub-chunks).
// Settling sub-chunk q (kShortPer = short_per<R>()):
//   known(i) = max level of i's writers before q (the last kShortRing
//              sub-chunks from an LDS ring, older ones loaded from global
//              memory a turn of every wave ahead);
//   level(i) = 1 + max(known(i), level(in-q writers)), the fixed point of
//              Jacobi rounds across the wave's lanes, one round per link of
//              the longest chain inside q (counted from the structure while
//              the wave waits for its turn).
// A round is a lane shuffle, where waiting on another workgroup's published
// level costs a device-scope round trip; a hand-over from wave to wave costs
// about a third of a sub-chunk's settling, hence several sub-chunks a turn.
// Visibility of the global levels: a wave waits for its own earlier stores
// (a workgroup-scope release) before it settles a turn, so once s_done has
// passed the first sub-chunk of turn u + kShortWaves the stores of turn u
// are complete.  A wave loads the global levels of turn t + kShortWaves
// right after settling turn t, and only of writers kShortRing sub-chunks or
// more before them: kShortRing >= 2 kShortWaves kShortPer puts those writers
// kShortWaves turns or more behind turn t.  A row with more than kShortR
// entries sets ctrl->bad and stops the block (the host then runs dataflow);
// every wait is bounded by the spin budget.
constexpr int kShortWaves = 16;
constexpr int kShortThreads = kShortWaves * 64;
constexpr int kShortR = 4;
constexpr int kShortRing = 256;  // sub-chunks whose levels stay in LDS
// sub-chunks a wave settles per turn (fewer for rows of up to kShortR
// entries, whose per-row state would otherwise spill registers)
template <int R>
constexpr int short_per() {
    return R <= 2 ? 8 : 4;
}
static_assert(kShortRing >= 2 * kShortWaves * short_per<2>() &&
                  kShortRing >= 2 * kShortWaves * short_per<kShortR>(),
              "loads of levels too recent");

// an LDS word by its byte address, so that which word a lane reads can be
// settled before the read, as plain data in a register
typedef __attribute__((address_space(3))) int lds_i32;
__device__ __forceinline__ int lds_addr(const int *p) {
    return (int)(uintptr_t)(const lds_i32 *)p;
}
__device__ __forceinline__ int lds_read_i32(int a) {
    return *(const lds_i32 *)(uintptr_t)(unsigned)a;
}

template <int R>
struct ShortRow {
    int m;        // entries (R + 1 stands for more)
    int pr[R];    // previous-writer rows, -1 none
    int v[R];     // levels of writers before row `old`, else 0
};

// row r0 + lane; levels of writers before `old` are final and visible
template <int R>
__device__ __forceinline__ ShortRow<R> short_fetch(const int64_t *__restrict__ row_ptr,
                                                const int32_t *__restrict__ prev_row,
                                                const int32_t *level, int64_t n, int64_t r0,
                                                int64_t old) {
    ShortRow<R> r;
    const int64_t i = r0 + lane_id();
    int64_t b0 = 0, b1 = 0;
    if (i < n) {
        b0 = row_ptr[i];
        b1 = row_ptr[i + 1];
    }
    r.m = (int)min(b1 - b0, (int64_t)R + 1);
#pragma unroll
    for (int k = 0; k < R; ++k) r.pr[k] = k < r.m ? prev_row[b0 + k] : -1;
#pragma unroll
    for (int k = 0; k < R; ++k) r.v[k] = (r.pr[k] >= 0 && r.pr[k] < old) ? level[r.pr[k]] : 0;
    return r;
}

template <int R>
__global__ __launch_bounds__(kShortThreads) void k_levels_short(const int64_t *__restrict__ row_ptr,
                                                                const int32_t *__restrict__ prev_row,
                                                                int64_t n, int32_t *level,
                                                                Ctrl *ctrl, int64_t timeout) {
    constexpr int kShortPer = short_per<R>();
    __shared__ int s_ring[kShortRing][64];
    __shared__ int s_done, s_stop, s_zero;
    const int lane = lane_id(), wave = wave_in_block();
    if (threadIdx.x == 0) {
        s_done = 0;
        s_stop = 0;
        s_zero = 0;
    }
    __syncthreads();
    const int64_t nsub = (n + 63) / 64;
    int64_t t = wave;  // this wave's turn
    if (kShortPer * t >= nsub) return;
    ShortRow<R> cur[kShortPer];
    auto fetch_turn = [&](int64_t u) {
#pragma unroll
        for (int j = 0; j < kShortPer; ++j) {
            const int64_t q = kShortPer * u + j;  // past the end: rows >= n, nothing loaded
            cur[j] = short_fetch<R>(row_ptr, prev_row, level, n, 64 * q, 64 * (q - kShortRing));
        }
    };
    fetch_turn(t);
    for (; kShortPer * t < nsub; t += kShortWaves) {
        const int64_t q0 = kShortPer * t;
        const int nq = (int)min((int64_t)kShortPer, nsub - q0);
        // this wave's earlier stores complete before it settles the turn (see above)
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        bool long_row = false;
#pragma unroll
        for (int j = 0; j < kShortPer; ++j) long_row = long_row || cur[j].m > R;
        if (__ballot(long_row) != 0ull) {
            if (lane == 0) {
                ctrl->bad = 1;
                __hip_atomic_store(&s_stop, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            }
            return;
        }
        // before the wait, from the structure alone: each row's writers
        // inside its sub-chunk (as a lane-shuffle address, and an increment
        // that is 1 for a writer and far below any level for none) and the
        // sub-chunk's depth, the most links on a chain of such writers -- the
        // settling then runs exactly that many Jacobi rounds; also the LDS
        // address of each writer's ring slot (a zero word when the writer is
        // not in the ring window) and the largest level of older writers
        int sha[kShortPer][R], inc[kShortPer][R], rad[kShortPer][R], old[kShortPer],
            depth[kShortPer];
#pragma unroll
        for (int j = 0; j < kShortPer; ++j) {
            const int64_t r0 = 64 * (q0 + j), ring0 = r0 - 64 * kShortRing;
            int bk = 0;
#pragma unroll
            for (int k = 0; k < R; ++k) {
                const int p = cur[j].pr[k];  // -1: no writer, or past the row's end
                const bool in = p >= r0;
                sha[j][k] = (in ? (int)(p - r0) : lane) * 4;
                inc[j][k] = in ? 1 : -(1 << 30);
                const bool ring = p >= 0 && p >= ring0 && p < r0;
                rad[j][k] = ring ? lds_addr(&s_ring[(p >> 6) & (kShortRing - 1)][p & 63])
                                 : lds_addr(&s_zero);
                if (p >= 0 && p < ring0) bk = max(bk, cur[j].v[k]);
            }
            old[j] = bk;
            // computed now, while the wave waits, and kept: the compiler
            // would otherwise redo the tests on the serial path after the wait
#pragma unroll
            for (int k = 0; k < R; ++k)
                __asm__ volatile("" : "+v"(rad[j][k]), "+v"(sha[j][k]), "+v"(inc[j][k]));
            __asm__ volatile("" : "+v"(old[j]));
            int d = 0;
            for (;;) {
                int nd = 0;
#pragma unroll
                for (int k = 0; k < R; ++k)
                    nd = max(nd, __builtin_amdgcn_ds_bpermute(sha[j][k], d) + inc[j][k]);
                const bool ch = nd != d;
                d = nd;
                if (__ballot(ch) == 0ull) break;
            }
            depth[j] = __builtin_amdgcn_readfirstlane(wave_max_dpp(d));
        }
        // wait for the sub-chunks before the turn: far from its turn a wave
        // sleeps between polls; the next in line polls s_done alone, and
        // looks at the stop flag and the clock every 32nd poll
        const int64_t t0 = now_ticks();
        for (int it = 1;; ++it) {
            const int dn = __hip_atomic_load(&s_done, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            if (dn == (int)q0) break;
            if ((int)q0 - dn > kShortPer) {
                __builtin_amdgcn_s_sleep(8);
                it = 0;
            }
            if ((it & 31) == 0) {
                if (__hip_atomic_load(&s_stop, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)) return;
                if (now_ticks() - t0 > timeout) {
                    if (lane == 0) {
                        record_error(ctrl, DERR_WAIT_TIMEOUT);
                        __hip_atomic_store(&s_stop, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                    }
                    return;
                }
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
        __builtin_amdgcn_s_setprio(3);  // the block waits on this wave: issue it first
        int lvs[kShortPer];
#pragma unroll
        for (int j = 0; j < kShortPer; ++j) {
            lvs[j] = 0;
            if (j >= nq) continue;
            // the ring reads (sub-chunks settled earlier in this turn are in
            // the ring already: one wave's LDS operations run in order)
            int known = old[j];
#pragma unroll
            for (int k = 0; k < R; ++k) known = max(known, lds_read_i32(rad[j][k]));
            // after r rounds every chain of at most r links inside the
            // sub-chunk has been followed: depth[j] rounds reach the fixed point
            const int base = known + 1;
            int lv = base;
            for (int round = 0; round < depth[j]; ++round) {
                int nl = base;
#pragma unroll
                for (int k = 0; k < R; ++k)
                    nl = max(nl, __builtin_amdgcn_ds_bpermute(sha[j][k], lv) + inc[j][k]);
                lv = nl;
            }
            s_ring[(q0 + j) & (kShortRing - 1)][lane] = lv;
            lvs[j] = lv;
        }
        __asm__ __volatile__("" ::: "memory");  // one wave's LDS operations run in order
        if (lane == 0)
            __hip_atomic_store(&s_done, (int)(q0 + nq), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        __builtin_amdgcn_s_setprio(0);
#pragma unroll
        for (int j = 0; j < kShortPer; ++j) {
            const int64_t r = 64 * (q0 + j) + lane;
            if (j < nq && r < n) level[r] = lvs[j];
        }
        // the wave's next turn: writers before its ring window were settled
        // at least kShortWaves turns before this one
        if (kShortPer * (t + kShortWaves) < nsub) fetch_turn(t + kShortWaves);
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

// ---- K3 walk ---------------------------------------------------------------
// Chain-like inputs, where most examples share a feature with the one before
// them: the dependency chain is about as long as the data, so one block
// walks the rows in order instead of crossing CUs per row.  Rows go in
// windows of at most kWalkRows rows and kWalkEnt entries.
//
// A run is a maximal stretch of rows each of which has the row before it as
// a previous writer.  Along a run levels rise by at least one per row, so a
// writer inside the run other than the row just before can never set a
// level: for row i of a run starting at a, with M_i the largest level among
// its writers before a,
//   level(a) = 1 + M_a,  level(i) = max(level(i-1), M_i) + 1,
// that is level(i) = i + 1 + max over a <= t <= i of (M_t - t): a prefix
// maximum.  The block stages a window (per entry: a writer before the window
// is folded into its row's M at once, from the levels already written or,
// for the window before, from LDS; a writer in the window is kept as a row
// index; the writer just before marks the row as continuing a run).  Then
// the window's runs go in order: the block folds the levels of writers in
// earlier runs into the run's M (one thread per entry), and wave 0 turns
// them into levels by a prefix maximum over 64 rows at a time.
constexpr int kWalkRows = 512;
constexpr int kWalkEnt = 16384;
constexpr int kWalkThreads = 1024;
constexpr int kWalkPer = kWalkEnt / kWalkThreads;  // entries per thread

struct WalkShared {
    int16_t ref[kWalkEnt];   // a writer in the window: its row; -1: none or already folded
    int16_t row[kWalkEnt];   // the entry's row in the window
    int16_t runs[kWalkRows + 1];  // first rows of the runs, then nr
    int nruns;
    int m[kWalkRows];        // largest level among the row's writers before the window
    int chain[kWalkRows];    // 1 when the row just before is one of the row's writers
    int rp[2][kWalkRows + 1];  // row bounds relative to a window's first entry (this, next)
    int lvl[2][kWalkRows];   // levels of this window and the previous one
    int nrows;               // rows of the next window
};

__device__ __forceinline__ int wave_prefix_max(int v) {
    const int l = lane_id();
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int t = __shfl_up(v, off);
        if (l >= off) v = max(v, t);
    }
    return v;
}

// Row bounds of the window starting at row r0 into S.rp[slot] (relative to
// its first entry), and its row count (as many rows as fit kWalkEnt
// entries) into S.nrows; S.nrows must be 0 beforehand.  One load per thread.
__device__ __forceinline__ void walk_bounds(const int64_t *__restrict__ row_ptr, int64_t n,
                                            int64_t r0, int64_t q0, int64_t rpt, WalkShared &S,
                                            int slot) {
    // the rows that fit are a prefix (row bounds never decrease): count them
    const int t = threadIdx.x;
    const int64_t rel = rpt - q0;
    const bool fits = t >= 1 && t <= kWalkRows && r0 + t <= n && rel <= kWalkEnt;
    if (t <= kWalkRows) S.rp[slot][t] = (int)min<int64_t>(rel, INT_MAX);
    const int c = __popcll(__ballot(fits));
    if (lane_id() == 0 && c > 0) atomicAdd(&S.nrows, c);
}

// A block barrier for LDS only: global loads may stay in flight across it
// (__syncthreads would wait for them).
__device__ __forceinline__ void lds_barrier() {
    __asm__ __volatile__("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    __asm__ __volatile__("" ::: "memory");
}

__global__ __launch_bounds__(kWalkThreads) void k_levels_walk(const int64_t *__restrict__ row_ptr,
                                                              int64_t n,
                                                              const int32_t *__restrict__ prow,
                                                              const int32_t *__restrict__ row_idx,
                                                              int32_t *__restrict__ level,
                                                              Ctrl *ctrl) {
    __shared__ WalkShared S;
    const int tid = threadIdx.x, lane = lane_id();
    constexpr int kNone = INT_MIN / 2;
    // The next window's row bounds and entries are loaded while the current
    // one is staged and solved: what a window loads does not depend on
    // earlier windows' levels, only the levels of writers before it do.
    int64_t r0 = 0, r0p = 0;  // first rows of this and the previous window
    int cur = 0, cb = 0;      // level buffer, row-bound buffer of this window
    if (tid == 0) S.nrows = 0;
    __syncthreads();
    int64_t q0 = row_ptr[0];
    walk_bounds(row_ptr, n, 0, q0, tid <= kWalkRows ? row_ptr[min((int64_t)tid, n)] : 0, S, 0);
    __syncthreads();
    int nr = S.nrows;
    int32_t pr[kWalkPer], row[kWalkPer], lvf[kWalkPer];
    auto load_entries = [&](int64_t wr0, int64_t wq0, int wE) {
#pragma unroll
        for (int u = 0; u < kWalkPer; ++u) {
            const int e = tid + u * kWalkThreads;
            const int64_t q = wq0 + min(e, max(wE - 1, 0));
            // raw rows: subtracting the window's first row here would wait
            // for the load; the staging does it
            pr[u] = e < wE ? prow[q] : -1;
            row[u] = e < wE ? row_idx[q] : (int32_t)wr0;
        }
    };
    if (nr > 0) load_entries(0, q0, S.rp[0][nr]);
#pragma unroll
    for (int u = 0; u < kWalkPer; ++u) lvf[u] = 0;  // no writers before the first window
    while (r0 < n) {
        if (nr == 0) {  // one row longer than a window: the caller uses another method
            if (tid == 0) ctrl->bad = 1;
            return;
        }
        const int E = S.rp[cb][nr];
        int *lc = S.lvl[cur];
        const int *lp = S.lvl[cur ^ 1];
        // lvf: levels of writers before the previous window, loaded during
        // the previous window; now the next window's row bounds
        const int64_t r0n = r0 + nr;
        const int64_t q0n = q0 + E;
        const int64_t rpn = tid <= kWalkRows ? row_ptr[min(r0n + tid, n)] : 0;
        if (tid < kWalkRows) {
            S.m[tid] = 0;
            S.chain[tid] = 0;
        }
        if (tid == 0) S.nrows = 0;
        lds_barrier();
        // stage this window
#pragma unroll
        for (int u = 0; u < kWalkPer; ++u) {
            const int e = tid + u * kWalkThreads;
            if (e < E) {
                int16_t ref = -1;
                const int rw = row[u] - (int32_t)r0;  // the entry's row in the window
                S.row[e] = (int16_t)rw;
                const int32_t p = pr[u];
                if (p >= r0) {
                    if (p == r0 + rw - 1) S.chain[rw] = 1;
                    else ref = (int16_t)(p - r0);
                } else if (p >= 0) {
                    atomicMax(&S.m[rw], p >= r0p ? lp[p - r0p] : lvf[u]);
                }
                S.ref[e] = ref;
            }
        }
        walk_bounds(row_ptr, n, r0n, q0n, rpn, S, cb ^ 1);
        lds_barrier();
        // the next window's entries, in flight while this one is solved
        const int nrn = S.nrows;
        if (r0n < n && nrn > 0) load_entries(r0n, q0n, S.rp[cb ^ 1][nrn]);
        // the runs' first rows (wave 0)
        if (tid < kWave) {
            int cnt = 0;
            for (int c0 = 0; c0 < nr; c0 += kWave) {
                const int j = c0 + lane;
                const bool st = j < nr && S.chain[j] == 0;
                const unsigned long long m = __ballot(st);
                if (st) S.runs[cnt + (int)lanes_below(m)] = (int16_t)j;
                cnt += __popcll(m);
            }
            if (lane == 0) {
                S.runs[cnt] = (int16_t)nr;
                S.nruns = cnt;
            }
        }
        lds_barrier();
        const int nruns = S.nruns;
        for (int k = 0; k < nruns; ++k) {
            const int a = S.runs[k], b = S.runs[k + 1];
            // writers in earlier runs of the window
            for (int e = S.rp[cb][a] + tid; e < S.rp[cb][b]; e += kWalkThreads) {
                const int r = S.ref[e];
                if (r >= 0 && r < a) atomicMax(&S.m[S.row[e]], lc[r]);
            }
            lds_barrier();
            // level(j) = j + 1 + max over a <= t <= j of (M_t - t)
            if (tid < kWave) {
                int carry = kNone;
                for (int c0 = a; c0 < b; c0 += kWave) {
                    const int j = c0 + lane;
                    const int pm = max(wave_prefix_max(j < b ? S.m[j] - j : kNone), carry);
                    if (j < b) lc[j] = j + 1 + pm;
                    carry = __shfl(pm, kWave - 1);
                }
            }
            lds_barrier();
        }
        // every load and store of the block done: the next window's
        // entries are in registers, the levels of earlier windows in memory
        __syncthreads();
        // the next window's writers before this window: their levels are
        // final (stored by this block before at least one barrier)
#pragma unroll
        for (int u = 0; u < kWalkPer; ++u) lvf[u] = (pr[u] >= 0 && pr[u] < r0) ? level[pr[u]] : 0;
        for (int i = tid; i < nr; i += kWalkThreads) level[r0 + i] = lc[i];
        r0p = r0;
        r0 = r0n;
        q0 = q0n;
        nr = nrn;
        cb ^= 1;
        cur ^= 1;
    }
}

// ---- K3 walk over few runs ---------------------------------------------------
// When a chain-like input has few runs (a run: rows each of which has the row
// before it as a previous writer), a grid settles the runs one after another
// instead of one block walking every window.  With M_t the largest level
// among row t's writers before the run's first row a (0 if none), the walk's
// prefix maximum gives level(j) = j + 1 + max over a <= t <= j of (M_t - t):
// writers inside the run never decide a level, since levels rise by one at
// least along it.  Each block owns a stretch of every run's rows, and a run
// takes one device barrier: each block raises M of its stretch's rows from
// their entries whose writer lies before the run (atomic maxima in LDS,
// 8192 rows at a time), scans the stretch -- prefix maxima of M_t - t,
// staged -- and publishes the stretch's maximum.  After the barrier every
// block forms the maxima of the stretches before each stretch; its levels
// are written at the start of the next run, whose gathers therefore form
// the level of a writer in the run just settled from that run's staged
// prefix maxima and stretch maxima.
constexpr int kRunThreads = 1024;
constexpr int kRunBlocks = 16;
constexpr int64_t kRunRowsPer = 512;  // at most one run per this many rows
constexpr int64_t kRunMinN = 65536;
constexpr int kRunChunk = 8192;  // rows whose M one block gathers in LDS at a time
constexpr int kRunPer = 8;       // entries a thread gathers at a time

// flag[i] = 1 when row i starts a run (no entry's previous writer in row i - 1)
__global__ __launch_bounds__(kBlock) void k_run_flags(const int64_t *__restrict__ row_ptr, int64_t n,
                                                      const int32_t *__restrict__ pn,
                                                      uint32_t *__restrict__ flag) {
    const int lane = lane_id();
    const int64_t nw = (int64_t)gridDim.x * (kBlock / kWave);
    for (int64_t i = blockIdx.x * (int64_t)(kBlock / kWave) + wave_in_block(); i < n; i += nw) {
        bool found = false;
        if (i > 0) {
            const int64_t lo = row_ptr[i - 1], b = row_ptr[i], e = row_ptr[i + 1];
            for (int64_t p = b + lane; p < e && !found; p += kWave) found = pn[p] >= lo;
        }
        const bool cont = __ballot(found) != 0ull;
        if (lane == 0) flag[i] = cont ? 0u : 1u;
    }
}

// starts[r] = first row of run r (pos: the exclusive scan of the flags, R runs),
// starts[R] = n
__global__ __launch_bounds__(kBlock) void k_run_starts(const uint32_t *__restrict__ pos, int64_t n,
                                                       int64_t R, int32_t *__restrict__ starts) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t next = i + 1 < n ? (int64_t)pos[i + 1] : R;
        if (next > (int64_t)pos[i]) starts[pos[i]] = (int32_t)i;
        if (i == n - 1) starts[R] = (int32_t)n;
    }
}

// Device barrier on an arrival counter that only grows (target: blocks times
// barriers so far); the host clears it afterwards.  The watchdog is read
// after the first poll and every 16th after it, the abort flag every 16th.
__device__ __forceinline__ bool runs_barrier(Ctrl *c, unsigned target, int64_t timeout) {
    __shared__ int ok_s;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    __syncthreads();
    if (threadIdx.x == 0) {
        int ok = 1;
        __hip_atomic_fetch_add(&c->bar_count, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        const int64_t t0 = now_ticks();
        for (int it = 1;
             __hip_atomic_load(&c->bar_count, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) < target;
             ++it) {
            if ((it & 15) == 1 && now_ticks() - t0 > timeout) {
                record_error(c, DERR_BARRIER_TIMEOUT);
                ok = 0;
                break;
            }
            if ((it & 15) == 0 && aborted(c)) {
                ok = 0;
                break;
            }
        }
        ok_s = ok;
    }
    __syncthreads();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    return ok_s != 0;
}

__global__ __launch_bounds__(kRunThreads) void k_levels_runs(
    const int64_t *__restrict__ row_ptr, const int32_t *__restrict__ prow,
    const int32_t *__restrict__ row_idx, int64_t R, const int32_t *__restrict__ starts,
    int32_t *stg, int32_t *level, int32_t *bmax, Ctrl *ctrl, int64_t timeout) {
    constexpr int kNone = INT_MIN / 2;
    __shared__ int s_m[kRunChunk];  // M_t of a chunk of this block's stretch
    __shared__ int s_w[kRunThreads / kWave];
    __shared__ int s_pre[kWave];  // the run just settled: max of the stretch maxima before each
    const int tid = threadIdx.x, lane = lane_id(), wave = wave_in_block();
    const int G = (int)gridDim.x, j = (int)blockIdx.x;
    unsigned target = 0;
    int64_t pa = 0, ps = 1, plo = 0, phi = 0;  // the run just settled, its span, this block's stretch
    for (int64_t k = 0; k <= R; ++k) {
        // levels of this block's stretch of the run just settled
        if (k > 0) {
            const int before = s_pre[j];
            for (int64_t t = plo + tid; t < phi; t += kRunThreads)
                level[t] = (int)t + 1 + max(before, stg[t]);
        }
        if (k == R) break;
        const int64_t a = starts[k], b = starts[k + 1];
        const int64_t span = (b - a + G - 1) / G;
        const int64_t lo = min(b, a + (int64_t)j * span), hi = min(b, lo + span);
        // this block's stretch, in chunks of rows: M_t from the writers before
        // the run (their levels are final, or formed from the run just
        // settled), then prefix maxima of M_t - t, staged
        int carry = kNone;
        for (int64_t c0 = lo; c0 < hi; c0 += kRunChunk) {
            const int64_t c1 = min(hi, c0 + (int64_t)kRunChunk);
            for (int i = tid; i < (int)(c1 - c0); i += kRunThreads) s_m[i] = 0;
            __syncthreads();
            // kRunPer entries a thread at a time, every load issued before
            // the first is used (the writers' level and staged value both
            // loaded, from row 0 when there is no writer before the run)
            const int64_t e1 = row_ptr[c1];
            for (int64_t p0 = row_ptr[c0] + tid; p0 < e1; p0 += kRunPer * kRunThreads) {
                int32_t w[kRunPer], r[kRunPer];
#pragma unroll
                for (int u = 0; u < kRunPer; ++u) {
                    const int64_t p = p0 + (int64_t)u * kRunThreads;
                    const bool in = p < e1;
                    w[u] = in ? prow[min(p, e1 - 1)] : -1;
                    r[u] = row_idx[min(p, e1 - 1)];
                }
                int lv[kRunPer], sv[kRunPer];
#pragma unroll
                for (int u = 0; u < kRunPer; ++u) {
                    const bool before = w[u] >= 0 && w[u] < a;
                    const int32_t q = before ? w[u] : 0;
                    lv[u] = level[q];
                    sv[u] = stg[q];
                }
#pragma unroll
                for (int u = 0; u < kRunPer; ++u) {
                    if (w[u] >= 0 && w[u] < a) {
                        const int lw = (k > 0 && w[u] >= pa)
                                           ? w[u] + 1 + max(s_pre[(int)((w[u] - pa) / ps)], sv[u])
                                           : lv[u];
                        atomicMax(&s_m[r[u] - (int)c0], lw);
                    }
                }
            }
            __syncthreads();
            for (int64_t s0 = c0; s0 < c1; s0 += kRunThreads) {
                const int64_t t = s0 + tid;
                int pm = wave_prefix_max(t < c1 ? s_m[t - c0] - (int)t : kNone);
                if (lane == kWave - 1) s_w[wave] = pm;
                __syncthreads();
                int before = carry, all = carry;
#pragma unroll
                for (int w2 = 0; w2 < kRunThreads / kWave; ++w2) {
                    if (w2 < wave) before = max(before, s_w[w2]);
                    all = max(all, s_w[w2]);
                }
                if (t < c1) stg[t] = max(pm, before);
                __syncthreads();
                carry = all;
            }
        }
        if (tid == 0) bmax[(k & 1) * kWave + j] = carry;
        target += (unsigned)G;
        if (!runs_barrier(ctrl, target, timeout)) return;
        // the maxima of the stretches before each stretch of this run
        if (wave == 0) {
            const int v = lane < G ? bmax[(k & 1) * kWave + lane] : kNone;
            const int incl = wave_prefix_max(v);
            const int excl = __shfl_up(incl, 1);
            s_pre[lane] = lane == 0 ? kNone : excl;
        }
        __syncthreads();
        pa = a;
        ps = span;
        plo = lo;
        phi = hi;
    }
}

// ---- K3 spine --------------------------------------------------------------
// When one feature f* is held by all rows but a few (the exceptional rows E),
// the rows holding it form a spine c_0 < c_1 < ... < c_{K-1}.  Consecutive
// spine rows share f*, so level(c_k) >= level(c_{k-1}) + 1; a previous writer
// of c_k that lies on the spine is some c_j, j < k, whose level is below
// level(c_{k-1}), so it cannot raise level(c_k).  Only previous writers in E
// can, through side edges e -> c_j (e's entry on some feature is followed in
// that feature's list by c_j's).  Hence
//   level(c_k) = k + M(k),
//   M(k) = max(1, max over side edges e -> c_j with j <= k of level(e) + 1 - j),
// and level(e) = 1 + max over e's previous writers (spine rows by the first
// formula, exceptional rows directly).  Starting from level(e) = 1 and
// applying both formulas repeatedly raises lower bounds to the least fixed
// point, the exact levels, in at most |E| + 1 rounds.  One block does this on
// the exceptional rows; a grid pass then writes the spine's levels.
constexpr int kSpineMaxE = 1024;    // exceptional rows
constexpr int kSpineMaxEnt = 4096;  // their stored entries
constexpr int kSpineThreads = 1024;

struct SpineWs {
    int e_rows[kSpineMaxE];       // exceptional rows (ascending once solved)
    int e_lv[kSpineMaxE];         // their levels
    int ent_pred[kSpineMaxEnt];   // per entry of an exceptional row: spine index of its
                                  // previous writer, -1 - (exceptional index), or kNone
    int ent_kt[kSpineMaxEnt];     // spine index of the entry's next writer, -1 if off the spine
    int ent_owner[kSpineMaxEnt];  // exceptional index of the entry's row
    int side_kt[kSpineMaxEnt];    // side edges sorted by spine index
    int side_pm[kSpineMaxEnt];    // prefix max of level(e) + 1 - kt along them
    int n_e, n_side, pad[2];
};

__global__ __launch_bounds__(kBlock) void k_top_feature(const int64_t *__restrict__ col_ptr,
                                                        int64_t d, Ctrl *ctrl) {
    unsigned long long best = 0;
    for (int64_t f = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; f < d;
         f += (int64_t)gridDim.x * blockDim.x) {
        const unsigned long long cnt = (unsigned long long)(col_ptr[f + 1] - col_ptr[f]);
        best = max(best, (cnt << 32) | (0xFFFFFFFFull - (unsigned long long)f));
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) best = max(best, (unsigned long long)__shfl_xor(best, off));
    if (lane_id() == 0 && best > 0) atomicMax(&ctrl->top_feature, best);
}

__global__ __launch_bounds__(kBlock) void k_spine_rows(const uint32_t *__restrict__ svals,
                                                       const int32_t *__restrict__ row_idx,
                                                       int64_t lo, int64_t K,
                                                       int32_t *__restrict__ rows) {
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < K;
         k += (int64_t)gridDim.x * blockDim.x)
        rows[k] = row_idx[svals[lo + k]];
}

// The exceptional rows are the gaps of the spine: rows strictly between
// consecutive spine rows, before the first and after the last.
__global__ __launch_bounds__(kBlock) void k_spine_gaps(const int32_t *__restrict__ rows, int64_t K,
                                                       int64_t n, SpineWs *sp) {
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k <= K;
         k += (int64_t)gridDim.x * blockDim.x) {
        const int64_t prev = k > 0 ? rows[k - 1] : -1;
        const int64_t cur = k < K ? rows[k] : n;
        const int64_t g = cur - prev - 1;
        if (g <= 0) continue;
        const int base = atomicAdd(&sp->n_e, (int)min(g, (int64_t)INT_MAX / 2));
        for (int64_t j = 0; j < g && base + j < kSpineMaxE; ++j)
            sp->e_rows[base + j] = (int)(prev + 1 + j);
    }
}

// index of row r in the ascending spine rows[0..K), or -1
__device__ __forceinline__ int64_t spine_find(const int32_t *rows, int64_t K, int64_t r) {
    int64_t lo = 0, hi = K;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (rows[mid] < r) lo = mid + 1;
        else hi = mid;
    }
    return (lo < K && rows[lo] == r) ? lo : -1;
}

// last j < cnt with kt[j] <= k, or -1
__device__ __forceinline__ int last_at_most(const int *kt, int cnt, int64_t k) {
    int lo = 0, hi = cnt;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (kt[mid] <= k) lo = mid + 1;
        else hi = mid;
    }
    return lo - 1;
}

// Block-wide exclusive max-scan of one value per thread (INT_MIN first).
__device__ int block_excl_max(int v, int *s_wave) {
    const int lane = lane_id(), wave = wave_in_block();
    int inc = v;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int y = __shfl_up(inc, off);
        if (lane >= off) inc = max(inc, y);
    }
    if (lane == kWave - 1) s_wave[wave] = inc;
    __syncthreads();
    int before = INT_MIN;
    for (int w = 0; w < wave; ++w) before = max(before, s_wave[w]);
    __syncthreads();
    const int prev = __shfl_up(inc, 1);
    return lane == 0 ? before : max(before, prev);
}

__device__ int block_excl_sum(int v, int *s_wave, int *total) {
    const int lane = lane_id(), wave = wave_in_block();
    int inc = v;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const int y = __shfl_up(inc, off);
        if (lane >= off) inc += y;
    }
    if (lane == kWave - 1) s_wave[wave] = inc;
    __syncthreads();
    int before = 0, all = 0;
    for (int w = 0; w < kSpineThreads / kWave; ++w) {
        if (w < wave) before += s_wave[w];
        all += s_wave[w];
    }
    __syncthreads();
    *total = all;
    return before + inc - v;
}

__global__ __launch_bounds__(kSpineThreads) void k_spine_solve(
    const int64_t *__restrict__ row_ptr, const int32_t *__restrict__ col,
    const int32_t *__restrict__ pn, const int32_t *__restrict__ row_idx,
    const uint32_t *__restrict__ svals, const int64_t *__restrict__ col_ptr,
    const int32_t *__restrict__ rows, int64_t K, SpineWs *sp, Ctrl *ctrl, int max_rounds) {
    __shared__ int s_e[kSpineMaxE];
    __shared__ int s_beg[kSpineMaxE + 1];
    __shared__ int s_lv[kSpineMaxE];
    __shared__ int s_skt[kSpineMaxEnt];
    __shared__ int s_pm[kSpineMaxEnt];
    __shared__ int s_wave[kSpineThreads / kWave];
    const int tid = threadIdx.x;
    const int n_e = sp->n_e;
    if (n_e > kSpineMaxE) {
        if (tid == 0) ctrl->spine_status = 1;
        return;
    }
    // the exceptional rows in ascending order (they are distinct)
    const int mine = tid < n_e ? sp->e_rows[tid] : INT_MAX;
    s_lv[tid] = mine;
    __syncthreads();
    if (tid < n_e) {
        int rank = 0;
        for (int j = 0; j < n_e; ++j) rank += s_lv[j] < mine;
        s_e[rank] = mine;
    }
    __syncthreads();
    // entry offsets
    const int m = tid < n_e ? (int)(row_ptr[s_e[tid] + 1] - row_ptr[s_e[tid]]) : 0;
    int n_ent = 0;
    const int beg = block_excl_sum(m, s_wave, &n_ent);
    if (n_ent > kSpineMaxEnt) {
        if (tid == 0) ctrl->spine_status = 1;
        return;
    }
    s_beg[tid] = beg;
    if (tid == 0) s_beg[n_e] = n_ent;
    __syncthreads();
    // previous writer and next writer of every entry
    for (int idx = tid; idx < n_ent; idx += kSpineThreads) {
        int lo = 0, hi = n_e;  // owner: last i with s_beg[i] <= idx
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (s_beg[mid] <= idx) lo = mid + 1;
            else hi = mid;
        }
        const int i = lo - 1;
        const int64_t p = row_ptr[s_e[i]] + (idx - s_beg[i]);
        int pred = kNone;
        const int32_t q = pn[p];
        if (q >= 0) {
            const int r = row_idx[q];
            const int64_t kb = spine_find(rows, K, r);
            if (kb >= 0) {
                pred = (int)kb;
            } else {
                int a = 0, b = n_e;  // r is an earlier exceptional row
                while (a < b) {
                    const int mid = (a + b) >> 1;
                    if (s_e[mid] < r) a = mid + 1;
                    else b = mid;
                }
                pred = -1 - a;
            }
        }
        const int f = col[p];
        int64_t a = col_ptr[f], b = col_ptr[f + 1];
        const int64_t end = b;
        while (a < b) {  // position of entry p in its feature's list
            const int64_t mid = (a + b) >> 1;
            if ((int64_t)svals[mid] < p) a = mid + 1;
            else b = mid;
        }
        int kt = -1;
        if (a + 1 < end) kt = (int)spine_find(rows, K, row_idx[svals[a + 1]]);
        sp->ent_pred[idx] = pred;
        sp->ent_kt[idx] = kt;
        sp->ent_owner[idx] = i;
    }
    __syncthreads();
    // side edges sorted by (spine index, entry)
    int n_side = 0;
    for (int idx = tid; idx < n_ent; idx += kSpineThreads) {
        const int kt = sp->ent_kt[idx];
        if (kt < 0) continue;
        int rank = 0;
        for (int j = 0; j < n_ent; ++j) {
            const int kj = sp->ent_kt[j];
            rank += kj >= 0 && (kj < kt || (kj == kt && j < idx));
        }
        s_skt[rank] = kt;
        sp->side_kt[rank] = kt;
        s_pm[rank] = sp->ent_owner[idx];  // owner for now
    }
    {
        int cnt = 0;
        for (int idx = tid; idx < n_ent; idx += kSpineThreads) cnt += sp->ent_kt[idx] >= 0;
        int total = 0;
        block_excl_sum(cnt, s_wave, &total);
        n_side = total;
    }
    __syncthreads();
    // owners of the sorted side edges, kept while the prefix max is recomputed
    constexpr int kPer = kSpineMaxEnt / kSpineThreads;
    int owner[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
        const int e = tid * kPer + j;
        owner[j] = e < n_side ? s_pm[e] : 0;
    }
    s_lv[tid] = 1;
    __syncthreads();
    int rounds = 0;
    bool converged = false;
    while (rounds < max_rounds) {
        ++rounds;
        // prefix max of level(owner) + 1 - kt over the sorted side edges
        // (thread tid holds edges tid * kPer .. tid * kPer + kPer - 1)
        int v[kPer];
        int run = INT_MIN;
#pragma unroll
        for (int j = 0; j < kPer; ++j) {
            const int e = tid * kPer + j;
            run = max(run, e < n_side ? s_lv[owner[j]] + 1 - s_skt[e] : INT_MIN);
            v[j] = run;
        }
        const int carry = block_excl_max(run, s_wave);
#pragma unroll
        for (int j = 0; j < kPer; ++j) {
            const int e = tid * kPer + j;
            if (e < n_side) s_pm[e] = max(v[j], carry);
        }
        __syncthreads();
        // levels of the exceptional rows from the current bounds
        int nl = 0;
        if (tid < n_e) {
            nl = 1;
            for (int idx = s_beg[tid]; idx < s_beg[tid + 1]; ++idx) {
                const int pred = sp->ent_pred[idx];
                if (pred >= 0) {
                    const int j = last_at_most(s_skt, n_side, pred);
                    const int M = max(1, j >= 0 ? s_pm[j] : INT_MIN);
                    nl = max(nl, pred + M + 1);
                } else if (pred != kNone) {
                    nl = max(nl, s_lv[-1 - pred] + 1);
                }
            }
        }
        const bool ch = tid < n_e && nl != s_lv[tid];
        __syncthreads();
        if (tid < n_e) s_lv[tid] = nl;
        if (!__syncthreads_or(ch)) {
            converged = true;
            break;
        }
    }
    if (tid < n_e) {
        sp->e_rows[tid] = s_e[tid];
        sp->e_lv[tid] = s_lv[tid];
    }
    for (int e = tid; e < n_side; e += kSpineThreads) sp->side_pm[e] = s_pm[e];
    if (tid == 0) {
        sp->n_side = n_side;
        ctrl->spine_rounds = rounds;
        ctrl->spine_status = converged ? 0 : 2;
    }
}

__global__ __launch_bounds__(kBlock) void k_spine_write(const int32_t *__restrict__ rows, int64_t K,
                                                        const SpineWs *__restrict__ sp,
                                                        int32_t *__restrict__ level) {
    const int n_side = sp->n_side;
    const int64_t i0 = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    for (int64_t k = i0; k < K; k += (int64_t)gridDim.x * blockDim.x) {
        const int j = last_at_most(sp->side_kt, n_side, k);
        const int M = max(1, j >= 0 ? sp->side_pm[j] : INT_MIN);
        level[rows[k]] = (int32_t)(k + M);
    }
    if (i0 < sp->n_e) level[sp->e_rows[i0]] = sp->e_lv[i0];
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

// Chain check: counts the rows i >= 1 none of whose entries has row i-1 as
// its previous writer.  An entry's previous writer lies in an earlier row, so
// it is row i-1 exactly when the previous entry's index is at least
// row_ptr[i-1].  One wave per row.
// The caller only needs to know whether there are no breaks, or at most n/4:
// every 64 rows a wave adds its count to the total and stops once the total
// is past n/4 (an input like config 4, where almost every example breaks,
// then reads a quarter of the previous writers instead of all of them).
constexpr int64_t kChainPrefix = 65536;  // rows the chain check reads first
// Rows 1 .. lim - 1 are checked (lim <= n): a prefix first, so that an input
// whose prefix already breaks often is not read further.
__global__ __launch_bounds__(kBlock) void k_chain_check(const int64_t *__restrict__ row_ptr,
                                                        int64_t lim, const int32_t *__restrict__ pn,
                                                        Ctrl *ctrl) {
    const int lane = lane_id();
    const int64_t nw = (int64_t)gridDim.x * (kBlock / kWave);
    const int64_t enough = lim / 4 + 1;
    int breaks = 0, rows = 0;
    for (int64_t i = 1 + blockIdx.x * (int64_t)(kBlock / kWave) + wave_in_block(); i < lim; i += nw) {
        const int64_t lo = row_ptr[i - 1], b = row_ptr[i], e = row_ptr[i + 1];
        bool found = false;
        for (int64_t p = b + lane; p < e && !found; p += kWave) found = pn[p] >= lo;
        if (__ballot(found) == 0ull) ++breaks;
        if (++rows == 64) {
            int total = 0;
            if (lane == 0) total = breaks ? atomicAdd(&ctrl->chain_breaks, breaks) + breaks
                                          : __hip_atomic_load(&ctrl->chain_breaks, __ATOMIC_RELAXED,
                                                              __HIP_MEMORY_SCOPE_AGENT);
            total = __builtin_amdgcn_readfirstlane(total);
            breaks = 0;
            rows = 0;
            if (total >= enough) return;
        }
    }
    if (lane == 0 && breaks) atomicAdd(&ctrl->chain_breaks, breaks);
}

// Levels of a chain: every example conflicts with the one before it, so
// levels increase strictly along the rows, the highest earlier conflicting
// example is always the previous one, and level(i) = i + 1.
__global__ __launch_bounds__(kBlock) void k_chain_levels(int64_t n, int32_t *__restrict__ level,
                                                         int32_t *__restrict__ perm,
                                                         int64_t *__restrict__ level_ptr,
                                                         int32_t *__restrict__ n_levels) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i <= n;
         i += (int64_t)gridDim.x * blockDim.x) {
        if (i < n) {
            level[i] = (int32_t)(i + 1);
            perm[i] = (int32_t)i;
        }
        level_ptr[i] = i;
        if (i == 0) *n_levels = (int32_t)n;
    }
}

// Schedule check, part 1: level_ptr non-decreasing from 0 to n, and every
// position e of level l (level_ptr[l-1] <= e < level_ptr[l]) holding an
// example p = perm[e] in [0, n) with level[p] = l, counted in seen[p] (a
// permutation leaves every count at 1).  The level of e by binary search.
__global__ __launch_bounds__(kBlock) void k_val_levels(const int32_t *__restrict__ level,
                                                       const int32_t *__restrict__ perm,
                                                       const int64_t *__restrict__ level_ptr,
                                                       int64_t n, int64_t L,
                                                       uint32_t *__restrict__ seen, Ctrl *ctrl) {
    int bad = 0;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e <= n;
         e += (int64_t)gridDim.x * blockDim.x) {
        if (e <= L) {
            const int64_t v = level_ptr[e];
            if (e == 0 && v != 0) bad = 1;
            if (e == L && v != n) bad = 1;
            if (e > 0 && v < level_ptr[e - 1]) bad = 1;
        }
        if (e == n) continue;
        // the last l in [0, L) with level_ptr[l] <= e: position e is in level l + 1
        int64_t lo = 0, hi = L;
        while (hi - lo > 1) {
            const int64_t mid = (lo + hi) >> 1;
            if (level_ptr[mid] <= e) lo = mid; else hi = mid;
        }
        const int32_t p = perm[e];
        if (p < 0 || (int64_t)p >= n) {
            bad = 1;
            continue;
        }
        if ((int64_t)level[p] != lo + 1) bad = 1;
        atomicAdd(&seen[p], 1u);
    }
    if (__ballot(bad) != 0ull && lane_id() == 0)
        __hip_atomic_store(&ctrl->bad, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Schedule check, part 2: every example seen once; every stored entry's
// example has a level above that of the example owning its previous entry on
// the same feature (pn, recomputed from the CSR), and the caller's prev_nz,
// when given, equals pn.
__global__ __launch_bounds__(kBlock) void k_val_order(const int32_t *__restrict__ level,
                                                      const uint32_t *__restrict__ seen, int64_t n,
                                                      const int32_t *__restrict__ pn,
                                                      const int32_t *__restrict__ row_idx,
                                                      const int32_t *__restrict__ prev_nz,
                                                      int64_t nnz, Ctrl *ctrl) {
    int bad = 0;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += stride)
        if (seen[i] != 1u) bad = 1;
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < nnz; p += stride) {
        const int32_t q = pn[p];
        if (prev_nz && prev_nz[p] != q) bad = 1;
        if (q >= 0 && level[row_idx[q]] >= level[row_idx[p]]) bad = 1;
    }
    if (__ballot(bad) != 0ull && lane_id() == 0)
        __hip_atomic_store(&ctrl->bad, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

int bit_length(uint64_t x) {
    int b = 0;
    while (x) {
        ++b;
        x >>= 1;
    }
    return b;
}

// compute units of the current device (queried per call: no cached state)
int device_cus() {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
        cus = 256;
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

// K0 + K1 + K2 into the workspace: previous-writer entries into pn, col_ptr,
// and csc_row when not null.
int build_conflicts(const pdb_csr *csr, int64_t n, int64_t d, SchedWs &w, int32_t *pn,
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
        // the radix pair not holding the sorted entries takes the pairs; the
        // sort's other buffers are the candidates array and pn itself
        uint32_t *fk = (sk == w.kA) ? w.kB : w.kA;
        uint32_t *fv = (sv == w.vA) ? w.vB : w.vA;
        k_prev_pairs<<<grid_for(nnz, kBlock, 1 << 16), kBlock, 0, s>>>(
            sk, sv, nnz, d, w.row_idx, fk, fv, col_ptr, csc_row);
        PDB_LAUNCHED();
        uint32_t *ok = nullptr, *ov = nullptr;
        PDB_HIP(radix_sort_pairs(fk, fv, nnz, bit_length((uint64_t)(nnz > 1 ? nnz - 1 : 1)),
                                 reinterpret_cast<uint32_t *>(w.cand),
                                 reinterpret_cast<uint32_t *>(pn), fk, fv, w.hist, w.scan_tmp,
                                 &ok, &ov, s, kPlaceBits));
        k_prev_place<<<(unsigned)cdiv(nnz, (int64_t)1 << kPlaceBits), kBlock, 0, s>>>(ok, ov, nnz,
                                                                                      pn);
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
    w.pn = reinterpret_cast<int32_t *>(take(std::max<int64_t>(nnz, 1) * 4));
    w.cand = reinterpret_cast<int32_t *>(take(std::max<int64_t>(nnz, 1) * 4));
    w.spine = take(sizeof(SpineWs));
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
    rc = build_conflicts(csr, n, d, w, w.pn, col_ptr, csc_row, &sk, &sv, stream);
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
    int32_t *pn = prev_nz ? prev_nz : w.pn;
    const uint32_t *sk, *sv;
    rc = build_conflicts(csr, n, d, w, pn, w.col_ptr, nullptr, &sk, &sv, stream);
    if (rc != PDB_OK) return rc;
    if (csr->nnz > 0) {
        k_prev_row<<<grid_for(csr->nnz, kBlock, 1 << 16), kBlock, 0, stream>>>(pn, csr->nnz,
                                                                              w.row_idx, prev_row);
        PDB_LAUNCHED();
    }
    PDB_HIP(hipStreamSynchronize(stream));
    return PDB_OK;
}

extern "C" int pdb_schedule(const pdb_csr *csr, const float *labels, int64_t n, int64_t d,
                            pdb_levels *lv, int method, pdb_schedule_info *info, void *ws,
                            size_t ws_bytes, const pdb_options *opt, hipStream_t s) {
    (void)labels;
    SchedWs w;
    int rc = sched_common_checks(csr, n, d, ws, ws_bytes, &w);
    if (rc != PDB_OK) return rc;
    Opts o;
    rc = resolve_opts(opt, &o);
    if (rc != PDB_OK) return rc;
    if (!lv || !lv->level_ptr || !lv->n_levels || (n > 0 && (!lv->level || !lv->perm)))
        return PDB_ERR_INVALID_ARG;
    if (method < PDB_SCHED_AUTO || method > PDB_SCHED_SHORT) return PDB_ERR_INVALID_ARG;
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
    int32_t *pn = lv->prev_nz ? lv->prev_nz : w.pn;
    const uint32_t *sk, *sv;
    rc = build_conflicts(csr, n, d, w, pn, w.col_ptr, nullptr, &sk, &sv, s);
    if (rc != PDB_OK) return rc;
    // the radix buffer pair that does not hold the sorted entries is free
    int32_t *free_k = reinterpret_cast<int32_t *>((sk == w.kA) ? w.kB : w.kA);
    const int64_t timeout = o.timeout;

    // a chain (every example conflicts with the one before it) is solved
    // outright; auto tries it first
    bool chain_like = false, chain_checked = false;
    if (method == PDB_SCHED_AUTO || method == PDB_SCHED_CHAIN) {
        chain_checked = true;
        // a prefix of the rows first: when more than a quarter of it breaks,
        // the input is no chain and is taken as not chain-like without
        // reading the rest (every method is exact; this only picks one)
        const int64_t lim0 = std::min<int64_t>(n, kChainPrefix);
        k_chain_check<<<grid_for(lim0, kBlock / kWave, 65536), kBlock, 0, s>>>(csr->row_ptr, lim0,
                                                                               pn, w.ctrl);
        PDB_LAUNCHED();
        rc = read_ctrl(w.ctrl, &host, s);
        if (rc != PDB_OK) return rc;
        const bool prefix_breaks = lim0 < n && 4 * (int64_t)host.chain_breaks > lim0;
        if (lim0 < n && !prefix_breaks) {
            k_fill_i32<<<1, 64, 0, s>>>(&w.ctrl->chain_breaks, 1, 0);
            k_chain_check<<<grid_for(n, kBlock / kWave, 65536), kBlock, 0, s>>>(csr->row_ptr, n,
                                                                                pn, w.ctrl);
            PDB_LAUNCHED();
            rc = read_ctrl(w.ctrl, &host, s);
            if (rc != PDB_OK) return rc;
        }
        if (host.chain_breaks == 0) {
            k_chain_levels<<<grid_for(n + 1, kBlock, 65536), kBlock, 0, s>>>(
                n, lv->level, lv->perm, lv->level_ptr, lv->n_levels);
            PDB_LAUNCHED();
            PDB_HIP(hipStreamSynchronize(s));
            lv->L_host = n;
            lv->max_width_host = 1;
            if (info) *info = pdb_schedule_info{PDB_SCHED_CHAIN, 0, n, 1};
            return PDB_OK;
        }
        if (method == PDB_SCHED_CHAIN) method = PDB_SCHED_DATAFLOW;
        // most examples conflict with their predecessor: the walk pays
        chain_like = !prefix_breaks && 4 * (int64_t)host.chain_breaks <= n;
    }

    // which method: the spine when the most frequent feature misses at most
    // kSpineMaxE rows, else the walk on chain-like inputs, else dataflow
    int use = method;
    int rounds = 0;
    int64_t top_count = 0, top_f = 0;
    if (method == PDB_SCHED_AUTO || method == PDB_SCHED_SPINE) {
        k_top_feature<<<grid_for(d, kBlock, 4096), kBlock, 0, s>>>(w.col_ptr, d, w.ctrl);
        PDB_LAUNCHED();
        rc = read_ctrl(w.ctrl, &host, s);
        if (rc != PDB_OK) return rc;
        top_count = (int64_t)(host.top_feature >> 32);
        top_f = (int64_t)(0xFFFFFFFFull - (host.top_feature & 0xFFFFFFFFull));
        const bool fits = top_count > 0 && n - top_count <= kSpineMaxE;
        use = fits ? PDB_SCHED_SPINE
                   : ((method == PDB_SCHED_AUTO && chain_like) ? PDB_SCHED_WALK : PDB_SCHED_DATAFLOW);
    }

    // rows of at most kShortR entries (matrix completion), where dataflow
    // would run: the short-row walk
    if ((method == PDB_SCHED_AUTO && use == PDB_SCHED_DATAFLOW) || method == PDB_SCHED_SHORT) {
        k_fill_i32<<<1, 64, 0, s>>>(reinterpret_cast<int32_t *>(&w.ctrl->max_width), 2, 0);
        k_max_diff<<<grid_for(n, kBlock, 4096), kBlock, 0, s>>>(csr->row_ptr, n, w.ctrl);
        PDB_LAUNCHED();
        rc = read_ctrl(w.ctrl, &host, s);
        if (rc != PDB_OK) return rc;
        use = host.max_width <= kShortR ? PDB_SCHED_SHORT : PDB_SCHED_DATAFLOW;
    }

    if (use == PDB_SCHED_SPINE) {
        SpineWs *sp = static_cast<SpineWs *>(w.spine);
        int32_t *rows = free_k;  // the spine rows, ascending
        // spine rows: the entries of top_f in feature order
        int64_t lo = 0;
        PDB_HIP(hipMemcpyAsync(&lo, w.col_ptr + top_f, sizeof(lo), hipMemcpyDeviceToHost, s));
        PDB_HIP(hipStreamSynchronize(s));
        k_spine_rows<<<grid_for(top_count, kBlock, 65536), kBlock, 0, s>>>(sv, w.row_idx, lo,
                                                                            top_count, rows);
        k_fill_i32<<<1, 64, 0, s>>>(&sp->n_e, 4, 0);
        k_spine_gaps<<<grid_for(top_count + 1, kBlock, 65536), kBlock, 0, s>>>(rows, top_count, n,
                                                                                sp);
        k_spine_solve<<<1, kSpineThreads, 0, s>>>(csr->row_ptr, csr->col, pn, w.row_idx, sv,
                                                  w.col_ptr, rows, top_count, sp, w.ctrl,
                                                  kSpineMaxE + 2);
        PDB_LAUNCHED();
        rc = read_ctrl(w.ctrl, &host, s);
        if (rc != PDB_OK) return rc;
        if (host.spine_status == 0) {
            k_spine_write<<<grid_for(std::max<int64_t>(top_count, kSpineMaxE), kBlock, 65536),
                            kBlock, 0, s>>>(rows, top_count, sp, lv->level);
            PDB_LAUNCHED();
            rounds = host.spine_rounds;
        } else {
            use = PDB_SCHED_DATAFLOW;  // too many exceptional rows or entries
        }
    }

    if (use == PDB_SCHED_WALK) {
        if (nnz > 0) {
            k_prev_row<<<grid_for(nnz, kBlock, 1 << 16), kBlock, 0, s>>>(pn, nnz, w.row_idx,
                                                                        w.cand);
            PDB_LAUNCHED();
        }
        // the number of runs is known exactly when the chain check counted
        // every break; few runs: the grid settles them one after another
        const int64_t R = (int64_t)host.chain_breaks + 1;
        if (chain_checked && n >= kRunMinN && R * kRunRowsPer <= n && n <= INT_MAX) {
            uint32_t *pos = reinterpret_cast<uint32_t *>(free_k);
            int32_t *stg = reinterpret_cast<int32_t *>(pos);  // the scan is spent by then
            int32_t *starts = lv->perm;  // R + 1 run starts, then 2 x 64 stretch maxima
            int32_t *bmax = lv->perm + R + 1;
            k_run_flags<<<grid_for(n, kBlock / kWave, 65536), kBlock, 0, s>>>(csr->row_ptr, n, pn,
                                                                              pos);
            PDB_HIP(exclusive_scan_u32(pos, pos, n, w.scan_tmp, s));
            k_run_starts<<<grid_for(n, kBlock, 65536), kBlock, 0, s>>>(pos, n, R, starts);
            PDB_LAUNCHED();
            int dev = 0, cus = 0;
            PDB_HIP(hipGetDevice(&dev));
            PDB_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
            const void *fn = reinterpret_cast<const void *>(&k_levels_runs);
            int per_cu = 0;
            PDB_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kRunThreads, 0));
            const int grid = std::max(1, std::min(kRunBlocks, cus * std::max(per_cu, 1)));
            const int64_t *rp = csr->row_ptr;
            const int32_t *prow = w.cand, *ridx = w.row_idx;
            const int32_t *st = starts;
            int32_t *lvl = lv->level;
            Ctrl *ctrl = w.ctrl;
            int64_t Rv = R, to = timeout;
            void *args[] = {&rp, &prow, &ridx, &Rv, &st, &stg, &lvl, &bmax, &ctrl, &to};
            PDB_HIP(hipLaunchCooperativeKernel(fn, dim3((unsigned)grid), dim3(kRunThreads), args, 0,
                                               s));
            // the barrier's arrival counter back to zero for later grid barriers
            k_fill_i32<<<1, 64, 0, s>>>(reinterpret_cast<int32_t *>(&w.ctrl->bar_count), 1, 0);
            PDB_LAUNCHED();
            rc = read_ctrl(w.ctrl, &host, s);
            if (rc != PDB_OK) return rc;
            if (host.err) return PDB_ERR_DEVICE;  // a barrier's wait gave up
        } else {
            k_levels_walk<<<1, kWalkThreads, 0, s>>>(csr->row_ptr, n, w.cand, w.row_idx,
                                                     lv->level, w.ctrl);
            PDB_LAUNCHED();
            rc = read_ctrl(w.ctrl, &host, s);
            if (rc != PDB_OK) return rc;
            if (host.bad) use = PDB_SCHED_DATAFLOW;  // a row longer than a window
        }
    }

    if (use == PDB_SCHED_SHORT) {
        if (n > kFlowMaxN) return PDB_ERR_UNSUPPORTED;
        // every row gets its level from the walk; zeros until then, so a walk
        // that stops early leaves no stale levels behind
        k_fill_i32<<<grid_for(n, kBlock, 65536), kBlock, 0, s>>>(lv->level, n, 0);
        PDB_LAUNCHED();
        if (nnz > 0) {
            k_prev_row<<<grid_for(nnz, kBlock, 1 << 16), kBlock, 0, s>>>(pn, nnz, w.row_idx,
                                                                        w.cand);
            PDB_LAUNCHED();
        }
        // rows of at most two entries (matrix completion) need half the lane shuffles
        if (host.max_width <= 2)
            k_levels_short<2><<<1, kShortThreads, 0, s>>>(csr->row_ptr, w.cand, n, lv->level,
                                                          w.ctrl, timeout);
        else
            k_levels_short<kShortR><<<1, kShortThreads, 0, s>>>(csr->row_ptr, w.cand, n, lv->level,
                                                                w.ctrl, timeout);
        PDB_LAUNCHED();
        rc = read_ctrl(w.ctrl, &host, s);
        if (rc != PDB_OK) return rc;
        if (host.err) return PDB_ERR_DEVICE;      // a wave's wait gave up
        if (host.bad) use = PDB_SCHED_DATAFLOW;  // a row longer than kShortR
    }

    if (use == PDB_SCHED_CHAINSCAN) {
        // csc_row[q] = row of the q-th entry in feature order
        int32_t *crow = free_k;
        if (nnz > 0)
            k_csc_row<<<grid_for(nnz, kBlock, 1 << 16), kBlock, 0, s>>>(sv, nnz, w.row_idx, crow);
        k_fill_i32<<<grid_for(n, kBlock, 65536), kBlock, 0, s>>>(lv->level, n, 1);
        PDB_LAUNCHED();
        const int64_t tiles = cdiv(std::max<int64_t>(nnz, 1), kTile);
        while (true) {
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
            if (!host.changed) break;  // at most n + 1 rounds
        }
    }
    if (use == PDB_SCHED_DATAFLOW) {
        // long rows, not chain-like (the chain check ran and found many
        // breaks): a wave per example
        const bool rowwave = chain_checked && !chain_like && nnz >= kRowWaveMinAvg * n;
        // previous-writer rows into cand (the wave-per-example form looks
        // them up itself)
        if (nnz > 0 && !rowwave) {
            k_prev_row<<<grid_for(nnz, kBlock, 1 << 16), kBlock, 0, s>>>(pn, nnz, w.row_idx,
                                                                        w.cand);
            PDB_LAUNCHED();
        }
        k_fill_i32<<<grid_for(n, kBlock, 65536), kBlock, 0, s>>>(lv->level, n, 0);
        PDB_LAUNCHED();
        if (n > kFlowMaxN) return PDB_ERR_UNSUPPORTED;
        const size_t lds = rowwave ? 0 : (size_t)kFlowWaveLds * 4 * (kBlock / kWave);
        const void *fn = rowwave ? reinterpret_cast<const void *>(&k_levels_rowwave)
                                 : reinterpret_cast<const void *>(&k_levels_dataflow);
        if (!rowwave)
            PDB_HIP(hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
        int per_cu = 0;
        PDB_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kBlock, lds));
        int64_t grid = std::min<int64_t>(
            (int64_t)device_cus() * std::max(per_cu, 1),
            cdiv(n, (int64_t)(rowwave ? 1 : kFlowB) * (kBlock / kWave)));
        // a wave per example: four waves per CU keep enough examples in
        // flight; more waves only add polling traffic (5M rows of 80 entries:
        // 128 -> 93 ms per schedule)
        if (rowwave) grid = std::min<int64_t>(grid, (int64_t)device_cus());
        {
            // cooperative: the whole grid resident (the waves wait on each other)
            const int64_t *a_rp = csr->row_ptr;
            const int32_t *a_prev = rowwave ? pn : w.cand;
            const int32_t *a_rows = w.row_idx;
            int32_t *a_level = lv->level;
            Ctrl *a_ctrl = w.ctrl;
            int64_t a_n = n, a_timeout = timeout;
            void *args_flow[] = {&a_rp, &a_prev, &a_n, &a_level, &a_ctrl, &a_timeout};
            void *args_row[] = {&a_rp, &a_prev, &a_rows, &a_n, &a_level, &a_ctrl, &a_timeout};
            PDB_HIP(hipLaunchCooperativeKernel(fn, dim3((unsigned)std::max<int64_t>(grid, 1)),
                                               dim3(kBlock), rowwave ? args_row : args_flow, lds,
                                               s));
        }
        rc = read_ctrl(w.ctrl, &host, s);
        if (rc != PDB_OK) return rc;
        if (host.err) return PDB_ERR_DEVICE;
    }

    // L, then K4
    k_max_level<<<grid_for(n, kBlock, 4096), kBlock, 0, s>>>(lv->level, n, w.ctrl);
    PDB_LAUNCHED();
    rc = read_ctrl(w.ctrl, &host, s);
    if (rc != PDB_OK) return rc;
    // any level kernel whose wait gave up has left levels unfinished
    if (host.err) return PDB_ERR_DEVICE;
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

extern "C" int pdb_validate_schedule(const pdb_csr *csr, int64_t n, int64_t d,
                                     const pdb_levels *lv, void *ws, size_t ws_bytes,
                                     hipStream_t s) {
    SchedWs w;
    int rc = sched_common_checks(csr, n, d, ws, ws_bytes, &w);
    if (rc != PDB_OK) return rc;
    if (!lv || !lv->level_ptr || !lv->n_levels || (n > 0 && (!lv->level || !lv->perm)))
        return PDB_ERR_INVALID_ARG;
    int32_t L = 0;
    PDB_HIP(hipMemcpyAsync(&L, lv->n_levels, sizeof(L), hipMemcpyDeviceToHost, s));
    PDB_HIP(hipStreamSynchronize(s));
    if (n == 0) {
        int64_t first = -1;
        PDB_HIP(hipMemcpyAsync(&first, lv->level_ptr, sizeof(first), hipMemcpyDeviceToHost, s));
        PDB_HIP(hipStreamSynchronize(s));
        return (L == 0 && first == 0) ? PDB_OK : PDB_ERR_DEVICE;
    }
    if (L < 1 || (int64_t)L > n) return PDB_ERR_DEVICE;
    const int64_t nnz = csr->nnz;
    Ctrl host{};
    k_ctrl_init<<<1, 64, 0, s>>>(w.ctrl);
    PDB_LAUNCHED();
    // previous writers from the CSR itself (nothing of the schedule is used)
    const uint32_t *sk, *sv;
    rc = build_conflicts(csr, n, d, w, w.pn, w.col_ptr, nullptr, &sk, &sv, s);
    if (rc != PDB_OK) return rc;
    // the radix buffer pair that does not hold the sorted entries is free
    uint32_t *seen = (sk == w.kA) ? w.kB : w.kA;
    k_fill_i32<<<grid_for(n, kBlock, 65536), kBlock, 0, s>>>(reinterpret_cast<int32_t *>(seen), n,
                                                             0);
    k_val_levels<<<grid_for(n + 1, kBlock, 65536), kBlock, 0, s>>>(lv->level, lv->perm,
                                                                    lv->level_ptr, n, L, seen,
                                                                    w.ctrl);
    k_val_order<<<grid_for(std::max(n, nnz), kBlock, 65536), kBlock, 0, s>>>(
        lv->level, seen, n, w.pn, w.row_idx, lv->prev_nz, nnz, w.ctrl);
    PDB_LAUNCHED();
    rc = read_ctrl(w.ctrl, &host, s);
    if (rc != PDB_OK) return rc;
    return host.bad ? PDB_ERR_DEVICE : PDB_OK;
}
