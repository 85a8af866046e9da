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
// example t wrote.  Runs of levels at most `chain_width` wide (default 4) go
// the same way, their examples one after another in level order, which is a
// sequential order of them (Theorem 2).  When every level is that narrow,
// the whole epoch is one such run over the rows in plain index order, the
// sequential order itself.  There one wave runs the chain and the three
// other waves
// of the block stage upcoming examples (columns, values, and the CSR index
// of each entry's previous writer) into LDS.  Weights of features below
// `hot` live in LDS for the whole run; a feature that example t just wrote is
// not re-read at all: example t+1 takes the old value and x from example t's
// lane (a cross-lane permute issued before example t's step is known) and
// applies example t's step itself with the same fma -- so the only work
// between two steps is arithmetic.  Features written a few examples back come
// from a small LDS ring; all other cold features are prefetched from global
// memory kD examples ahead (their last writer finished before the prefetch).
#include <atomic>
#include <climits>

#include "pdb_math.h"
#include "pdb_words.h"

namespace pdbk {

namespace {

constexpr int kWavesPerBlock = kBlock / kWave;

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
    // the pipeline's select-free step is checked for logistic loss only
    static constexpr bool kFastCheck = LOSS == PDB_LOGISTIC;

    __device__ __forceinline__ void operator()(int64_t e, int64_t end) const {
        (void)end;
        row(perm[e]);
    }
    // example i (a row index), by one wave
    __device__ __forceinline__ void row(int64_t i) const {
        const int lane = lane_id();
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
            const float s = sgd_scale<LOSS>(wave_sum64(acc), yi, lr);
            if (lane < m) w[c] = __builtin_fmaf(-s, x, wv);
        } else {
            float acc = 0.0f;
            for (int k = lane; k < m; k += kWave) {
                const int c = col[b + k];
                acc = __builtin_fmaf(w[c], VAL ? val[b + k] : 1.0f, acc);
            }
            const float s = sgd_scale<LOSS>(wave_sum64(acc), yi, lr);
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
    static constexpr bool kFastCheck = false;

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

constexpr int kD = 16;           // window of fresh values and cold-prefetch distance
constexpr int kRB = 64;          // staged examples (power of two, >= 2 kD + kPB)
constexpr int kPB = 16;          // examples per producer batch
constexpr int kRing = kD * 64;   // LDS ring of recent cold writes
constexpr int kChainMin = 32;    // shorter runs take the plain path
// staged records the consumer holds in registers (examples t, t+1, t+2): a
// slot is read a full step before its read source is needed, so the LDS
// latency of that read never stalls the chain
constexpr int kMirror = 3;
// buffer offset past the end of any weight vector: a load there returns 0
// and a store is dropped (buffer range checking), so lanes with nothing to
// load or store still issue the instruction
constexpr unsigned kOOR = 0x80000000u;

typedef __attribute__((address_space(3))) float lds_f32;
__device__ __forceinline__ unsigned lds_addr(const float *p) {
    return (unsigned)(uintptr_t)(const lds_f32 *)p;
}
__device__ __forceinline__ float lds_read(unsigned a) { return *(const lds_f32 *)(uintptr_t)a; }
__device__ __forceinline__ void lds_write(unsigned a, float v) { *(lds_f32 *)(uintptr_t)a = v; }

// Fixed part of the pipeline's LDS; the cached weights live in dynamic LDS.
struct ChainShared {
    // per staged example (slot t mod kRB) and lane: {x bits, LDS write
    // address, read source, buffer offset of the global write}.  The read
    // source is 4 x the lane to take a forwarded value from (< 256), the
    // address of zero[1] for a value to prefetch from global memory, or an
    // LDS address to read (cache, ring, zero[0] for lanes without an entry).
    // The write address is the cache slot of a hot feature, the ring slot of
    // a cold one, or lsink.  The write offset has bit 31 set (out of range:
    // dropped) unless the feature is cold.  Slots kRB .. kRB + 2 repeat
    // slots 0 .. 2, so that the consumer reads a block of kD + 3
    // consecutive slots without wrapping.
    uint4 st[(kRB + kMirror) * 64];
    float mt_t[kRB + kMirror];  // target: [y > 0] (logistic) or y (least squares)
    int seq[kRB];         // position t staged in the slot, ~t when its example has more
                          // than 64 entries, INT_MIN none
    int ctl[4];           // [0] consumer no longer needs positions < ctl[0]; [1] stop
    float ring[kRing];    // new weights of cold features written within kD examples
    float lsink[64];      // LDS write target of lanes without an entry
    float zero[4];        // [0] read by lanes without an entry; [1] marks global sources
};

extern __shared__ __align__(16) float g_wcache[];

__device__ __forceinline__ int lds_load(const int *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void lds_store(int *p, int v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void compiler_fence() { __asm__ __volatile__("" ::: "memory"); }

template <int LOSS>
__device__ __forceinline__ float target_of(float y) {
    return LOSS == PDB_LOGISTIC ? (y > 0.0f ? 1.0f : 0.0f) : y;
}

// Producer wave pid (0..2): stages examples t of the run (batches of kPB, in
// turn), never more than kRB ahead of the consumer.  For every entry it finds
// whether the previous writer is among the kD examples before it and picks
// where the consumer will read the current weight: forwarded from the
// previous example's lane, the LDS cache (hot feature), the ring (cold
// feature written within kD examples), or the prefetched global value.
//
// DENSE: the run is the consecutive rows r0, r0 + 1, ..., so the entries of
// the kD examples before position t are the CSR range [b(t - kD), b(t)): one
// comparison tells whether the previous writer is in the window, and the ring
// is indexed by the writer's CSR index (the window spans at most kD * 64
// entries, so no two of them share a ring slot).  Otherwise each entry is
// matched against the kD preceding examples' entry ranges and the ring is
// indexed by (position mod kD, lane).
// Row bounds and targets of the positions a producer batch at t0 needs:
// lane i describes position t0 - kD + i (the window before the batch, the
// batch, and for DENSE one more that ends the batch's last example).
struct BatchMeta {
    int b, m;
    float tg;  // label of the position (clamped into the run)
};

template <int LOSS, bool VAL, bool DENSE>
__device__ __forceinline__ BatchMeta batch_meta(const SgdOp<LOSS, VAL> &op, int64_t t0,
                                                int64_t e_beg, int64_t len, int64_t r0) {
    // every lane loads (positions clamped into the run), so no load sits in
    // a branch and none has to complete before the batch's entry loads
    const int lane = lane_id();
    const int64_t q = t0 - kD + lane;
    const int64_t qc = min(max(q, (int64_t)0), len - 1);
    BatchMeta mt;
    if (DENSE) {
        // b of positions clamped to [0, len]; m comes later from the next lane
        mt.b = (int)op.row_ptr[r0 + min(max(q, (int64_t)0), len)];
        mt.m = 0;
        mt.tg = op.y[r0 + qc];
    } else {
        const int64_t r = op.perm[e_beg + qc];
        const int64_t b0 = op.row_ptr[r], b1 = op.row_ptr[r + 1];
        const float yv = op.y[r];
        const bool ok = lane < kD + kPB && q >= 0 && q < len;
        mt.b = ok ? (int)b0 : 0;
        mt.m = ok ? (int)(b1 - b0) : 0;
        mt.tg = yv;
    }
    return mt;
}

template <int LOSS, bool VAL, bool DENSE>
__device__ void chain_producer(const SgdOp<LOSS, VAL> &op, int pid, int64_t e_beg, int64_t len,
                               int64_t r0, int hot, ChainShared &S) {
    const int lane = lane_id();
    const unsigned wc_base = lds_addr(&g_wcache[0]);
    const unsigned zero_a = lds_addr(&S.zero[0]);
    const unsigned gsrc_a = lds_addr(&S.zero[1]);
    const unsigned lsink_a = lds_addr(&S.lsink[lane]);
    const unsigned ring_a = lds_addr(&S.ring[0]);
    // lanes without an entry load from here (a valid address) and ignore it
    const int32_t *dummy_i = reinterpret_cast<const int32_t *>(op.row_ptr);
    const float *dummy_f = reinterpret_cast<const float *>(op.row_ptr);
    int64_t t0 = (int64_t)pid * kPB;
    BatchMeta nxt = batch_meta<LOSS, VAL, DENSE>(op, t0, e_beg, len, r0);
    for (; t0 < len; t0 += 3 * kPB) {
        while (t0 + kPB - 1 >= (int64_t)lds_load(&S.ctl[0]) + kRB) {
            if (lds_load(&S.ctl[1])) return;
            __builtin_amdgcn_s_sleep(1);
        }
        if (lds_load(&S.ctl[1])) return;
        const int b = nxt.b;
        const int m = DENSE ? __shfl_down(b, 1) - b : nxt.m;
        const float tg = target_of<LOSS>(nxt.tg);
        // every entry load of the batch first (unconditional, so they all go
        // out before the first wait), then this wave's next batch
        int c[kPB], pn[kPB];
        float x[kPB];
#pragma unroll
        for (int i = 0; i < kPB; ++i) {
            const int bi = __builtin_amdgcn_readlane(b, kD + i);
            const int mi = __builtin_amdgcn_readlane(m, kD + i);
            const bool live = lane < mi;  // mi = 0 past the end of the run
            const int64_t e = (int64_t)bi + lane;
            c[i] = *(live ? op.col + e : dummy_i);
            pn[i] = *(live ? op.prev_nz + e : dummy_i);
            x[i] = VAL ? *(live ? op.val + e : dummy_f) : 1.0f;
        }
        nxt = batch_meta<LOSS, VAL, DENSE>(op, t0 + 3 * kPB, e_beg, len, r0);
        // classify every entry with comparisons on all lanes and a chain of
        // selects (no branch holds a use of the loaded values, so the loads
        // stay where they were issued)
        uint4 A[kPB];
#pragma unroll
        for (int i = 0; i < kPB; ++i) {
            const int bi = __builtin_amdgcn_readlane(b, kD + i);
            const int mi = __builtin_amdgcn_readlane(m, kD + i);
            const bool live = lane < mi;
            const bool is_hot = live & ((unsigned)c[i] < (unsigned)hot);
            const unsigned cache = wc_base + ((unsigned)c[i] << 2);
            unsigned rd, laddr;
            if (DENSE) {
                // previous example starts at bprev, the window at bwin (both
                // clamp to the run's first example at its start)
                const int bprev = __builtin_amdgcn_readlane(b, kD + i - 1);
                const int bwin = __builtin_amdgcn_readlane(b, i);
                const bool fwd = pn[i] >= bprev;
                const bool win = pn[i] >= bwin;
                rd = win ? ring_a + (((unsigned)pn[i] & (kRing - 1)) << 2) : gsrc_a;
                rd = is_hot ? cache : rd;
                rd = fwd ? (unsigned)(pn[i] - bprev) << 2 : rd;
                rd = live ? rd : zero_a;
                laddr = ring_a + (((unsigned)(bi + lane) & (kRing - 1)) << 2);
            } else {
                int rel = 0, off = 0;
#pragma unroll
                for (int j = 1; j <= kD; ++j) {
                    const int bj = __builtin_amdgcn_readlane(b, kD + i - j);
                    const int mj = __builtin_amdgcn_readlane(m, kD + i - j);
                    const unsigned o = (unsigned)(pn[i] - bj);
                    const bool hit = o < (unsigned)mj;
                    rel = hit ? j : rel;
                    off = hit ? (int)o : off;
                }
                const int64_t t = t0 + i;
                const unsigned wslot = (unsigned)(t - rel) & (kD - 1);
                rd = rel >= 2 ? ring_a + (wslot << 8) + ((unsigned)off << 2) : gsrc_a;
                rd = is_hot ? cache : rd;
                rd = rel == 1 ? (unsigned)off << 2 : rd;
                rd = live ? rd : zero_a;
                laddr = ring_a + (((unsigned)t & (kD - 1)) << 8) + ((unsigned)lane << 2);
            }
            laddr = is_hot ? cache : laddr;
            laddr = live ? laddr : lsink_a;
            const unsigned goff = ((unsigned)c[i] << 2) | ((live & !is_hot) ? 0u : kOOR);
            // without stored values every x is 1 and the word carries the
            // example's target instead, saving the consumer a read
            const unsigned xw = VAL ? __float_as_uint(live ? x[i] : 0.0f)
                                    : (unsigned)__builtin_amdgcn_readlane(__float_as_int(tg), kD + i);
            A[i] = make_uint4(xw, laddr, rd, goff);
        }
        const int sb = (int)(t0 & (kRB - 1));  // a multiple of kPB: no wrap inside the batch
#pragma unroll
        for (int i = 0; i < kPB; ++i) S.st[(sb + i) * 64 + lane] = A[i];
        if (sb == 0) {
            S.st[kRB * 64 + lane] = A[0];
            S.st[(kRB + 1) * 64 + lane] = A[1];
            S.st[(kRB + 2) * 64 + lane] = A[2];
        }
        {
            // every lane stores (lanes outside the batch into the sink), so
            // the label load is never moved into a branch
            const bool in_batch = lane >= kD && lane < kD + kPB;
            const int slot = sb + lane - kD;
            const int64_t q = t0 - kD + lane;  // the position this lane describes
            lds_write(in_batch ? lds_addr(&S.mt_t[slot]) : lsink_a, tg);
            lds_write((in_batch && slot < kMirror) ? lds_addr(&S.mt_t[kRB + slot]) : lsink_a, tg);
            compiler_fence();  // LDS executes one wave's operations in order
            if (in_batch && q < len)
                lds_store(&S.seq[slot], m > kWave ? ~(int)q : (int)q);
        }
        compiler_fence();
    }
}

// Waits until positions lo .. hi-1 (hi - lo <= kRB) are staged; returns the
// first of them holding an example with more than 64 entries, or INT64_MAX.
__device__ __forceinline__ int64_t wait_staged(ChainShared &S, int64_t lo, int64_t hi,
                                               long long *waited) {
    const int64_t t = lo + lane_id();
    const int slot = (int)(t & (kRB - 1));
    const bool want = t < hi;
    long long c0 = 0;
    bool first = true;
    int v;
    for (;;) {
        v = lds_load(&S.seq[slot]);
        const bool ok = !want || v == (int)t || v == ~(int)t;
        if (__ballot(!ok) == 0ull) break;
        if (first) c0 = (long long)__builtin_readcyclecounter();
        first = false;
        __builtin_amdgcn_s_sleep(0);
    }
    if (!first) *waited += (long long)__builtin_readcyclecounter() - c0;
    compiler_fence();
    const unsigned long long longrow = __ballot(want && v == ~(int)t);
    return longrow ? lo + __ffsll(longrow) - 1 : INT64_MAX;
}

struct Stg {
    uint4 a;  // x bits, LDS write address, read source, global write offset
    float t;  // target
};

// slot in [0, kRB + kMirror)
__device__ __forceinline__ Stg read_slot(const ChainShared &S, int slot) {
    Stg r;
    r.a = S.st[slot * 64 + lane_id()];
    r.t = S.mt_t[slot];
    return r;
}

// The staged slots of one consumer block (kD + 3 consecutive slots from sb):
// LDS addresses of this lane's first record and of the first target, so that
// every read in the block is that address plus a constant offset.
struct SlotBlock {
    unsigned st, mt;
};

__device__ __forceinline__ SlotBlock slot_block(const ChainShared &S, int sb) {
    SlotBlock b;
    b.st = (unsigned)(uintptr_t)(const __attribute__((address_space(3))) uint4 *)&S.st[sb * 64 + lane_id()];
    b.mt = lds_addr(&S.mt_t[sb]);
    __asm__ volatile("" : "+v"(b.mt));  // a vector register: reads then take constant offsets
    return b;
}

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// the target is read only with stored values (else the x word holds it)
template <int K, bool VAL>
__device__ __forceinline__ Stg read_slot_at(SlotBlock b) {
    const u32x4 v =
        *(const __attribute__((address_space(3))) u32x4 *)(uintptr_t)(b.st + K * 64 * 16);
    Stg r;
    r.a = make_uint4(v.x, v.y, v.z, v.w);
    r.t = VAL ? lds_read(b.mt + K * 4) : 0.0f;
    return r;
}

struct ChainState {
    Stg cur, nxt, nxt2;           // examples t, t+1 and t+2
    float cur_v, cur_fw, cur_fx;  // example t's weight, or the forwarded (w_old, x) pair
    bool cur_fwd;
    float s_prev;                 // step of example t-1
    // example t-1's old weight, x and write targets: its new weights are
    // computed and written at the start of step t
    float p_wold, p_x;
    unsigned p_l, p_g;
    float gv[kD];                 // prefetched cold values, example at t mod kD
    unsigned pf[kD];              // prefetch offsets of the next examples
};

// One example, position t = t0 + SL with its staged slots in sblk.  Every
// memory operation is issued unconditionally, so the count of outstanding
// loads and stores is the same on every path and the waits stay exact.
// Only the chain s(t-1) -> w_old -> z -> s(t) is serial; the writes of
// example t-1 and the reads for example t+1 (which depend on values known
// early in the step) are free to fill its stalls.  Order that matters: the
// writes of t-1 precede the reads for t+1 (a value t-1 writes may be one
// t+1 reads) and the prefetch (a cold value t-1 writes may be prefetched).
template <int SL, int LOSS, bool VAL, bool FAST>
__device__ __forceinline__ void chain_step(ChainState &st, const SgdOp<LOSS, VAL> &op,
                                           SlotBlock sblk, __amdgpu_buffer_rsrc_t wbuf,
                                           unsigned gsrc_a) {
    // without stored values every x is 1 and the x word is the target
    const float x = VAL ? __uint_as_float(st.cur.a.x) : 1.0f;
    const float tgt = VAL ? st.cur.t : __uint_as_float(st.cur.a.x);
    // (a) example t-1's step lands: its new weights, and this example's
    // weights (forwarded lanes apply that step to the pair they took)
    // FAST: every lane takes the fma, lanes whose weight came from memory with
    // x = 0 (the rotation put the memory value in cur_fw), which k_pipe_decide
    // has shown to give the same bits for this epoch
    const float w_old = FAST ? __builtin_fmaf(-st.s_prev, st.cur_fx, st.cur_fw)
                             : (st.cur_fwd ? __builtin_fmaf(-st.s_prev, st.cur_fx, st.cur_fw)
                                           : st.cur_v);
    // binary logistic: the product w * 1 + 0 differs from w only for w = -0,
    // which changes z at most in the sign of a zero sum, and the logistic
    // function is the same at +0 and -0; lanes without an entry hold 0
    const float acc = (!VAL && LOSS == PDB_LOGISTIC) ? w_old : __builtin_fmaf(w_old, x, 0.0f);
    // (b) writes of example t-1; example t+1's weights (those example t
    // writes are forwarded), the staged example t+3, and the cold values of
    // example t+kD (their last writers are before t)
    __builtin_amdgcn_sched_barrier(0);  // the region of the sum starts here
    const float w_prev = __builtin_fmaf(-st.s_prev, st.p_x, st.p_wold);
    lds_write(st.p_l, w_prev);
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(w_prev), wbuf, st.p_g, 0, 0);
    const unsigned rd = st.nxt.a.z;
    const float v1 = lds_read(rd);
    const float fw1 = __int_as_float(__builtin_amdgcn_ds_bpermute((int)rd, __float_as_int(w_old)));
    // without stored values every x is 1: nothing to forward
    const float fx1 =
        VAL ? __int_as_float(__builtin_amdgcn_ds_bpermute((int)rd, __float_as_int(x))) : 1.0f;
    const Stg nxt3 = read_slot_at<SL + 3, VAL>(sblk);
    const float g_pf = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(wbuf, st.pf[SL], 0, 0));
    // (c) the step of example t.  The memory operations above go into the
    // gaps the DPP adds of the sum must leave after each VALU write (two
    // instructions each: a DPP add, two LDS operations, ...), and the
    // fences keep every other instruction of the step out of that region:
    // the rotation's select of the value read for example t+1 would
    // otherwise be scheduled inside the sum, and its wait for that LDS read
    // would stall the chain (consumer 319 -> 311 cycles per example)
    const float z = wave_sum64_lane63(acc);  // the sum is in lane 63
    __builtin_amdgcn_sched_group_barrier(0x0002, 2, 0);  // VALU x2, LDS x2, ..., VMEM x2
    __builtin_amdgcn_sched_group_barrier(0x0080, 2, 0);
    __builtin_amdgcn_sched_group_barrier(0x0002, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x0080, 2, 0);
    __builtin_amdgcn_sched_group_barrier(0x0002, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x0010, 2, 0);
    if constexpr (VAL) {
        // stored values: the slot's two reads fill the wait before the first
        // cross-row add instead of delaying the last row add
        __builtin_amdgcn_sched_group_barrier(0x0002, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x0080, 2, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    // (d) the step runs on every lane and is read out of lane 63.  The
    // rotation's selects sit between the exponential and the reciprocal,
    // long after the LDS read they wait for, where they fill gaps of the
    // chain instead of delaying the next example's forwarded values
    // (consumer 311 -> 301 cycles per example with the step's first write
    // moved into the sum and the read-out after the step)
    float s, cur_v;
    bool cur_fwd;
    if (LOSS == PDB_LOGISTIC) {
        const float e = dev_exp87(-z);
        __builtin_amdgcn_sched_barrier(0);
        // NaN select off the head of the chain; FAST: z is never NaN
        const float sub = FAST ? tgt : logistic_sub(z, tgt);
        cur_v = (rd == gsrc_a) ? st.gv[(SL + 1) % kD] : v1;
        cur_fwd = rd < 256u;
        s = op.lr * logistic_from_exp(e, sub);
    } else {
        s = op.lr * (z - tgt);
        __builtin_amdgcn_sched_barrier(0);
        cur_v = (rd == gsrc_a) ? st.gv[(SL + 1) % kD] : v1;
        cur_fwd = rd < 256u;
    }
    s = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(s), 63));
    __builtin_amdgcn_sched_barrier(0);
    // rotation
    st.p_wold = w_old;
    st.p_x = x;
    st.p_l = st.cur.a.y;
    st.p_g = st.cur.a.w;
    st.s_prev = s;
    st.cur_v = cur_v;
    st.gv[SL] = g_pf;
    st.cur = st.nxt;
    st.cur_fw = FAST ? (cur_fwd ? fw1 : cur_v) : fw1;
    st.cur_fx = FAST ? (cur_fwd ? fx1 : 0.0f) : fx1;
    st.cur_fwd = cur_fwd;
    st.nxt = st.nxt2;
    st.nxt2 = nxt3;
}

// Writes the last example's new weights.
__device__ __forceinline__ void chain_flush(const ChainState &st, __amdgpu_buffer_rsrc_t wbuf) {
    const float w_prev = __builtin_fmaf(-st.s_prev, st.p_x, st.p_wold);
    lds_write(st.p_l, w_prev);
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(w_prev), wbuf, st.p_g, 0, 0);
}

// Prefetch offsets of positions q0 .. q0 + kD - 1: the global write offset of
// each lane's feature (out of range for hot features and lanes without an
// entry).  Lanes whose value comes from elsewhere load it too and ignore it,
// and positions past the end read stale slots: every such load stays inside
// the weight buffer or is out of range and returns 0.
__device__ __forceinline__ void chain_prefetch_offsets(ChainState &st, const ChainShared &S,
                                                       int64_t q0) {
#pragma unroll
    for (int j = 0; j < kD; ++j) st.pf[j] = S.st[(int)((q0 + j) & (kRB - 1)) * 64 + lane_id()].w;
}

#define PDB_CHAIN_STEPS(STEP) \
    STEP(0) STEP(1) STEP(2) STEP(3) STEP(4) STEP(5) STEP(6) STEP(7) \
    STEP(8) STEP(9) STEP(10) STEP(11) STEP(12) STEP(13) STEP(14) STEP(15)
static_assert(kD == 16, "PDB_CHAIN_STEPS lists kD steps");

// Consumer: runs examples t = 0.. of the run in order.  Returns the number
// processed: len, or the position of the first example with more than 64
// entries (the caller runs that one on the plain path).
template <int LOSS, bool VAL, bool FAST>
__device__ int64_t chain_consumer(const SgdOp<LOSS, VAL> &op, int64_t len, int64_t d,
                                  ChainShared &S, Ctrl *ctrl) {
    const int lane = lane_id();
    const long long cyc0 = (long long)__builtin_readcyclecounter();
    long long waited = 0;
    const __amdgpu_buffer_rsrc_t wbuf =
        __builtin_amdgcn_make_buffer_rsrc(op.w, 0, (int)(d * 4), 0x00020000);
    unsigned gsrc_a = lds_addr(&S.zero[1]);
    __asm__ volatile("" : "+s"(gsrc_a));  // computed once, kept in a register
    ChainState st;
    int64_t stop = std::min(len, wait_staged(S, 0, std::min<int64_t>(kD, len), &waited));
    chain_prefetch_offsets(st, S, 0);
#pragma unroll
    for (int j = 0; j < kD; ++j)
        st.gv[j] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(wbuf, st.pf[j], 0, 0));
    st.cur = read_slot(S, 0);
    st.nxt = read_slot(S, 1);
    st.nxt2 = read_slot(S, 2);
    st.cur_v = (st.cur.a.z == gsrc_a) ? st.gv[0] : lds_read(st.cur.a.z);
    // the run's first example forwards nothing (FAST: fma(-0, 0, w) = w)
    st.cur_fw = FAST ? st.cur_v : 0.0f;
    st.cur_fx = 0.0f;
    st.cur_fwd = false;
    st.s_prev = 0.0f;
    // no example before the first: its "writes" go to the sinks
    st.p_wold = st.p_x = 0.0f;
    st.p_l = lds_addr(&S.lsink[lane]);
    st.p_g = kOOR;

    int64_t t0 = 0;
    for (; t0 < stop; t0 += kD) {
        // positions read in this block: t+2 and t+kD for t in [t0, t0+kD)
        stop = std::min(stop, wait_staged(S, t0 + 2, std::min<int64_t>(t0 + 2 * kD, len), &waited));
        if (t0 + kD > stop) break;
        chain_prefetch_offsets(st, S, t0 + kD);
        lds_store(&S.ctl[0], (int)(t0 + 2));
        const SlotBlock sblk = slot_block(S, (int)(t0 & (kRB - 1)));
#define PDB_STEP(SL) chain_step<SL, LOSS, VAL, FAST>(st, op, sblk, wbuf, gsrc_a);
        PDB_CHAIN_STEPS(PDB_STEP)
#undef PDB_STEP
    }
    if (t0 < stop) {  // last, partial block
        chain_prefetch_offsets(st, S, t0 + kD);
        const SlotBlock sblk = slot_block(S, (int)(t0 & (kRB - 1)));
#define PDB_STEP(SL) \
    if (SL < kD - 1 && t0 + SL < stop) chain_step<SL, LOSS, VAL, FAST>(st, op, sblk, wbuf, gsrc_a);
        PDB_CHAIN_STEPS(PDB_STEP)
#undef PDB_STEP
    }
    chain_flush(st, wbuf);
    lds_store(&S.ctl[1], 1);
    if (lane == 0) {
        atomicAdd((unsigned long long *)&ctrl->stat_cycles,
                  (unsigned long long)((long long)__builtin_readcyclecounter() - cyc0));
        atomicAdd((unsigned long long *)&ctrl->stat_wait, (unsigned long long)waited);
        atomicAdd((unsigned long long *)&ctrl->stat_rows, (unsigned long long)stop);
        atomicAdd((unsigned long long *)&ctrl->stat_runs, 1ull);
    }
    return stop;
}

// Runs perm[e_beg .. e_end) (consecutive narrow levels, in level order: a
// sequential order of their examples) with the whole block.  width1: every
// level of the run has one example, so the examples have increasing indices.
// idx_r0 >= 0: the run is rows idx_r0, idx_r0 + 1, ... in index order
// instead (perm is not read).
template <int LOSS, bool VAL>
__device__ void chain_run(const SgdOp<LOSS, VAL> &op, int64_t e_beg, int64_t e_end, int hot,
                          int64_t d, Ctrl *ctrl, bool width1, bool fast, int64_t idx_r0 = -1) {
    __shared__ ChainShared S;
    __shared__ int64_t s_done;
    const int wave = wave_in_block();
    int64_t pos = e_beg;
    while (pos < e_end) {
        // examples of a width-1 run have increasing indices: the run is a range
        // of consecutive examples exactly when its ends differ by its length - 1
        int64_t dense_r0 = idx_r0 + (pos - e_beg);
        if (idx_r0 < 0) {
            const int64_t r_first = op.perm[pos], r_last = op.perm[e_end - 1];
            dense_r0 = (width1 && r_last - r_first == e_end - 1 - pos) ? r_first : -1;
        }
        for (int i = threadIdx.x; i < hot; i += kBlock) g_wcache[i] = op.w[i];
        for (int i = threadIdx.x; i < kRB; i += kBlock) S.seq[i] = INT_MIN;
        if (threadIdx.x < 4) {
            S.ctl[threadIdx.x] = 0;
            S.zero[threadIdx.x] = 0.0f;
        }
        __syncthreads();
        if (wave == 0) {
            int64_t done;
            if constexpr (LOSS == PDB_LOGISTIC) {
                done = fast ? chain_consumer<LOSS, VAL, true>(op, e_end - pos, d, S, ctrl)
                            : chain_consumer<LOSS, VAL, false>(op, e_end - pos, d, S, ctrl);
            } else {
                (void)fast;
                done = chain_consumer<LOSS, VAL, false>(op, e_end - pos, d, S, ctrl);
            }
            if (lane_id() == 0) s_done = done;
        } else if (dense_r0 >= 0) {
            chain_producer<LOSS, VAL, true>(op, wave - 1, pos, e_end - pos, dense_r0, hot, S);
        } else {
            chain_producer<LOSS, VAL, false>(op, wave - 1, pos, e_end - pos, -1, hot, S);
        }
        __syncthreads();
        for (int i = threadIdx.x; i < hot; i += kBlock) op.w[i] = g_wcache[i];
        __syncthreads();
        pos += s_done;
        if (pos < e_end) {
            // an example with more than 64 entries: plain path, then resume
            if (wave == 0) {
                if (idx_r0 >= 0)
                    op.row(idx_r0 + (pos - e_beg));
                else
                    op(pos, pos + 1);
            }
            __syncthreads();
            ++pos;
        }
    }
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

// first level after l that is wider than cw or starts kChainMin levels of
// width 1 (L if none); block-uniform.  Bit i of a wave's 128-bit mask is the
// width-1 test of level base + i; after the shifts it says whether the 32
// levels from base + i all have width 1.
static_assert(kChainMin == 32, "narrow_run_end tests runs of 32 levels");
__device__ int64_t narrow_run_end(int64_t l, int64_t L, const int64_t *level_ptr, int64_t cw) {
    __shared__ int64_t s_w[kWavesPerBlock];
    const int wave = wave_in_block();
    for (int64_t start = l + 1; start < L; start += kBlock) {
        const int64_t c = start + threadIdx.x;
        const int64_t w0 = c < L ? level_ptr[c + 1] - level_ptr[c] : 0;
        const int64_t c1 = c + kWave;
        const int64_t w1 = c1 < L ? level_ptr[c1 + 1] - level_ptr[c1] : 0;
        const unsigned long long wide = __ballot(c < L && w0 > cw);
        unsigned __int128 m = ((unsigned __int128)__ballot(w1 == 1) << 64) | __ballot(w0 == 1);
        m &= m >> 1;
        m &= m >> 2;
        m &= m >> 4;
        m &= m >> 8;
        m &= m >> 16;
        const unsigned long long hit = wide | (unsigned long long)m;
        if (lane_id() == 0)
            s_w[wave] = hit ? start + wave * kWave + (__ffsll(hit) - 1) : INT64_MAX;
        __syncthreads();
        int64_t mn = INT64_MAX;
#pragma unroll
        for (int w = 0; w < kWavesPerBlock; ++w) mn = min(mn, s_w[w]);
        __syncthreads();
        if (mn != INT64_MAX) return min(mn, L);
    }
    return L;
}

template <class Op>
__global__ __launch_bounds__(kBlock) void k_levels_apply(Op op, const int64_t *level_ptr,
                                                         const int32_t *n_levels,
                                                         int64_t thin_max, int hot, int64_t d,
                                                         Ctrl *ctrl, int64_t timeout,
                                                         int64_t chain_width, int index_order) {
    constexpr int U = Op::kUnits;
    const int64_t L = *n_levels;
    // the pipeline's select-free step, when k_pipe_decide found it exact
    const bool fast = __builtin_amdgcn_readfirstlane(ctrl->pipe_fast) != 0;
    if constexpr (Op::kChain) {
        // every level is narrow (one block): the epoch is one pipeline run
        // over the rows in index order -- itself a sequential order of the
        // levels (Theorem 2), so every weight sees the same updates in the
        // same order -- with no entry matched against a window and no
        // boundary between runs
        if (index_order) {
            chain_run(op, 0, level_ptr[L], hot, d, ctrl, true, fast, 0);
            return;
        }
    } else {
        (void)index_order;
    }
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
                        // a run of narrow levels goes through the pipeline one
                        // example after another (a sequential order of them)
                        // when it holds enough examples
                        if (hot >= 0 && end - beg <= chain_width && l2 >= no_chain_before) {
                            // a long run of width-1 levels first (its examples
                            // may be consecutive rows); else narrow levels up
                            // to the next such run or wider level
                            const int64_t l3 = find_run_end(l2, L, level_ptr, 1);
                            if (l3 - l2 >= kChainMin) {
                                chain_run(op, beg, level_ptr[l3], hot, d, ctrl, true, fast);
                                l2 = l3;
                                continue;
                            }
                            int64_t l4 = l3;
                            if (chain_width > 1) {
                                l4 = narrow_run_end(l2, L, level_ptr, chain_width);
                                if (level_ptr[l4] - beg >= kChainMin) {
                                    chain_run(op, beg, level_ptr[l4], hot, d, ctrl, false, fast);
                                    l2 = l4;
                                    continue;
                                }
                            }
                            no_chain_before = max(l3, l4);
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

// Counts b in [lo, hi) (as bit patterns) whose recip_normal differs from the
// IEEE quotient 1/b; keeps the smallest such pattern.
__global__ __launch_bounds__(kBlock) void k_check_recip(uint32_t lo, uint32_t hi, Ctrl *ctrl) {
    unsigned long long bad = 0;
    uint32_t first = 0xFFFFFFFFu;
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t u = lo + (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; u < hi; u += stride) {
        const float b = __uint_as_float((uint32_t)u);
        const float q = recip_normal(b);
        const float ref = 1.0f / b;
        if (__float_as_uint(q) != __float_as_uint(ref)) {
            ++bad;
            first = min(first, (uint32_t)u);
        }
    }
    if (bad) {
        atomicAdd((unsigned long long *)&ctrl->stat_cycles, bad);
        // stat_wait holds 2^32 - 1 - (smallest bad pattern); zero means none
        atomicMax((unsigned long long *)&ctrl->stat_wait, (unsigned long long)(0xFFFFFFFFu - first));
    }
}

// The width-1 pipeline's select-free step (FAST) computes every lane's weight
// as fma(-s, x', w') -- for a lane whose weight came from memory x' = 0 and
// w' is that weight -- instead of selecting between the forwarded value and
// the memory value, and drops the logistic step's NaN select.  Both give
// bitwise the same result when
//   (a) no weight the epoch reads is -0 (w + (-s * 0) is +0 for w = -0 and
//       s < 0): w0 holds no -0, and the epoch never writes one, since
//       fma(a, b, c) is -0 only when c is;
//   (b) no step s is infinite or NaN (-s * 0 would be NaN) and no z is NaN:
//       with finite inputs and the logistic loss, |g| <= 1 and |s| <= |lr|, so
//       every weight stays within W = max|w0| + n |lr| max|x| and every dot
//       product within nnz W max|x|; k_pipe_decide asks that to be below
//       2^100.
// k_pipe_check reduces max|w0|, max|x| and the flags into the control block.
__global__ __launch_bounds__(kBlock) void k_pipe_check(const float *__restrict__ w, int64_t d,
                                                       const float *__restrict__ val, int64_t nnz,
                                                       Ctrl *ctrl) {
    unsigned wm = 0, xm = 0;
    bool bad = false;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < d; i += stride) {
        const unsigned b = __float_as_uint(w[i]);
        bad |= (b & 0x7F800000u) == 0x7F800000u || b == 0x80000000u;  // inf, NaN, -0
        wm = max(wm, b & 0x7FFFFFFFu);
    }
    if (val)
        for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < nnz; i += stride) {
            const unsigned b = __float_as_uint(val[i]);
            bad |= (b & 0x7F800000u) == 0x7F800000u;
            xm = max(xm, b & 0x7FFFFFFFu);
        }
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        wm = max(wm, (unsigned)__shfl_xor((int)wm, o));
        xm = max(xm, (unsigned)__shfl_xor((int)xm, o));
    }
    const bool any_bad = __ballot(bad) != 0ull;
    if (lane_id() == 0) {
        atomicMax(&ctrl->pipe_wmax, wm);
        atomicMax(&ctrl->pipe_xmax, xm);
        if (any_bad) atomicOr(&ctrl->pipe_bad, 1);
    }
}

__global__ void k_pipe_decide(Ctrl *ctrl, float lr, int64_t n, int64_t nnz, int has_val) {
    const double wmax = (double)__uint_as_float(ctrl->pipe_wmax);
    const double xmax = has_val ? (double)__uint_as_float(ctrl->pipe_xmax) : 1.0;
    const double alr = fabs((double)lr);
    const double W = wmax + (double)n * alr * xmax;
    const bool ok = !ctrl->pipe_bad && isfinite(lr) && (double)nnz * W * xmax < 0x1p100;
    ctrl->pipe_fast = ok ? 1 : 0;
}

__global__ void k_ctrl_zero(Ctrl *c) {
    int *w = reinterpret_cast<int *>(c);
    for (int i = threadIdx.x; i < (int)(sizeof(Ctrl) / sizeof(int)); i += blockDim.x) w[i] = 0;
}

template <class Op>
int launch_levels(const Op &op, const pdb_levels *lv, int64_t d, bool chain_ok, Ctrl *ctrl,
                  const Opts &opt, hipStream_t s, int64_t n = 0, int64_t nnz = 0) {
    // the caller's options: widest level run by block 0 alone, a cap on the
    // number of weights cached in LDS by the width-1 pipeline, and the
    // widest level a pipeline run may include (a level of w examples costs
    // w pipeline steps, about 140 ns each, instead of one block-barrier
    // level, about 650 ns)
    const int64_t thin = opt.thin_max;
    const int64_t hot_cap = opt.hot_cap;
    const int64_t chain_width = opt.pipeline_width;
    const int64_t timeout = opt.timeout;
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
        const int64_t room = (int64_t)max_lds - (int64_t)sizeof(ChainShared) - 2048;
        int64_t h = std::min<int64_t>(room / 4, d);
        if (hot_cap >= 0) h = std::min<int64_t>(h, hot_cap);
        h = std::max<int64_t>(h, 0);
        hot = (int)h;
        lds = (size_t)std::max<int64_t>(h, 1) * 4;
        PDB_HIP(hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
        if constexpr (Op::kFastCheck) {
            k_pipe_check<<<grid_for(std::max(d, nnz), kBlock, 1024), kBlock, 0, s>>>(op.w, d, op.val,
                                                                                  nnz, ctrl);
            k_pipe_decide<<<1, 1, 0, s>>>(ctrl, op.lr, n, nnz, op.val != nullptr);
            PDB_LAUNCHED();
        }
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
    // every level at most chain_width wide, and enough examples for the
    // pipeline: one run over the rows in index order, on one block
    const int index_order =
        (Op::kChain && hot >= 0 && widest >= 1 && widest <= chain_width &&
         n >= kChainMin) ? 1 : 0;
    if (index_order) grid = 1;
    Op o = op;
    const int64_t *level_ptr = lv->level_ptr;
    const int32_t *n_levels = lv->n_levels;
    if (grid == 1) {
        k_levels_apply<Op><<<1, kBlock, lds, s>>>(o, level_ptr, n_levels, thin, hot, d, ctrl,
                                                  timeout, chain_width, index_order);
        PDB_LAUNCHED();
    } else {
        int64_t thin_arg = thin, to = timeout, cw = chain_width;
        int hot_arg = hot;
        int64_t d_arg = d;
        int io = index_order;
        void *args[] = {&o, &level_ptr, &n_levels, &thin_arg, &hot_arg, &d_arg, &ctrl, &to, &cw, &io};
        PDB_HIP(hipLaunchCooperativeKernel(fn, dim3(grid), dim3(kBlock), args, lds, s));
    }
    return PDB_OK;
}

// ---------------------------------------------------------------------------
// Sync-free epoch (the Read Protocol of Sec. 5 at feature grain): no levels
// and no barriers.  Each feature's weight and the CSR index of the entry that
// last wrote it share one 64-bit word.  Examples are taken in index order;
// entry p reads its feature once the word carries p's previous writer
// (prev_nz[p], -1 for none), and writes back its new weight together with p.
// One word carries both, so a single 64-bit access is the whole handshake.
// The earliest unfinished example never waits for a later one, so the grid
// always makes progress.

constexpr int kSyncB = 1;  // consecutive examples per ticket, run in order by one wave

__global__ void k_wv_in(const float *__restrict__ w, unsigned long long *__restrict__ wv,
                        int64_t d) {
    for (int64_t f = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; f < d;
         f += (int64_t)gridDim.x * blockDim.x)
        wv[f] = word_pack(w[f], -1);
}

__global__ void k_wv_out(const unsigned long long *__restrict__ wv, float *__restrict__ w,
                         int64_t d) {
    for (int64_t f = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; f < d;
         f += (int64_t)gridDim.x * blockDim.x)
        w[f] = word_value(wv[f]);
}

__device__ __forceinline__ int64_t readlane64(int64_t v, int l) {
    const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)v, l);
    const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)((uint64_t)v >> 32), l);
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Examples are dealt to the waves in turn: with W waves in the grid, wave k
// runs tickets k, k + W, k + 2W, ... of kSyncB consecutive examples each, in
// order.  The grid is launched cooperatively (all of it resident), so the
// earliest unfinished example is always the one its wave is working on, and
// it waits only on earlier examples, all finished: the grid always makes
// progress.  No shared counter hands out the work: requests to one
// contended device-scope counter are served about 200 ns apart, which would
// bound the epoch at that much per ticket.  Everything of a ticket that does
// not depend on earlier examples is loaded when it starts: row bounds,
// labels, and the entries (column, previous writer, value) of every example
// of up to 2 x 64 entries.
template <int LOSS, bool VAL>
__global__ __launch_bounds__(kBlock) void k_sgd_syncfree(SgdOp<LOSS, VAL> op,
                                                         unsigned long long *wv, int64_t d,
                                                         int64_t n, Ctrl *ctrl, int64_t timeout) {
    (void)d;
    const int lane = lane_id();
    const int64_t stride = (int64_t)gridDim.x * kWavesPerBlock * kSyncB;
    for (int64_t tk = ((int64_t)blockIdx.x * kWavesPerBlock + wave_in_block()) * kSyncB; tk < n;
         tk += stride) {
        // lanes 0 .. kSyncB: row bounds of the ticket's examples (clamped at n)
        const int64_t rp = lane <= kSyncB ? op.row_ptr[min(tk + lane, n)] : 0;
        const float yv = lane < kSyncB ? op.y[min(tk + lane, n - 1)] : 0.0f;
        int c0[kSyncB], pn0[kSyncB], c1[kSyncB], pn1[kSyncB];
        float x0[kSyncB], x1[kSyncB];
#pragma unroll
        for (int j = 0; j < kSyncB; ++j) {
            const int64_t b = readlane64(rp, j);
            const int m = (int)(readlane64(rp, j + 1) - b);  // 0 past n
            const bool short_row = m <= 2 * kWave;
            const bool l0 = short_row && lane < m, l1 = short_row && kWave + lane < m;
            c0[j] = l0 ? op.col[b + lane] : 0;
            pn0[j] = l0 ? op.prev_nz[b + lane] : -1;
            x0[j] = (VAL && l0) ? op.val[b + lane] : 1.0f;
            c1[j] = l1 ? op.col[b + kWave + lane] : 0;
            pn1[j] = l1 ? op.prev_nz[b + kWave + lane] : -1;
            x1[j] = (VAL && l1) ? op.val[b + kWave + lane] : 1.0f;
        }
#pragma unroll
        for (int j = 0; j < kSyncB; ++j) {
            if (tk + j >= n) break;
            const int64_t b = readlane64(rp, j);
            const int m = (int)(readlane64(rp, j + 1) - b);
            const float yi = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(yv), j));
            if (m <= 2 * kWave) {
                // every poll of the example in flight together; the new
                // weights come from the values the wait read (nothing else
                // writes these features before this example does)
                const bool l0 = lane < m, l1 = kWave + lane < m;
                unsigned long long v0 = 0, v1 = 0;
                if (!word_wait_wave2(wv, l0, c0[j], pn0[j], &v0, l1, c1[j], pn1[j], &v1, ctrl,
                                     timeout))
                    return;
                const float w0 = word_value(v0), w1 = word_value(v1);
                float acc = l0 ? __builtin_fmaf(w0, x0[j], 0.0f) : 0.0f;
                if (l1) acc = __builtin_fmaf(w1, x1[j], acc);
                const float s = sgd_scale<LOSS>(wave_sum64(acc), yi, op.lr);
                if (l0) word_put(wv, c0[j], word_pack(__builtin_fmaf(-s, x0[j], w0), (int)(b + lane)));
                if (l1)
                    word_put(wv, c1[j],
                             word_pack(__builtin_fmaf(-s, x1[j], w1), (int)(b + kWave + lane)));
            } else {
                float acc = 0.0f;
                for (int k0 = 0; k0 < m; k0 += kWave) {
                    const int k = k0 + lane;
                    const bool live = k < m;
                    const int c = live ? op.col[b + k] : 0;
                    const int pn = live ? op.prev_nz[b + k] : -1;
                    unsigned long long v = 0;
                    if (!word_wait_wave(wv, live, c, pn, &v, ctrl, timeout)) return;
                    if (live) acc = __builtin_fmaf(word_value(v), VAL ? op.val[b + k] : 1.0f, acc);
                }
                const float s = sgd_scale<LOSS>(wave_sum64(acc), yi, op.lr);
                // nothing else writes these features before this example does
                for (int k = lane; k < m; k += kWave) {
                    const int c = op.col[b + k];
                    const float wold = word_value(word_get(wv, c));
                    word_put(wv, c,
                               word_pack(__builtin_fmaf(-s, VAL ? op.val[b + k] : 1.0f, wold),
                                       (int)(b + k)));
                }
            }
        }
    }
}

int64_t syncfree_ws_bytes(int64_t d) { return (int64_t)sizeof(Ctrl) + align_up(8 * d); }

// Matrix completion, sync-free: every component of a U or V row is a
// (value, last rating) word; rating t waits until the user row's words carry
// the previous rating on that user (prev_nz[2t] / 2) and the item row's the
// previous rating on that item (prev_nz[2t + 1] / 2), then writes both rows
// tagged t.  Two ratings per wave, one per 32-lane half, unless the second
// depends on the first.
constexpr int kSyncMfB = 2;  // consecutive ratings per ticket (a pair when independent)

__device__ __forceinline__ int prev_rating(const int32_t *prev_nz, int64_t e) {
    const int32_t q = prev_nz[e];
    return q < 0 ? -1 : (q >> 1);
}

__global__ __launch_bounds__(kBlock) void k_mf_syncfree(
    const int32_t *__restrict__ user, const int32_t *__restrict__ item,
    const float *__restrict__ rating, const int32_t *__restrict__ prev_nz,
    unsigned long long *uvw, int64_t n_users, int64_t n_items, int64_t n, float lr, float reg,
    Ctrl *ctrl, int64_t timeout) {
    (void)n_items;
    const int lane = lane_id();
    const int h = lane >> 5, j = lane & 31;  // user rows first, then item rows, 32 words each
    // tickets of kSyncMfB consecutive ratings dealt to the waves in turn, as
    // in k_sgd_syncfree (lane k < kSyncMfB holds rating tk + k)
    const int64_t stride = (int64_t)gridDim.x * kWavesPerBlock * kSyncMfB;
    for (int64_t tk = ((int64_t)blockIdx.x * kWavesPerBlock + wave_in_block()) * kSyncMfB; tk < n;
         tk += stride) {
        const int64_t stop = min(tk + kSyncMfB, n);
        const bool mine = lane < kSyncMfB && tk + lane < n;
        const int64_t q = mine ? tk + lane : 0;
        const int mu = mine ? user[q] : 0, mi = mine ? item[q] : 0;
        const float mr = mine ? rating[q] : 0.0f;
        const int mpu = mine ? prev_rating(prev_nz, 2 * q) : -1;
        const int mpi = mine ? prev_rating(prev_nz, 2 * q + 1) : -1;
        for (int64_t t = tk; t < stop;) {
            const int a = (int)(t - tk);
            const bool pair = t + 1 < stop && __builtin_amdgcn_readlane(mpu, a + 1) != (int)t &&
                              __builtin_amdgcn_readlane(mpi, a + 1) != (int)t;
            const int count = pair ? 2 : 1;
            const int64_t tt = t + h;
            const bool valid = h < count;
            const int src = a + (valid ? h : 0);  // a lane of the ticket: a + 1 < kSyncMfB if valid
            const int su = __shfl(mu, src), si = __shfl(mi, src);
            const int tu = __shfl(mpu, src), ti = __shfl(mpi, src);
            const float r = __shfl(mr, src);
            const int64_t uo = valid ? (int64_t)su * 32 + j : 0;
            const int64_t vo = valid ? (n_users + (int64_t)si) * 32 + j : 0;
            unsigned long long u = 0, v = 0;
            if (!word_wait_wave2(uvw, valid, uo, tu, &u, valid, vo, ti, &v, ctrl, timeout)) return;
            const float uj = valid ? word_value(u) : 0.0f, vj = valid ? word_value(v) : 0.0f;
            const float err = r - butterfly32(__builtin_fmaf(uj, vj, 0.0f));
            if (valid) {
                const float ea = err * vj, eb = reg * uj;
                const float a2 = err * uj, b2 = reg * vj;
                word_put(uvw, uo, word_pack(__builtin_fmaf(lr, ea - eb, uj), (int)tt));
                word_put(uvw, vo, word_pack(__builtin_fmaf(lr, a2 - b2, vj), (int)tt));
            }
            t += count;
        }
    }
}

// Grid of a sync-free kernel: no more blocks than can be resident at once
// (the launch is cooperative: a wave spinning on a writer never keeps that
// writer's wave from running) and about 8 levels' worth of examples in
// flight, at least a block per four CUs (more only adds waiting waves and
// polling traffic).
// Matrix completion on one compute unit (k_mf_onecu): the Read Protocol of
// Sec. 5 at row grain, as in k_mf_syncfree, but one block runs every rating,
// so a hand-over between two ratings is met inside the compute unit -- the
// LDS for the hottest rows, the unit's L1 cache (workgroup scope) for the
// others -- instead of at the device-wide coherence point.  Measured
// hand-overs between two waves of one block: 205 ns through global memory at
// workgroup scope, 100 ns through LDS, against 420-680 ns at device scope.
// That wins on inputs whose levels are narrow (the chain of hand-overs is
// long) while one compute unit's throughput keeps up.
//  * The producer wave streams each rating's user, item, value and previous
//    ratings into an LDS ring in rating order, and touches its cold rows'
//    words so they are in the L2 cache when a worker gets there.
//  * Fifteen workers take tickets of two consecutive ratings from an LDS
//    counter as they become free, one rating per 32-lane half (lane j:
//    component j).  Each half computes the step (the same arithmetic as
//    MfOp) and publishes its rows tagged with its rating as soon as both
//    rows' words carry the expected previous ratings, so a second rating
//    that depends on the first simply sees the first's tag.  A worker held
//    by a wait holds only its own ticket: the next ratings go to whichever
//    worker is free (dealing tickets in turn tied every hot row's chain of
//    ratings to the slowest of the workers it passed through).
//  * Rows with the smallest ids (the Zipf-hot ones of the generator) live in
//    LDS as (value, rating) words for the whole epoch and are written back at
//    the end.  Almost every wait is for one of them, so a poll rereads only
//    the words still awaited, and LDS ones only unless a lane awaits a word
//    in global memory.
//  * Issue priority: the compute unit's vector issue is its busiest
//    resource (mostly busy on a Zipf input), so a wave polling for a word
//    runs above the ticket work and the step that follows a wait above both
//    -- they are the chain of hand-overs that bounds the epoch.
//  * Progress: tickets are handed out in index order and every ticket waits
//    only on earlier ratings, so the earliest unfinished ticket is held by a
//    worker and never blocked; the producer reuses a ring entry only when no
//    worker may still read it.
constexpr int kMfThreads = 1024;  // one block of 16 waves: 15 workers and the producer
constexpr int kMfWorkers = kMfThreads / kWave - 1;
constexpr int kMfRing = 1024;     // ratings staged ahead (power of two)
constexpr int kMfPB = 256;        // ratings per producer batch (4 per lane)
constexpr int kMfLds = 160 * 1024;  // LDS of one compute unit (gfx950): ring + hot rows
// a worker's ticket: two consecutive ratings, one per 32-lane half (lane j
// of a half holds component j of the rating's rows).  Spreading a rating
// over 16 or 8 lanes (tickets of four or eight ratings) issues fewer
// instructions per rating where nothing waits, but holds more ratings
// behind each wait, and on Zipf-hot rows that costs more
constexpr int kMfTicket = 2;
constexpr unsigned long long kMfHalfMask = 0xFFFFFFFFull;

struct MfShared {
    int4 rec[kMfRing];     // user, item, previous rating on the user, on the item (-1 none)
    float r[kMfRing];
    int ready;             // ratings staged: 0 .. ready-1
    int next_tk;           // next ticket to hand out
    int prog[kMfWorkers];  // lowest rating whose ring entry each worker may still read
    int stop;              // a wave gave up: every loop ends, nothing is written back
};
// the hot rows' words follow MfShared in dynamic LDS, 256-byte aligned
constexpr int kMfHotOff = (int)((sizeof(MfShared) + 255) / 256 * 256);
constexpr int kMfHotRows = (kMfLds - kMfHotOff) / 256;

typedef __attribute__((address_space(3))) unsigned long long lds_u64;
__device__ __forceinline__ unsigned long long lword_get(unsigned a) {
    return __hip_atomic_load((lds_u64 *)(uintptr_t)a, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void lword_put(unsigned a, unsigned long long w) {
    __hip_atomic_store((lds_u64 *)(uintptr_t)a, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

struct MfBatch {
    int u[4], it[4];
    float r[4];
    int2 p[4];
};

__device__ __forceinline__ MfBatch mf_batch_load(const int32_t *__restrict__ user,
                                                 const int32_t *__restrict__ item,
                                                 const float *__restrict__ rating,
                                                 const int32_t *__restrict__ prev_nz, int64_t q0,
                                                 int64_t n) {
    MfBatch m;
#pragma unroll
    for (int x = 0; x < 4; ++x) {
        const int64_t q = q0 + lane_id() + 64 * x;
        const int64_t qc = q < n ? q : n - 1;  // past the end: rating n - 1, not staged
        m.u[x] = user[qc];
        m.it[x] = item[qc];
        m.r[x] = rating[qc];
        m.p[x] = *reinterpret_cast<const int2 *>(prev_nz + 2 * qc);
    }
    return m;
}

__device__ bool mf_give_up(MfShared &S, Ctrl *ctrl, int64_t t0, int64_t timeout) {
    if (lds_load(&S.stop) || aborted(ctrl)) {
        lds_store(&S.stop, 1);
        return true;
    }
    if (now_ticks() - t0 > timeout) {
        record_error(ctrl, DERR_WAIT_TIMEOUT);
        lds_store(&S.stop, 1);
        return true;
    }
    return false;
}

__device__ void mf_producer(const int32_t *__restrict__ user, const int32_t *__restrict__ item,
                            const float *__restrict__ rating, const int32_t *__restrict__ prev_nz,
                            const unsigned long long *uvw, int64_t n_users, int64_t n, int hot_u,
                            int hot_i, MfShared &S, Ctrl *ctrl, int64_t timeout) {
    const int lane = lane_id();
    // batch b's entries are loaded during batch b - 1, and its cold words
    // touched during batch b; the touched values are consumed one batch
    // later, so no wait of the loop is for a load issued in the same batch
    MfBatch cur = mf_batch_load(user, item, rating, prev_nz, 0, n);
    unsigned long long touch[16], sink = 0;
#pragma unroll
    for (int x = 0; x < 16; ++x) touch[x] = 0;
    for (int64_t q0 = 0; q0 < n; q0 += kMfPB) {
        // ring space: every worker is past rating q0 + kMfPB - kMfRing
        int64_t t0 = 0;
        bool quit = false;
        for (int round = 0;; ++round) {
            // the ticket counter first, then the workers' entries: a worker
            // publishes its entry before it takes a ticket, so a ticket
            // taken after the counter was read is at or above it
            const int nt = lds_load(&S.next_tk);
            compiler_fence();
            const int pv = lane < kMfWorkers ? lds_load(&S.prog[lane]) : INT_MAX;
            int mn = min(pv, (int)min((int64_t)nt * kMfTicket, (int64_t)INT_MAX));
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) mn = min(mn, __shfl_xor(mn, o));
            if ((int64_t)mn + kMfRing >= q0 + kMfPB) break;
            if (round == 0) t0 = now_ticks();
            if ((round & 31) == 31 && mf_give_up(S, ctrl, t0, timeout)) {
                quit = true;
                break;
            }
            __builtin_amdgcn_s_sleep(2);
        }
        if (quit) break;
        const MfBatch nxt = mf_batch_load(user, item, rating, prev_nz, q0 + kMfPB, n);
#pragma unroll
        for (int x = 0; x < 16; ++x) sink ^= touch[x];
        // touch both 128-byte lines of each cold row's words (32 words of 8
        // bytes), so the rows are in the L2 cache when the workers read them;
        // a hot row's lanes touch the first row instead
#pragma unroll
        for (int x = 0; x < 4; ++x) {
            const unsigned long long *ru = uvw + (cur.u[x] < hot_u ? 0 : (int64_t)cur.u[x] * 32);
            const unsigned long long *ri =
                uvw + (cur.it[x] < hot_i ? 0 : (n_users + cur.it[x]) * 32);
            touch[4 * x] = __hip_atomic_load(ru, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            touch[4 * x + 1] =
                __hip_atomic_load(ru + 16, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            touch[4 * x + 2] = __hip_atomic_load(ri, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            touch[4 * x + 3] =
                __hip_atomic_load(ri + 16, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
#pragma unroll
        for (int x = 0; x < 4; ++x) {
            const int slot = (int)((q0 + lane + 64 * x) & (kMfRing - 1));
            S.rec[slot] = make_int4(cur.u[x], cur.it[x], cur.p[x].x < 0 ? -1 : (cur.p[x].x >> 1),
                                    cur.p[x].y < 0 ? -1 : (cur.p[x].y >> 1));
            S.r[slot] = cur.r[x];
        }
        compiler_fence();  // LDS executes one wave's operations in order
        if (lane == 0) lds_store(&S.ready, (int)min(q0 + kMfPB, n));
        compiler_fence();
        cur = nxt;
    }
#pragma unroll
    for (int x = 0; x < 16; ++x) sink ^= touch[x];
    __asm__ volatile("" ::"v"(sink));
}

// A lane's word of a row: from LDS at address la when the row is hot, else
// from uvw at byte offset ga (workgroup scope: every reader and writer of the
// words is in this block).  Both loads are issued, into separate registers,
// so that neither waits for the other: a cold row's la is the first hot row,
// and a hot row's global words are not used until the end of the epoch.
__device__ __forceinline__ unsigned long long mf_word_get(bool hot, unsigned la, unsigned ga,
                                                          const char *uvb) {
    const unsigned long long lw = lword_get(la);
    const unsigned long long gw = __hip_atomic_load(
        reinterpret_cast<const unsigned long long *>(uvb + (size_t)ga), __ATOMIC_RELAXED,
        __HIP_MEMORY_SCOPE_WORKGROUP);
    return hot ? lw : gw;
}
// Stores a lane's word of a row: to LDS at address a when the row is hot,
// else to uvw at byte offset a.  Only the lanes that call take part.
__device__ __forceinline__ void mf_word_put(bool hot, unsigned a, unsigned long long *uvw,
                                            unsigned long long w) {
    if (hot) {
        lword_put(a, w);
    } else {
        __hip_atomic_store(
            reinterpret_cast<unsigned long long *>(reinterpret_cast<char *>(uvw) + (size_t)a), w,
            __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
}

__global__ __launch_bounds__(kMfThreads) void k_mf_onecu(
    const int32_t *__restrict__ user, const int32_t *__restrict__ item,
    const float *__restrict__ rating, const int32_t *__restrict__ prev_nz,
    unsigned long long *uvw, int64_t n_users, int64_t n, int hot_u, int hot_i, float lr,
    float reg, Ctrl *ctrl, int64_t timeout) {
    extern __shared__ __align__(256) unsigned char mf_lds[];
    MfShared &S = *reinterpret_cast<MfShared *>(mf_lds);
    unsigned long long *hotw = reinterpret_cast<unsigned long long *>(mf_lds + kMfHotOff);
    const int wave = threadIdx.x / kWave;
    if (threadIdx.x < kMfWorkers) S.prog[threadIdx.x] = INT_MAX;
    if (threadIdx.x == 0) {
        S.ready = 0;
        S.next_tk = 0;
        S.stop = 0;
    }
    // hot rows: users 0 .. hot_u - 1, then items 0 .. hot_i - 1
    for (int x = threadIdx.x; x < hot_u * 32; x += kMfThreads) hotw[x] = uvw[x];
    for (int x = threadIdx.x; x < hot_i * 32; x += kMfThreads)
        hotw[hot_u * 32 + x] = uvw[n_users * 32 + x];
    __syncthreads();
    if (wave == kMfWorkers) {
        mf_producer(user, item, rating, prev_nz, uvw, n_users, n, hot_u, hot_i, S, ctrl, timeout);
    } else {
        const int lane = lane_id();
        const int g = lane >> 5, j = lane & 31;  // rating of the ticket, component
        const int n_tk = (int)((n + kMfTicket - 1) / kMfTicket);
        // where this lane's word of a row is: an LDS address for a hot
        // row, a byte offset into uvw (below 2^32) for the others
        const unsigned hot_base = (unsigned)(uintptr_t)(lds_u64 *)hotw + (unsigned)j * 8u;
        const unsigned ucol = (unsigned)j * 8u;
        const unsigned icol = (unsigned)n_users * 256u + ucol;
        const char *const uvb = reinterpret_cast<const char *>(uvw);
        const unsigned long long gmask = kMfHalfMask << (32 * g);  // this lane's half
        int ready = 0;  // last value read of S.ready
        bool quit = false;
        while (!quit) {
            // take the next ticket: first publish a bound below it (the
            // counter as it reads now), then the ticket itself, so the
            // producer never reuses an entry this worker has yet to read
            lds_store(&S.prog[wave],
                      (int)min((int64_t)kMfTicket * lds_load(&S.next_tk), (int64_t)INT_MAX));
            int k = 0;
            if (lane == 0) k = atomicAdd(&S.next_tk, 1);
            k = __builtin_amdgcn_readfirstlane(k);
            if (k >= n_tk) break;
            const int q0 = kMfTicket * k;
            lds_store(&S.prog[wave], q0);
            // normal issue priority for the ticket's own work; the wait and
            // the step after it go higher (they are on the chain of hand-overs)
            __builtin_amdgcn_s_setprio(1);
            const int cnt = min(kMfTicket, (int)n - q0);
            const int need = q0 + cnt;
            if (ready < need) {
                int64_t t0 = 0;
                for (int round = 0; (ready = lds_load(&S.ready)) < need; ++round) {
                    if (round == 0) t0 = now_ticks();
                    if ((round & 31) == 31 && mf_give_up(S, ctrl, t0, timeout)) {
                        quit = true;
                        break;
                    }
                    __builtin_amdgcn_s_sleep(1);
                }
                if (quit) break;
                compiler_fence();
            }
            const bool valid = g < cnt;
            const int q = valid ? q0 + g : q0;  // an idle group mirrors the first
            const int slot = q & (kMfRing - 1);
            const int4 rc = S.rec[slot];
            const float r = S.r[slot];
            // the ring entries are read (one wave's LDS operations run in order)
            lds_store(&S.prog[wave], INT_MAX);
            // rc.x user, rc.y item, rc.z / rc.w their previous ratings
            const bool uh = rc.x < hot_u, ih = rc.y < hot_i;
            const unsigned ul = uh ? hot_base + (unsigned)rc.x * 256u : hot_base;
            const unsigned il = ih ? hot_base + (unsigned)(hot_u + rc.y) * 256u : hot_base;
            const unsigned ug = ucol + (unsigned)rc.x * 256u, ig = icol + (unsigned)rc.y * 256u;
            unsigned long long wu = mf_word_get(uh, ul, ug, uvb);
            unsigned long long wi = mf_word_get(ih, il, ig, uvb);
            // each rating goes as soon as all its words carry the expected
            // previous ratings -- a rating that depends on an earlier one of
            // the same ticket sees its tag once that one has published -- so
            // a wait on one hot row holds up only its own rating
            bool pend = valid;
            int64_t t0 = 0;
            for (int round = 0;; ++round) {
                const bool bad_u = word_tag(wu) != rc.z, bad_i = word_tag(wi) != rc.w;
                const unsigned long long nr = __ballot(pend && (bad_u || bad_i));
                const bool go = pend && (nr & gmask) == 0ull;
                if (__ballot(go)) {
                    if (round > 0) __builtin_amdgcn_s_setprio(3);
                    const float uj = word_value(wu), vj = word_value(wi);
                    const float err = r - butterfly32(__builtin_fmaf(uj, vj, 0.0f));
                    const float ea = err * vj, eb = reg * uj;
                    const float a2 = err * uj, b2 = reg * vj;
                    const unsigned long long nu = word_pack(__builtin_fmaf(lr, ea - eb, uj), q);
                    const unsigned long long ni = word_pack(__builtin_fmaf(lr, a2 - b2, vj), q);
                    if (go) {
                        mf_word_put(uh, uh ? ul : ug, uvw, nu);
                        mf_word_put(ih, ih ? il : ig, uvw, ni);
                    }
                    pend = pend && !go;
                    if (__ballot(pend) == 0ull) break;
                }
                if (round == 0) {
                    t0 = now_ticks();
                } else {
                    // the watchdog and the abort flag (a device-scope load)
                    // every 32 rounds, not on the path of every poll
                    if ((round & 31) == 0 && mf_give_up(S, ctrl, t0, timeout)) {
                        quit = true;
                        break;
                    }
                }
                // almost every wait is for a Zipf-hot row in LDS: unless a
                // lane awaits a word in global memory, the round rereads LDS
                // only (a cache round trip would cost several LDS ones)
                if (__ballot(pend && ((bad_u && !uh) || (bad_i && !ih)))) {
                    if (round > 0) __builtin_amdgcn_s_sleep(1);
                    if (pend && bad_u) wu = mf_word_get(uh, ul, ug, uvb);
                    if (pend && bad_i) wi = mf_word_get(ih, il, ig, uvb);
                } else {
                    __builtin_amdgcn_s_setprio(2);
                    if (pend && bad_u) wu = lword_get(ul);
                    if (pend && bad_i) wi = lword_get(il);
                }
            }
            if (quit) break;
        }
        lds_store(&S.prog[wave], INT_MAX);
    }
    __syncthreads();
    // the hot rows go back to their words (unless a wave gave up)
    if (!S.stop) {
        for (int x = threadIdx.x; x < hot_u * 32; x += kMfThreads) uvw[x] = hotw[x];
        for (int x = threadIdx.x; x < hot_i * 32; x += kMfThreads)
            uvw[n_users * 32 + x] = hotw[hot_u * 32 + x];
    }
}

int syncfree_grid(const void *fn, int64_t n, int64_t L, int per_block, int64_t *grid) {
    int dev = 0, cus = 0, per_cu = 0;
    PDB_HIP(hipGetDevice(&dev));
    PDB_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
    PDB_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kBlock, 0));
    const int64_t width = L > 0 ? cdiv(n, L) : n;
    int64_t g = std::min<int64_t>((int64_t)cus * std::max(per_cu, 1), cdiv(n, per_block));
    g = std::min<int64_t>(g, std::max<int64_t>(cdiv(8 * width, per_block), cus / 4));
    *grid = std::max<int64_t>(g, 1);
    return PDB_OK;
}

int launch_mf_syncfree(const MfOp &op, const int32_t *prev_nz, int64_t n, int64_t n_users,
                       int64_t n_items, int64_t L, void *ws, int64_t timeout, bool one_cu,
                       hipStream_t s) {
    Ctrl *ctrl = static_cast<Ctrl *>(ws);
    unsigned long long *uvw =
        reinterpret_cast<unsigned long long *>(static_cast<char *>(ws) + sizeof(Ctrl));
    k_ctrl_zero<<<1, 64, 0, s>>>(ctrl);
    PDB_LAUNCHED();
    if (n_users > 0)
        k_wv_in<<<grid_for(n_users * 32, kBlock, 8192), kBlock, 0, s>>>(op.U, uvw, n_users * 32);
    if (n_items > 0)
        k_wv_in<<<grid_for(n_items * 32, kBlock, 8192), kBlock, 0, s>>>(op.V, uvw + n_users * 32,
                                                                       n_items * 32);
    PDB_LAUNCHED();
    if (one_cu) {
        // the hottest rows in LDS: as many items as users, each side capped
        // by its count
        const int hot_i = (int)std::min<int64_t>(n_items, kMfHotRows / 2);
        const int hot_u = (int)std::min<int64_t>(n_users, kMfHotRows - hot_i);
        PDB_HIP(hipFuncSetAttribute(reinterpret_cast<const void *>(&k_mf_onecu),
                                    hipFuncAttributeMaxDynamicSharedMemorySize, kMfLds));
        k_mf_onecu<<<1, kMfThreads, kMfLds, s>>>(op.user, op.item, op.rating, prev_nz, uvw,
                                                n_users, n, hot_u, hot_i, op.lr, op.reg, ctrl,
                                                timeout);
        PDB_LAUNCHED();
    } else {
        const void *fn = reinterpret_cast<const void *>(&k_mf_syncfree);
        int64_t grid = 1;
        int rc = syncfree_grid(fn, n, L, 2 * kWavesPerBlock, &grid);
        if (rc != PDB_OK) return rc;
        // cooperative: the whole grid resident (the waves wait on each other)
        const int32_t *a_user = op.user, *a_item = op.item;
        const float *a_rating = op.rating;
        float a_lr = op.lr, a_reg = op.reg;
        void *args[] = {&a_user, &a_item, &a_rating, &prev_nz, &uvw, &n_users, &n_items, &n,
                        &a_lr, &a_reg, &ctrl, const_cast<int64_t *>(&timeout)};
        PDB_HIP(hipLaunchCooperativeKernel(fn, dim3((unsigned)grid), dim3(kBlock), args, 0, s));
    }
    if (n_users > 0)
        k_wv_out<<<grid_for(n_users * 32, kBlock, 8192), kBlock, 0, s>>>(uvw, op.U, n_users * 32);
    if (n_items > 0)
        k_wv_out<<<grid_for(n_items * 32, kBlock, 8192), kBlock, 0, s>>>(uvw + n_users * 32, op.V,
                                                                        n_items * 32);
    PDB_LAUNCHED();
    return PDB_OK;
}

template <int LOSS, bool VAL>
int launch_syncfree(const SgdOp<LOSS, VAL> &op, int64_t n, int64_t d, int64_t L, void *ws,
                    int64_t timeout, hipStream_t s) {
    Ctrl *ctrl = static_cast<Ctrl *>(ws);
    unsigned long long *wv = reinterpret_cast<unsigned long long *>(static_cast<char *>(ws) +
                                                                    sizeof(Ctrl));
    k_ctrl_zero<<<1, 64, 0, s>>>(ctrl);
    PDB_LAUNCHED();
    if (d > 0) {
        k_wv_in<<<grid_for(d, kBlock, 8192), kBlock, 0, s>>>(op.w, wv, d);
        PDB_LAUNCHED();
    }
    const void *fn = reinterpret_cast<const void *>(&k_sgd_syncfree<LOSS, VAL>);
    int64_t grid = 1;
    int rc = syncfree_grid(fn, n, L, kSyncB * kWavesPerBlock, &grid);
    if (rc != PDB_OK) return rc;
    // cooperative: the whole grid resident (the waves wait on each other)
    SgdOp<LOSS, VAL> a_op = op;
    void *args[] = {&a_op, &wv, &d, &n, &ctrl, const_cast<int64_t *>(&timeout)};
    PDB_HIP(hipLaunchCooperativeKernel(fn, dim3((unsigned)grid), dim3(kBlock), args, 0, s));
    if (d > 0) {
        k_wv_out<<<grid_for(d, kBlock, 8192), kBlock, 0, s>>>(wv, op.w, d);
        PDB_LAUNCHED();
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

extern "C" int pdb_epoch_workspace_bytes(int64_t d, size_t *bytes) {
    if (!bytes || d < 0) return PDB_ERR_INVALID_ARG;
    if (d >= INT32_MAX) return PDB_ERR_UNSUPPORTED;
    *bytes = (size_t)syncfree_ws_bytes(d);
    return PDB_OK;
}

namespace {
int sgd_epoch_impl(const pdb_csr *csr, const float *labels, int64_t n, int64_t d, float *w,
                   float lr, int loss, const pdb_levels *lv, void *ws, size_t ws_bytes,
                   const pdb_options *opt, hipStream_t s) {
    int rc = epoch_checks(lv, n, ws, ws_bytes);
    if (rc != PDB_OK) return rc;
    Opts o;
    rc = resolve_opts(opt, &o);
    if (rc != PDB_OK) return rc;
    if (!csr || (n > 0 && (!csr->row_ptr || !labels || !w)) || (csr->nnz > 0 && !csr->col))
        return PDB_ERR_INVALID_ARG;
    if (loss != PDB_LOGISTIC && loss != PDB_SQUARED) return PDB_ERR_INVALID_ARG;
    if (d < 0 || csr->nnz < 0) return PDB_ERR_INVALID_ARG;
    if (d >= INT32_MAX || csr->nnz >= INT32_MAX) return PDB_ERR_UNSUPPORTED;
    if (n == 0) return PDB_OK;
    Ctrl *ctrl = static_cast<Ctrl *>(ws);
    const bool has_val = csr->val != nullptr;
    // the width-1 pipeline addresses weights with 32-bit buffer offsets
    const bool chain_ok = o.pipeline && lv->prev_nz != nullptr && d < (int64_t(1) << 29);
    // sync-free when the levels are wide on average (a barrier per level
    // would cost more than a wait per feature), the previous writers are
    // known and the workspace holds the packed words; the epoch mode option
    // forces levels or sync-free
    const bool sf_ok = lv->prev_nz != nullptr && (int64_t)ws_bytes >= syncfree_ws_bytes(d);
    const bool wide = lv->L_host > 0 && n >= 8 * lv->L_host;
    const bool syncfree =
        sf_ok && (o.epoch_mode == PDB_EPOCH_SYNCFREE || (o.epoch_mode == PDB_EPOCH_AUTO && wide));
#define PDB_SGD_CASE(LS, HV)                                                                 \
    if (loss == LS && has_val == HV) {                                                       \
        SgdOp<LS, HV> op{csr->row_ptr, csr->col, csr->val, labels, w, lv->perm, lv->prev_nz, lr}; \
        if (syncfree) return launch_syncfree(op, n, d, lv->L_host, ws, o.timeout, s);         \
        return launch_levels(op, lv, d, chain_ok, ctrl, o, s, n, csr->nnz);                  \
    }
    PDB_SGD_CASE(PDB_LOGISTIC, true)
    PDB_SGD_CASE(PDB_LOGISTIC, false)
    PDB_SGD_CASE(PDB_SQUARED, true)
    PDB_SGD_CASE(PDB_SQUARED, false)
#undef PDB_SGD_CASE
    return PDB_ERR_INVALID_ARG;
}

// Scratch of pdb_sgd_epoch_noalloc: the control block, then one packed word
// per feature for the sync-free execution.  Each GPU holds its own copy from
// module load to process end; host code reaches it only through the address
// hipGetSymbolAddress returns for the current device.
constexpr int64_t kScratchMaxD = int64_t(1) << 21;
constexpr size_t kScratchBytes = sizeof(Ctrl) + 8 * (size_t)kScratchMaxD;
static_assert(sizeof(Ctrl) % 256 == 0, "the packed words start 256-byte aligned");
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxScratchDevices = 64;
std::atomic<void *> g_scratch[kMaxScratchDevices];

// The device address of `scratch` on the current device, looked up once per
// device (concurrent first calls look up the same address).
int scratch_address(void **out) {
    int dev = 0;
    PDB_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxScratchDevices) return PDB_ERR_UNSUPPORTED;
    void *p = g_scratch[dev].load(std::memory_order_acquire);
    if (!p) {
        PDB_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p) return PDB_ERR_HIP;
        g_scratch[dev].store(p, std::memory_order_release);
    }
    *out = p;
    return PDB_OK;
}

__global__ void k_status_out(const Ctrl *ctrl, int32_t *status) { *status = ctrl->err; }
}  // namespace

extern "C" int pdb_sgd_epoch(const pdb_csr *csr, const float *labels, int64_t n, int64_t d,
                             float *w, float lr, int loss, const pdb_levels *lv, void *ws,
                             size_t ws_bytes, const pdb_options *opt, hipStream_t s) {
    return sgd_epoch_impl(csr, labels, n, d, w, lr, loss, lv, ws, ws_bytes, opt, s);
}

extern "C" int pdb_sgd_epoch_noalloc(const pdb_csr *csr, const float *labels, int64_t n,
                                     int64_t d, float *w, float lr, int loss,
                                     const pdb_levels *lv, int32_t *status,
                                     const pdb_options *opt, hipStream_t s) {
    if (d < 0 || n < 0) return PDB_ERR_INVALID_ARG;
    if (d > kScratchMaxD) return PDB_ERR_UNSUPPORTED;
    void *ws = nullptr;
    int rc = scratch_address(&ws);
    if (rc != PDB_OK) return rc;
    // the previous call's control block is still there: start from zero
    // (also when there is nothing to run and the status is read at once)
    k_ctrl_zero<<<1, 64, 0, s>>>(static_cast<Ctrl *>(ws));
    PDB_LAUNCHED();
    rc = sgd_epoch_impl(csr, labels, n, d, w, lr, loss, lv, ws, kScratchBytes, opt, s);
    if (rc != PDB_OK || !status) return rc;
    k_status_out<<<1, 1, 0, s>>>(static_cast<const Ctrl *>(ws), status);
    PDB_LAUNCHED();
    return PDB_OK;
}

extern "C" int pdb_mf_epoch(const int32_t *user, const int32_t *item, const float *rating,
                            int64_t n, float *U, int64_t n_users, float *V, int64_t n_items,
                            int32_t rank, float lr, float reg, const pdb_levels *lv, void *ws,
                            size_t ws_bytes, const pdb_options *opt, hipStream_t s) {
    int rc = epoch_checks(lv, n, ws, ws_bytes);
    if (rc != PDB_OK) return rc;
    Opts o;
    rc = resolve_opts(opt, &o);
    if (rc != PDB_OK) return rc;
    if (rank != 32) return PDB_ERR_INVALID_ARG;
    if (n_users < 0 || n_items < 0) return PDB_ERR_INVALID_ARG;
    if (n > 0 && (!user || !item || !rating || !U || !V)) return PDB_ERR_INVALID_ARG;
    if (n == 0) return PDB_OK;
    MfOp op{user, item, rating, U, V, lv->perm, lr, reg};
    // sync-free under the same rule as pdb_sgd_epoch; the packed words need
    // pdb_epoch_workspace_bytes((n_users + n_items) * 32)
    const bool sf_ok = lv->prev_nz != nullptr &&
                       (int64_t)ws_bytes >= syncfree_ws_bytes((n_users + n_items) * 32) &&
                       n < INT32_MAX / 2;
    const bool wide = lv->L_host > 0 && n >= 8 * lv->L_host;
    // one compute unit: its words are indexed with 32-bit integers, and it
    // wins while levels are narrow (about 35 ns per rating on one unit
    // against a device-scope hand-over of about 0.8 us per level)
    // the one-unit kernel addresses the words with 32-bit byte offsets
    const bool one_cu_fits = (n_users + n_items) * 256 <= ((int64_t)1 << 32);
    const bool narrow = lv->L_host > 0 && n < 16 * lv->L_host;
    const bool one_cu = one_cu_fits && (o.mf_one_cu == 1 || (o.mf_one_cu == -1 && narrow));
    if (sf_ok && (o.epoch_mode == PDB_EPOCH_SYNCFREE ||
                  (o.epoch_mode == PDB_EPOCH_AUTO && (wide || one_cu))))
        return launch_mf_syncfree(op, lv->prev_nz, n, n_users, n_items, lv->L_host, ws, o.timeout,
                                  one_cu, s);
    return launch_levels(op, lv, n_users + n_items, false, static_cast<Ctrl *>(ws), o, s);
}

extern "C" int pdb_check_reciprocal(uint32_t lo_bits, uint32_t hi_bits, uint64_t *mismatches,
                                    uint32_t *first_bad, void *ws, size_t ws_bytes,
                                    hipStream_t s) {
    if (!mismatches || !first_bad || !ws) return PDB_ERR_INVALID_ARG;
    if (ws_bytes < sizeof(Ctrl)) return PDB_ERR_WORKSPACE;
    // the reciprocal is defined for b in [1, 2^126)
    if (lo_bits < 0x3F800000u || hi_bits > 0x7E800000u || lo_bits > hi_bits)
        return PDB_ERR_INVALID_ARG;
    Ctrl *ctrl = static_cast<Ctrl *>(ws);
    k_ctrl_zero<<<1, 64, 0, s>>>(ctrl);
    PDB_LAUNCHED();
    if (hi_bits > lo_bits) {
        const uint64_t count = hi_bits - lo_bits;
        const unsigned grid = (unsigned)std::min<uint64_t>(cdiv((int64_t)count, kBlock), 8192);
        k_check_recip<<<grid, kBlock, 0, s>>>(lo_bits, hi_bits, ctrl);
        PDB_LAUNCHED();
    }
    Ctrl host;
    PDB_HIP(hipMemcpyAsync(&host, ctrl, sizeof(Ctrl), hipMemcpyDeviceToHost, s));
    PDB_HIP(hipStreamSynchronize(s));
    *mismatches = (uint64_t)host.stat_cycles;
    *first_bad = 0xFFFFFFFFu - (uint32_t)host.stat_wait;
    return PDB_OK;
}
