// Packed (value, tag) words of the sync-free kernels (gfx950, wave64): a
// binary32 value and the 32-bit tag of the writer that produced it share one
// 64-bit word, so a single device-scope access reads or publishes both and
// a reader never sees a value with another writer's tag.  Internal header,
// not installed.
#pragma once

#include "pdb_internal.h"

namespace pdbk {

__device__ __forceinline__ unsigned long long word_pack(float v, int tag) {
    return ((unsigned long long)(unsigned)tag << 32) | (unsigned long long)__float_as_uint(v);
}
__device__ __forceinline__ float word_value(unsigned long long w) {
    return __uint_as_float((unsigned)w);
}
__device__ __forceinline__ int word_tag(unsigned long long w) { return (int)(unsigned)(w >> 32); }

// device-scope 64-bit accesses: single-copy atomic
__device__ __forceinline__ unsigned long long word_get(unsigned long long *base, int64_t i) {
    return __hip_atomic_load(&base[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void word_put(unsigned long long *base, int64_t i,
                                         unsigned long long w) {
    __hip_atomic_store(&base[i], w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// workgroup-scope 64-bit accesses: the waves of one block share the compute
// unit's vector L1 cache, which serves these without a trip to the L2
__device__ __forceinline__ unsigned long long word_get_wg(const unsigned long long *base,
                                                          int64_t i) {
    return __hip_atomic_load(&base[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void word_put_wg(unsigned long long *base, int64_t i,
                                            unsigned long long w) {
    __hip_atomic_store(&base[i], w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Sleeps about 2^min(round, 3) x 64 cycles (s_sleep takes a constant):
// for waits where many words of many blocks are polled at once (mini-batch
// unions, dense partial sums), so that waiting waves do not crowd the
// frontier's accesses.
__device__ __forceinline__ void word_backoff(int round) {
    switch (round < 3 ? round : 3) {
        case 0: __builtin_amdgcn_s_sleep(1); break;
        case 1: __builtin_amdgcn_s_sleep(2); break;
        case 2: __builtin_amdgcn_s_sleep(4); break;
        default: __builtin_amdgcn_s_sleep(8); break;
    }
}

// Sleeps 64 cycles, then 128 from the second round on: for the per-example
// waits of the sync-free epochs, where a longer back-off only delays the wave
// that is next on the chain (capped at 512 cycles it cost the config-4 epoch
// 12%: 38.9 ms against 34.7 ms; the mini-batch epoch's union waits instead
// lost 30% with this one).
__device__ __forceinline__ void word_backoff_short(int round) {
    if (round == 0) __builtin_amdgcn_s_sleep(1);
    else __builtin_amdgcn_s_sleep(2);
}

// The abort flag and the watchdog are read every 8 poll rounds: the flag is
// a device-scope load, and reading it every round put one more such load on
// every poll.
__device__ __forceinline__ bool word_check_due(int round) { return (round & 7) == 7; }

// Polls word idx (one per lane; lanes with want = false only take part in
// the rounds) until it carries tag; the whole wave backs off while nothing
// arrives.  False on timeout or abort.
__device__ __forceinline__ bool word_wait_wave(unsigned long long *base, bool want, int64_t idx,
                                               int tag, unsigned long long *out, Ctrl *ctrl,
                                               int64_t timeout) {
    bool ready = !want;
    int64_t t0 = 0;
    for (int round = 0;; ++round) {
        if (!ready) {
            const unsigned long long v = word_get(base, idx);
            if (word_tag(v) == tag) {
                *out = v;
                ready = true;
            }
        }
        if (__ballot(!ready) == 0ull) return true;
        if (round == 0) t0 = now_ticks();
        if (word_check_due(round)) {
            if (aborted(ctrl)) return false;
            if (now_ticks() - t0 > timeout) {
                record_error(ctrl, DERR_WAIT_TIMEOUT);
                return false;
            }
        }
        word_backoff_short(round);
        __asm__ __volatile__("" ::: "memory");  // the next round loads again
    }
}

// Polls two words per lane as word_wait_wave does one (want0/want1 say which
// this lane needs); both polls are in flight together every round.
__device__ __forceinline__ bool word_wait_wave2(unsigned long long *base, bool want0, int64_t idx0,
                                                int tag0, unsigned long long *out0, bool want1,
                                                int64_t idx1, int tag1, unsigned long long *out1,
                                                Ctrl *ctrl, int64_t timeout) {
    bool ready0 = !want0, ready1 = !want1;
    int64_t t0 = 0;
    for (int round = 0;; ++round) {
        unsigned long long v0 = 0, v1 = 0;
        if (!ready0) v0 = word_get(base, idx0);
        if (!ready1) v1 = word_get(base, idx1);
        if (!ready0 && word_tag(v0) == tag0) {
            *out0 = v0;
            ready0 = true;
        }
        if (!ready1 && word_tag(v1) == tag1) {
            *out1 = v1;
            ready1 = true;
        }
        if (__ballot(!(ready0 && ready1)) == 0ull) return true;
        if (round == 0) t0 = now_ticks();
        if (word_check_due(round)) {
            if (aborted(ctrl)) return false;
            if (now_ticks() - t0 > timeout) {
                record_error(ctrl, DERR_WAIT_TIMEOUT);
                return false;
            }
        }
        word_backoff_short(round);
        __asm__ __volatile__("" ::: "memory");  // the next round loads again
    }
}

}  // namespace pdbk
