// Per-example arithmetic shared by the epoch kernels (gfx950, wave64): the
// exponential and reciprocal of the logistic step, the lane reductions of
// the matched summation order, and the step scale s = lr * g.  Internal
// header, not installed.
#pragma once

#include "pdb_internal.h"

namespace pdbk {

// e^x for x <= 87 (larger x count as 87): k = rint(x log2 e), r = x - k ln 2
// with ln 2 in two binary32 pieces, e^r from its Taylor series through r^7
// (pairs c_j + c_{j+1} r, combined by Horner's rule in r^2: one instruction
// fewer than Estrin's r^4 at the same depth of four, which counts on the
// width-1 pipeline's one wave -- 6 cycles per example), times 2^k by ldexp:
// one rounding into the subnormals.  A NaN x gives some
// finite value: the callers carry NaN past this function (logistic_grad), so
// that no select sits on the serial path of a dependent chain.
__device__ __forceinline__ float dev_exp87(float x) {
    // branch-free: the arithmetic runs on x clamped to [-104, 87] (one med3);
    // below the bottom that gives the same answer (e^-104 rounds to 0)
    const float xc = __builtin_amdgcn_fmed3f(x, -104.0f, 87.0f);
    const float kf = __builtin_rintf(xc * 0x1.715476p+0f);
    float r = __builtin_fmaf(-kf, 0x1.62e430p-1f, xc);
    r = __builtin_fmaf(-kf, -0x1.05c610p-29f, r);
    const float r2 = r * r;
    const float p01 = __builtin_fmaf(1.0f, r, 1.0f);
    const float p23 = __builtin_fmaf(0x1.555556p-3f, r, 0.5f);            // 1/6, 1/2
    const float p45 = __builtin_fmaf(0x1.111112p-7f, r, 0x1.555556p-5f);  // 1/120, 1/24
    const float p67 = __builtin_fmaf(0x1.a01a02p-13f, r, 0x1.6c16c2p-10f);  // 1/5040, 1/720
    const float q = __builtin_fmaf(__builtin_fmaf(__builtin_fmaf(p67, r2, p45), r2, p23), r2, p01);
    return __builtin_amdgcn_ldexpf(q, (int)kf);
}

// 1/b, correctly rounded, for b in [1, 2^126) (NaN gives NaN): y0 = v_rcp,
// then one Newton step y0 + y0 (1 - b y0) with the residual exact in an fma.
// On gfx950 this gives the IEEE quotient for every b in the range -- an
// exhaustive property of the hardware reciprocal, not a theorem: v_rcp alone
// is off in about a tenth of the cases, the corrected value in none.
// pdb_check_reciprocal repeats that comparison on the device at hand.  The
// range keeps the quotient a normal number, so no scaling is needed.
__device__ __forceinline__ float recip_normal(float b) {
    const float y0 = __builtin_amdgcn_rcpf(b);
    return __builtin_fmaf(__builtin_fmaf(-b, y0, 1.0f), y0, y0);
}

// The gradient factor of the logistic loss, g = 1/(1 + e^min(-z, 87)) - tgt:
// the cap keeps 1 + e below 2^126 (e^87 < 2^126), where recip_normal is
// exact.  A NaN z gives a NaN g (the logistic function of NaN is NaN); the
// NaN enters through the subtrahend, chosen while the exponential is still
// being evaluated.
__device__ __forceinline__ float logistic_sub(float z, float tgt) { return (z == z) ? tgt : -z; }
__device__ __forceinline__ float logistic_from_exp(float e, float sub) {
    return recip_normal(1.0f + e) - sub;
}
__device__ __forceinline__ float logistic_grad(float z, float tgt) {
    return logistic_from_exp(dev_exp87(-z), logistic_sub(z, tgt));
}

// v + v[partner] with the partner chosen by a DPP lane pattern
template <int CTRL>
__device__ __forceinline__ float dpp_add(float v) {
    return v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, true));
}

// Intra-row part of the butterfly p_l <- p_l + p_{l xor o}, o = 1, 2, 4, 8:
// o = 1, 2 are quad permutations; o = 4 is the mirror within each group of 8
// lanes -- once the quads hold equal values the mirrored partner holds the
// same value as lane l xor 4; o = 8 is the mirror within each row of 16,
// likewise.  Every lane of row r ends with the row's sum R_r.
__device__ __forceinline__ float butterfly16(float v) {
    v = dpp_add<0xB1>(v);   // quad_perm [1,0,3,2]
    v = dpp_add<0x4E>(v);   // quad_perm [2,3,0,1]
    v = dpp_add<0x141>(v);  // row_half_mirror
    return dpp_add<0x140>(v);  // row_mirror
}

// Sum over the 64 lanes, bitwise the xor butterfly for o = 1, ..., 32, whose
// common result is (R_0 + R_1) + (R_2 + R_3).  After the intra-row part,
// row_bcast:15 adds lane 15 of the previous row (row 3 then holds R_3 + R_2,
// row 1 R_1 + R_0) and row_bcast:31 adds lane 31 to rows 2 and 3, so lane 63
// holds (R_3 + R_2) + (R_1 + R_0): the same sums, each with its operands
// swapped, which IEEE addition does not notice.  Rows without a source lane
// add their own value; they are not read.  The result is read out of lane 63
// as a wave-uniform value: two DPP adds and a readlane instead of two
// cross-row swaps.  wave_sum64_lane63 leaves the sum in lane 63 (a caller
// that computes on from there reads its result out of lane 63 later).
__device__ __forceinline__ float wave_sum64_lane63(float v) {
    v = butterfly16(v);
    v = dpp_add<0x142>(v);  // row_bcast:15
    return dpp_add<0x143>(v);  // row_bcast:31
}
__device__ __forceinline__ float wave_sum64(float v) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wave_sum64_lane63(v)), 63));
}

// The butterfly over each 32-lane half (o = 1..16); lanes of half h get half
// h's sum R_{2h} + R_{2h+1} (the row swap pairs rows 0-1 and 2-3).
__device__ __forceinline__ float butterfly32(float v) {
    v = butterfly16(v);
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int LOSS>
__device__ __forceinline__ float sgd_scale(float z, float y, float lr) {
    float g;
    if (LOSS == PDB_LOGISTIC) {
        g = logistic_grad(z, y > 0.0f ? 1.0f : 0.0f);
    } else {
        g = z - y;
    }
    return lr * g;
}

}  // namespace pdbk
