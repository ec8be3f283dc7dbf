// score_mods.h -- device helpers for the Score and Norm stages of attention.
//
// Score modifications act on the scaled raw score s = scale * q . k before
// the mask (Appendix A, "Score Modifications"): the soft-cap C * tanh(s / C)
// ("Softcap Attention"), then the additive position biases: ALiBi
// -slope_h * |i' - j| and the relative position term (i' - j) ("Relative
// Position Embeddings"). The softmax kernels run in base 2, so their scores
// carry a factor log2(e) ("unit"); ReLU and Sigmoid normalisation (Appendix
// A, "Normalization Variants") work on natural scores (unit 1).
#pragma once

#include <hip/hip_runtime.h>

namespace attn {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Additive position bias selected at compile time.
enum : int {
    kBiasNone = 0,
    kBiasAlibi = 1,    // bias_abs * |i' - j|, bias_abs = -slope_h * unit
    kBiasRelPos = 2,   // bias_lin * (jref - j), bias_lin = unit
    kBiasGeneral = 3,  // both terms, coefficients possibly zero
};

// Normalisation selected at compile time.
enum : int { kNormSoftmax = 0, kNormRelu = 1, kNormSigmoid = 2 };

// tanh for fp32 with small relative error over the whole line (<= ~2e-6,
// so the soft-capped score C tanh(s/C) keeps a relative error of that order
// whatever C is). |x| < 1/16: x - x^3/3 (the first dropped term, 2x^5/15, is
// below 2.1e-6 x there). Elsewhere, for either sign, 1 - 2/(1 + e^(2x)):
// with |tanh x| >= 0.0624 its absolute error (about 2e-7 from the exp and
// reciprocal) is below 3.3e-6 relative; it tends to +-1 without overflow.
__device__ __forceinline__ float tanh_f32(float x)
{
    const float x2 = x * x;
    const float cubic = __builtin_fmaf(x2 * x, -1.0f / 3.0f, x);
    const float e = __builtin_amdgcn_exp2f(x * (2.0f * kLog2e));
    const float t = __builtin_fmaf(-2.0f, __builtin_amdgcn_rcpf(1.0f + e), 1.0f);
    return __builtin_fabsf(x) < 0.0625f ? cubic : t;
}

// Final score, in units, of a raw dot product `dot` for the query at key-axis
// position ip and key j. The relative-position term is taken against jref:
// softmax is unchanged by a per-row constant, so the softmax kernels use
// jref = the row's first visible key (the largest bias, keeping the dominant
// scores small in magnitude) and add (ip - jref) back to the LSE; the other
// normalisations use jref = ip, the literal (i' - j).
template <bool SOFTCAP, int BIAS>
__device__ __forceinline__ float score_u(float dot, float scale_u, float softcap_pre,
                                         float softcap_post_u, float bias_abs, float bias_lin,
                                         int ip, int jref, int j)
{
    float t;
    if constexpr (SOFTCAP)
        t = softcap_post_u * tanh_f32(dot * softcap_pre);
    else
        t = dot * scale_u;
    if constexpr (BIAS == kBiasAlibi || BIAS == kBiasGeneral)
        t = __builtin_fmaf(bias_abs, __builtin_fabsf((float)(ip - j)), t);
    if constexpr (BIAS == kBiasRelPos || BIAS == kBiasGeneral)
        t = __builtin_fmaf(bias_lin, (float)(jref - j), t);
    return t;
}

// C' tanh(dot * pre) with C' = C * unit, the soft-cap of score_u with the
// outer product folded into the last step of each branch: for |y| < 1/16,
// C' y (1 - y^2 / 3); elsewhere C' - 2 C' / (1 + e^(2y)) (same accuracy as
// tanh_f32).
__device__ __forceinline__ float softcap_u(float dot, float pre, float cu)
{
    const float y = dot * pre;
    const float small = y * __builtin_fmaf(y * y, cu * (-1.0f / 3.0f), cu);
    const float e = __builtin_amdgcn_exp2f(y * (2.0f * kLog2e));
    const float big = __builtin_fmaf(-2.0f * cu, __builtin_amdgcn_rcpf(1.0f + e), cu);
    return __builtin_fabsf(y) < 0.0625f ? small : big;
}

// Soft-cap forms of the bf16 kernels, chosen per launch by C.
enum : int {
    kCapOff = 0,
    kCapShort = 1,  // C <= kCapShortMax: C' - 2 C' / (1 + e^(2y)) alone
    kCapExact = 2,  // softcap_u, both branches
};
// Near y = 0 the short form cancels: its absolute error stays about
// 2.4e-7 C' (1 ulp of the reciprocal and of e^(2y) around 1/2 and 1), which
// is at most 1e-4 in log2 units for C <= 256, below every tolerance of the
// outputs (the ALiBi and relative-position terms, and the row max, are exact).
// Larger C need the cubic branch.
constexpr float kCapShortMax = 256.0f;

// C' tanh(y) as C' - 2 C' / (1 + e^(2y)) with e^(2y) = 2^(dot * pre2),
// pre2 = 2 log2(e) scale / C.
__device__ __forceinline__ float softcap_short_u(float dot, float pre2, float cu)
{
    const float e = __builtin_amdgcn_exp2f(dot * pre2);
    return __builtin_fmaf(-2.0f * cu, __builtin_amdgcn_rcpf(1.0f + e), cu);
}

// score_u for the bf16 kernels, with the position terms taken as floats:
// dabs = i' - j and dlin = jref - j, which the kernels form as a per-tile
// base minus the key's compile-time offset within the tile. `softcap_pre` is
// scale / C for kCapExact and 2 log2(e) scale / C for kCapShort.
template <int CAP, int BIAS>
__device__ __forceinline__ float score_tile_u(float dot, float scale_u, float softcap_pre,
                                              float softcap_post_u, float bias_abs, float bias_lin,
                                              float dabs, float dlin)
{
    float t;
    if constexpr (CAP == kCapShort)
        t = softcap_short_u(dot, softcap_pre, softcap_post_u);
    else if constexpr (CAP == kCapExact)
        t = softcap_u(dot, softcap_pre, softcap_post_u);
    else
        t = dot * scale_u;
    if constexpr (BIAS == kBiasAlibi || BIAS == kBiasGeneral)
        t = __builtin_fmaf(bias_abs, __builtin_fabsf(dabs), t);
    if constexpr (BIAS == kBiasRelPos || BIAS == kBiasGeneral)
        t = __builtin_fmaf(bias_lin, dlin, t);
    return t;
}

// ReLU(x) and Sigmoid(x) of a natural score; a masked score (-inf) maps to 0.
template <int NORM>
__device__ __forceinline__ float activation(float x)
{
    if constexpr (NORM == kNormRelu) {
        return __builtin_fmaxf(x, 0.0f);
    } else {
        // 1 / (1 + e^-x); e^-x = +inf for x = -inf gives 0
        return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(x * -kLog2e));
    }
}

}  // namespace attn
