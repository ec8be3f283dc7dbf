// score_mods.h -- device helpers for the Score stage of attention.
//
// Score modifications act on the scaled raw score s = scale * q . k before
// the mask (Appendix A, "Score Modifications"): the soft-cap C * tanh(s / C)
// ("Softcap Attention"), then the ALiBi bias -slope_h * |i' - j|. The kernels
// run the softmax in base 2, so a score leaves here multiplied by log2(e).
#pragma once

#include <hip/hip_runtime.h>

namespace attn {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// tanh for fp32 with small absolute and relative error over the whole line.
// |x| < 0.4: Taylor series of tanh about 0 (coefficients from the Bernoulli
// numbers, 2^{2n}(2^{2n}-1)B_{2n}/(2n)!) through x^13; the first dropped term
// is below 2e-9 there. |x| >= 0.4: tanh|x| = (1 - e)/(1 + e) with
// e = exp(-2|x|) <= 0.45, so the subtraction loses no significant bits.
__device__ __forceinline__ float tanh_f32(float x)
{
    float ax = __builtin_fabsf(x);
    float x2 = x * x;
    float poly = 21844.0f / 6081075.0f;
    poly = __builtin_fmaf(poly, x2, -1382.0f / 155925.0f);
    poly = __builtin_fmaf(poly, x2, 62.0f / 2835.0f);
    poly = __builtin_fmaf(poly, x2, -17.0f / 315.0f);
    poly = __builtin_fmaf(poly, x2, 2.0f / 15.0f);
    poly = __builtin_fmaf(poly, x2, -1.0f / 3.0f);
    float small = __builtin_fmaf(ax * x2, poly, ax);
    float e = __builtin_amdgcn_exp2f(-2.0f * kLog2e * ax);
    float big = (1.0f - e) * __builtin_amdgcn_rcpf(1.0f + e);
    float r = ax < 0.4f ? small : big;
    return __builtin_copysignf(r, x);
}

// Final score in log2 units for a raw dot product `dot` of query position ip
// (on the key axis) and key j.
template <bool SOFTCAP, bool ALIBI>
__device__ __forceinline__ float score_log2(float dot, float scale_log2, float softcap_pre,
                                            float softcap_post, float slope_log2, int ip, int j)
{
    float t;
    if constexpr (SOFTCAP) {
        t = softcap_post * tanh_f32(dot * softcap_pre);
    } else {
        t = dot * scale_log2;
    }
    if constexpr (ALIBI) {
        int rel = ip - j;
        t = __builtin_fmaf(-slope_log2, (float)(rel < 0 ? -rel : rel), t);
    }
    return t;
}

}  // namespace attn
