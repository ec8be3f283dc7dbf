// softcap_poly.h -- the soft-cap (Appendix A, "Softcap Attention") as a short
// polynomial, for the kernels that fold the running max into the scores.
//
// tanh(y) / y ~= a0 + a1 y^2 + a2 y^4 on |y| <= R: fits minimising the
// relative error over y^2 in [0, R^2] (linear-programming minimax on a fine
// grid), coefficients rounded to float; rel is the largest relative error of
// the rounded polynomial on that interval. With s = scale / C and C' the
// cap in score units, C' tanh(s dot) = dot (b0 + z (b1 + z b2)), z = dot^2,
// b_k = C' s^(2k+1) a_k, for z <= (R / s)^2. The score then errs by at most
// C' R rel (|tanh y| <= |y| <= R): the host takes the widest range whose
// bound stays within kCapPolyMaxErr, so a larger C gets a narrower range
// (tiles with a larger |y| are recomputed with the exact form).
#pragma once

struct CapPolyFit {
    float r;        // range of |y|
    float a[3];     // a0, a1, a2
    double rel;     // max relative error of a0 + a1 y^2 + a2 y^4 against tanh(y) / y
};

// widest range first
constexpr CapPolyFit kCapPolyFits[] = {
    {0.50f, {0.99997741f, -0.331691504f, 0.115209743f}, 2.26e-05},
    {0.45f, {0.999987662f, -0.332226396f, 0.11834956f}, 1.24e-05},
    {0.40f, {0.999993742f, -0.332625359f, 0.121274538f}, 6.26e-06},
    {0.35f, {0.999997139f, -0.332909465f, 0.123949632f}, 2.88e-06},
    {0.30f, {0.999998868f, -0.333101213f, 0.126346782f}, 1.17e-06},
    {0.25f, {0.999999583f, -0.333218783f, 0.1284118f}, 4.17e-07},
    {0.20f, {0.999999881f, -0.333287358f, 0.130173713f}, 1.45e-07},
};
constexpr int kCapPolyFitCount = sizeof(kCapPolyFits) / sizeof(kCapPolyFits[0]);

// Largest error allowed in a soft-capped score from the polynomial, in score
// units (log2 units for softmax): 1e-4 changes P by under 7e-5 relative,
// about 1/28 of the bf16 rounding of P that the P V product sees anyway.
constexpr double kCapPolyMaxErr = 1.0e-4;
