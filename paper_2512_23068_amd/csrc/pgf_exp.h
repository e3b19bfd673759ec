// Exponentials of the transitions, shared by the selective-SSM and the
// linear-attention kernels.
//
// The per-step transition Abar = exp(Delta A) is taken on the hardware
// exponential 2^x (v_exp_f32), with x = Delta * A * log2(e).  Measured on
// gfx950 over every f32 argument of each binade 2^-20 <= |x| < 2^-9 (against
// fp64 exp2), v_exp_f32 returns results in [1/2, 1) 0.1175 ulp below the
// exact value on average: a relative bias of -7.0e-9 per step (0.26 ulp mean
// absolute error, 0.66 ulp at most).  A lane with Abar close to 1 multiplies
// its state by one such factor every step, so the bias compounds linearly in
// the lane's memory: a decay held for 131072 steps came out 9e-4 low.
// Raising the argument by kExp2Lift = 0.1175 * 2^-24 / ln 2 moves the mean
// to within 2e-10 relative for |x| < 2^-10 (and leaves 2^(0 + kExp2Lift)
// rounded to exactly 1, so a step with Delta = 0 is still the identity); for
// larger |x| it overshoots by at most 8e-9 relative, where a lane forgets
// within a few hundred steps.  The fma that forms Delta * A * log2(e) absorbs
// the addition, so the transition costs what it did.
//
// The segment transitions P = exp(A * sum Delta) of the carries take larger
// arguments, where the hardware's bias differs from binade to binade; they are
// evaluated once per segment and lane (not per step), by exp2_series, whose
// result carries only round-to-nearest errors.
#pragma once

#include <hip/hip_runtime.h>

namespace pgf {

constexpr float kExp2Lift = 1.0104e-8f;

// exp(delta * a) for at = a * log2(e): the per-step transition.
__device__ __forceinline__ float transition(float delta, float at) {
    return __builtin_amdgcn_exp2f(fmaf(delta, at, kExp2Lift));
}

// 2^v without the hardware exponential: v = k + f with k = rint(v),
// |f| <= 1/2; 2^f = sum_j (f ln 2)^j / j! to j = 8 (the first omitted term is
// below 2e-10 relative), in Horner form on f with the coefficients
// (ln 2)^j / j!; 2^k is applied exactly by ldexp.  Arguments below -200
// give 0 (as 2^v does in f32), above 128 give +inf; NaN stays NaN.
__device__ __forceinline__ float exp2_series(float v) {
    const float vc = v < -200.0f ? -200.0f : (v > 128.0f ? 128.0f : v);
    const float k = rintf(vc);
    const float f = vc - k;   // exact
    float p = fmaf(f, 1.3215487e-06f, 1.5252734e-05f);   // (ln2)^8/8!, (ln2)^7/7!
    p = fmaf(f, p, 1.5403530e-04f);                      // (ln2)^6/6!
    p = fmaf(f, p, 1.3333558e-03f);                      // (ln2)^5/5!
    p = fmaf(f, p, 9.6181291e-03f);                      // (ln2)^4/4!
    p = fmaf(f, p, 5.5504109e-02f);                      // (ln2)^3/3!
    p = fmaf(f, p, 2.4022651e-01f);                      // (ln2)^2/2!
    p = fmaf(f, p, 6.9314718e-01f);                      // ln2
    p = fmaf(f, p, 1.0f);
    return __builtin_amdgcn_ldexpf(p, vc == vc ? (int)k : 0);
}

// e^v through exp2_series: v log2(e) = p + lo with p = fl(v log2e_hi) and
// lo recovering its rounding (an fma) and the low part of log2(e), so the
// argument carries no rounding of its own; 2^lo ~ 1 + lo ln 2 (|lo| is
// below 2^-23 |p|).
__device__ __forceinline__ float exp_series(float v) {
    constexpr float kHi = 1.44269502162933349609375f;  // log2(e) rounded to f32
    constexpr float kLo = 1.925963033500011079e-08f;   // log2(e) - kHi
    const float p = v * kHi;
    const float lo = fmaf(v, kHi, -p) + v * kLo;
    const float e = exp2_series(p);
    return fmaf(e, lo * 0.693147180559945309f, e);
}

}  // namespace pgf
