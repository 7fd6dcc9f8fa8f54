// Surrogate derivative of the firing function and the membrane-potential
// gradient dH = grad_spikes * sigma'(H - V_th) (surrogate-gradient training,
// Sec. Introduction; the arctan and rational surrogates of the appendix
// Setting of Experiments; sigmoid), as one fixed sequence of
// float operations shared by every kernel that needs it, so that all of them
// give the same bits.  Internal to the library; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mfpsn {

// ---------------------------------------------------------------------------
// surrogate derivative (float, fixed operation sequence)
// ---------------------------------------------------------------------------
// exp(y) for y <= 0: Cody-Waite reduction with ln 2 = hi + lo (hi has 15
// significant bits), degree-7 Taylor polynomial of e^r by fma Horner steps,
// scaling by 2^n.  y < -86 (or NaN) gives 0.
__device__ __forceinline__ float mf_exp_nonpos(float y)
{
    const float log2e = 0x1.715476p+0f;
    const float ln2hi = 0x1.62e4p-1f;
    const float ln2lo = 0x1.7f7d1cp-20f;
    const bool zero = !(y >= -86.0f);
    float n = rintf(y * log2e);
    float r = __builtin_fmaf(n, -ln2hi, y);
    r = __builtin_fmaf(n, -ln2lo, r);
    float p = 0x1.a01a02p-13f;
    p = __builtin_fmaf(p, r, 0x1.6c16c2p-10f);
    p = __builtin_fmaf(p, r, 0x1.111112p-7f);
    p = __builtin_fmaf(p, r, 0x1.555556p-5f);
    p = __builtin_fmaf(p, r, 0x1.555556p-3f);
    p = __builtin_fmaf(p, r, 0.5f);
    p = __builtin_fmaf(p, r, 1.0f);
    p = __builtin_fmaf(p, r, 1.0f);
    float e = ldexpf(p, (int)n);
    return zero ? 0.0f : e;
}

// n / b rounded to nearest, for b in [1, 4] and n zero or in [2^-100, 2^62]:
// the reciprocal refined by one Newton step, then the quotient corrected
// twice by its exact residual.  These are the operations of the general
// correctly rounded float division, whose operand scaling and special-case
// fixup leave values in this range unchanged (they act on zero, infinite,
// subnormal and near-limit operands and quotients only).  b == 1 is exact
// for any n: the refined reciprocal is 1 and every residual is 0.
__device__ __forceinline__ float quot_1_4(float n, float b)
{
    float r = __builtin_amdgcn_rcpf(b);
    const float e = __builtin_fmaf(-b, r, 1.0f);
    r = __builtin_fmaf(e, r, r);
    float q = n * r;
    float t = __builtin_fmaf(-b, q, n);
    q = __builtin_fmaf(t, r, q);
    t = __builtin_fmaf(-b, q, n);
    return __builtin_fmaf(t, r, q);
}

// sigmoid: alpha e / (1 + e)^2 with e = exp(-alpha |u|)
// atan:    (alpha / 2) / (1 + (pi/2 alpha u)^2)
// rational: 1 / (1 + alpha u^2)
// atan and rational share one operation sequence: z = m u, den = 1 + q z^2,
// num / den, with (m, q, num) = (float(pi/2) alpha, 1, alpha/2) or
// (1, alpha, 1); the multiplications by 1 are exact, so each result is
// bit-identical to its own formula.
//
// The sigmoid's quotient has den^2 in [1, 4] (e in [0, 1]); its numerator
// alpha e is 0, or at least alpha 2^-24 wherever den^2 > 1 (1 + e rounds to
// 1 below that).  For alpha = 0 or alpha >= 2^-60 (and alpha <= 1024, which
// the descriptor's validation guarantees) quot_1_4 therefore gives the
// correctly rounded quotient; smaller alphas take the general division.
struct Surrogate {
    int quick;    // 1: sigmoid with the quotient of quot_1_4
    int sigmoid;  // 1: sigmoid, 0: atan or rational
    float alpha;
    float m, q, num;
    __device__ void init(int kind, float a)
    {
        sigmoid = kind == 0;
        quick = kind == 0 && (a == 0.0f || a >= 0x1p-60f);
        alpha = a;
        m = kind == 1 ? 0x1.921fb6p+0f * a : 1.0f;
        q = kind == 1 ? 1.0f : a;
        num = kind == 1 ? 0.5f * a : 1.0f;
    }
    // kQuick = false keeps the general division only (the same results; the
    // code of both quotients costs registers where a kernel holds many)
    template <bool kQuick = true>
    __device__ __forceinline__ float operator()(float u) const
    {
        if (sigmoid) {
            float a = alpha * fabsf(u);
            float e = mf_exp_nonpos(-a);
            float den = 1.0f + e;
            float nm = alpha * e;
            float den2 = den * den;
            if (kQuick && __builtin_expect(quick, 1))
                return quot_1_4(nm, den2);
            return nm / den2;
        }
        float z = m * u;
        float z2 = z * z;
        float t = q * z2;
        float den = 1.0f + t;
        return num / den;
    }
};

// Surrogate factor of a potential: float sigma'(H - v_th); Q8.8 the integer
// L = round-half-even(2^15 sigma'((H - v_th) / 256)).
template <bool kQuick = true>
__device__ __forceinline__ float sg_factor(const Surrogate& sg, float h, float v_th, int)
{
    float u = h - v_th;
    return sg.template operator()<kQuick>(u);
}
__device__ __forceinline__ int32_t sg_factor_q(const Surrogate& sg, int32_t u)
{
    float uf = (float)u * 0.00390625f;
    float s = sg(uf);
    return (int32_t)rintf(s * 32768.0f);
}
__device__ __forceinline__ int32_t sg_factor(const Surrogate& sg, int32_t h, float, int v_th_q)
{
    return sg_factor_q(sg, (int32_t)((uint32_t)h - (uint32_t)v_th_q));
}

// dH = grad_spikes * factor (Q8.8: floor((g * L) / 2^15))
__device__ __forceinline__ float delta_h(float g, float f) { return g * f; }
__device__ __forceinline__ int32_t delta_h(int32_t g, int32_t L)
{
    int64_t p = (int64_t)g * (int64_t)L;
    return (int32_t)(p >> 15);
}

}  // namespace mfpsn
