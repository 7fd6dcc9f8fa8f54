/*
 * Oracle for the mul-free channel-wise Parallel Spiking Neuron (arXiv 2501.14490).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, plain, single-threaded CPU
 * statement of what the neuron's training step computes.  Only the test suite,
 * the smoke check and the CPU-baseline leg of the benchmark may load it.  It
 * shares no code, header, table or constant with the HIP library: every
 * constant below is written out here from its definition.
 *
 * Conventions (all arrays are dense, row-major, caller-owned host memory):
 *   x, H, spikes, grad_spikes, dH, grad_x : [T][N][C][S]  (time-first layout,
 *                                           S = product of spatial dims)
 *   sign, shift : [C][k] int8   (tap i of channel c is sign * 2^-shift)
 *   bias        : [C]
 *   grad_w      : [C][k],  grad_b : [C]
 * Tap i of an order-k neuron with dilation d looks back (k-1-i)*d steps, so
 * tap k-1 is "now" (Sec. 4.1, Eq. GPSN-charge; also the Toeplitz weight of
 * App. A.2).  Inputs at negative time are absent (the sliding PSN convention
 * X[j] = 0 for j < 0, Sec. 3.2), so their terms are omitted from the sum.
 *
 * Floating-point order (the paper does not fix one): taps are added in
 * ascending i to an accumulator that starts at +0.0f, each term is the exact
 * power-of-two scaling of x (Sec. 4.2, Eq. bitshift: scaling an FP32 value by
 * a power of two only moves its exponent), the bias is added last, every add
 * is one IEEE single-precision round-to-nearest operation and nothing is
 * contracted into an FMA.  Build with -ffp-contract=off.
 *
 * Parity is pinned by the tests under tests/ (closed forms, invariants, a
 * dense Toeplitz formulation, finite differences, exact rational arithmetic
 * and the paper's printed numbers); see each function's comment.
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>
#include <string.h>

#define ORC_SG_SIGMOID 0
#define ORC_SG_ATAN 1
#define ORC_SG_RATIONAL 2

/* ------------------------------------------------------------------------ */
/* Elementary functions, single precision, pinned operation sequence.        */
/* ------------------------------------------------------------------------ */

/* exp(y) in float: Cody-Waite reduction y = n*ln2 + r with ln2 split into a
 * short high part (exact products n*hi for |n| < 2^15) and a low part, then
 * the degree-7 Taylor polynomial of e^r (coefficients 1/j! rounded to float)
 * by fused multiply-add Horner steps, then scaling by 2^n.  y below -86 (or
 * NaN) gives 0: e^-86 is still a normal float, so the scaling never rounds.
 * y above 88 is clamped to 88 (e^88 is the largest power the scaling keeps
 * finite).  Pinned against double-precision exp in the tests. */
float orc_exp(float y)
{
    if (!(y >= -86.0f))
        return 0.0f;
    if (y > 88.0f)
        y = 88.0f;
    const float log2e = 0x1.715476p+0f;          /* float(1/ln 2)       = 0x3FB8AA3B */
    const float ln2_hi = 0x1.62e4p-1f;           /* 0x3F317200, 15 significant bits */
    const float ln2_lo = 0x1.7f7d1cp-20f;        /* float(ln 2 - ln2_hi) = 0x35BFBE8E */
    float n = rintf(y * log2e);                  /* round half to even */
    float r = fmaf(n, -ln2_hi, y);
    r = fmaf(n, -ln2_lo, r);
    float p = 0x1.a01a02p-13f;                   /* float(1/7!) */
    p = fmaf(p, r, 0x1.6c16c2p-10f);             /* float(1/6!) */
    p = fmaf(p, r, 0x1.111112p-7f);              /* float(1/5!) */
    p = fmaf(p, r, 0x1.555556p-5f);              /* float(1/4!) */
    p = fmaf(p, r, 0x1.555556p-3f);              /* float(1/3!) */
    p = fmaf(p, r, 0.5f);                        /* 1/2! */
    p = fmaf(p, r, 1.0f);                        /* 1/1! */
    p = fmaf(p, r, 1.0f);                        /* 1/0! */
    return ldexpf(p, (int)n);
}

/* Surrogate derivative sigma'(u) of the firing function, evaluated in float.
 *   sigmoid  : derivative of sigmoid(alpha*u): alpha*e/(1+e)^2, e = exp(-alpha|u|)
 *              (the surrogate the workloads use);
 *   arctan   : alpha / (2 (1 + (pi/2 alpha u)^2))   (App. E, sequential CIFAR, SHD);
 *   rational : 1 / (1 + alpha u^2)                   (App. E, DVS-Lip).
 * Each line is one rounded float operation; the division is correctly
 * rounded. */
float orc_surrogate(int kind, float alpha, float u)
{
    if (kind == ORC_SG_SIGMOID) {
        float a = alpha * fabsf(u);
        float e = orc_exp(-a);
        float den = 1.0f + e;
        float num = alpha * e;
        float den2 = den * den;
        return num / den2;
    }
    if (kind == ORC_SG_ATAN) {
        float c = 0x1.921fb6p+0f * alpha;  /* float(pi/2) * alpha */
        float z = c * u;
        float z2 = z * z;
        float den = 1.0f + z2;
        float num = 0.5f * alpha;
        return num / den;
    }
    /* rational */
    float u2 = u * u;
    float au2 = alpha * u2;
    float den = 1.0f + au2;
    return 1.0f / den;
}

/* float -> bfloat16 bits, round to nearest even (NaN stays a quiet NaN). */
uint16_t orc_f32_to_bf16(float f)
{
    uint32_t b;
    memcpy(&b, &f, 4);
    if ((b & 0x7F800000u) == 0x7F800000u && (b & 0x007FFFFFu) != 0u)
        return (uint16_t)((b >> 16) | 0x0040u);
    uint32_t lsb = (b >> 16) & 1u;
    uint32_t rounded = b + 0x7FFFu + lsb;
    return (uint16_t)(rounded >> 16);
}

float orc_bf16_to_f32(uint16_t h)
{
    uint32_t b = ((uint32_t)h) << 16;
    float f;
    memcpy(&f, &b, 4);
    return f;
}

/* ------------------------------------------------------------------------ */
/* Power-of-two quantizer  Q(W) = sign(W) * 2^round(log2 |W|)  (Sec. 4.2,    */
/* Eq. round_w).                                                              */
/* ------------------------------------------------------------------------ */

/* sign(W) returns +1 or -1 (Eq. round_w); W = 0 (either sign) counts as +1.
 * round(log2|W|) is the exact rounding of the real logarithm: writing
 * |W| = f * 2^m with f in [1, 2), the result is m when f < sqrt(2) and m+1
 * otherwise (f = sqrt(2) cannot occur, sqrt(2) being irrational).  The
 * comparison f >= sqrt(2) is done as f*f >= 2 in double, where f*f is exact
 * (f has at most 24 significant bits).  The stored shift is -round(log2|W|)
 * clamped into [lo, hi]; W = 0 and NaN map to shift = hi (the smallest
 * magnitude), +-Inf to shift = lo. */
void orc_quantize(const float* w, int64_t count, int lo, int hi, int8_t* sign, int8_t* shift)
{
    for (int64_t j = 0; j < count; ++j) {
        float v = w[j];
        sign[j] = (v < 0.0f) ? (int8_t)-1 : (int8_t)1;
        int s;
        if (isnan(v) || v == 0.0f) {
            s = hi;
        } else if (isinf(v)) {
            s = lo;
        } else {
            int m;
            float f = frexpf(fabsf(v), &m); /* |v| = f * 2^m, f in [0.5, 1) */
            double f2 = 2.0 * (double)f;    /* in [1, 2) */
            int e = (m - 1) + ((f2 * f2 >= 2.0) ? 1 : 0);
            s = -e;
            if (s < lo) s = lo;
            if (s > hi) s = hi;
        }
        shift[j] = (int8_t)s;
    }
}

/* Gradient of the latent weight from the gradient of the quantized weight
 * (Sec. 4.2).  mode 0, the whole-quantizer straight-through estimator the
 * paper trains with: dWq/dW = 1, so grad_w = grad_wq.  mode 1, the estimator
 * that only replaces round()'s derivative by 1 (Eq. ste, Eq. ste_q):
 * dWq/dW = 2^round(log2|W|) / |W| = |Wq| / |W|, with |Wq| = 2^-shift (the
 * clamped shift the quantizer chose), so grad_w = grad_wq * (2^-shift / |W|),
 * each operation one correctly rounded float operation in that order.  Where
 * the factor is undefined or not finite (W = 0, W not finite) grad_w is 0. */
void orc_quantizer_grad(const float* w, const int8_t* shift, int lo, int hi, const float* grad_wq,
                        int64_t count, int mode, float* grad_w)
{
    for (int64_t j = 0; j < count; ++j) {
        if (mode == 0) {
            grad_w[j] = grad_wq[j];
            continue;
        }
        const float a = fabsf(w[j]);
        if (!(a > 0.0f) || isinf(a)) {
            grad_w[j] = 0.0f;
            continue;
        }
        int s = shift[j];
        if (s < lo) s = lo;
        if (s > hi) s = hi;
        const float q = ldexpf(1.0f, -s);   /* |Wq|, exact */
        const float f = q / a;              /* rounded once */
        grad_w[j] = isfinite(f) ? grad_wq[j] * f : 0.0f;
    }
}

/* ------------------------------------------------------------------------ */
/* Forward: charge (Eq. mfdpsn_charge) + fire (Eq. mfdpsn_fire).             */
/* ------------------------------------------------------------------------ */

static int clamp_shift(int s, int lo, int hi)
{
    return s < lo ? lo : (s > hi ? hi : s);
}

/* floor(v / 2^s) for s >= 0, written out as a floor division so that it does
 * not lean on how C shifts negative numbers (Sec. 4.2: a right shift of a
 * two's-complement integer rounds toward minus infinity). */
static int64_t floor_div_pow2(int64_t v, int s)
{
    int64_t p = (int64_t)1 << s;
    int64_t q = v / p;              /* truncates toward zero */
    if ((v % p) != 0 && v < 0)
        q -= 1;
    return q;
}

/* Threshold of channel c: the learnable channel-wise V_th[c] of
 * Eq. mfdpsn_fire when a per-channel array is given, else the one scalar
 * threshold shared by every channel (Sec. 3.1, Eq. fire). */
static float thr_f32(const float* v_th_c, float v_th, int c)
{
    return v_th_c ? v_th_c[c] : v_th;
}

static int32_t thr_q88(const int32_t* v_th_c, int32_t v_th, int c)
{
    return v_th_c ? v_th_c[c] : v_th;
}

/* Float potentials and spikes.
 *   H[t,n,c,s] = (sum_{i=0..k-1, tau>=0} sign[c,i] * ldexp(x[tau,n,c,s], -shift[c,i])) + bias[c],
 *   tau = t - (k-1-i) d;   spike = (H >= V_th) ? 1 : 0   (Heaviside, Theta(0) = 1, Sec. 3.1),
 * with V_th = v_th_c[c] when v_th_c is given (the channel-wise threshold of
 * Eq. mfdpsn_fire), else the scalar v_th.  The threshold is compared with H
 * as is: it is not folded into the bias, so the comparison sees the rounded
 * sum acc + bias[c] itself.
 * Shifts are clamped into [lo, hi].  *tap_count receives the number of
 * (non-omitted) tap terms evaluated, i.e. the SHIFT count of Table
 * "params and shape" summed over all columns. */
void orc_forward_f32(const float* x, int T, int N, int C, int S, int k, int d,
                     const int8_t* sign, const int8_t* shift, int lo, int hi,
                     const float* bias, float v_th, const float* v_th_c, float* H, uint8_t* spikes,
                     int64_t* tap_count)
{
    int64_t taps = 0;
    const int64_t M = (int64_t)N * C * S;
    for (int t = 0; t < T; ++t)
        for (int n = 0; n < N; ++n)
            for (int c = 0; c < C; ++c)
                for (int s = 0; s < S; ++s) {
                    const int64_t col = ((int64_t)n * C + c) * S + s;
                    float acc = 0.0f;
                    for (int i = 0; i < k; ++i) {
                        const int64_t tau = (int64_t)t - (int64_t)(k - 1 - i) * d;
                        if (tau < 0)
                            continue;
                        float term = ldexpf(x[tau * M + col], -clamp_shift(shift[c * k + i], lo, hi));
                        if (sign[c * k + i] < 0)
                            term = -term;
                        acc = acc + term;
                        ++taps;
                    }
                    const float h = acc + bias[c];
                    if (H)
                        H[t * M + col] = h;
                    if (spikes)
                        spikes[t * M + col] = (h >= thr_f32(v_th_c, v_th, c)) ? 1 : 0;
                }
    if (tap_count)
        *tap_count = taps;
}

/* Q8.8 fixed-point potentials and spikes: every term is the arithmetic right
 * shift (floor) of the int16 input, negated for a negative tap; the int32
 * accumulator starts at the Q8.8 bias.  Shifts are clamped into [lo, hi]
 * (lo >= 0).  The spike compares H with v_th_c[c] (Q8.8) when given, else
 * with the scalar v_th. */
void orc_forward_q88(const int16_t* x, int T, int N, int C, int S, int k, int d,
                     const int8_t* sign, const int8_t* shift, int lo, int hi,
                     const int32_t* bias, int32_t v_th, const int32_t* v_th_c, int32_t* H, uint8_t* spikes,
                     int64_t* tap_count)
{
    int64_t taps = 0;
    const int64_t M = (int64_t)N * C * S;
    for (int t = 0; t < T; ++t)
        for (int n = 0; n < N; ++n)
            for (int c = 0; c < C; ++c)
                for (int s = 0; s < S; ++s) {
                    const int64_t col = ((int64_t)n * C + c) * S + s;
                    int64_t acc = bias[c];
                    for (int i = 0; i < k; ++i) {
                        const int64_t tau = (int64_t)t - (int64_t)(k - 1 - i) * d;
                        if (tau < 0)
                            continue;
                        int64_t term = floor_div_pow2(x[tau * M + col], clamp_shift(shift[c * k + i], lo, hi));
                        acc += (sign[c * k + i] < 0) ? -term : term;
                        ++taps;
                    }
                    if (H)
                        H[t * M + col] = (int32_t)acc;
                    if (spikes)
                        spikes[t * M + col] = (acc >= thr_q88(v_th_c, v_th, c)) ? 1 : 0;
                }
    if (tap_count)
        *tap_count = taps;
}

/* ------------------------------------------------------------------------ */
/* Backward (App. A.3, Eqs. backward_X, backward_W, backward_b, with the     */
/* dilation d carried through).                                               */
/* ------------------------------------------------------------------------ */

/* Float path.  dH = grad_spikes * sigma'(H - V_th) (surrogate gradient of the
 * Heaviside), V_th the channel's threshold (v_th_c[c] when given, else v_th);
 * H is recomputed by orc_forward_f32 into the caller's H buffer.
 *   grad_x[t] = sum_{i ascending, t+(k-1-i)d < T} sign*ldexp(dH[t+(k-1-i)d], -shift)
 *                (transposed dilated convolution; float, same rules as the charge)
 *   grad_w[c,i] = sum_{t,n,s, tau>=0} x[tau] * dH[t]     (double; products of two
 *                 floats are exact in double)
 *   grad_b[c]   = sum_{t,n,s} dH[t]                      (double)
 * grad_w is the gradient of the quantized weight, which the whole-quantizer
 * straight-through estimator passes unchanged to the latent weight
 * (Sec. 4.2).
 *   grad_vth[c] = sum_{t,n,s} -dH[t]                     (double; optional)
 * is the gradient of the channel's threshold: H - V_th[c] enters the
 * surrogate with V_th[c] negated (Eq. mfdpsn_fire). */
void orc_backward_f32(const float* x, const float* grad_spikes, int T, int N, int C, int S,
                      int k, int d, const int8_t* sign, const int8_t* shift, int lo, int hi,
                      const float* bias, float v_th, const float* v_th_c, int kind, float alpha,
                      float* H, float* dH, float* grad_x, double* grad_w, double* grad_b,
                      double* grad_vth)
{
    const int64_t M = (int64_t)N * C * S;
    const int64_t total = (int64_t)T * M;
    orc_forward_f32(x, T, N, C, S, k, d, sign, shift, lo, hi, bias, v_th, v_th_c, H, NULL, NULL);
    for (int64_t e = 0; e < total; ++e) {
        const int c = (int)((e / S) % C);
        const float u = H[e] - thr_f32(v_th_c, v_th, c);
        dH[e] = grad_spikes[e] * orc_surrogate(kind, alpha, u);
    }
    for (int t = 0; t < T; ++t)
        for (int n = 0; n < N; ++n)
            for (int c = 0; c < C; ++c)
                for (int s = 0; s < S; ++s) {
                    const int64_t col = ((int64_t)n * C + c) * S + s;
                    float acc = 0.0f;
                    for (int i = 0; i < k; ++i) {
                        const int64_t tau = (int64_t)t + (int64_t)(k - 1 - i) * d;
                        if (tau >= T)
                            continue;
                        float term = ldexpf(dH[tau * M + col], -clamp_shift(shift[c * k + i], lo, hi));
                        if (sign[c * k + i] < 0)
                            term = -term;
                        acc = acc + term;
                    }
                    grad_x[t * M + col] = acc;
                }
    for (int c = 0; c < C; ++c) {
        for (int i = 0; i < k; ++i) {
            double sum = 0.0;
            for (int t = 0; t < T; ++t) {
                const int64_t tau = (int64_t)t - (int64_t)(k - 1 - i) * d;
                if (tau < 0)
                    continue;
                for (int n = 0; n < N; ++n)
                    for (int s = 0; s < S; ++s) {
                        const int64_t col = ((int64_t)n * C + c) * S + s;
                        sum += (double)x[tau * M + col] * (double)dH[t * M + col];
                    }
            }
            grad_w[c * k + i] = sum;
        }
        double sb = 0.0, sv = 0.0;
        for (int t = 0; t < T; ++t)
            for (int n = 0; n < N; ++n)
                for (int s = 0; s < S; ++s) {
                    const double v = (double)dH[t * M + ((int64_t)n * C + c) * S + s];
                    sb += v;
                    sv += -v;
                }
        grad_b[c] = sb;
        if (grad_vth)
            grad_vth[c] = sv;
    }
}

/* Integer surrogate factor of the Q8.8 path: round-half-even of
 * 2^15 * sigma'(u / 256), sigma' evaluated by orc_surrogate in float (u is the
 * Q8.8 distance to the threshold; the float conversion rounds to nearest). */
int32_t orc_surrogate_q15(int kind, float alpha, int32_t u)
{
    const float uf = (float)u * 0.00390625f;
    const float sg = orc_surrogate(kind, alpha, uf);
    return (int32_t)rintf(sg * 32768.0f);
}

/* Q8.8 path.  dH = floor(grad_spikes * L(H - V_th) / 2^15) with L the Q0.15
 * surrogate factor above (grad_spikes and dH are Q8.8) and V_th the channel's
 * threshold (v_th_c[c] when given, else v_th); grad_x uses the same
 * floor-shift taps as the charge (int32, Q8.8); grad_w = sum x*dH exactly in
 * int64 (Q16.16); grad_b = sum dH in int64 (Q8.8); grad_vth = sum -dH
 * (optional). */
void orc_backward_q88(const int16_t* x, const int16_t* grad_spikes, int T, int N, int C, int S,
                      int k, int d, const int8_t* sign, const int8_t* shift, int lo, int hi,
                      const int32_t* bias, int32_t v_th, const int32_t* v_th_c, int kind, float alpha,
                      int32_t* H, int32_t* dH, int32_t* grad_x, int64_t* grad_w, int64_t* grad_b,
                      int64_t* grad_vth)
{
    const int64_t M = (int64_t)N * C * S;
    const int64_t total = (int64_t)T * M;
    orc_forward_q88(x, T, N, C, S, k, d, sign, shift, lo, hi, bias, v_th, v_th_c, H, NULL, NULL);
    for (int64_t e = 0; e < total; ++e) {
        const int c = (int)((e / S) % C);
        const int32_t L = orc_surrogate_q15(kind, alpha, H[e] - thr_q88(v_th_c, v_th, c));
        dH[e] = (int32_t)floor_div_pow2((int64_t)grad_spikes[e] * (int64_t)L, 15);
    }
    for (int t = 0; t < T; ++t)
        for (int n = 0; n < N; ++n)
            for (int c = 0; c < C; ++c)
                for (int s = 0; s < S; ++s) {
                    const int64_t col = ((int64_t)n * C + c) * S + s;
                    int64_t acc = 0;
                    for (int i = 0; i < k; ++i) {
                        const int64_t tau = (int64_t)t + (int64_t)(k - 1 - i) * d;
                        if (tau >= T)
                            continue;
                        int64_t term = floor_div_pow2(dH[tau * M + col], clamp_shift(shift[c * k + i], lo, hi));
                        acc += (sign[c * k + i] < 0) ? -term : term;
                    }
                    grad_x[t * M + col] = (int32_t)acc;
                }
    for (int c = 0; c < C; ++c) {
        for (int i = 0; i < k; ++i) {
            int64_t sum = 0;
            for (int t = 0; t < T; ++t) {
                const int64_t tau = (int64_t)t - (int64_t)(k - 1 - i) * d;
                if (tau < 0)
                    continue;
                for (int n = 0; n < N; ++n)
                    for (int s = 0; s < S; ++s) {
                        const int64_t col = ((int64_t)n * C + c) * S + s;
                        sum += (int64_t)x[tau * M + col] * (int64_t)dH[t * M + col];
                    }
            }
            grad_w[c * k + i] = sum;
        }
        int64_t sb = 0, sv = 0;
        for (int t = 0; t < T; ++t)
            for (int n = 0; n < N; ++n)
                for (int s = 0; s < S; ++s) {
                    const int64_t v = dH[t * M + ((int64_t)n * C + c) * S + s];
                    sb += v;
                    sv -= v;
                }
        grad_b[c] = sb;
        if (grad_vth)
            grad_vth[c] = sv;
    }
}

/* ------------------------------------------------------------------------ */
/* Step-by-step inference (Sec. 3.2: the sliding PSN emits H[t] at step t;    */
/* Sec. 5, Table "inference memory": the neuron keeps an input history whose  */
/* length grows with its order).                                              */
/* ------------------------------------------------------------------------ */

/* One time step t of the charge and fire, for inputs that arrive one step at
 * a time.  The neuron keeps the inputs of its receptive field in a history
 * ring hist[R][N][C][S] with R = (k-1)*d + 1 slots, the input of time tau in
 * slot tau mod R: tap i reads time tau = t - (k-1-i) d, and the oldest one,
 * tap 0, reaches back (k-1) d steps.  The step first stores x_t (the inputs
 * of time t, [N][C][S]) in slot t mod R, then evaluates the same sum as
 * orc_forward_f32 at this t: ascending taps from +0.0f, terms with tau < 0
 * omitted, bias last.  Calling it for t = 0, 1, ..., T-1 gives the
 * potentials and spikes of orc_forward_f32 over the whole sequence. */
void orc_stream_step_f32(const float* x_t, int N, int C, int S, int k, int d, int64_t t,
                         float* hist, const int8_t* sign, const int8_t* shift, int lo, int hi,
                         const float* bias, float v_th, float* H_t, uint8_t* spikes_t)
{
    const int64_t M = (int64_t)N * C * S;
    const int64_t R = (int64_t)(k - 1) * d + 1;
    memcpy(hist + (t % R) * M, x_t, (size_t)M * sizeof(float));
    for (int n = 0; n < N; ++n)
        for (int c = 0; c < C; ++c)
            for (int s = 0; s < S; ++s) {
                const int64_t col = ((int64_t)n * C + c) * S + s;
                float acc = 0.0f;
                for (int i = 0; i < k; ++i) {
                    const int64_t tau = t - (int64_t)(k - 1 - i) * d;
                    if (tau < 0)
                        continue;
                    float term = ldexpf(hist[(tau % R) * M + col], -clamp_shift(shift[c * k + i], lo, hi));
                    if (sign[c * k + i] < 0)
                        term = -term;
                    acc = acc + term;
                }
                const float h = acc + bias[c];
                if (H_t)
                    H_t[col] = h;
                if (spikes_t)
                    spikes_t[col] = (h >= v_th) ? 1 : 0;
            }
}

/* Q8.8 version of the step: int16 history, floor shifts, negation after the
 * shift, int32 accumulator starting at the bias (as orc_forward_q88). */
void orc_stream_step_q88(const int16_t* x_t, int N, int C, int S, int k, int d, int64_t t,
                         int16_t* hist, const int8_t* sign, const int8_t* shift, int lo, int hi,
                         const int32_t* bias, int32_t v_th, int32_t* H_t, uint8_t* spikes_t)
{
    const int64_t M = (int64_t)N * C * S;
    const int64_t R = (int64_t)(k - 1) * d + 1;
    memcpy(hist + (t % R) * M, x_t, (size_t)M * sizeof(int16_t));
    for (int n = 0; n < N; ++n)
        for (int c = 0; c < C; ++c)
            for (int s = 0; s < S; ++s) {
                const int64_t col = ((int64_t)n * C + c) * S + s;
                int64_t acc = bias[c];
                for (int i = 0; i < k; ++i) {
                    const int64_t tau = t - (int64_t)(k - 1 - i) * d;
                    if (tau < 0)
                        continue;
                    int64_t term = floor_div_pow2(hist[(tau % R) * M + col], clamp_shift(shift[c * k + i], lo, hi));
                    acc += (sign[c * k + i] < 0) ? -term : term;
                }
                if (H_t)
                    H_t[col] = (int32_t)acc;
                if (spikes_t)
                    spikes_t[col] = (acc >= v_th) ? 1 : 0;
            }
}

/* ------------------------------------------------------------------------ */
/* Batch-normalized threshold with fused-weight quantization (App. C,        */
/* Eqs. weight fuse, bias fuse): the training step the paper runs.            */
/* ------------------------------------------------------------------------ */

/* The convolution with the latent (real-valued) weights, the intermediate
 * variable of App. C whose statistics the batch normalization uses:
 *   Tv[t,n,c,s] = sum_{i, tau >= 0} W[c,i] * x[tau,n,c,s],  tau = t-(k-1-i)d,
 * in double: each product of two floats is exact in double, the sum runs in
 * ascending i from +0.0 (no FMA contraction). */
static double bn_conv_value(const float* x, int64_t M, int64_t t, int64_t col, int c, int k, int d,
                            const float* w)
{
    double acc = 0.0;
    for (int i = 0; i < k; ++i) {
        const int64_t tau = t - (int64_t)(k - 1 - i) * d;
        if (tau < 0)
            continue;
        acc = acc + (double)w[c * k + i] * (double)x[tau * M + col];
    }
    return acc;
}

/* Training-mode statistics and fusion.  Per channel c, over all (t, n, s):
 *   mean mu = sum Tv / n_c,  biased variance var = sum (Tv - mu)^2 / n_c,
 *   n_c = T*N*S (App. C normalizes with these per-channel batch statistics,
 *   the variance divided by the count, not by the count minus one);
 *   s = gamma / sqrt(var + eps),  W_f = s * W,  b_f = beta - s * mu
 * (Eq. weight fuse, Eq. bias fuse).  The sums are sequential in (t, n, s)
 * order, in double; the variance takes the two-pass form.  W_f and b_f are
 * rounded once to float (the quantizer and the charge consume floats); aux
 * keeps [mu, var, s, 1/sqrt(var + eps)] per channel in double for the
 * backward.  stats (optional) receives [sum Tv, sum Tv^2] per channel. */
void orc_bn_forward_stats(const float* x, int T, int N, int C, int S, int k, int d, const float* w,
                          const float* gamma, const float* beta, float eps, float* w_f, float* b_f,
                          double* aux, double* stats)
{
    const int64_t M = (int64_t)N * C * S;
    const double nc = (double)T * N * S;
    for (int c = 0; c < C; ++c) {
        double s1 = 0.0, s2 = 0.0;
        for (int t = 0; t < T; ++t)
            for (int n = 0; n < N; ++n)
                for (int sp = 0; sp < S; ++sp) {
                    const double v = bn_conv_value(x, M, t, ((int64_t)n * C + c) * S + sp, c, k, d, w);
                    s1 += v;
                    s2 += v * v;
                }
        const double mu = nc > 0 ? s1 / nc : 0.0;
        double dev = 0.0;
        for (int t = 0; t < T; ++t)
            for (int n = 0; n < N; ++n)
                for (int sp = 0; sp < S; ++sp) {
                    const double v = bn_conv_value(x, M, t, ((int64_t)n * C + c) * S + sp, c, k, d, w) - mu;
                    dev += v * v;
                }
        const double var = nc > 0 ? dev / nc : 0.0;
        const double inv = 1.0 / sqrt(var + (double)eps);
        const double sc = (double)gamma[c] * inv;
        for (int i = 0; i < k; ++i)
            w_f[c * k + i] = (float)(sc * (double)w[c * k + i]);
        b_f[c] = (float)((double)beta[c] - sc * mu);
        aux[4 * c + 0] = mu;
        aux[4 * c + 1] = var;
        aux[4 * c + 2] = sc;
        aux[4 * c + 3] = inv;
        if (stats) {
            stats[2 * c + 0] = s1;
            stats[2 * c + 1] = s2;
        }
    }
}

/* Backward of the fusion and the statistics.  Inputs: the gradients of the
 * fused (quantized) weight and bias, grad_wf [C][k] and grad_bf [C] (the
 * quantizer passes grad_wf to W_f unchanged, Sec. 4.2), and grad_xq, the
 * input gradient through the quantized convolution (App. A.3 Eq. backward_X),
 * all in double.  With n_c, mu, var, s, inv from the forward:
 *   dL/ds   = sum_i grad_wf[c,i] W[c,i] - grad_bf[c] mu
 *   dL/dgamma = dL/ds * inv,   dL/dbeta = grad_bf
 *   dL/dvar = -dL/ds * s / (2 (var + eps)),   dL/dmu (through b_f) = -s grad_bf
 *   dTv = dL/dmu / n_c + dL/dvar * 2 (Tv - mu) / n_c      (per element)
 *   grad_x = grad_xq + sum_i W[c,i] dTv[t + (k-1-i)d]      (transposed conv, latent W)
 *   grad_w = s grad_wf + sum_{t,n,s} dTv[t] x[t-(k-1-i)d]
 * (the derivative of var through mu vanishes: sum (Tv - mu) = 0).  Every sum
 * in double; grad_x, grad_w, grad_gamma, grad_beta returned in double. */
void orc_bn_backward(const float* x, int T, int N, int C, int S, int k, int d, const float* w,
                     const float* gamma, float eps, const double* aux, const double* grad_wf,
                     const double* grad_bf, const double* grad_xq, double* grad_x, double* grad_w,
                     double* grad_gamma, double* grad_beta)
{
    const int64_t M = (int64_t)N * C * S;
    const double nc = (double)T * N * S;
    (void)gamma;
    for (int c = 0; c < C; ++c) {
        const double mu = aux[4 * c + 0], var = aux[4 * c + 1], sc = aux[4 * c + 2], inv = aux[4 * c + 3];
        double dsc = 0.0;
        for (int i = 0; i < k; ++i)
            dsc += grad_wf[c * k + i] * (double)w[c * k + i];
        dsc -= grad_bf[c] * mu;
        grad_gamma[c] = dsc * inv;
        grad_beta[c] = grad_bf[c];
        const double dvar = -dsc * sc / (2.0 * (var + (double)eps));
        const double dmu = -sc * grad_bf[c];
        const double b = nc > 0 ? 2.0 * dvar / nc : 0.0;
        const double a = nc > 0 ? dmu / nc - b * mu : 0.0;
        for (int i = 0; i < k; ++i)
            grad_w[c * k + i] = sc * grad_wf[c * k + i];
        for (int n = 0; n < N; ++n)
            for (int sp = 0; sp < S; ++sp) {
                const int64_t col = ((int64_t)n * C + c) * S + sp;
                for (int t = 0; t < T; ++t) {
                    /* input gradient at time t: dTv of the outputs its taps feed */
                    double gx = 0.0;
                    for (int i = 0; i < k; ++i) {
                        const int64_t to = (int64_t)t + (int64_t)(k - 1 - i) * d;
                        if (to >= T)
                            continue;
                        const double dtv = a + b * bn_conv_value(x, M, to, col, c, k, d, w);
                        gx = gx + (double)w[c * k + i] * dtv;
                    }
                    grad_x[t * M + col] = grad_xq[t * M + col] + gx;
                }
            }
        for (int i = 0; i < k; ++i) {
            double acc = 0.0;
            for (int t = 0; t < T; ++t)
                for (int n = 0; n < N; ++n)
                    for (int sp = 0; sp < S; ++sp) {
                        const int64_t tau = (int64_t)t - (int64_t)(k - 1 - i) * d;
                        if (tau < 0)
                            continue;
                        const int64_t col = ((int64_t)n * C + c) * S + sp;
                        const double dtv = a + b * bn_conv_value(x, M, t, col, c, k, d, w);
                        acc += dtv * (double)x[tau * M + col];
                    }
            grad_w[c * k + i] += acc;
        }
    }
}

/* Sawtooth dilation schedule (Sec. 4.1, Eq. d): d^0 = 1, d^{l+1} = d^l mod P + 1
 * (the paper uses P = 3), computed by iterating the recurrence. */
int orc_sawtooth_dilation(int layer, int period)
{
    int d = 1;
    for (int l = 0; l < layer; ++l)
        d = d % period + 1;
    return d;
}
