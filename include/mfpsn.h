/*
 * mfpsn.h — C ABI of libmfpsn.so, the gfx950 (MI355X) implementation of the
 * training step of the mul-free channel-wise Parallel Spiking Neuron
 * (arXiv 2501.14490, "Multiplication-Free Parallelizable Spiking Neurons with
 * Efficient Spatio-Temporal Dynamics").
 *
 * Problem statement (Sec. 4.1 Eq. GPSN-charge, Sec. 4.2 Eqs. round_w,
 * mfdpsn_charge, mfdpsn_fire; App. A.3 Eqs. forward_H, backward_X/W/b):
 *
 *   H[t,n,c,s] = sum_{i=0..k-1, t-(k-1-i)d >= 0} sign[c,i] * 2^-shift[c,i] * x[t-(k-1-i)d, n,c,s]
 *                + bias[c]
 *   spikes     = (H >= V_th[c])                    (Heaviside, Theta(0) = 1)
 *   dH         = grad_spikes * sigma'(H - V_th[c]) (surrogate gradient)
 *   grad_x[t]  = sum_{i, t+(k-1-i)d < T} sign[c,i] * 2^-shift[c,i] * dH[t+(k-1-i)d]
 *   grad_w[c,i]= sum_{t,n,s} x[t-(k-1-i)d] * dH[t]  (gradient of the quantized
 *                weight, passed unchanged to the latent weight by the
 *                whole-quantizer straight-through estimator)
 *   grad_b[c]  = sum_{t,n,s} dH[t]
 *   grad_vth[c]= -grad_b[c]                        (gradient of the threshold)
 * V_th[c] is the learnable channel-wise threshold of Eq. mfdpsn_fire when a
 * per-channel array is passed, else the one scalar threshold of the
 * descriptor (Sec. 3.1, Eq. fire); the comparison and the surrogate see the
 * rounded potential H itself (the threshold is not folded into the bias).
 *
 * Every product by a tap is a power-of-two scaling: an exponent move (ldexp)
 * for float data, an arithmetic right shift (floor) for Q8.8 integers
 * (Sec. 4.2, Eq. bitshift).  Float sums run in ascending tap order from +0,
 * bias last, each add rounded to nearest; grad_w and grad_b are accumulated
 * from exact double-precision products and rounded once.
 *
 * Layouts (all device memory, owned by the caller, dense, row-major):
 *   x, grad_spikes, spikes, h_out, grad_x : [T][N][C][S]   time-first; S is the
 *                                            product of the spatial dimensions
 *   sign, shift : int8 [C][k]   weight = sign * 2^-shift (sign < 0 means -1,
 *                               anything else +1; shift is clamped into
 *                               [shift_lo, shift_hi])
 *   bias        : float [C] (F32, BF16) or int32 [C] Q8.8 (Q8_8)
 *   grad_w      : float [C][k] (F32, BF16) or int64 [C][k] Q16.16 (Q8_8)
 *   grad_b      : float [C]    (F32, BF16) or int64 [C] Q8.8 (Q8_8)
 * Storage types per dtype:
 *   MFPSN_F32  : x, grad_spikes, grad_x float; h_out float
 *   MFPSN_BF16 : x, grad_spikes, grad_x bfloat16 (arithmetic in float, grad_x
 *                rounded to nearest even); h_out float
 *   MFPSN_Q8_8 : x, grad_spikes int16 Q8.8; grad_x int32 Q8.8; h_out int32 Q8.8
 *
 * Error behaviour: every entry point validates its arguments on the host
 * before touching the GPU; on error it returns a negative mfpsn_status and
 * launches nothing.  Launch failures return MFPSN_ERR_HIP.  All work is
 * enqueued asynchronously on `stream` (a hipStream_t; NULL is the null
 * stream).  Outputs are overwritten, never accumulated into.  The library
 * keeps no per-call state and allocates no device memory; calls on different
 * streams with disjoint outputs may overlap.
 */
#ifndef MFPSN_H
#define MFPSN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MFPSN_ABI_VERSION 10
#define MFPSN_MAX_K 32

typedef enum mfpsn_status {
    MFPSN_OK = 0,
    MFPSN_ERR_NULL = -1,      /* a required pointer is NULL                      */
    MFPSN_ERR_SHAPE = -2,     /* a size is negative or too large                 */
    MFPSN_ERR_PARAM = -3,     /* k, dilation, shift range, v_th or alpha invalid */
    MFPSN_ERR_DTYPE = -4,     /* unknown dtype or surrogate                      */
    MFPSN_ERR_WORKSPACE = -5, /* workspace too small or misaligned               */
    MFPSN_ERR_ALIGN = -6,     /* a tensor pointer is misaligned for its type     */
    MFPSN_ERR_HIP = -7        /* the HIP runtime reported an error               */
} mfpsn_status;

typedef enum mfpsn_dtype {
    MFPSN_F32 = 0,
    MFPSN_BF16 = 1,
    MFPSN_Q8_8 = 2
} mfpsn_dtype;

/* Surrogate derivative sigma'(u) used by the backward (Sec. 1 and App. E):
 *   SIGMOID : alpha*e/(1+e)^2, e = exp(-alpha*|u|)   (derivative of sigmoid(alpha*u))
 *   ATAN    : alpha / (2 (1 + (pi/2 * alpha * u)^2))
 *   RATIONAL: 1 / (1 + alpha * u^2)
 * Evaluated in float with a fixed operation sequence (own exp: Cody-Waite
 * reduction, degree-7 Taylor polynomial); the Q8.8 path uses the integer
 * factor L(u) = round_half_even(2^15 * sigma'(u/256)) and
 * dH = floor(grad_spikes * L / 2^15). */
typedef enum mfpsn_surrogate {
    MFPSN_SG_SIGMOID = 0,
    MFPSN_SG_ATAN = 1,
    MFPSN_SG_RATIONAL = 2
} mfpsn_surrogate;

typedef struct mfpsn_desc {
    int32_t T, N, C, S;  /* sizes, each >= 0; N*C*S*elem_bytes < 2^31        */
    int32_t k;           /* order, 1..MFPSN_MAX_K                              */
    int32_t dilation;    /* this layer's d >= 1 (see mfpsn_sawtooth_dilation)  */
    int32_t dtype;       /* mfpsn_dtype                                        */
    int32_t surrogate;   /* mfpsn_surrogate                                    */
    float alpha;         /* surrogate parameter, 0 <= alpha <= 1024            */
    float v_th;          /* threshold, float paths (finite); used when no      */
                         /* per-channel thresholds are passed                  */
    int32_t v_th_q;      /* threshold, Q8.8 path (256 == 1.0), |v_th_q| <= 2^30 */
    int32_t shift_lo;    /* shifts are clamped into [shift_lo, shift_hi];      */
    int32_t shift_hi;    /* float: -126..126, Q8.8: 0..31                      */
} mfpsn_desc;

/* Forward: charge (Eq. mfdpsn_charge) and fire (Eq. mfdpsn_fire).
 *   x      : [T][N][C][S] storage type of desc->dtype
 *   sign, shift : int8 [C][k];  bias : float[C] or int32[C] (Q8.8)
 *   v_th_c : optional (may be NULL) per-channel thresholds V_th[c], the
 *            learnable channel-wise threshold of Eq. mfdpsn_fire: float[C]
 *            (F32, BF16) or int32[C] Q8.8 (|V_th[c]| <= 2^30); NULL means
 *            desc->v_th (desc->v_th_q) for every channel.  Device values are
 *            not validated: a NaN threshold never fires.
 *   spikes : uint8 [T][N][C][S], 1 where H >= V_th[c] else 0 (NaN -> 0)
 *   h_out  : optional (may be NULL) membrane potential H, float (F32, BF16)
 *            or int32 (Q8.8), [T][N][C][S].  Passed to mfpsn_backward, it
 *            spares the backward the charge.
 *   sg_out : optional (may be NULL) surrogate factor of H, [T][N][C][S]:
 *            float sigma'(H - V_th[c]) (F32, BF16), or int32
 *            L = round_half_even(2^15 * sigma'((H - V_th[c]) / 256)) (Q8.8).
 *            Passed to mfpsn_backward, it spares the backward the charge and
 *            the surrogate (dH = grad_spikes * factor there).
 * Alignment: x 4 bytes (F32) / 2 bytes (BF16, Q8.8); h_out, sg_out, bias,
 * v_th_c 4 bytes. */
int mfpsn_forward(const mfpsn_desc* desc, const void* x, const int8_t* sign, const int8_t* shift,
                  const void* bias, const void* v_th_c, uint8_t* spikes, void* h_out, void* sg_out,
                  void* stream);

/* Bytes of device workspace mfpsn_backward needs for this problem (per-block
 * partial sums of grad_w and grad_b: double, or int64 for Q8.8).  Returns a
 * status; *bytes is written on success. */
int mfpsn_backward_workspace_size(const mfpsn_desc* desc, size_t* bytes);

/* Backward: dH, grad_x (App. A.3 Eq. backward_X), grad_w (Eq. backward_W)
 * and grad_b (Eq. backward_b).
 *   grad_spikes : [T][N][C][S] storage type of desc->dtype (the upstream
 *                 gradient of the spikes)
 *   h           : optional (may be NULL) potentials H of this x, taps and
 *                 bias, as written by mfpsn_forward's h_out
 *   sg          : optional (may be NULL) surrogate factor of this x, taps,
 *                 bias, thresholds and surrogate, as written by
 *                 mfpsn_forward's sg_out
 *   v_th_c      : optional per-channel thresholds, as for mfpsn_forward (the
 *                 same array the forward used)
 *   The backward uses sg if given, else h if given, else recomputes H and
 *   the factor from x.  All three give identical results; a saved tensor
 *   trades 4 bytes per element of memory traffic for the recomputation.
 *   grad_x      : [T][N][C][S] float (F32), bfloat16 (BF16), int32 (Q8.8)
 *   grad_w      : float [C][k] or int64 [C][k] (Q8.8, Q16.16)
 *   grad_b      : float [C]    or int64 [C]    (Q8.8)
 *   grad_vth    : optional (may be NULL) gradient of the thresholds,
 *                 -grad_b: float [C] or int64 [C] (Q8.8)
 *   workspace   : >= mfpsn_backward_workspace_size bytes, 8-byte aligned;
 *                 contents on entry are ignored (every word used is written)
 * grad_x follows the sum of the definition exactly, every term included.
 * grad_w and grad_b do not depend on the order in which the GPU runs its
 * blocks: partial sums are reduced in a fixed order, so repeated calls give
 * identical bits.  The Q8.8 path is exact (int64 sums); the call fails with
 * MFPSN_ERR_SHAPE when T*N*S*32768*max|dH| could reach 2^62. */
int mfpsn_backward(const mfpsn_desc* desc, const void* x, const void* grad_spikes, const void* h,
                   const void* sg, const int8_t* sign, const int8_t* shift, const void* bias,
                   const void* v_th_c, void* grad_x, void* grad_w, void* grad_b, void* grad_vth,
                   void* workspace, size_t workspace_bytes, void* stream);

/* mfpsn_backward for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same computation, arguments and results as mfpsn_backward, without the
 * workspace arguments.  Its workspace is a fixed array of
 * MFPSN_NO_ALLOC_WORKSPACE_BYTES of device memory inside the library, one per
 * GPU, held until the process ends; the call allocates nothing.  Problems
 * whose mfpsn_backward_workspace_size exceeds that size fail with
 * MFPSN_ERR_WORKSPACE before anything is launched.  Every word of the array
 * a call uses is written by that call before it is read, so nothing carries
 * over between calls; but all calls on one GPU share the array, so calls
 * that may overlap on one GPU (different streams, or host threads without an
 * order between their streams) race and must not be issued. */
#define MFPSN_NO_ALLOC_WORKSPACE_BYTES (64u << 20)
int mfpsn_backward_no_alloc(const mfpsn_desc* desc, const void* x, const void* grad_spikes, const void* h,
                            const void* sg, const int8_t* sign, const int8_t* shift, const void* bias,
                            const void* v_th_c, void* grad_x, void* grad_w, void* grad_b, void* grad_vth,
                            void* stream);

/* Power-of-two quantizer Q(W) = sign(W) * 2^round(log2|W|) (Sec. 4.2,
 * Eq. round_w), applied elementwise to `count` (< 2^31) floats w (device):
 *   sign  = -1 if w < 0 else +1 (so sign(0) = +1)
 *   shift = clamp(-round(log2|w|), shift_lo, shift_hi), with the exact
 *           rounding of the real logarithm (|w| = f 2^m, f in [1,2):
 *           m + (f >= sqrt 2)); w = 0 or NaN -> shift_hi; +-Inf -> shift_lo.
 * The gradient of the latent weight is grad_w itself (straight-through). */
int mfpsn_quantize_weights(const float* w, int64_t count, int32_t shift_lo, int32_t shift_hi,
                           int8_t* sign, int8_t* shift, void* stream);

/* Batch-normalized threshold with fused-weight quantization, the training
 * step of App. C (Eq. weight fuse, Eq. bias fuse), for float x (MFPSN_F32):
 * the spike rule is Theta(gamma (H - mu)/sqrt(var + eps) + beta) on the
 * latent-weight convolution H, trained through the fused, quantized weight.
 *   forward:  mfpsn_bn_forward_stats -> mfpsn_quantize_weights(w_f) ->
 *             mfpsn_forward(bias = b_f, v_th = 0, saving the factor)
 *   backward: mfpsn_backward (grad_x, grad of W_f = grad of the quantized
 *             weight, grad of b_f) -> mfpsn_bn_backward
 * mfpsn_bn_forward_stats: per channel c, over all (t, n, s), the mean mu and
 * the biased variance var of Tv = latent W * x (Tv in double: exact float
 * products, ascending taps), then s = gamma/sqrt(var + eps),
 * w_f = s * w (float [C][k]), b_f = beta - s * mu (float [C]),
 * aux = [mu, var, s, 1/sqrt(var + eps)] (double [C][4], for the backward),
 * stats = [sum Tv, sum Tv^2] (double [C][2], optional).  Sums are added in a
 * fixed order (bitwise reproducible), as sums of the deviations e = Tv - p
 * from a pivot p (Tv of the channel's last step at its first column):
 * mu = p + sum e/n, var = sum e^2/n - (sum e/n)^2, at least 0, which keeps
 * var accurate when |mu| is much larger than the standard deviation.
 * mfpsn_bn_backward: from grad_wf (float [C][k]) and grad_bf (float [C])
 * of the fused weight and bias, adds the statistics path to grad_x (float
 * [T][N][C][S], in: the quantized path's input gradient, out: the total)
 * and writes grad_w (float [C][k], latent weight), grad_gamma, grad_beta
 * (float [C]):  ds = sum_i grad_wf W - grad_bf mu, grad_gamma = ds/sqrt(var +
 * eps), grad_beta = grad_bf, dvar = -ds s / (2 (var + eps)), dmu = -s grad_bf,
 * dTv = dmu/n + dvar 2 (Tv - mu)/n, grad_x += W^T * dTv (latent weights,
 * double, ascending taps), grad_w = s grad_wf + sum dTv x (n = T*N*S).
 * Both need mfpsn_bn_workspace_size bytes of workspace (8-byte aligned,
 * caller-owned, contents not kept between calls: per-thread partial sums of
 * the reductions and the per-channel coefficients of dTv).  x, w, gamma,
 * beta, the gradients and aux are device memory, not written except the
 * outputs named above.  eps > 0 and finite, else MFPSN_ERR_PARAM; empty
 * batches are MFPSN_ERR_SHAPE; dtypes other than f32 MFPSN_ERR_DTYPE. */
int mfpsn_bn_workspace_size(const mfpsn_desc* desc, size_t* bytes);
int mfpsn_bn_forward_stats(const mfpsn_desc* desc, const float* x, const float* w, const float* gamma,
                           const float* beta, float eps, float* w_f, float* b_f, double* aux, double* stats,
                           void* workspace, size_t workspace_bytes, void* stream);
int mfpsn_bn_backward(const mfpsn_desc* desc, const float* x, const float* w, const double* aux, float eps,
                      const float* grad_wf, const float* grad_bf, float* grad_x, float* grad_w, float* grad_gamma,
                      float* grad_beta, void* workspace, size_t workspace_bytes, void* stream);

/* Gradient of the latent weight from the gradient of the quantized weight
 * (Sec. 4.2), elementwise over `count` (< 2^31) weights, device memory:
 *   MFPSN_STE_WHOLE : the whole-quantizer straight-through estimator the paper
 *                     trains with, dWq/dW = 1: grad_w = grad_wq (w, shift unused)
 *   MFPSN_STE_ROUND : only round()'s derivative replaced by 1 (Eq. ste), so
 *                     dWq/dW = 2^round(log2|W|)/|W| = |Wq|/|W| (Eq. ste_q):
 *                     grad_w = grad_wq * (2^-shift / |w|), shift clamped into
 *                     [shift_lo, shift_hi] as by the quantizer; the quotient and
 *                     the product each rounded once; 0 where w = 0, w is not
 *                     finite or the quotient overflows.
 * w, grad_wq, grad_w: float [count]; shift: int8 [count] (from
 * mfpsn_quantize_weights).  grad_w may alias grad_wq. */
enum { MFPSN_STE_WHOLE = 0, MFPSN_STE_ROUND = 1 };
int mfpsn_quantizer_grad(const float* w, const int8_t* shift, int32_t shift_lo, int32_t shift_hi,
                         const float* grad_wq, int64_t count, int32_t mode, float* grad_w, void* stream);

/* Step-by-step (streaming) inference: one time step of the charge
 * (Eq. mfdpsn_charge) and fire (Eq. mfdpsn_fire) per call, for inputs that
 * arrive one step at a time (the sliding PSN emits H[t] at step t, Sec. 3.2;
 * the input history it stores grows with the order, Sec. 5, Table
 * "inference memory").  The neuron keeps the last (k-1)*dilation + 1 inputs
 * of every column, its receptive field, in a history ring owned by the
 * caller:
 *   ring : [R][N][C][S] storage type of desc->dtype, R = (k-1)*dilation + 1;
 *          the input of time tau is in slot tau mod R.  Never read before it
 *          is written, so it needs no initialization.
 * mfpsn_stream_ring_bytes writes R to *steps and the ring's size in bytes to
 * *bytes (either pointer may be NULL, not both).  desc->T is ignored by both
 * streaming calls; every other field means what it means above.
 *
 * mfpsn_stream_step, for time step t >= 0:
 *   x_t      : [N][C][S] storage type of desc->dtype, the inputs of time t;
 *              stored into ring slot t mod R
 *   spikes_t : uint8 [N][C][S];  h_t : optional (NULL) float / int32 [N][C][S]
 *   H_t = sum over taps i with t-(k-1-i)d >= 0 of sign*2^-shift*x[t-(k-1-i)d]
 *         + bias, in the same order and arithmetic as mfpsn_forward, so
 *   calls for t = 0, 1, ..., T-1 (in that order, on one stream, on one ring)
 *   give mfpsn_forward's spikes and H over the sequence bit for bit.
 * The call reads the ring slots of times t-d, t-2d, ..., so steps of one ring
 * must not overlap: issue them in order on one stream.  Errors: t < 0 is
 * MFPSN_ERR_PARAM; alignment as for mfpsn_forward (ring like x). */
int mfpsn_stream_ring_bytes(const mfpsn_desc* desc, int32_t* steps, size_t* bytes);
int mfpsn_stream_step(const mfpsn_desc* desc, int64_t t, const void* x_t, void* ring,
                      const int8_t* sign, const int8_t* shift, const void* bias,
                      uint8_t* spikes_t, void* h_t, void* stream);

/* Sawtooth dilation of layer `layer` (0-based) for a period P (Sec. 4.1,
 * Eq. d with P = 3): d^0 = 1, d^{l+1} = d^l mod P + 1, i.e. (layer mod P) + 1.
 * Returns 0 if layer < 0 or period < 1. */
int32_t mfpsn_sawtooth_dilation(int32_t layer, int32_t period);

/* Static description of a status code. */
const char* mfpsn_status_string(int status);

/* Forward (Eq. mfdpsn_charge, Eq. mfdpsn_fire) in the time-last layout, time
 * innermost (the paper's second layout):
 *   x      : [N][C][S][T] storage type of desc->dtype
 *   spikes : uint8 [N][C][S][T];  h_out : optional (may be NULL), [N][C][S][T]
 *            float (F32, BF16) or int32 (Q8.8)
 * sign, shift, bias, desc (sizes T, N, C, S as for mfpsn_forward) and the
 * values computed are those of mfpsn_forward: the outputs are its outputs
 * with the time axis moved last, bit for bit.  Same alignment and errors as
 * mfpsn_forward; MFPSN_ERR_SHAPE also when N*C*S*ceil(T/64) >= 2^33.  The
 * library keeps no state; the call is asynchronous on `stream`. */
int mfpsn_forward_time_last(const mfpsn_desc* desc, const void* x, const int8_t* sign, const int8_t* shift,
                            const void* bias, uint8_t* spikes, void* h_out, void* stream);

/* Bytes of device workspace mfpsn_backward_time_last needs: 8-byte sums,
 * (k+1)*C of them plus (k+1) per partial-sum slot; the slots are
 * ceil(N*C*S/64) + N*C when T <= 64, else C plus the segment kernel's
 * waves (at most 4 * min(ceil(N*C*S*ceil(T/L)/4), 8192), L as below).
 * Depends on desc only.  Returns a status; *bytes is written on success. */
int mfpsn_backward_time_last_workspace_size(const mfpsn_desc* desc, size_t* bytes);

/* Backward (App. A.3 Eqs. backward_X, backward_W, backward_b, with the taps
 * dilated by d) in the time-last layout:
 *   x, grad_spikes : [N][C][S][T] storage type of desc->dtype
 *   grad_x         : [N][C][S][T] float (F32), bfloat16 (BF16, rounded to
 *                    nearest even) or int32 (Q8.8)
 *   grad_w [C][k], grad_b [C] : float, or int64 (Q8.8: Q16.16 and Q8.8);
 *                    overwritten
 *   workspace      : >= mfpsn_backward_time_last_workspace_size bytes,
 *                    8-byte aligned; contents on entry are ignored
 * H is recomputed from x (the charge of mfpsn_forward), dH = grad_spikes *
 * sigma'(H - v_th) with the surrogate of mfpsn_backward, and grad_x is the
 * definition's sum over the taps in ascending order, every term included.
 * grad_w and grad_b are sums of exact products in double (int64 for Q8.8)
 * rounded once to float; the double sums are added in a fixed order for a
 * given desc and device, so repeated calls give the same bits (the Q8.8
 * sums are exact).  Errors as
 * mfpsn_backward; MFPSN_ERR_SHAPE also for N*C*S >= 2^37 and, when T > 64,
 * for (k-1)*dilation > 1024 or N*C*S*ceil(T/L) >= 2^33, L = 256 (1024 when
 * (k-1)*dilation > 64).  Asynchronous on `stream`. */
int mfpsn_backward_time_last(const mfpsn_desc* desc, const void* x, const void* grad_spikes, const int8_t* sign,
                             const int8_t* shift, const void* bias, void* grad_x, void* grad_w, void* grad_b,
                             void* workspace, size_t workspace_bytes, void* stream);

/* Chaining layers: one layer's spikes as the next layer's input, for a
 * stack of neuron layers joined by identity stateless layers (the sawtooth
 * stack of Sec. 4.1, dilations 1..P one layer after the other).
 * x[i] = spikes[i] != 0 ? 1 : 0 in the storage type `dtype` (MFPSN_F32
 * float 1.0, MFPSN_BF16 bfloat16 1.0, MFPSN_Q8_8 int16 256), elementwise
 * over `count` elements of device memory (spikes uint8, x 2 or 4 bytes,
 * aligned to its element size, not overlapping spikes).  In the backward,
 * the next layer's grad_x is this layer's grad_spikes unchanged for the
 * float storage types (the derivative of the identity).  Errors:
 * MFPSN_ERR_SHAPE for count < 0, MFPSN_ERR_DTYPE, MFPSN_ERR_NULL,
 * MFPSN_ERR_ALIGN; count = 0 does nothing. */
int mfpsn_spikes_to_input(const uint8_t* spikes, int64_t count, int32_t dtype, void* x, void* stream);

/* MFPSN_ABI_VERSION of the loaded library. */
int32_t mfpsn_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MFPSN_H */
