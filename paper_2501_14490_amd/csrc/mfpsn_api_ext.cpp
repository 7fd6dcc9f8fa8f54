// C ABI of libmfpsn.so beside the training step: the batch-normalized
// threshold with fused-weight quantization, the quantizer's latent-weight
// gradient, step-by-step inference, the chaining of layers and the forward
// in the time-last layout.  Declarations and the contract of
// every entry point are in include/mfpsn.h.
#include "mfpsn.h"

#include <math.h>
#include <stdint.h>

#include "mfpsn_bn.h"
#include "mfpsn_chain.h"
#include "mfpsn_internal.h"
#include "mfpsn_qgrad.h"
#include "mfpsn_stream.h"
#include "mfpsn_tl.h"
#include "mfpsn_validate.h"

using namespace mfpsn;

namespace {

// The streaming step looks at one time step: the descriptor's T plays no
// part, every other field is checked as for the whole-sequence calls.
int validate_stream(const mfpsn_desc* d)
{
    if (!d)
        return MFPSN_ERR_NULL;
    mfpsn_desc one = *d;
    one.T = 0;
    return validate(&one);
}

// History slots of the streaming step: the receptive field (k-1)*d + 1.
int64_t ring_steps(const mfpsn_desc* d) { return (int64_t)(d->k - 1) * d->dilation + 1; }

}  // namespace

namespace {
// The batch-normalization entry points take float x (MFPSN_F32) and one
// layer's shapes; T is used.
int validate_bn(const mfpsn_desc* d, BnGeom* g)
{
    const int st = validate(d);
    if (st != MFPSN_OK)
        return st;
    if (d->dtype != MFPSN_F32)
        return MFPSN_ERR_DTYPE;
    g->T = d->T;
    g->N = d->N;
    g->C = d->C;
    g->S = d->S;
    g->k = d->k;
    g->d = d->dilation;
    g->M = (size_t)d->N * d->C * d->S;
    g->tq = d->T / d->dilation;
    g->tr = d->T % d->dilation;
    // Walk plan: a grid of about three waves per SIMD (256 CUs x 4 SIMDs),
    // chunks of each residue class such that each thread has two or three
    // items (each chunk at least 2k steps), and a thread count that spreads
    // the items evenly and keeps every thread in one channel
    constexpr int64_t kTarget = 256 * 4 * 3 * 64;
    const int64_t L = ((int64_t)d->T + d->dilation - 1) / d->dilation;
    const int64_t walks = (int64_t)g->M * d->dilation;
    int64_t nch = walks > 0 ? (2 * kTarget + walks - 1) / walks : 1;
    const int64_t max_nch = L / (2 * (int64_t)d->k);
    if (nch > max_nch)
        nch = max_nch;
    if (nch < 1)
        nch = 1;
    g->lc = L > 0 ? (int32_t)((L + nch - 1) / nch) : 1;  // an empty sequence has no chunks
    g->nch = (int32_t)((L + g->lc - 1) / g->lc);
    g->items = (size_t)g->nch * d->dilation * g->M;
    const int64_t SC = (int64_t)d->S * d->C;
    int64_t a = SC, b = kBnThreads;  // base = lcm(SC, block size)
    while (b != 0) {
        const int64_t t = a % b;
        a = b;
        b = t;
    }
    const int64_t base = SC / a * kBnThreads;
    const int64_t items = (int64_t)g->items;
    int64_t G;
    if (items == 0)
        G = kBnThreads;
    else if (base > items)
        G = (items + kBnThreads - 1) / kBnThreads * kBnThreads;  // one item per thread
    else {
        const int64_t per = (items + kTarget - 1) / kTarget;  // items per thread
        G = ((items + per - 1) / per + base - 1) / base * base;
    }
    g->G = (size_t)G;
    g->R = SC > 0 ? (int32_t)((G + SC - 1) / SC) : 1;
    g->NG = (g->R + kBnRowGroup - 1) / kBnRowGroup;
    return MFPSN_OK;
}

// Range [lo, hi) of |v| in which v * 2^-s stays a normal float for every s
// in [shift_lo, shift_hi]: exponent field E with max(1, hi+1) <= E <=
// 254 + min(0, lo) (empty when no E qualifies)
void fast_range(const mfpsn_desc* desc, float* lo, float* hi)
{
    const int emin = desc->shift_hi + 1 > 1 ? desc->shift_hi + 1 : 1;
    const int emax = 254 + (desc->shift_lo < 0 ? desc->shift_lo : 0);
    if (emin > emax) {
        *lo = INFINITY;
        *hi = 0.0f;
    } else {
        *lo = ldexpf(1.0f, emin - 127);
        *hi = emax == 254 ? INFINITY : ldexpf(1.0f, emax - 126);
    }
}
}  // namespace

int mfpsn_bn_workspace_size(const mfpsn_desc* desc, size_t* bytes)
{
    BnGeom g;
    const int st = validate_bn(desc, &g);
    if (st != MFPSN_OK)
        return st;
    if (!bytes)
        return MFPSN_ERR_NULL;
    *bytes = g.M > 0 && g.T > 0 ? bn_workspace_bytes(g) : 0;
    return MFPSN_OK;
}

int mfpsn_bn_forward_stats(const mfpsn_desc* desc, const float* x, const float* w, const float* gamma,
                           const float* beta, float eps, float* w_f, float* b_f, double* aux, double* stats,
                           void* workspace, size_t workspace_bytes, void* stream)
{
    BnGeom g;
    const int st = validate_bn(desc, &g);
    if (st != MFPSN_OK)
        return st;
    if (!(eps > 0.0f) || !isfinite(eps))
        return MFPSN_ERR_PARAM;
    if (g.M == 0 || g.T == 0)
        return MFPSN_ERR_SHAPE;  // statistics of an empty batch are undefined
    if (!x || !w || !gamma || !beta || !w_f || !b_f || !aux)
        return MFPSN_ERR_NULL;
    if (!aligned(x, 4) || !aligned(w, 4) || !aligned(gamma, 4) || !aligned(beta, 4) || !aligned(w_f, 4) ||
        !aligned(b_f, 4) || !aligned(aux, 8) || !aligned(stats, 8))
        return MFPSN_ERR_ALIGN;
    if (!workspace || workspace_bytes < bn_workspace_bytes(g) || !aligned(workspace, 8))
        return MFPSN_ERR_WORKSPACE;
    if (launch_bn_forward_stats(g, x, w, gamma, beta, eps, w_f, b_f, aux, stats, workspace, (hipStream_t)stream) !=
        hipSuccess)
        return MFPSN_ERR_HIP;
    return MFPSN_OK;
}

int mfpsn_bn_backward(const mfpsn_desc* desc, const float* x, const float* w, const double* aux, float eps,
                      const float* grad_wf, const float* grad_bf, float* grad_x, float* grad_w, float* grad_gamma,
                      float* grad_beta, void* workspace, size_t workspace_bytes, void* stream)
{
    BnGeom g;
    const int st = validate_bn(desc, &g);
    if (st != MFPSN_OK)
        return st;
    if (!(eps > 0.0f) || !isfinite(eps))
        return MFPSN_ERR_PARAM;
    if (g.M == 0 || g.T == 0)
        return MFPSN_ERR_SHAPE;
    if (!x || !w || !aux || !grad_wf || !grad_bf || !grad_x || !grad_w || !grad_gamma || !grad_beta)
        return MFPSN_ERR_NULL;
    if (!aligned(x, 4) || !aligned(w, 4) || !aligned(aux, 8) || !aligned(grad_wf, 4) || !aligned(grad_bf, 4) ||
        !aligned(grad_x, 4) || !aligned(grad_w, 4) || !aligned(grad_gamma, 4) || !aligned(grad_beta, 4))
        return MFPSN_ERR_ALIGN;
    if (!workspace || workspace_bytes < bn_workspace_bytes(g) || !aligned(workspace, 8))
        return MFPSN_ERR_WORKSPACE;
    if (launch_bn_backward(g, x, w, aux, eps, grad_wf, grad_bf, grad_x, grad_w, grad_gamma, grad_beta, workspace,
                           (hipStream_t)stream) != hipSuccess)
        return MFPSN_ERR_HIP;
    return MFPSN_OK;
}

int mfpsn_quantizer_grad(const float* w, const int8_t* shift, int32_t shift_lo, int32_t shift_hi,
                         const float* grad_wq, int64_t count, int32_t mode, float* grad_w, void* stream)
{
    if (count < 0 || count >= ((int64_t)1 << 31))
        return MFPSN_ERR_SHAPE;
    if (shift_lo > shift_hi || shift_lo < -128 || shift_hi > 127 || (mode != MFPSN_STE_WHOLE && mode != MFPSN_STE_ROUND))
        return MFPSN_ERR_PARAM;
    if (count > 0 && (!grad_wq || !grad_w || (mode == MFPSN_STE_ROUND && (!w || !shift))))
        return MFPSN_ERR_NULL;
    if (!aligned(w, 4) || !aligned(grad_wq, 4) || !aligned(grad_w, 4))
        return MFPSN_ERR_ALIGN;
    if (launch_quantizer_grad(w, shift, shift_lo, shift_hi, grad_wq, count, mode, grad_w, (hipStream_t)stream) !=
        hipSuccess)
        return MFPSN_ERR_HIP;
    return MFPSN_OK;
}

int mfpsn_stream_ring_bytes(const mfpsn_desc* desc, int32_t* steps, size_t* bytes)
{
    int st = validate_stream(desc);
    if (st != MFPSN_OK)
        return st;
    if (!steps && !bytes)
        return MFPSN_ERR_NULL;
    const int64_t R = ring_steps(desc);
    const int64_t M = (int64_t)desc->N * desc->C * desc->S;
    if (steps)
        *steps = (int32_t)R;
    if (bytes)
        *bytes = (size_t)R * (size_t)M * (size_t)elem_bytes(desc->dtype);
    return MFPSN_OK;
}

int mfpsn_stream_step(const mfpsn_desc* desc, int64_t t, const void* x_t, void* ring, const int8_t* sign,
                      const int8_t* shift, const void* bias, uint8_t* spikes_t, void* h_t, void* stream)
{
    int st = validate_stream(desc);
    if (st != MFPSN_OK)
        return st;
    if (t < 0)
        return MFPSN_ERR_PARAM;
    const int64_t M = (int64_t)desc->N * desc->C * desc->S;
    if (M > 0 && (!x_t || !ring || !spikes_t))
        return MFPSN_ERR_NULL;
    if (desc->C > 0 && (!sign || !shift || !bias))
        return MFPSN_ERR_NULL;
    const int es = elem_bytes(desc->dtype);
    if (!aligned(x_t, es) || !aligned(ring, es) || !aligned(bias, 4) || !aligned(h_t, 4))
        return MFPSN_ERR_ALIGN;
    if (M == 0)
        return MFPSN_OK;
    const int64_t R = ring_steps(desc);
    StreamArgs a;
    a.M = M;
    a.C = desc->C;
    a.S = desc->S;
    a.k = desc->k;
    a.d = desc->dilation;
    a.R = (int32_t)R;
    a.slot = (int32_t)(t % R);
    const int64_t reach = t / desc->dilation;  // taps that look back at most t steps
    a.m_max = (int32_t)(reach < desc->k - 1 ? reach : desc->k - 1);
    for (int m = 0; m < MFPSN_MAX_K; ++m) {
        int64_t sl = m < desc->k ? a.slot - (int64_t)m * desc->dilation : 0;  // >= -(R-1)
        if (sl < 0)
            sl += R;
        a.rows[m] = sl * M;
    }
    a.shift_lo = desc->shift_lo;
    a.shift_hi = desc->shift_hi;
    a.v_th = desc->v_th;
    a.v_th_q = desc->v_th_q;
    a.x_t = x_t;
    a.ring = ring;
    a.sign = sign;
    a.shift = shift;
    a.bias = bias;
    a.spikes = spikes_t;
    a.h_t = h_t;
    if (launch_stream_step(a, desc->dtype, (hipStream_t)stream) != hipSuccess)
        return MFPSN_ERR_HIP;
    return MFPSN_OK;
}


int mfpsn_spikes_to_input(const uint8_t* spikes, int64_t count, int32_t dtype, void* x, void* stream)
{
    if (count < 0)
        return MFPSN_ERR_SHAPE;
    if (dtype != MFPSN_F32 && dtype != MFPSN_BF16 && dtype != MFPSN_Q8_8)
        return MFPSN_ERR_DTYPE;
    if (count == 0)
        return MFPSN_OK;
    if (!spikes || !x)
        return MFPSN_ERR_NULL;
    if (!aligned(x, elem_bytes(dtype)))
        return MFPSN_ERR_ALIGN;
    if (launch_spikes_to_input(spikes, count, dtype, x, (hipStream_t)stream) != hipSuccess)
        return MFPSN_ERR_HIP;
    return MFPSN_OK;
}

int mfpsn_forward_time_last(const mfpsn_desc* desc, const void* x, const int8_t* sign, const int8_t* shift,
                            const void* bias, uint8_t* spikes, void* h_out, void* stream)
{
    const int st = validate(desc);
    if (st != MFPSN_OK)
        return st;
    const int64_t M = (int64_t)desc->N * desc->C * desc->S;
    // long columns with histories of at most kTlBwdMaxSpan steps: segments of
    // 256 steps (1024 for histories above 64); longer histories: segments of
    // 256 time steps, or of 64 for short sequences (fewer idle lanes)
    const int64_t span = (int64_t)(desc->k - 1) * desc->dilation;
    const int seg = desc->T > kTlColsMaxT && span <= kTlBwdMaxSpan ? (span > 64 ? kTlBwdSegLong : kTlBwdSeg) : 0;
    const int spl = desc->T > 96 ? 4 : 1;
    const int64_t nseg = seg > 0 ? ((int64_t)desc->T + seg - 1) / seg : ((int64_t)desc->T + 64 * spl - 1) / (64 * spl);
    if (M * (((int64_t)desc->T + 63) / 64) >= ((int64_t)1 << 33))  // segments must fit the grid
        return MFPSN_ERR_SHAPE;
    if (M == 0 || desc->T == 0)
        return MFPSN_OK;
    if (!x || !sign || !shift || !bias || !spikes)
        return MFPSN_ERR_NULL;
    const int es = elem_bytes(desc->dtype);
    if (!aligned(x, es) || !aligned(bias, 4) || !aligned(h_out, 4))
        return MFPSN_ERR_ALIGN;
    TlArgs a;
    a.x = x;
    a.sign = sign;
    a.shift = shift;
    a.bias = bias;
    a.spikes = spikes;
    a.h_out = h_out;
    a.M = M;
    a.T = desc->T;
    a.C = desc->C;
    a.S = desc->S;
    a.k = desc->k;
    a.d = desc->dilation;
    a.steps_per_lane = spl;
    a.seg = seg;
    a.nseg = (int32_t)nseg;
    a.halo = span <= kTlMaxHalo ? (int32_t)span : 0;
    a.shift_lo = desc->shift_lo;
    a.shift_hi = desc->shift_hi;
    a.v_th = desc->v_th;
    a.v_th_q = desc->v_th_q;
    fast_range(desc, &a.fast_lo, &a.fast_hi);
    a.tdiv = desc->T >= 2 ? (uint32_t)((((uint64_t)1) << 32) / (uint64_t)desc->T + 1) : 0;
    a.vec_x = aligned(x, 4 * es) ? 1 : 0;
    a.vec_s = aligned(spikes, 16) ? 1 : 0;
    if (launch_forward_time_last(a, desc->dtype, (hipStream_t)stream) != hipSuccess)
        return MFPSN_ERR_HIP;
    return MFPSN_OK;
}

// Workspace of the time-last backward: the [k+1][C] sums, then the
// partial-sum slots (tl_bwd_slots) of k+1 sums each, 8 bytes per sum.
static size_t tl_bwd_workspace(const mfpsn_desc* desc)
{
    const int64_t M = (int64_t)desc->N * desc->C * desc->S;
    const int seg = (int64_t)(desc->k - 1) * desc->dilation > 64 ? kTlBwdSegLong : kTlBwdSeg;
    const int64_t nseg = ((int64_t)desc->T + seg - 1) / seg;
    const int64_t slots = tl_bwd_slots(M, desc->T, desc->C, desc->N, nseg);
    return (size_t)(desc->k + 1) * ((size_t)desc->C + (size_t)slots) * 8;
}

int mfpsn_backward_time_last_workspace_size(const mfpsn_desc* desc, size_t* bytes)
{
    const int st = validate(desc);
    if (st != MFPSN_OK)
        return st;
    if (!bytes)
        return MFPSN_ERR_NULL;
    *bytes = tl_bwd_workspace(desc);
    return MFPSN_OK;
}

int mfpsn_backward_time_last(const mfpsn_desc* desc, const void* x, const void* grad_spikes, const int8_t* sign,
                             const int8_t* shift, const void* bias, void* grad_x, void* grad_w, void* grad_b,
                             void* workspace, size_t ws_bytes, void* stream)
{
    const int st = validate(desc);
    if (st != MFPSN_OK)
        return st;
    const int64_t M = (int64_t)desc->N * desc->C * desc->S;
    // long histories: longer segments, so that the dH recomputed over the
    // history after each segment is a smaller share of its work
    const int seg = (int64_t)(desc->k - 1) * desc->dilation > 64 ? kTlBwdSegLong : kTlBwdSeg;
    const int64_t nseg = ((int64_t)desc->T + seg - 1) / seg;
    if (M >= ((int64_t)1 << 37))
        return MFPSN_ERR_SHAPE;
    if (desc->T > kTlColsMaxT &&
        ((int64_t)(desc->k - 1) * desc->dilation > kTlBwdMaxSpan || M * nseg >= ((int64_t)1 << 33)))
        return MFPSN_ERR_SHAPE;
    const int64_t total = M * desc->T;
    if (total > 0 && (!x || !grad_spikes || !grad_x))
        return MFPSN_ERR_NULL;
    if (desc->C > 0 && (!sign || !shift || !bias || !grad_w || !grad_b))
        return MFPSN_ERR_NULL;
    const int es = elem_bytes(desc->dtype);
    const size_t wb = desc->dtype == MFPSN_Q8_8 ? 8 : 4;
    if (!aligned(x, es) || !aligned(grad_spikes, es) || !aligned(grad_x, desc->dtype == MFPSN_BF16 ? 2 : 4) ||
        !aligned(bias, 4) || !aligned(grad_w, wb) || !aligned(grad_b, wb))
        return MFPSN_ERR_ALIGN;
    if (desc->dtype == MFPSN_Q8_8) {
        // every partial sum of grad_w must fit int64
        const double reach = (double)desc->T * desc->N * desc->S * 32768.0 * q88_max_dh(desc);
        if (reach >= 4611686018427387904.0)
            return MFPSN_ERR_SHAPE;
    }
    const size_t need = tl_bwd_workspace(desc);
    if (need > 0 && (!workspace || ws_bytes < need || !aligned(workspace, 8)))
        return MFPSN_ERR_WORKSPACE;
    if (desc->C == 0)
        return MFPSN_OK;
    TlBwdArgs a;
    a.x = x;
    a.g = grad_spikes;
    a.sign = sign;
    a.shift = shift;
    a.bias = bias;
    a.grad_x = grad_x;
    a.acc = workspace;
    a.part = (char*)workspace + (size_t)(desc->k + 1) * (size_t)desc->C * 8;
    a.M = M;
    a.T = desc->T;
    a.C = desc->C;
    a.S = desc->S;
    a.k = desc->k;
    a.d = desc->dilation;
    a.shift_lo = desc->shift_lo;
    a.shift_hi = desc->shift_hi;
    a.v_th = desc->v_th;
    a.v_th_q = desc->v_th_q;
    a.sg = desc->surrogate;
    a.alpha = desc->alpha;
    fast_range(desc, &a.fast_lo, &a.fast_hi);
    a.tdiv = desc->T >= 2 ? (uint32_t)((((uint64_t)1) << 32) / (uint64_t)desc->T + 1) : 0;
    a.vec_x = aligned(x, 4 * es) && aligned(grad_spikes, 4 * es) ? 1 : 0;
    a.seg = seg;
    a.nseg = (int32_t)nseg;
    a.chunk = 0;
    hipStream_t s = (hipStream_t)stream;
    if (launch_backward_time_last(a, desc->dtype, s) != hipSuccess)
        return MFPSN_ERR_HIP;
    FinArgs f;
    f.C = desc->C;
    f.k = desc->k;
    f.blocks = 1;
    f.dtype = desc->dtype;
    f.partial = (const double*)workspace;
    f.grad_w = grad_w;
    f.grad_b = grad_b;
    f.grad_vth = nullptr;
    if (launch_finalize(f, s) != hipSuccess)
        return MFPSN_ERR_HIP;
    return MFPSN_OK;
}
