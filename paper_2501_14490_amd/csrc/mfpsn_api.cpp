// C ABI of libmfpsn.so, the training step: argument validation, launch
// planning and dispatch of the forward, the backward and the quantizer.
// Declarations and the contract of every entry point are in include/mfpsn.h.
#include "mfpsn.h"

#include <math.h>
#include <stdint.h>
#include <string.h>

#include <initializer_list>

#include "mfpsn_internal.h"
#include "mfpsn_validate.h"

using namespace mfpsn;

namespace {

int grad_x_bytes(int dtype) { return dtype == MFPSN_BF16 ? 2 : 4; }

// Longest chunk of a residue class (a multiple of k) whose rows, with the
// halo and prefetch rows around it, keep every 32-bit buffer offset of an
// item in range; row_es is the widest element of the streams the call
// moves (4 covers every call).
int64_t max_chunk(const mfpsn_desc* d, int row_es = 4)
{
    const int64_t row = (int64_t)d->N * d->C * d->S * row_es * d->dilation;
    if (row <= 0)
        return INT64_MAX;
    const int64_t rows = (((int64_t)1 << 31) - 1) / row - 3 * (int64_t)d->k - 8;
    return rows >= d->k ? rows / d->k * d->k : 0;
}

}  // namespace

namespace mfpsn {
int validate(const mfpsn_desc* d)
{
    if (!d)
        return MFPSN_ERR_NULL;
    if (d->dtype != MFPSN_F32 && d->dtype != MFPSN_BF16 && d->dtype != MFPSN_Q8_8)
        return MFPSN_ERR_DTYPE;
    if (d->surrogate != MFPSN_SG_SIGMOID && d->surrogate != MFPSN_SG_ATAN &&
        d->surrogate != MFPSN_SG_RATIONAL)
        return MFPSN_ERR_DTYPE;
    if (d->T < 0 || d->N < 0 || d->C < 0 || d->S < 0)
        return MFPSN_ERR_SHAPE;
    if (d->k < 1 || d->k > MFPSN_MAX_K || d->dilation < 1)
        return MFPSN_ERR_PARAM;
    if ((int64_t)(d->k - 1) * d->dilation > (int64_t)1 << 30)
        return MFPSN_ERR_PARAM;
    // one time step of any tensor fits a 31-bit offset (the product of three
    // int32 sizes is formed in 128 bits, so it cannot overflow)
    const __int128 cols = (__int128)d->N * d->C * d->S;
    if (cols * 4 >= ((__int128)1 << 31))
        return MFPSN_ERR_SHAPE;
    const int64_t M = (int64_t)cols;
    if (d->C > 65535 && !(d->S == 1))  // plane mode puts one channel per grid row
        return MFPSN_ERR_SHAPE;
    if (M > 0 && d->T > 0 && max_chunk(d) == 0)  // k rows of one class do not fit 31-bit offsets
        return MFPSN_ERR_SHAPE;
    if (d->shift_lo > d->shift_hi)
        return MFPSN_ERR_PARAM;
    if (d->dtype == MFPSN_Q8_8) {
        if (d->shift_lo < 0 || d->shift_hi > 31)
            return MFPSN_ERR_PARAM;
        if (d->v_th_q < -(1 << 30) || d->v_th_q > (1 << 30))  // H - v_th_q fits int32
            return MFPSN_ERR_PARAM;
    } else {
        if (d->shift_lo < -126 || d->shift_hi > 126)
            return MFPSN_ERR_PARAM;
        if (!isfinite(d->v_th))
            return MFPSN_ERR_PARAM;
    }
    if (!(d->alpha >= 0.0f && d->alpha <= 1024.0f))
        return MFPSN_ERR_PARAM;
    return MFPSN_OK;
}
}  // namespace mfpsn

namespace {

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

constexpr int64_t kFwdTargetItems = 8192;
// Waves take contiguous ranges of items.  Taking every nw-th item instead
// (so that the waves running together walk neighbouring tiles) measured
// slower on MI355X for three of the four workloads (event vision 215 against
// 226 G elements/s, long fixed point 123 against 131), and faster only for
// the sequential-image shape (201 against 195).
constexpr bool kStridedItems = false;
// Items of one group (channel or channel group) are counted in 31 bits.
constexpr int64_t kMaxItems = ((int64_t)1 << 31) - 1;

// Two adjacent columns per lane (one 2x-wide access per stream and step):
// plane mode with an even S (a lane's two positions share one row of S
// columns), orders the two-column kernels are built for, and tensors aligned
// for the wide accesses.
bool pair_layout(const mfpsn_desc* d)
{
    return !(d->S == 1 && d->C >= 64) && d->S % 2 == 0 && d->k <= kPairMaxK;
}

bool pair_aligned(std::initializer_list<const void*> ptrs)
{
    for (const void* p : ptrs)
        if (p != nullptr && ((uintptr_t)p & 7u) != 0)
            return false;
    return true;
}

// The flat forward (16- or 8-byte accesses over the flattened rows): an
// order it is built for, S a multiple of its columns per lane, and tensors
// aligned for its accesses.
int flat_layout(const mfpsn_desc* d, const void* x, const void* spikes, const void* h_out, const void* sg_out)
{
    const int nv = flat_nv(d->k, d->dtype);
    if (nv == 0 || d->S % nv != 0)
        return 0;
    const uintptr_t wx = (uintptr_t)nv * elem_bytes(d->dtype), ws = (uintptr_t)nv;
    const uintptr_t ww = 4u * nv < 16u ? 4u * nv : 16u;
    if (((uintptr_t)x % wx) != 0 || ((uintptr_t)spikes % ws) != 0 || ((uintptr_t)h_out % ww) != 0 ||
        ((uintptr_t)sg_out % ww) != 0)
        return 0;
    return nv;
}

// flat: the flat forward's columns per lane (0: lane-channel or plane mode);
// row_es: the widest element of the call's streams (bounds the chunks)
Geom plan(const mfpsn_desc* d, bool backward, int nv, int flat = 0, int row_es = 4)
{
    Geom g;
    memset(&g, 0, sizeof(g));
    g.T = d->T;
    g.N = d->N;
    g.C = d->C;
    g.S = d->S;
    g.k = d->k;
    g.d = d->dilation;
    g.M = (uint32_t)((int64_t)d->N * d->C * d->S);
    g.tq = d->T / d->dilation;
    g.tr = d->T % d->dilation;
    g.esize = elem_bytes(d->dtype);
    g.shift_lo = d->shift_lo;
    g.shift_hi = d->shift_hi;
    g.sg = d->surrogate;
    g.alpha = d->alpha;
    g.v_th = d->v_th;
    g.v_th_q = d->v_th_q;
    {
        // x * 2^-s stays a normal float for every s in [lo, hi] when its
        // exponent field E satisfies max(1, hi+1) <= E <= 254 + min(0, lo)
        const int emin = d->shift_hi + 1 > 1 ? d->shift_hi + 1 : 1;
        const int emax = 254 + (d->shift_lo < 0 ? d->shift_lo : 0);
        if (emin > emax) {
            g.fast_lo = INFINITY;
            g.fast_hi = 0.0f;
        } else {
            g.fast_lo = ldexpf(1.0f, emin - 127);
            g.fast_hi = emax == 254 ? INFINITY : ldexpf(1.0f, emax - 126);
        }
        g.x_exact = d->dtype == MFPSN_BF16 && d->shift_lo >= 0 && d->shift_hi <= 16;
    }
    if (flat > 0) {
        g.mode = kFlat;
        g.nv = flat;
        g.groups = 1;
        g.tiles = (int32_t)ceil_div((int64_t)g.M, 64 * flat);
    } else if (d->S == 1 && d->C >= 64) {
        g.mode = kLaneChannel;
        g.nv = 1;
        g.groups = (int32_t)ceil_div(d->C, 64);
        g.tiles = d->N;
    } else {
        g.mode = kPlane;
        g.nv = nv;
        g.groups = d->C;
        g.tiles = (int32_t)ceil_div((int64_t)d->N * d->S, 64 * nv);
        // Rows whose length is not a multiple of 128 bytes start mid-line, so
        // tiles over the flattened plane straddle lines and neighbouring tiles
        // fetch the shared lines twice.  Long enough rows get tiles of their
        // own that start on lines, at the price of a few shadow lanes.
        const int64_t width = 64 * nv, line = 128 / g.esize;
        const int64_t per_row = ceil_div(d->S + line - 1, width);
        if (((int64_t)d->S * g.esize) % 128 != 0 && per_row * width * 8 <= (int64_t)d->S * 9) {
            g.row_tiles = (int32_t)per_row;
            g.tiles = (int32_t)(per_row * d->N);
        }
    }
    g.line_elems = 128 / g.esize;
    // Backward: each residue class is one chunk (at most the offset cap), and
    // the launcher cuts the classes finer for the kernel's resident waves
    // (balance_chunks), so the block bound allows the finest cut, chunks of k
    // steps.  Forward: classes are cut into chunks (multiples of k, of at
    // least 4k steps) only while the columns give fewer than kFwdTargetItems
    // items over all groups; the halo of a chunk is k-1 loads.
    const int64_t K = d->k;
    const int64_t class_len = d->T > 0 ? ceil_div(d->T, d->dilation) : 0;
    // residue classes that hold a step: d, or T when the dilation exceeds the
    // sequence (classes r >= T are empty)
    g.ncls = d->dilation < d->T ? d->dilation : (d->T > 0 ? d->T : 1);
    const int64_t base = (int64_t)g.tiles * g.ncls;
    int64_t cap = max_chunk(d, row_es);
    if (cap > ((int64_t)1 << 30))
        cap = ((int64_t)1 << 30) / K * K;
    int64_t chunk = ceil_div(class_len > 0 ? class_len : 1, K) * K;
    if (chunk > cap)
        chunk = cap;
    int64_t nchunks = ceil_div(class_len, chunk);
    if (!backward) {
        while ((int64_t)g.groups * base * nchunks < kFwdTargetItems && ceil_div(chunk / 2, K) * K >= 4 * K &&
               ceil_div(chunk / 2, K) * K < chunk) {
            chunk = ceil_div(chunk / 2, K) * K;
            nchunks = ceil_div(class_len, chunk);
        }
    }
    if (nchunks < 1)
        nchunks = 1;
    g.cap = (int32_t)cap;
    g.chunk = (int32_t)chunk;
    g.nchunks = (int32_t)nchunks;
    g.run_max = 1;
    g.items = base * g.nchunks;
    g.strided = kStridedItems ? 1 : 0;
    // upper bound of the persistent grid (the launcher picks the actual size)
    int64_t blocks = ceil_div(kMaxResidentBlocks, g.groups);
    const int64_t need = ceil_div(base * ceil_div(class_len > 0 ? class_len : 1, K), kWaves);
    if (blocks > need)
        blocks = need;
    g.blocks = (int32_t)(blocks > 0 ? blocks : 1);
    return g;
}

size_t workspace_bytes(const Geom& g)
{
    return (size_t)g.blocks * (size_t)(g.k + 1) * (size_t)g.C * sizeof(double);
}

// Workspace of the backward: enough for either column layout (the layout
// also depends on the pointers, which the size query does not see).
size_t backward_workspace(const mfpsn_desc* d)
{
    size_t b = workspace_bytes(plan(d, true, 1));
    if (pair_layout(d)) {
        const size_t b2 = workspace_bytes(plan(d, true, 2));
        b = b2 > b ? b2 : b;
    }
    return b;
}

}  // namespace

extern "C" {

int32_t mfpsn_abi_version(void) { return MFPSN_ABI_VERSION; }

const char* mfpsn_status_string(int status)
{
    switch (status) {
    case MFPSN_OK: return "ok";
    case MFPSN_ERR_NULL: return "a required pointer is NULL";
    case MFPSN_ERR_SHAPE: return "a size is negative or too large";
    case MFPSN_ERR_PARAM: return "invalid order, dilation, shift range, threshold or alpha";
    case MFPSN_ERR_DTYPE: return "unknown dtype or surrogate";
    case MFPSN_ERR_WORKSPACE: return "workspace too small or misaligned";
    case MFPSN_ERR_ALIGN: return "tensor pointer misaligned for its element type";
    case MFPSN_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
    }
}

int32_t mfpsn_sawtooth_dilation(int32_t layer, int32_t period)
{
    if (layer < 0 || period < 1)
        return 0;
    return (layer % period) + 1;
}

int mfpsn_forward(const mfpsn_desc* desc, const void* x, const int8_t* sign, const int8_t* shift,
                  const void* bias, const void* v_th_c, uint8_t* spikes, void* h_out, void* sg_out,
                  void* stream)
{
    int st = validate(desc);
    if (st != MFPSN_OK)
        return st;
    const int64_t total = (int64_t)desc->T * desc->N * desc->C * desc->S;
    if (total > 0 && (!x || !spikes))
        return MFPSN_ERR_NULL;
    if (desc->C > 0 && (!sign || !shift || !bias))
        return MFPSN_ERR_NULL;
    if (!aligned(x, elem_bytes(desc->dtype)) || !aligned(bias, 4) || !aligned(v_th_c, 4) ||
        !aligned(h_out, 4) || !aligned(sg_out, 4))
        return MFPSN_ERR_ALIGN;
    if (total == 0)
        return MFPSN_OK;
    FwdArgs a;
    a.g = plan(desc, false, pair_layout(desc) && pair_aligned({x, spikes, h_out, sg_out}) ? 2 : 1,
               flat_layout(desc, x, spikes, h_out, sg_out),
               h_out || sg_out ? 4 : elem_bytes(desc->dtype));
    if (a.g.items > kMaxItems)
        return MFPSN_ERR_SHAPE;
    a.x = x;
    a.sign = sign;
    a.shift = shift;
    a.bias = bias;
    a.v_th_c = v_th_c;
    a.spikes = spikes;
    a.h_out = h_out;
    a.sg_out = sg_out;
    if (launch_forward(a, desc->dtype, (hipStream_t)stream) != hipSuccess)
        return MFPSN_ERR_HIP;
    return MFPSN_OK;
}

int mfpsn_backward_workspace_size(const mfpsn_desc* desc, size_t* bytes)
{
    int st = validate(desc);
    if (st != MFPSN_OK)
        return st;
    if (!bytes)
        return MFPSN_ERR_NULL;
    const int64_t total = (int64_t)desc->T * desc->N * desc->C * desc->S;
    if (total > 0 && (plan(desc, true, 1).items > kMaxItems || plan(desc, true, 2).items > kMaxItems))
        return MFPSN_ERR_SHAPE;
    *bytes = total > 0 ? backward_workspace(desc) : 0;
    return MFPSN_OK;
}

int mfpsn_backward(const mfpsn_desc* desc, const void* x, const void* grad_spikes, const void* h,
                   const void* sg, const int8_t* sign, const int8_t* shift, const void* bias,
                   const void* v_th_c, void* grad_x, void* grad_w, void* grad_b, void* grad_vth,
                   void* workspace, size_t ws_bytes, void* stream)
{
    int st = validate(desc);
    if (st != MFPSN_OK)
        return st;
    const int64_t total = (int64_t)desc->T * desc->N * desc->C * desc->S;
    if (total > 0 && (!x || !grad_spikes || !grad_x))
        return MFPSN_ERR_NULL;
    if (desc->C > 0 && (!sign || !shift || !bias || !grad_w || !grad_b))
        return MFPSN_ERR_NULL;
    const int es = elem_bytes(desc->dtype);
    if (!aligned(x, es) || !aligned(grad_spikes, es) || !aligned(grad_x, grad_x_bytes(desc->dtype)) ||
        !aligned(bias, 4) || !aligned(v_th_c, 4) || !aligned(h, 4) || !aligned(sg, 4) ||
        !aligned(grad_w, desc->dtype == MFPSN_Q8_8 ? 8 : 4) || !aligned(grad_b, desc->dtype == MFPSN_Q8_8 ? 8 : 4) ||
        !aligned(grad_vth, desc->dtype == MFPSN_Q8_8 ? 8 : 4))
        return MFPSN_ERR_ALIGN;
    if (desc->dtype == MFPSN_Q8_8) {
        // every partial sum of grad_w must fit int64
        const double reach = (double)desc->T * desc->N * desc->S * 32768.0 * q88_max_dh(desc);
        if (reach >= 4611686018427387904.0)
            return MFPSN_ERR_SHAPE;
    }
    BwdArgs a;
    // (the block bound, and with it the workspace, does not depend on the
    // row width: it allows the finest cut of the classes)
    const int row_es = h || sg ? 4 : (es > grad_x_bytes(desc->dtype) ? es : grad_x_bytes(desc->dtype));
    a.g = plan(desc, true, pair_layout(desc) && pair_aligned({x, grad_spikes, h, sg, grad_x}) ? 2 : 1, 0, row_es);
    if (total > 0 && a.g.items > kMaxItems)
        return MFPSN_ERR_SHAPE;
    const size_t need = total > 0 ? backward_workspace(desc) : 0;
    if (need > 0 && (!workspace || ws_bytes < need || !aligned(workspace, 8)))
        return MFPSN_ERR_WORKSPACE;
    a.x = x;
    a.gs = grad_spikes;
    a.h = h;
    a.sg = sg;
    a.sign = sign;
    a.shift = shift;
    a.bias = bias;
    a.v_th_c = v_th_c;
    a.grad_x = grad_x;
    a.partial = (double*)workspace;
    hipStream_t s = (hipStream_t)stream;
    if (total > 0 && launch_backward(a, desc->dtype, s) != hipSuccess)
        return MFPSN_ERR_HIP;
    FinArgs f;
    f.C = desc->C;
    f.k = desc->k;
    f.blocks = total > 0 ? a.g.blocks : 0;
    f.dtype = desc->dtype;
    f.partial = (const double*)workspace;
    f.grad_w = grad_w;
    f.grad_b = grad_b;
    f.grad_vth = grad_vth;
    if (launch_finalize(f, s) != hipSuccess)
        return MFPSN_ERR_HIP;
    return MFPSN_OK;
}

int mfpsn_quantize_weights(const float* w, int64_t count, int32_t shift_lo, int32_t shift_hi,
                           int8_t* sign, int8_t* shift, void* stream)
{
    if (count < 0 || count >= ((int64_t)1 << 31))
        return MFPSN_ERR_SHAPE;
    if (shift_lo > shift_hi || shift_lo < -128 || shift_hi > 127)
        return MFPSN_ERR_PARAM;
    if (count > 0 && (!w || !sign || !shift))
        return MFPSN_ERR_NULL;
    if (!aligned(w, 4))
        return MFPSN_ERR_ALIGN;
    if (launch_quantize(w, count, shift_lo, shift_hi, sign, shift, (hipStream_t)stream) != hipSuccess)
        return MFPSN_ERR_HIP;
    return MFPSN_OK;
}

}  // extern "C"
