// gfx950 kernels of the mul-free channel-wise Parallel Spiking Neuron
// (arXiv 2501.14490): forward charge + fire, fused surrogate-gradient
// backward, deterministic reduction of the weight/bias gradients, and the
// power-of-two weight quantizer.
//
// Work decomposition.  x is time-first, [T][N][C][S]; the M = N*C*S columns
// are independent time series.  A dilated order-k convolution only couples
// time steps of one residue class t = r (mod d), so each lane walks one
// column along one residue class (class step j <-> time r + j*d), optionally
// restricted to a chunk [j0, j1) of class steps.  The lane keeps the last k
// inputs of its walk in a register ring, so every input is read from HBM once
// per pass (plus a (k-1)-step halo per chunk).  The ring is indexed with
// compile-time slots: the walk is unrolled by k, and class step j lives in
// slot (j - j0 + k - 1) mod k.
//
// Taps never multiply: a float tap is an exact exponent move (v_ldexp_f32)
// followed by a sign flip (xor of the sign bit) and one rounded add; a Q8.8
// tap is an arithmetic right shift and an xor-add (the -1 that xor-negation
// leaves per negative tap is folded into the starting value).  Sums run in
// ascending tap order from +0 with the bias added last, so the float
// potentials are bit-identical to a sequential evaluation of the definition.
//
// The backward recomputes H from the x ring (H is not stored), evaluates the
// surrogate, pushes dH into a second ring, emits grad_x (k-1) class steps
// late (when the last dH it needs exists), and accumulates grad_w / grad_b
// from exact double products (Q8.8: exact integers in double).  Per-lane sums
// are reduced inside the block in a fixed order and written as per-block
// partials; a finalize kernel adds the partials in block order, so the
// gradients are bitwise reproducible.
#include <hip/hip_runtime.h>
#include <hip/hip_bf16.h>
#include <stdint.h>

#include <utility>

#include "mfpsn_internal.h"


namespace mfpsn {
namespace {

constexpr uint32_t kOutOfRange = 0x80000000u;  // buffer offset past every num_records we use
constexpr int kRsrcWord3 = 0x00020000;         // raw (untyped) buffer, gfx9 family

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, uint64_t byte_off,
                                                       uint32_t nbytes)
{
    return __builtin_amdgcn_make_buffer_rsrc((void*)((const char*)base + byte_off), (short)0,
                                             (int)nbytes, kRsrcWord3);
}

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// ---------------------------------------------------------------------------
// storage types
// ---------------------------------------------------------------------------
template <int DT> struct IO;

template <> struct IO<kF32> {
    using V = float;    // register value of x / grad_spikes
    using D = float;    // dH
    static constexpr int es = 4;
    __device__ static V load(__amdgpu_buffer_rsrc_t r, uint32_t vo)
    {
        return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, vo, 0, 0));
    }
    static constexpr int gx_es = 4;
    __device__ static void store_gx(__amdgpu_buffer_rsrc_t r, uint32_t vo, D v)
    {
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), r, vo, 0, 0);
    }
};

template <> struct IO<kBF16> {
    using V = float;
    using D = float;
    static constexpr int es = 2;
    __device__ static V load(__amdgpu_buffer_rsrc_t r, uint32_t vo)
    {
        uint32_t h = __builtin_amdgcn_raw_buffer_load_b16(r, vo, 0, 0);
        return __builtin_bit_cast(float, h << 16);
    }
    static constexpr int gx_es = 2;
    __device__ static void store_gx(__amdgpu_buffer_rsrc_t r, uint32_t vo, D v)
    {
        __bf16 h = (__bf16)v;  // round to nearest even (v_cvt_pk_bf16_f32)
        __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, h), r, vo, 0, 0);
    }
};

template <> struct IO<kQ88> {
    using V = int32_t;
    using D = int32_t;
    static constexpr int es = 2;
    __device__ static V load(__amdgpu_buffer_rsrc_t r, uint32_t vo)
    {
        uint32_t h = __builtin_amdgcn_raw_buffer_load_b16(r, vo, 0, 0);
        return (int32_t)(int16_t)(uint16_t)h;
    }
    static constexpr int gx_es = 4;
    __device__ static void store_gx(__amdgpu_buffer_rsrc_t r, uint32_t vo, D v)
    {
        __builtin_amdgcn_raw_buffer_store_b32((uint32_t)v, r, vo, 0, 0);
    }
};

// ---------------------------------------------------------------------------
// taps: weight sign * 2^-shift
// ---------------------------------------------------------------------------
template <int K, int DT> struct Taps;

template <int K> struct TapsF {
    int nsh[K];        // -shift
    uint32_t sm[K];    // sign bit to xor in
    __device__ void load(const int8_t* sign, const int8_t* shift, int c, int lo, int hi)
    {
#pragma unroll
        for (int i = 0; i < K; ++i) {
            int s = shift[c * K + i];
            s = s < lo ? lo : (s > hi ? hi : s);
            nsh[i] = -s;
            sm[i] = sign[c * K + i] < 0 ? 0x80000000u : 0u;
        }
    }
    // sign * 2^-shift * v: exact exponent move, then sign flip.
    __device__ __forceinline__ float apply(float v, int i) const
    {
        float y = ldexpf(v, nsh[i]);
        return __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, y) ^ sm[i]);
    }
};
template <int K> struct Taps<K, kF32> : TapsF<K> {};
template <int K> struct Taps<K, kBF16> : TapsF<K> {};

template <int K> struct Taps<K, kQ88> {
    int sh[K];         // shift, 0..31
    int m[K];          // 0 (positive tap) or -1 (negative tap)
    int cneg;          // number of negative taps
    __device__ void load(const int8_t* sign, const int8_t* shift, int c, int lo, int hi)
    {
        cneg = 0;
#pragma unroll
        for (int i = 0; i < K; ++i) {
            int s = shift[c * K + i];
            s = s < lo ? lo : (s > hi ? hi : s);
            sh[i] = s;
            m[i] = sign[c * K + i] < 0 ? -1 : 0;
            cneg -= m[i];
        }
    }
    // (v >> s) ^ m equals +(v >> s) or -(v >> s) - 1; the -1s are cancelled by
    // starting the sum at cneg.
    __device__ __forceinline__ int apply(int v, int i) const { return (v >> sh[i]) ^ m[i]; }
};

// ---------------------------------------------------------------------------
// surrogate derivative (float, fixed operation sequence)
// ---------------------------------------------------------------------------
// exp(y): Cody-Waite reduction with ln 2 = hi + lo (hi has 15 significant
// bits), degree-7 Taylor polynomial of e^r by fma Horner steps, scaling by
// 2^n.  y < -86 (or NaN) gives 0, y > 88 is clamped to 88.
__device__ __forceinline__ float mf_exp(float y)
{
    const float log2e = 0x1.715476p+0f;
    const float ln2hi = 0x1.62e4p-1f;
    const float ln2lo = 0x1.7f7d1cp-20f;
    const bool zero = !(y >= -86.0f);
    y = y > 88.0f ? 88.0f : y;
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

struct Surrogate {
    int kind;
    float alpha;
    float c_atan;   // float(pi/2) * alpha
    __device__ __forceinline__ float operator()(float u) const
    {
        if (kind == 0) {
            float a = alpha * fabsf(u);
            float e = mf_exp(-a);
            float den = 1.0f + e;
            float num = alpha * e;
            float den2 = den * den;
            return num / den2;
        }
        if (kind == 1) {
            float z = c_atan * u;
            float z2 = z * z;
            float den = 1.0f + z2;
            float num = 0.5f * alpha;
            return num / den;
        }
        float u2 = u * u;
        float au2 = alpha * u2;
        float den = 1.0f + au2;
        return 1.0f / den;
    }
};

__device__ __forceinline__ float delta_h(const Surrogate& sg, float g, float h, float v_th, int)
{
    float u = h - v_th;
    return g * sg(u);
}

__device__ __forceinline__ int32_t delta_h(const Surrogate& sg, int32_t g, int32_t h, float,
                                           int v_th_q)
{
    int32_t u = h - v_th_q;
    float uf = (float)u * 0.00390625f;
    float s = sg(uf);
    int32_t L = (int32_t)rintf(s * 32768.0f);
    int64_t p = (int64_t)g * (int64_t)L;
    return (int32_t)(p >> 15);
}

// ---------------------------------------------------------------------------
// lane -> column
// ---------------------------------------------------------------------------
struct Item {
    int r;        // residue class
    int Lr;       // class length
    int j0, j1;   // class-step chunk
    bool active;  // this lane's column exists
    uint32_t col; // column index in [0, M)
};

template <int MODE>
__device__ __forceinline__ Item decode_item(const Geom& g, int64_t q, int grp, int lane)
{
    Item it;
    const int chunk_id = (int)(q % g.nchunks);
    const int64_t q2 = q / g.nchunks;
    it.r = (int)(q2 % g.d);
    const int tile = (int)(q2 / g.d);
    it.Lr = it.r < g.T ? (g.T - it.r + g.d - 1) / g.d : 0;
    it.j0 = chunk_id * g.chunk;
    it.j1 = min(it.Lr, it.j0 + g.chunk);
    if (MODE == kLaneChannel) {
        const int c = grp * 64 + lane;
        it.active = c < g.C;
        it.col = (uint32_t)tile * (uint32_t)g.C + (uint32_t)c;
    } else if (g.S >= 64) {
        const int n = tile / g.spw;
        const int s = (tile % g.spw) * 64 + lane;
        it.active = s < g.S;
        it.col = ((uint32_t)n * (uint32_t)g.C + (uint32_t)grp) * (uint32_t)g.S + (uint32_t)s;
    } else {
        const int n = tile * g.gpw + lane / g.S;
        const int s = lane % g.S;
        it.active = (lane < g.gpw * g.S) && (n < g.N);
        it.col = ((uint32_t)n * (uint32_t)g.C + (uint32_t)grp) * (uint32_t)g.S + (uint32_t)s;
    }
    return it;
}

__device__ __forceinline__ uint32_t voff(const Item& it, int es)
{
    return it.active ? it.col * (uint32_t)es : kOutOfRange;
}

// ---------------------------------------------------------------------------
// forward
// ---------------------------------------------------------------------------
template <int K, int DT, int MODE>
__global__ __launch_bounds__(kThreads) void fwd_kernel(FwdArgs a)
{
    using V = typename IO<DT>::V;
    const Geom& g = a.g;
    const int lane = threadIdx.x & 63;
    const int wave = uniform(threadIdx.x >> 6);
    const int grp = blockIdx.y;
    const int c = (MODE == kLaneChannel) ? min(grp * 64 + lane, g.C - 1) : grp;

    Taps<K, DT> tp;
    tp.load(a.sign, a.shift, c, g.shift_lo, g.shift_hi);
    V start;  // value the tap sum starts from
    V bias;
    if constexpr (DT == kQ88) {
        bias = ((const int32_t*)a.bias)[c];
        start = bias + tp.cneg;
    } else {
        bias = ((const float*)a.bias)[c];
        start = 0.0f;
    }
    const uint32_t xstep = g.M * (uint32_t)IO<DT>::es;
    const uint32_t hstep = g.M * 4u;

    for (int rep = 0; rep < g.R; ++rep) {
        const int64_t q = ((int64_t)blockIdx.x * kWaves + wave) * g.R + rep;
        if (q >= g.items)
            break;
        const Item it = decode_item<MODE>(g, q, grp, lane);
        if (it.j0 >= it.j1)
            continue;
        const uint32_t vx = voff(it, IO<DT>::es);
        const uint32_t v1 = voff(it, 1);
        const uint32_t v4 = voff(it, 4);
        const int r = it.r, d = g.d;

        auto xat = [&](int j) -> V {
            const int t = r + j * d;
            return IO<DT>::load(rsrc(a.x, (uint64_t)t * xstep, xstep), vx);
        };
        auto out = [&](int j, V h) {
            const int t = r + j * d;
            bool fire;
            if constexpr (DT == kQ88)
                fire = h >= g.v_th_q;
            else
                fire = h >= g.v_th;
            __builtin_amdgcn_raw_buffer_store_b8((uint8_t)(fire ? 1 : 0),
                                                 rsrc(a.spikes, (uint64_t)t * g.M, g.M), v1, 0, 0);
            if (a.h_out)
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, h),
                                                      rsrc(a.h_out, (uint64_t)t * hstep, hstep), v4,
                                                      0, 0);
        };

        V ring[K];
#pragma unroll
        for (int m = 0; m < K - 1; ++m) {
            const int j = it.j0 - (K - 1) + m;
            const V v = xat(max(j, 0));  // never address before the tensor
            ring[m] = j >= 0 ? v : V(0);
        }
        // one block = K class steps; its K loads are issued before any use
        // (indices clamped into the chunk) so their latencies overlap.
        auto block = [&](int jb, auto full_c) {
            constexpr bool full = decltype(full_c)::value;
            V xin[K];
#pragma unroll
            for (int u = 0; u < K; ++u)
                xin[u] = xat(min(jb + u, it.j1 - 1));
            [&]<int... U>(std::integer_sequence<int, U...>) {
                (([&] {
                     constexpr int u = U;
                     if (!full && jb + u >= it.j1)
                         return;
                     ring[(u + K - 1) % K] = xin[u];
                     V acc = start;
#pragma unroll
                     for (int i = 0; i < K; ++i)
                         acc = acc + tp.apply(ring[(u + i) % K], i);
                     V h;
                     if constexpr (DT == kQ88)
                         h = acc;
                     else
                         h = acc + bias;
                     out(jb + u, h);
                 }()),
                 ...);
            }(std::make_integer_sequence<int, K>{});
        };
        int j = it.j0;
        for (; j + K <= it.j1; j += K)
            block(j, std::true_type{});
        if (j < it.j1)
            block(j, std::false_type{});
    }
}

// ---------------------------------------------------------------------------
// backward
// ---------------------------------------------------------------------------
__device__ __forceinline__ double wave_sum(double v)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1)
        v += __shfl_xor(v, m, 64);
    return v;
}

template <int K, int DT, int MODE>
__global__ __launch_bounds__(kThreads) void bwd_kernel(BwdArgs a)
{
    using V = typename IO<DT>::V;
    using D = typename IO<DT>::D;
    const Geom& g = a.g;
    const int lane = threadIdx.x & 63;
    const int wave = uniform(threadIdx.x >> 6);
    const int grp = blockIdx.y;
    const int c_lane = (MODE == kLaneChannel) ? grp * 64 + lane : grp;
    const int c = min(c_lane, g.C - 1);

    Taps<K, DT> tp;
    tp.load(a.sign, a.shift, c, g.shift_lo, g.shift_hi);
    V start, bias;
    D dstart;
    if constexpr (DT == kQ88) {
        bias = ((const int32_t*)a.bias)[c];
        start = bias + tp.cneg;
        dstart = tp.cneg;
    } else {
        bias = ((const float*)a.bias)[c];
        start = 0.0f;
        dstart = 0.0f;
    }
    Surrogate sg;
    sg.kind = g.sg;
    sg.alpha = g.alpha;
    sg.c_atan = 0x1.921fb6p+0f * g.alpha;

    const uint32_t xstep = g.M * (uint32_t)IO<DT>::es;
    const uint32_t gxstep = g.M * (uint32_t)IO<DT>::gx_es;

    double gw[K];
#pragma unroll
    for (int i = 0; i < K; ++i)
        gw[i] = 0.0;
    double gb = 0.0;

    for (int rep = 0; rep < g.R; ++rep) {
        const int64_t q = ((int64_t)blockIdx.x * kWaves + wave) * g.R + rep;
        if (q >= g.items)
            break;
        const Item it = decode_item<MODE>(g, q, grp, lane);
        if (it.j0 >= it.j1)
            continue;
        const uint32_t vx = voff(it, IO<DT>::es);
        const uint32_t vgx = voff(it, IO<DT>::gx_es);
        const int r = it.r, d = g.d;
        const int j0 = it.j0, j1 = it.j1, Lr = it.Lr;

        auto at = [&](const void* base, int j) -> V {
            const int t = r + j * d;
            return IO<DT>::load(rsrc(base, (uint64_t)t * xstep, xstep), vx);
        };

        V xr[K];
        double xd[K];
        D dr[K];
#pragma unroll
        for (int m = 0; m < K - 1; ++m) {
            const int j = j0 - (K - 1) + m;
            const V v = at(a.x, max(j, 0));  // never address before the tensor
            xr[m] = j >= 0 ? v : V(0);
            xd[m] = (double)xr[m];
        }
        const int jend = j1 + K - 1;
        auto block = [&](int jb, auto full_c) {
            constexpr bool full = decltype(full_c)::value;
            V xin[K], gin[K];
#pragma unroll
            for (int u = 0; u < K; ++u) {
                const int jl = min(jb + u, Lr - 1);
                xin[u] = at(a.x, jl);
                gin[u] = at(a.gs, jl);
            }
            [&]<int... U>(std::integer_sequence<int, U...>) {
                (([&] {
                     constexpr int u = U;
                     constexpr int slot = (u + K - 1) % K;
                     const int j = jb + u;
                     if (!full && j >= jend)
                         return;
                     D dh = D(0);
                     if (full || j < Lr) {
                         xr[slot] = xin[u];
                         xd[slot] = (double)xin[u];
                         V acc = start;
#pragma unroll
                         for (int i = 0; i < K; ++i)
                             acc = acc + tp.apply(xr[(u + i) % K], i);
                         V h;
                         if constexpr (DT == kQ88)
                             h = acc;
                         else
                             h = acc + bias;
                         dh = delta_h(sg, gin[u], h, g.v_th, g.v_th_q);
                     } else {
                         xr[slot] = V(0);
                         xd[slot] = 0.0;
                     }
                     dr[slot] = dh;
                     if (full || j < j1) {
                         const double dd = (double)dh;
#pragma unroll
                         for (int i = 0; i < K; ++i)
                             gw[i] = __builtin_fma(xd[(u + i) % K], dd, gw[i]);
                         gb += dd;
                     }
                     if (full || j >= j0 + K - 1) {
                         D acc = dstart;
#pragma unroll
                         for (int i = 0; i < K; ++i)
                             acc = acc + tp.apply(dr[(u + K - 1 - i) % K], i);
                         const int t = r + (j - (K - 1)) * d;
                         IO<DT>::store_gx(rsrc(a.grad_x, (uint64_t)t * gxstep, gxstep), vgx, acc);
                     }
                 }()),
                 ...);
            }(std::make_integer_sequence<int, K>{});
        };
        // blocks strictly inside [j0 + K - 1, j1) need no per-step checks
        int j = j0;
        block(j, std::false_type{});
        j += K;
        for (; j + K <= j1; j += K)
            block(j, std::true_type{});
        for (; j < jend; j += K)
            block(j, std::false_type{});
    }

    // block reduction in a fixed order, then one partial row per block
    const int C = g.C;
    if constexpr (MODE == kLaneChannel) {
        __shared__ double red[K + 1][64];
        for (int w = 0; w < kWaves; ++w) {
            if (wave == w) {
#pragma unroll
                for (int i = 0; i < K; ++i)
                    red[i][lane] = (w == 0) ? gw[i] : red[i][lane] + gw[i];
                red[K][lane] = (w == 0) ? gb : red[K][lane] + gb;
            }
            __syncthreads();
        }
        for (int e = threadIdx.x; e < (K + 1) * 64; e += kThreads) {
            const int i = e >> 6, l = e & 63;
            const int cc = grp * 64 + l;
            if (cc < C)
                a.partial[((size_t)blockIdx.x * (K + 1) + i) * C + cc] = red[i][l];
        }
    } else {
        __shared__ double red[kWaves][K + 1];
#pragma unroll
        for (int i = 0; i < K; ++i) {
            const double v = wave_sum(gw[i]);
            if (lane == 0)
                red[wave][i] = v;
        }
        {
            const double v = wave_sum(gb);
            if (lane == 0)
                red[wave][K] = v;
        }
        __syncthreads();
        if (threadIdx.x < K + 1) {
            double s = red[0][threadIdx.x];
            for (int w = 1; w < kWaves; ++w)
                s += red[w][threadIdx.x];
            a.partial[((size_t)blockIdx.x * (K + 1) + threadIdx.x) * C + grp] = s;
        }
    }
}

// ---------------------------------------------------------------------------
// finalize: grad_w[c,i] = sum_b partial[b][i][c], grad_b[c] = sum_b partial[b][k][c]
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void fin_kernel(FinArgs a)
{
    const int e = blockIdx.x * 256 + threadIdx.x;
    const int kk = a.k + 1;
    if (e >= kk * a.C)
        return;
    const int i = e / a.C, c = e % a.C;
    double s = 0.0;
    for (int b = 0; b < a.blocks; ++b)
        s += a.partial[((size_t)b * kk + i) * a.C + c];
    if (a.dtype == kQ88) {
        const int64_t v = (int64_t)s;
        if (i < a.k)
            ((int64_t*)a.grad_w)[c * a.k + i] = v;
        else
            ((int64_t*)a.grad_b)[c] = v;
    } else {
        const float v = (float)s;
        if (i < a.k)
            ((float*)a.grad_w)[c * a.k + i] = v;
        else
            ((float*)a.grad_b)[c] = v;
    }
}

// ---------------------------------------------------------------------------
// quantizer Q(W) = sign(W) 2^round(log2|W|), exact rounding of the logarithm
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void quant_kernel(const float* w, int64_t count, int lo, int hi,
                                                    int8_t* sign, int8_t* shift)
{
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= count)
        return;
    const float v = w[e];
    const uint32_t bits = __builtin_bit_cast(uint32_t, v);
    const uint32_t mag = bits & 0x7FFFFFFFu;
    int s;
    if (mag == 0u || mag > 0x7F800000u) {          // zero or NaN
        s = hi;
    } else if (mag == 0x7F800000u) {               // infinity
        s = lo;
    } else {
        int m;            // floor(log2|v|)
        uint32_t frac;    // 23-bit fraction of |v| / 2^m
        const uint32_t E = mag >> 23;
        if (E != 0u) {
            m = (int)E - 127;
            frac = mag & 0x7FFFFFu;
        } else {          // subnormal: |v| = mag * 2^-149
            const int top = 31 - __builtin_clz(mag);
            m = top - 149;
            frac = (mag << (23 - top)) & 0x7FFFFFu;
        }
        // 1 + 0x3504F3 / 2^23 < sqrt(2) < 1 + 0x3504F4 / 2^23
        const int e2 = m + (frac >= 0x3504F4u ? 1 : 0);
        s = -e2;
        s = s < lo ? lo : (s > hi ? hi : s);
    }
    sign[e] = v < 0.0f ? (int8_t)-1 : (int8_t)1;
    shift[e] = (int8_t)s;
}

// ---------------------------------------------------------------------------
// launchers.  This file is compiled once per storage type and range of k
// (MFPSN_TU_DTYPE, MFPSN_TU_KLO..MFPSN_TU_KHI) so the instantiations build in
// parallel; the translation unit with MFPSN_TU_MISC also holds the finalize
// and quantize launchers.
// ---------------------------------------------------------------------------
}  // namespace

template <int K, int DT>
hipError_t fwd_k(const FwdArgs& a, hipStream_t st)
{
    dim3 grid(a.g.blocks, a.g.groups), block(kThreads);
    if (a.g.mode == kLaneChannel)
        hipLaunchKernelGGL((fwd_kernel<K, DT, kLaneChannel>), grid, block, 0, st, a);
    else
        hipLaunchKernelGGL((fwd_kernel<K, DT, kPlane>), grid, block, 0, st, a);
    return hipGetLastError();
}

template <int K, int DT>
hipError_t bwd_k(const BwdArgs& a, hipStream_t st)
{
    dim3 grid(a.g.blocks, a.g.groups), block(kThreads);
    if (a.g.mode == kLaneChannel)
        hipLaunchKernelGGL((bwd_kernel<K, DT, kLaneChannel>), grid, block, 0, st, a);
    else
        hipLaunchKernelGGL((bwd_kernel<K, DT, kPlane>), grid, block, 0, st, a);
    return hipGetLastError();
}

#ifdef MFPSN_TU_DTYPE
#define MFPSN_INST(K)                                                                      \
    template hipError_t fwd_k<K, MFPSN_TU_DTYPE>(const FwdArgs&, hipStream_t);           \
    template hipError_t bwd_k<K, MFPSN_TU_DTYPE>(const BwdArgs&, hipStream_t);
#define MFPSN_IN_TU(K) (MFPSN_TU_KLO <= (K) && (K) <= MFPSN_TU_KHI)
#if MFPSN_IN_TU(1)
MFPSN_INST(1)
#endif
#if MFPSN_IN_TU(2)
MFPSN_INST(2)
#endif
#if MFPSN_IN_TU(3)
MFPSN_INST(3)
#endif
#if MFPSN_IN_TU(4)
MFPSN_INST(4)
#endif
#if MFPSN_IN_TU(5)
MFPSN_INST(5)
#endif
#if MFPSN_IN_TU(6)
MFPSN_INST(6)
#endif
#if MFPSN_IN_TU(7)
MFPSN_INST(7)
#endif
#if MFPSN_IN_TU(8)
MFPSN_INST(8)
#endif
#if MFPSN_IN_TU(9)
MFPSN_INST(9)
#endif
#if MFPSN_IN_TU(10)
MFPSN_INST(10)
#endif
#if MFPSN_IN_TU(11)
MFPSN_INST(11)
#endif
#if MFPSN_IN_TU(12)
MFPSN_INST(12)
#endif
#if MFPSN_IN_TU(13)
MFPSN_INST(13)
#endif
#if MFPSN_IN_TU(14)
MFPSN_INST(14)
#endif
#if MFPSN_IN_TU(15)
MFPSN_INST(15)
#endif
#if MFPSN_IN_TU(16)
MFPSN_INST(16)
#endif
#if MFPSN_IN_TU(17)
MFPSN_INST(17)
#endif
#if MFPSN_IN_TU(18)
MFPSN_INST(18)
#endif
#if MFPSN_IN_TU(19)
MFPSN_INST(19)
#endif
#if MFPSN_IN_TU(20)
MFPSN_INST(20)
#endif
#if MFPSN_IN_TU(21)
MFPSN_INST(21)
#endif
#if MFPSN_IN_TU(22)
MFPSN_INST(22)
#endif
#if MFPSN_IN_TU(23)
MFPSN_INST(23)
#endif
#if MFPSN_IN_TU(24)
MFPSN_INST(24)
#endif
#if MFPSN_IN_TU(25)
MFPSN_INST(25)
#endif
#if MFPSN_IN_TU(26)
MFPSN_INST(26)
#endif
#if MFPSN_IN_TU(27)
MFPSN_INST(27)
#endif
#if MFPSN_IN_TU(28)
MFPSN_INST(28)
#endif
#if MFPSN_IN_TU(29)
MFPSN_INST(29)
#endif
#if MFPSN_IN_TU(30)
MFPSN_INST(30)
#endif
#if MFPSN_IN_TU(31)
MFPSN_INST(31)
#endif
#if MFPSN_IN_TU(32)
MFPSN_INST(32)
#endif
#endif  // MFPSN_TU_DTYPE

#ifdef MFPSN_TU_MISC
hipError_t launch_finalize(const FinArgs& a, hipStream_t st)
{
    const int n = (a.k + 1) * a.C;
    if (n == 0)
        return hipSuccess;
    hipLaunchKernelGGL(fin_kernel, dim3((n + 255) / 256), dim3(256), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_quantize(const float* w, int64_t count, int32_t lo, int32_t hi, int8_t* sign,
                           int8_t* shift, hipStream_t st)
{
    if (count == 0)
        return hipSuccess;
    hipLaunchKernelGGL(quant_kernel, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, st, w,
                       count, lo, hi, sign, shift);
    return hipGetLastError();
}
#endif  // MFPSN_TU_MISC

}  // namespace mfpsn
