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
// compile-time slots: the walk is unrolled by k.  The grid is persistent:
// as many blocks as fit on the GPU at once, each wave striding over items
// (column tile, residue class, chunk).
//
// Taps never multiply: a float tap moves the exponent, either with one
// integer add of ((-shift) << 23) ^ sign-bit to the bit pattern (normal
// inputs whose result stays normal) or with v_ldexp_f32 and a sign flip (any
// other input: zero, subnormal, infinite, NaN); a Q8.8 tap is an arithmetic
// right shift and an xor-add (the -1 that xor-negation leaves per negative
// tap is folded into the starting value).  Sums run in ascending tap order
// from +0 with the bias added last, so the float potentials are
// bit-identical to a sequential evaluation of the definition.
//
// The backward walks each class backwards in time: the dH ring then already
// holds the future values grad_x needs, so grad_x of step j is emitted at
// step j.  H comes from the forward's saved potentials when the caller
// passes them, else it is recomputed from the x ring.  grad_w / grad_b are
// accumulated from exact double products (Q8.8: exact integers in double),
// reduced inside the block in a fixed order and written as per-block
// partials; a finalize kernel adds the partials in block order, so the
// gradients are bitwise reproducible.
#include <hip/hip_runtime.h>
#include <hip/hip_bf16.h>
#include <stdint.h>

#include <utility>

#include "mfpsn_internal.h"


namespace mfpsn {
namespace {

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Loads run P class steps ahead of their use.  P divides k so that the
// prefetch slot of a step is a compile-time index inside the k-step unrolled
// block; orders with no divisor in [2, 8] fall back to one step ahead.
constexpr int prefetch_depth(int K, int cap = 8)
{
    if (K <= cap)
        return K;
    for (int p = cap; p >= 2; --p)
        if (K % p == 0)
            return p;
    return 1;
}

// ---------------------------------------------------------------------------
// storage types.  Every access is (row: uniform 64-bit address of one time
// step of a tensor, rbytes: that step's size) + (lane byte offset): a raw
// buffer access whose descriptor the scalar unit rebuilds from the row.
// ---------------------------------------------------------------------------
constexpr int kRsrcWord3 = 0x00020000;  // raw (untyped) buffer, gfx9 family

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_at(uint64_t row, uint32_t rbytes)
{
    return __builtin_amdgcn_make_buffer_rsrc((void*)row, (short)0, (int)rbytes, kRsrcWord3);
}

template <int DT> struct IO;

template <> struct IO<kF32> {
    using V = float;    // register value of x / grad_spikes
    using D = float;    // dH
    static constexpr int es = 4;
    static constexpr int gx_es = 4;
    __device__ static V load(uint64_t row, uint32_t rb, uint32_t off)
    {
        return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsrc_at(row, rb), off, 0, 0));
    }
    __device__ static void store_gx(uint64_t row, uint32_t rb, uint32_t off, D v)
    {
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), rsrc_at(row, rb), off, 0, 0);
    }
};

template <> struct IO<kBF16> {
    using V = float;
    using D = float;
    static constexpr int es = 2;
    static constexpr int gx_es = 2;
    __device__ static V load(uint64_t row, uint32_t rb, uint32_t off)
    {
        const uint32_t h = __builtin_amdgcn_raw_buffer_load_b16(rsrc_at(row, rb), off, 0, 0);
        return __builtin_bit_cast(float, h << 16);
    }
    __device__ static void store_gx(uint64_t row, uint32_t rb, uint32_t off, D v)
    {
        const __bf16 h = (__bf16)v;  // round to nearest even (v_cvt_pk_bf16_f32)
        __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, h), rsrc_at(row, rb), off, 0,
                                              0);
    }
};

template <> struct IO<kQ88> {
    using V = int32_t;
    using D = int32_t;
    static constexpr int es = 2;
    static constexpr int gx_es = 4;
    __device__ static V load(uint64_t row, uint32_t rb, uint32_t off)
    {
        const uint32_t h = __builtin_amdgcn_raw_buffer_load_b16(rsrc_at(row, rb), off, 0, 0);
        return (int32_t)(int16_t)(uint16_t)h;
    }
    __device__ static void store_gx(uint64_t row, uint32_t rb, uint32_t off, D v)
    {
        __builtin_amdgcn_raw_buffer_store_b32((uint32_t)v, rsrc_at(row, rb), off, 0, 0);
    }
};

// 32-bit words (H, saved or stored) and bytes (spikes)
__device__ __forceinline__ uint32_t load_w(uint64_t row, uint32_t rb, uint32_t off)
{
    return __builtin_amdgcn_raw_buffer_load_b32(rsrc_at(row, rb), off, 0, 0);
}
__device__ __forceinline__ void store_w(uint64_t row, uint32_t rb, uint32_t off, uint32_t v)
{
    __builtin_amdgcn_raw_buffer_store_b32(v, rsrc_at(row, rb), off, 0, 0);
}
__device__ __forceinline__ void store_b(uint64_t row, uint32_t rb, uint32_t off, uint8_t v)
{
    __builtin_amdgcn_raw_buffer_store_b8(v, rsrc_at(row, rb), off, 0, 0);
}

// H as saved by the forward: float for the float paths, int32 for Q8.8
template <int DT> using HVal = typename IO<DT>::V;

// ---------------------------------------------------------------------------
// taps: weight sign * 2^-shift
// ---------------------------------------------------------------------------
template <int K, int DT> struct Taps;

template <int K> struct TapsF {
    static constexpr bool kHasFast = true;
    // ((-shift) << 23) ^ (sign bit of a negative tap): the value added to a
    // float's bit pattern to scale it by sign * 2^-shift (shift in -126..126)
    uint32_t kc[K];
    __device__ void load(const int8_t* sign, const int8_t* shift, int c, int lo, int hi)
    {
#pragma unroll
        for (int i = 0; i < K; ++i) {
            int s = shift[c * K + i];
            s = s < lo ? lo : (s > hi ? hi : s);
            kc[i] = ((uint32_t)(-s) << 23) ^ (sign[c * K + i] < 0 ? 0x80000000u : 0u);
        }
    }
    // sign * 2^-shift * v for any float: exact exponent move (v_ldexp_f32),
    // then sign flip.  Bits 23..30 of kc are -shift (sign-extended); bit 31 of
    // ((-shift) << 23) alone is set exactly when shift > 0, so the tap's sign
    // bit is bit 31 of kc xor (shift > 0).
    __device__ __forceinline__ float apply(float v, int i) const
    {
        const int nsh = (int)(kc[i] << 1) >> 24;
        const uint32_t neg = (kc[i] ^ (nsh < 0 ? 0x80000000u : 0u)) & 0x80000000u;
        float y = ldexpf(v, nsh);
        return __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, y) ^ neg);
    }
    // The same value for a normal v whose result stays normal: adding kc to
    // the bit pattern subtracts the shift from the exponent field and flips
    // the sign bit.
    __device__ __forceinline__ float apply_fast(float v, int i) const
    {
        return __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, v) + kc[i]);
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
    static constexpr bool kHasFast = false;
    // (v >> s) ^ m equals +(v >> s) or -(v >> s) - 1; the -1s are cancelled by
    // starting the sum at cneg.
    __device__ __forceinline__ int apply(int v, int i) const { return (v >> sh[i]) ^ m[i]; }
    __device__ __forceinline__ int apply_fast(int v, int i) const { return apply(v, i); }
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

// True (wave-uniform) when some active lane's value is outside the range in
// which the exponent-add tap is exact (lane masks straight from v_cmp).
__device__ __forceinline__ bool any_slow(float v, const Geom& g, uint64_t act)
{
    const float m = __builtin_fabsf(v);
    const uint64_t ok = __builtin_amdgcn_fcmpf(m, g.fast_lo, 3 /* >= */) &
                        __builtin_amdgcn_fcmpf(m, g.fast_hi, 4 /* < */);
    return (act & ~ok) != 0;
}
__device__ __forceinline__ bool any_slow(int, const Geom&, uint64_t) { return false; }

// ---------------------------------------------------------------------------
// lane -> column.  Lane-channel tiles: 64 consecutive channels of one sample.
// Plane tiles: 64 consecutive positions p = n*S + s of one channel's (n, s)
// plane, so every lane is busy except in the plane's last tile.  A lane whose
// column does not exist reads and writes the column of the last existing
// lane of its wave: it computes that lane's values, so its stores duplicate
// that lane's in the same instruction.  Its grad_w / grad_b contribution is
// dropped: lane-channel lanes past C write no partial row; in a partial plane
// tile the backward zeroes the lane's dH before accumulating.
// ---------------------------------------------------------------------------
struct Item {
    int r;        // residue class
    int Lr;       // class length
    int j0, j1;   // class-step chunk
    bool active;  // this lane's column exists
    bool partial; // plane tile with missing columns (wave-uniform)
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
        it.partial = false;
        it.col = (uint32_t)tile * (uint32_t)g.C + (uint32_t)min(c, g.C - 1);
    } else {
        const uint32_t NS = (uint32_t)g.N * (uint32_t)g.S;
        const uint32_t pos = (uint32_t)tile * 64u + (uint32_t)lane;
        it.active = pos < NS;
        it.partial = (uint32_t)tile * 64u + 64u > NS;
        const uint32_t pc = min(pos, NS - 1u);
        const uint32_t n = pc / (uint32_t)g.S, s = pc % (uint32_t)g.S;
        it.col = (n * (uint32_t)g.C + (uint32_t)grp) * (uint32_t)g.S + s;
    }
    return it;
}

// addr += inc, kept opaque so the compiler updates one running SGPR pair per
// stream instead of precomputing (and spilling) an address per unrolled step
__device__ __forceinline__ void advance(uint64_t& addr, int64_t inc)
{
    addr += (uint64_t)inc;
    asm volatile("" : "+s"(addr));
}

// ---------------------------------------------------------------------------
// forward
// ---------------------------------------------------------------------------
template <int K, int DT, int MODE>
__global__ __launch_bounds__(kThreads) void fwd_kernel(FwdArgs a)
{
    using V = typename IO<DT>::V;
    using TP = Taps<K, DT>;
    constexpr int P = prefetch_depth(K);
    constexpr int es = IO<DT>::es;
    const Geom& g = a.g;
    const int lane = threadIdx.x & 63;
    const int wave = uniform(threadIdx.x >> 6);
    const int grp = blockIdx.y;
    const int c = (MODE == kLaneChannel) ? min(grp * 64 + lane, g.C - 1) : grp;

    TP tp;
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
    const int64_t xrow = (int64_t)g.M * es;  // bytes per time step
    const uint32_t xrb = (uint32_t)xrow, srb = g.M, hrb = g.M * 4u;
    const int want_h = a.h_out != nullptr ? 1 : 0;
    const int64_t stride = (int64_t)gridDim.x * kWaves;

    for (int64_t q = (int64_t)blockIdx.x * kWaves + wave; q < g.items; q += stride) {
        const Item it = decode_item<MODE>(g, q, grp, lane);
        if (it.j0 >= it.j1)
            continue;
        const uint32_t ox = it.col * es, o1 = it.col, o4 = it.col * 4u;
        const uint64_t act = __builtin_amdgcn_ballot_w64(it.active);
        const int r = it.r, d = g.d, j0 = it.j0, j1 = it.j1, Lr = it.Lr;

        const int64_t xcls = d * xrow, scls = (int64_t)d * g.M, hcls = (int64_t)d * g.M * 4;
        const uint64_t x0 = (uint64_t)a.x + (uint64_t)(r * xrow);
        auto xat = [&](int j) -> V { return IO<DT>::load(x0 + (uint64_t)(j * xcls), xrb, ox); };
        uint64_t xnext = x0 + (uint64_t)((j0 + P) * xcls);  // prefetch of step j + P
        uint64_t srow = (uint64_t)a.spikes + (uint64_t)(r * (int64_t)g.M + j0 * scls);
        uint64_t hrow = (uint64_t)a.h_out + (uint64_t)((r * (int64_t)g.M + j0 * scls) * 4);

        V ring[K];
        int slow = 0;  // steps left before every ring entry is in the fast range
#pragma unroll
        for (int m = 0; m < K - 1; ++m) {
            const int j = j0 - (K - 1) + m;
            const V v = xat(max(j, 0));  // never address before the tensor
            ring[m] = j >= 0 ? v : V(0);
            if (TP::kHasFast && any_slow(ring[m], g, act))
                slow = m + 1;
        }
        V pf[P];
#pragma unroll
        for (int p = 0; p < P; ++p)
            pf[p] = xat(min(j0 + p, Lr - 1));

        // one step: take the prefetched input into the ring, sum the taps,
        // fire, store; full blocks need no index checks and no clamping
        auto step = [&](auto uc, int j, auto full_c) __attribute__((always_inline)) {
            constexpr int u = decltype(uc)::value;
            constexpr bool full = decltype(full_c)::value;
            const V xv = pf[u % P];
            if constexpr (full)
                pf[u % P] = IO<DT>::load(xnext, xrb, ox);
            else
                pf[u % P] = xat(min(j + P, Lr - 1));
            advance(xnext, xcls);
            ring[(u + K - 1) % K] = xv;
            V acc = start;
            if constexpr (TP::kHasFast) {
                if (any_slow(xv, g, act))
                    slow = K;
                if (__builtin_expect(slow > 0, 0)) {
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        acc = acc + tp.apply(ring[(u + i) % K], i);
                    --slow;
                } else {
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        acc = acc + tp.apply_fast(ring[(u + i) % K], i);
                }
            } else {
#pragma unroll
                for (int i = 0; i < K; ++i)
                    acc = acc + tp.apply(ring[(u + i) % K], i);
            }
            V h;
            bool fire;
            if constexpr (DT == kQ88) {
                h = acc;
                fire = h >= g.v_th_q;
            } else {
                h = acc + bias;
                fire = h >= g.v_th;
            }
            store_b(srow, srb, o1, fire ? 1 : 0);
            if (want_h != 0)
                store_w(hrow, hrb, o4, __builtin_bit_cast(uint32_t, h));
            advance(srow, scls);
            advance(hrow, hcls);
        };
        auto block = [&](int jb, auto full_c) __attribute__((always_inline)) {
            constexpr bool full = decltype(full_c)::value;
            [&]<int... U>(std::integer_sequence<int, U...>) __attribute__((always_inline)) {
                (void)((full || jb + U < j1
                            ? (step(std::integral_constant<int, U>{}, jb + U, full_c), true)
                            : false) &&
                       ...);
            }(std::make_integer_sequence<int, K>{});
        };
        // orders above 16 keep a single (checked) copy of the block to bound
        // the code size
        int j = j0;
        if constexpr (K <= 16)
            for (; j + K <= j1 && j + K + P <= Lr; j += K)
                block(j, std::true_type{});
        for (; j < j1; j += K)
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

// Reverse walk over class steps j = jtop, jtop-1, ..., j0 (walk index
// s = jtop - j, slot u = s mod k).  Rings: x[t] for t in [j-k+1, j] at slot
// (jtop - t) mod k; dH[t] for t in [j, j+k-1] at slot (jtop - t) mod k, zero
// for t past the sequence.  Steps above j1 - 1 are the halo of a lower chunk:
// only their dH is computed.
template <int K, int DT, int MODE, bool HS>
__global__ __launch_bounds__(kThreads) void bwd_kernel(BwdArgs a)
{
    using V = typename IO<DT>::V;
    using D = typename IO<DT>::D;
    using TP = Taps<K, DT>;
    constexpr int P = prefetch_depth(K, 4);  // three streams: keep the queues short
    constexpr int es = IO<DT>::es;
    constexpr int gxs = IO<DT>::gx_es;
    constexpr bool kRecompute = !HS;
    // x stays a float ring; each grad_w product widens its x operand at use
    constexpr bool kWide = false;
    const Geom& g = a.g;
    const int lane = threadIdx.x & 63;
    const int wave = uniform(threadIdx.x >> 6);
    const int grp = blockIdx.y;
    const int c_lane = (MODE == kLaneChannel) ? grp * 64 + lane : grp;
    const int c = min(c_lane, g.C - 1);

    TP tp;
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

    const int64_t xrow = (int64_t)g.M * es, gxrow = (int64_t)g.M * gxs, hrow = (int64_t)g.M * 4;
    const uint32_t xrb = (uint32_t)xrow, gxrb = (uint32_t)gxrow, hrb = (uint32_t)hrow;
    const int64_t stride = (int64_t)gridDim.x * kWaves;

    double gw[K];
#pragma unroll
    for (int i = 0; i < K; ++i)
        gw[i] = 0.0;
    double gb = 0.0;

    for (int64_t q = (int64_t)blockIdx.x * kWaves + wave; q < g.items; q += stride) {
        const Item it = decode_item<MODE>(g, q, grp, lane);
        if (it.j0 >= it.j1)
            continue;
        const uint32_t ox = it.col * es, ogx = it.col * gxs, oh = it.col * 4u;
        const uint64_t act = __builtin_amdgcn_ballot_w64(it.active);
        const int r = it.r, d = g.d;
        const int j0 = it.j0, j1 = it.j1, Lr = it.Lr;
        const int jtop = min(j1 + K - 1, Lr) - 1;

        const int64_t xcls = d * xrow, gxcls = d * gxrow, hcls = d * hrow;
        const uint64_t x0 = (uint64_t)a.x + (uint64_t)(r * xrow);
        const uint64_t g0 = (uint64_t)a.gs + (uint64_t)(r * xrow);
        const uint64_t h0 = (uint64_t)a.h + (uint64_t)(r * hrow);
        auto xat = [&](int j) -> V { return IO<DT>::load(x0 + (uint64_t)(j * xcls), xrb, ox); };
        auto gat = [&](int j) -> V { return IO<DT>::load(g0 + (uint64_t)(j * xcls), xrb, ox); };
        auto hat = [&](int j) -> V {
            return __builtin_bit_cast(V, load_w(h0 + (uint64_t)(j * hcls), hrb, oh));
        };
        // running addresses: prefetch of walk index s + P (step j - P, its
        // x-ring entry j - P - k + 1) and the grad_x row of step j
        uint64_t gnext = g0 + (uint64_t)((jtop - P) * xcls);
        uint64_t hnext = h0 + (uint64_t)((jtop - P) * hcls);
        uint64_t xnext = x0 + (uint64_t)((jtop - P - K + 1) * xcls);
        uint64_t gxrow_j = (uint64_t)a.grad_x + (uint64_t)(r * gxrow + (int64_t)jtop * gxcls);

        V xr[K];
        double xd[kWide ? K : 1];
        D dr[K];
        int slow_x = 0;      // steps left on the exact recompute path
        int slow_d = K - 1;  // steps left on the exact grad_x path (the zero dH past the top)
#pragma unroll
        for (int i = 0; i < K; ++i)
            dr[i] = D(0);
#pragma unroll
        for (int m = 0; m < K - 1; ++m) {
            const int t = jtop - m;
            const V v0 = xat(max(t, 0));  // never address before the tensor
            const V v = t >= 0 ? v0 : V(0);
            xr[m] = v;
            if constexpr (kWide)
                xd[m] = (double)v;
            if (kRecompute && TP::kHasFast && any_slow(v, g, act))
                slow_x = m + 1;
        }
        V pfx[P], pfg[P], pfh[HS ? P : 1];
#pragma unroll
        for (int p = 0; p < P; ++p) {
            const int jp = max(jtop - p, 0);
            pfg[p] = gat(jp);
            if constexpr (HS)
                pfh[p] = hat(jp);
            pfx[p] = xat(max(jtop - p - K + 1, 0));
        }

        auto step = [&](auto uc, int j, auto full_c) __attribute__((always_inline)) {
            constexpr int u = decltype(uc)::value;
            constexpr bool full = decltype(full_c)::value;
            constexpr int xslot = (u + K - 1) % K;
            const V gv = pfg[u % P];
            V xv = pfx[u % P];
            V hv = V(0);
            if constexpr (HS)
                hv = pfh[u % P];
            if constexpr (full) {
                pfg[u % P] = IO<DT>::load(gnext, xrb, ox);
                if constexpr (HS)
                    pfh[u % P] = __builtin_bit_cast(V, load_w(hnext, hrb, oh));
                pfx[u % P] = IO<DT>::load(xnext, xrb, ox);
            } else {
                const int jn = max(j - P, 0);
                pfg[u % P] = gat(jn);
                if constexpr (HS)
                    pfh[u % P] = hat(jn);
                pfx[u % P] = xat(max(j - P - K + 1, 0));
                if (j - K + 1 < 0)  // x ring entry before the start of time
                    xv = V(0);
            }
            advance(gnext, -xcls);
            if constexpr (HS)
                advance(hnext, -hcls);
            advance(xnext, -xcls);
            xr[xslot] = xv;
            if constexpr (kWide)
                xd[xslot] = (double)xv;
            V h;
            if constexpr (kRecompute) {
                V acc = start;
                if constexpr (TP::kHasFast) {
                    if (any_slow(xv, g, act))
                        slow_x = K;
                    if (__builtin_expect(slow_x > 0, 0)) {
#pragma unroll
                        for (int i = 0; i < K; ++i)
                            acc = acc + tp.apply(xr[(u + K - 1 - i) % K], i);
                        --slow_x;
                    } else {
#pragma unroll
                        for (int i = 0; i < K; ++i)
                            acc = acc + tp.apply_fast(xr[(u + K - 1 - i) % K], i);
                    }
                } else {
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        acc = acc + tp.apply(xr[(u + K - 1 - i) % K], i);
                }
                if constexpr (DT == kQ88)
                    h = acc;
                else
                    h = acc + bias;
            } else {
                h = hv;
            }
            const D dh = delta_h(sg, gv, h, g.v_th, g.v_th_q);
            dr[u] = dh;
            if (TP::kHasFast && any_slow(dh, g, act))
                slow_d = K;
            if (full || j < j1) {
                double dd = (double)dh;
                if (!full && it.partial)
                    dd = it.active ? dd : 0.0;  // no contribution from shadow lanes
#pragma unroll
                for (int i = 0; i < K; ++i) {
                    double xi;
                    if constexpr (kWide)
                        xi = xd[(u + K - 1 - i) % K];
                    else
                        xi = (double)xr[(u + K - 1 - i) % K];
                    gw[i] = __builtin_fma(xi, dd, gw[i]);
                }
                gb += dd;
                D acc = dstart;
                if constexpr (TP::kHasFast) {
                    if (__builtin_expect(slow_d > 0, 0)) {
#pragma unroll
                        for (int i = 0; i < K; ++i)
                            acc = acc + tp.apply(dr[(u + 1 + i) % K], i);
                    } else {
#pragma unroll
                        for (int i = 0; i < K; ++i)
                            acc = acc + tp.apply_fast(dr[(u + 1 + i) % K], i);
                    }
                } else {
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        acc = acc + tp.apply(dr[(u + 1 + i) % K], i);
                }
                IO<DT>::store_gx(gxrow_j, gxrb, ogx, acc);
            }
            advance(gxrow_j, -gxcls);
            if (slow_d > 0)
                --slow_d;
            // keep the scheduler from hoisting later steps' loads above this
            // step (which would hold them in registers for a whole block)
            __builtin_amdgcn_sched_barrier(0);
        };
        auto block = [&](int jb, auto full_c) __attribute__((always_inline)) {
            constexpr bool full = decltype(full_c)::value;
            [&]<int... U>(std::integer_sequence<int, U...>) __attribute__((always_inline)) {
                (void)((full || jb - U >= j0
                            ? (step(std::integral_constant<int, U>{}, jb - U, full_c), true)
                            : false) &&
                       ...);
            }(std::make_integer_sequence<int, K>{});
        };
        // full blocks: every step owned (j < j1, j >= j0), x-ring entries and
        // prefetches at or after the start of time.  The first block holds the
        // halo (or the zero dH past the top); orders above 16 keep one
        // checked copy only.
        int jb = jtop;
        block(jb, std::false_type{});
        jb -= K;
        if constexpr (K <= 16)
            if (!it.partial)
                for (; jb - K + 1 >= j0 && jb < j1 && jb >= 2 * K - 2 + P; jb -= K)
                    block(jb, std::true_type{});
        for (; jb >= j0; jb -= K)
            block(jb, std::false_type{});
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
// One block of 16 waves per 64 outputs: wave w adds the partial rows of a
// fixed contiguous range of blocks, then wave 0 adds the 16 sums in order,
// so the result does not depend on scheduling.
constexpr int kFinWaves = 16;

__global__ __launch_bounds__(64 * kFinWaves) void fin_kernel(FinArgs a)
{
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int n_out = (a.k + 1) * a.C;
    const int e = blockIdx.x * 64 + lane;
    const bool ok = e < n_out;
    const int ec = ok ? e : n_out - 1;  // loads stay inside the workspace
    const int per = (a.blocks + kFinWaves - 1) / kFinWaves;
    const int b0 = min(w * per, a.blocks);
    const int b1 = min(b0 + per, a.blocks);
    double s = 0.0;
    int b = b0;
    for (; b + 8 <= b1; b += 8) {
        double v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            v[u] = a.partial[(size_t)(b + u) * n_out + ec];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            s += v[u];
    }
    for (; b < b1; ++b)
        s += a.partial[(size_t)b * n_out + ec];
    __shared__ double red[kFinWaves][64];
    red[w][lane] = s;
    __syncthreads();
    if (w != 0 || !ok)
        return;
    double t = red[0][lane];
    for (int q = 1; q < kFinWaves; ++q)
        t += red[q][lane];
    const int i = e / a.C, c = e % a.C;
    if (a.dtype == kQ88) {
        const int64_t v = (int64_t)t;
        if (i < a.k)
            ((int64_t*)a.grad_w)[c * a.k + i] = v;
        else
            ((int64_t*)a.grad_b)[c] = v;
    } else {
        const float v = (float)t;
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

// Blocks of `kern` that fit on the current device at once (cached per kernel
// and device).
template <typename Kern>
int resident_blocks(Kern kern, int (&cache)[16])
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0)
        dev = 0;
    const int slot = dev & 15;
    if (cache[slot] == 0) {
        int per_cu = 0, cus = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, kThreads, 0) != hipSuccess)
            per_cu = 1;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            cus = 1;
        cache[slot] = (per_cu > 0 ? per_cu : 1) * (cus > 0 ? cus : 1);
    }
    return cache[slot];
}

// Persistent grid: as many blocks per group as fit at once, at most one per
// kWaves items and never more than the planner's bound.
inline int persistent_blocks(const Geom& g, int resident)
{
    int64_t per_group = resident / g.groups;
    if (per_group < 1)
        per_group = 1;
    const int64_t need = (g.items + kWaves - 1) / kWaves;
    if (per_group > need)
        per_group = need;
    if (per_group > g.blocks)
        per_group = g.blocks;
    return (int)(per_group > 0 ? per_group : 1);
}

template <int K, int DT>
hipError_t fwd_k(FwdArgs& a, hipStream_t st)
{
    static int cache[2][16];
    const bool lc = a.g.mode == kLaneChannel;
    auto kern = lc ? fwd_kernel<K, DT, kLaneChannel> : fwd_kernel<K, DT, kPlane>;
    a.g.blocks = persistent_blocks(a.g, resident_blocks(kern, cache[lc ? 0 : 1]));
    hipLaunchKernelGGL(kern, dim3(a.g.blocks, a.g.groups), dim3(kThreads), 0, st, a);
    return hipGetLastError();
}

template <int K, int DT>
hipError_t bwd_k(BwdArgs& a, hipStream_t st)
{
    static int cache[4][16];
    const bool lc = a.g.mode == kLaneChannel;
    const bool hs = a.h != nullptr;
    auto kern = lc ? (hs ? bwd_kernel<K, DT, kLaneChannel, true> : bwd_kernel<K, DT, kLaneChannel, false>)
                   : (hs ? bwd_kernel<K, DT, kPlane, true> : bwd_kernel<K, DT, kPlane, false>);
    a.g.blocks = persistent_blocks(a.g, resident_blocks(kern, cache[(lc ? 0 : 2) + (hs ? 1 : 0)]));
    hipLaunchKernelGGL(kern, dim3(a.g.blocks, a.g.groups), dim3(kThreads), 0, st, a);
    return hipGetLastError();
}

#ifdef MFPSN_TU_DTYPE
#define MFPSN_INST(K)                                                                      \
    template hipError_t fwd_k<K, MFPSN_TU_DTYPE>(FwdArgs&, hipStream_t);                 \
    template hipError_t bwd_k<K, MFPSN_TU_DTYPE>(BwdArgs&, hipStream_t);
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
    hipLaunchKernelGGL(fin_kernel, dim3((n + 63) / 64), dim3(64 * kFinWaves), 0, st, a);
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
