// gfx950 kernels of the mul-free channel-wise Parallel Spiking Neuron
// (arXiv 2501.14490): forward charge + fire, fused surrogate-gradient
// backward, deterministic reduction of the weight/bias gradients, and the
// power-of-two weight quantizer.
//
// Work decomposition.  x is time-first, [T][N][C][S]; the M = N*C*S columns
// are independent time series.  A dilated order-k convolution only couples
// time steps of one residue class t = r (mod d), so each lane walks one
// column along one residue class (class step j <-> time r + j*d), or a run of
// consecutive chunks of it [j0, j1) (chunks start at multiples of k).  Each
// wave owns a contiguous range of these items whose length differs from the
// others' by at most one, so the persistent grid finishes together.  Register
// rings are indexed by the class step mod k, and the walks are unrolled in
// blocks of k steps, so every ring slot is a compile-time register.  Block
// variants: full (no bounds checks), checked (per-step uniform guards and
// clamped prefetches), the forward's block at the start of the sequence,
// where the taps that would read before time 0 are left out at compile time,
// and the backward's last block, which stops at the item's end.
//
// Memory: one raw buffer resource per tensor and item, a per-lane column
// offset, and a per-step running scalar offset (one SALU add per stream and
// step).  Loads run P class steps ahead of their use.
//
// Taps: a float tap's term is the input times w = sign * 2^-shift, the tap's
// exponent move, which is exact when the input is zero or far enough from the
// exponent limits; there fma(x, w, acc) is the definition's sum acc + term
// with its one rounding.  A wave holding an input outside that range (tiny,
// huge, infinite, NaN) rounds the product and then adds for the k steps the
// input reaches.  A Q8.8 tap is an arithmetic right shift and an xor-add (the
// -1 that xor-negation leaves per negative tap is folded into the starting
// value).  Sums run in ascending tap order (starting from +0 in the
// definition; the first term is taken as is, which can only differ in the
// sign of a zero, and a zero bias is added as +0), bias last, so the float
// potentials and input gradients are bit-identical to a sequential
// evaluation of the definition.
//
// The forward can also save the potentials H or the surrogate factor
// sigma'(H - v_th) (Q8.8: the integer factor L).  From saved H the backward
// skips the recompute of the charge; from the saved factor it also skips the
// surrogate, dH = grad_spikes * factor.  Either trades 8 bytes of traffic per
// element for arithmetic; which pass gets the surrogate decides which pass
// the arithmetic lands in.
//
// Backward.  Each class is walked backwards in time.  dH[j] is computed once
// (from the forward's saved factor, or from H recomputed out of the x ring) and
// scattered into the k open grad_x accumulators it feeds (outputs j-k+1..j);
// contributions reach every output in ascending tap order, so the sum order
// is the definition's.  Output j is complete after step j and is stored.
// Lanes whose dH has exact tap products (zero included: its terms change no
// bit of an accumulator that starts at +0) add them with fused multiply-adds;
// lanes whose dH lies outside that range round each product, then add, on
// their own lanes only.  grad_x therefore equals the sequential definition
// bit for bit.
// grad_w / grad_b are accumulated from exact products: double for float data
// (the x ring is kept in double), int64 for Q8.8; they are reduced inside the
// block in a fixed order and written as per-block partials, which a finalize
// kernel adds in block order, so the gradients are bitwise reproducible.
#include <hip/hip_runtime.h>
#include <hip/hip_bf16.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

#include "mfpsn_internal.h"
#include "mfpsn_surrogate.h"


namespace mfpsn {
namespace {

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ uint32_t uniform_u(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_readfirstlane((int)v);
}

// Prefetch distance: a divisor of k (so the prefetch slot of a step is a
// compile-time index inside a k-step block), at most `cap`.
constexpr int prefetch_depth(int K, int cap)
{
    if (K <= cap)
        return K;
    for (int p = cap; p >= 2; --p)
        if (K % p == 0)
            return p;
    return 1;
}

// Loads in flight per wave decide how close a pass gets to HBM bandwidth:
// the forward has one input stream, the backward three.
#ifndef MFPSN_FWD_PREFETCH
#define MFPSN_FWD_PREFETCH 8
#endif
#ifndef MFPSN_FWD_PREFETCH_F32_PAIR
#define MFPSN_FWD_PREFETCH_F32_PAIR 2
#endif
#ifndef MFPSN_FWD_PREFETCH_WIDE
#define MFPSN_FWD_PREFETCH_WIDE 4
#endif
#ifndef MFPSN_BWD_PREFETCH
#define MFPSN_BWD_PREFETCH 2
#endif
#ifndef MFPSN_BWD_PREFETCH_HIGH_K
#define MFPSN_BWD_PREFETCH_HIGH_K 8
#endif
#ifndef MFPSN_BWD_PAIR_BYTES
#define MFPSN_BWD_PAIR_BYTES 16
#endif
constexpr int kFwdPrefetch = MFPSN_FWD_PREFETCH;
constexpr int kFwdPrefetchF32Pair = MFPSN_FWD_PREFETCH_F32_PAIR;
constexpr int kFwdPrefetchWide = MFPSN_FWD_PREFETCH_WIDE;  // 16-byte accesses
constexpr int kBwdPrefetch = MFPSN_BWD_PREFETCH;
constexpr int kBwdPrefetchHighK = MFPSN_BWD_PREFETCH_HIGH_K;  // orders 24 and up
constexpr int kBwdPairBytes = MFPSN_BWD_PAIR_BYTES;  // plane mode, two columns per lane

// What the scheduler may move across the end of a step (the mask of
// __builtin_amdgcn_sched_barrier): 0 keeps every instruction in its step, so
// no later step's loads are hoisted and held in registers for a whole block.
#ifndef MFPSN_FWD_STEP_BARRIER
#define MFPSN_FWD_STEP_BARRIER 0
#endif
#ifndef MFPSN_BWD_STEP_BARRIER
#define MFPSN_BWD_STEP_BARRIER 0
#endif

// Highest order built with unguarded full blocks (higher orders walk only
// guarded blocks: smaller code, a few scalar instructions more per step).
#ifndef MFPSN_FULL_BLOCK_MAX_K
#define MFPSN_FULL_BLOCK_MAX_K 16
#endif
constexpr int kFullBlockMaxK = MFPSN_FULL_BLOCK_MAX_K;

template <int V> using ic = std::integral_constant<int, V>;
// Block kinds (flags): kFull runs every step unguarded; kChecked clamps its
// prefetches (the backward's also selects what reaches before time 0; the
// forward's also stops at the item's end); kEdge is the forward's first
// block, whose taps before time 0 are left out; kLast is the backward's
// final block, the only one of its walk that stops at the item's end, run
// outside every loop (a block loop that could stop mid-block carries the
// registers of prefetches issued but never used, and reconciles them with
// moves that each wait for the pending load).
enum BlockKind : int { kFull = 0, kChecked = 1, kEdge = 2 | 1, kLast = 4 | 1 };

// ---------------------------------------------------------------------------
// buffers: raw buffer resource over [tensor + off, tensor end), per-lane
// voffset, uniform soffset.  Every access the kernels issue lies inside the
// tensor by construction (prefetches are clamped in checked blocks).
// ---------------------------------------------------------------------------
constexpr int kRsrcWord3 = 0x00020000;  // raw (untyped) buffer, gfx9 family

struct Buf {
    __amdgpu_buffer_rsrc_t rs;
};

__device__ __forceinline__ Buf make_buf(const void* tensor, uint64_t tensor_bytes, uint64_t off)
{
    const uint64_t rem = off < tensor_bytes ? tensor_bytes - off : 0;
    uint32_t n = rem > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)rem;
    // opaque, so descriptors of equal-sized tensors do not share (and then
    // copy every step) their size and flag words
    asm volatile("" : "+s"(n));
    Buf b;
    b.rs = __builtin_amdgcn_make_buffer_rsrc((void*)((const char*)tensor + off), (short)0, (int)n, kRsrcWord3);
    return b;
}

// Cache-policy bits of the streaming accesses (every element is read or
// written once per pass).
#ifndef MFPSN_LD_CPOL
#define MFPSN_LD_CPOL 0
#endif
#ifndef MFPSN_ST_CPOL
#define MFPSN_ST_CPOL 2  // nt: streaming stores
#endif
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32x4 ld128(Buf b, uint32_t v, int32_t s)
{
    return __builtin_amdgcn_raw_buffer_load_b128(b.rs, v, s, MFPSN_LD_CPOL);
}
__device__ __forceinline__ u32x2 ld64(Buf b, uint32_t v, int32_t s)
{
    return __builtin_amdgcn_raw_buffer_load_b64(b.rs, v, s, MFPSN_LD_CPOL);
}
__device__ __forceinline__ uint32_t ld32(Buf b, uint32_t v, int32_t s)
{
    return __builtin_amdgcn_raw_buffer_load_b32(b.rs, v, s, MFPSN_LD_CPOL);
}
__device__ __forceinline__ uint16_t ld16(Buf b, uint32_t v, int32_t s)
{
    return __builtin_amdgcn_raw_buffer_load_b16(b.rs, v, s, MFPSN_LD_CPOL);
}
__device__ __forceinline__ void st128(Buf b, uint32_t v, int32_t s, u32x4 x)
{
    __builtin_amdgcn_raw_buffer_store_b128(x, b.rs, v, s, MFPSN_ST_CPOL);
}
__device__ __forceinline__ void st64(Buf b, uint32_t v, int32_t s, u32x2 x)
{
    __builtin_amdgcn_raw_buffer_store_b64(x, b.rs, v, s, MFPSN_ST_CPOL);
}
__device__ __forceinline__ void st32(Buf b, uint32_t v, int32_t s, uint32_t x)
{
    __builtin_amdgcn_raw_buffer_store_b32(x, b.rs, v, s, MFPSN_ST_CPOL);
}
__device__ __forceinline__ void st16(Buf b, uint32_t v, int32_t s, uint16_t x)
{
    __builtin_amdgcn_raw_buffer_store_b16(x, b.rs, v, s, MFPSN_ST_CPOL);
}
__device__ __forceinline__ void st8(Buf b, uint32_t v, int32_t s, uint8_t x)
{
    __builtin_amdgcn_raw_buffer_store_b8(x, b.rs, v, s, MFPSN_ST_CPOL);
}

// The NV adjacent columns a lane holds (NV = 1, 2, 4 or 8, neighbours in
// memory): every stream moves them with one access (two for eight 32-bit
// words), so a wave's access covers 64 * NV elements.
template <typename T, int NV> struct Pk {
    T v[NV];
};
// NV adjacent 32-bit words (potentials, surrogate factors, Q8.8 grad_x)
template <int NV>
__device__ __forceinline__ Pk<uint32_t, NV> ld_words(Buf b, uint32_t v, int32_t s)
{
    Pk<uint32_t, NV> r;
    if constexpr (NV == 1) {
        r.v[0] = ld32(b, v, s);
    } else if constexpr (NV == 2) {
        const u32x2 w = ld64(b, v, s);
        r.v[0] = w.x;
        r.v[1] = w.y;
    } else {
#pragma unroll
        for (int q = 0; q < NV / 4; ++q) {
            const u32x4 w = ld128(b, v + 16u * q, s);
            r.v[4 * q] = w.x;
            r.v[4 * q + 1] = w.y;
            r.v[4 * q + 2] = w.z;
            r.v[4 * q + 3] = w.w;
        }
    }
    return r;
}
template <int NV>
__device__ __forceinline__ void st_words(Buf b, uint32_t v, int32_t s, const Pk<uint32_t, NV>& x)
{
    if constexpr (NV == 1) {
        st32(b, v, s, x.v[0]);
    } else if constexpr (NV == 2) {
        u32x2 w;
        w.x = x.v[0];
        w.y = x.v[1];
        st64(b, v, s, w);
    } else {
#pragma unroll
        for (int q = 0; q < NV / 4; ++q) {
            u32x4 w;
            w.x = x.v[4 * q];
            w.y = x.v[4 * q + 1];
            w.z = x.v[4 * q + 2];
            w.w = x.v[4 * q + 3];
            st128(b, v + 16u * q, s, w);
        }
    }
}
// NV adjacent bytes, byte e in bits 8(e mod 4).. of word e / 4
template <int NV>
__device__ __forceinline__ void st_bytes(Buf b, uint32_t v, int32_t s, const uint32_t (&x)[(NV + 3) / 4])
{
    if constexpr (NV == 1) {
        st8(b, v, s, (uint8_t)x[0]);
    } else if constexpr (NV == 2) {
        st16(b, v, s, (uint16_t)x[0]);
    } else if constexpr (NV == 4) {
        st32(b, v, s, x[0]);
    } else {
        u32x2 w;
        w.x = x[0];
        w.y = x[1];
        st64(b, v, s, w);
    }
}
// 16-bit values packed two to a 32-bit word (bf16, Q8.8): NV values in
// (NV + 1) / 2 words.  A single value stays a 16-bit one until it is used:
// widening it where it is loaded would wait for the load there.
template <int NV> using Halves = Pk<std::conditional_t<NV == 1, uint16_t, uint32_t>, (NV + 1) / 2>;
template <int NV>
__device__ __forceinline__ Halves<NV> ld_halves(Buf b, uint32_t v, int32_t s)
{
    Halves<NV> r;
    if constexpr (NV == 1) {
        r.v[0] = ld16(b, v, s);
    } else if constexpr (NV == 2) {
        r.v[0] = ld32(b, v, s);
    } else if constexpr (NV == 4) {
        const u32x2 w = ld64(b, v, s);
        r.v[0] = w.x;
        r.v[1] = w.y;
    } else {
        const u32x4 w = ld128(b, v, s);
        r.v[0] = w.x;
        r.v[1] = w.y;
        r.v[2] = w.z;
        r.v[3] = w.w;
    }
    return r;
}
template <int NV>
__device__ __forceinline__ void st_halves(Buf b, uint32_t v, int32_t s, const Pk<uint32_t, (NV + 1) / 2>& x)
{
    if constexpr (NV == 1) {
        st16(b, v, s, (uint16_t)x.v[0]);
    } else if constexpr (NV == 2) {
        st32(b, v, s, x.v[0]);
    } else if constexpr (NV == 4) {
        u32x2 w;
        w.x = x.v[0];
        w.y = x.v[1];
        st64(b, v, s, w);
    } else {
        u32x4 w;
        w.x = x.v[0];
        w.y = x.v[1];
        w.z = x.v[2];
        w.w = x.v[3];
        st128(b, v, s, w);
    }
}

// s += inc, kept opaque so the compiler keeps one running SGPR per stream
// instead of precomputing (and spilling) an offset per unrolled step
__device__ __forceinline__ void advance(int32_t& s, int32_t inc)
{
    s += inc;
    asm volatile("" : "+s"(s));
}

// Makes v opaque at this point: the code that produces it cannot be sunk
// past here (the compiler would otherwise defer the grad_w updates of a whole
// unrolled block to its end and keep every step's operands live).
template <typename T>
__device__ __forceinline__ void pin(T& v)
{
    asm volatile("" : "+v"(v));
}

// ---------------------------------------------------------------------------
// storage types
// ---------------------------------------------------------------------------
template <int DT> struct IO;

template <> struct IO<kF32> {
    using V = float;     // value of x / grad_spikes / H / dH in registers
    using W = double;    // exact product accumulator of grad_w, grad_b
    static constexpr int es = 4;     // bytes per stored x / grad_spikes
    static constexpr int gx_es = 4;  // bytes per stored grad_x
    template <int NV> using Raw = Pk<uint32_t, NV>;
    template <int NV>
    __device__ static Raw<NV> load_raw(Buf b, uint32_t v, int32_t s)
    {
        return ld_words<NV>(b, v, s);
    }
    template <int NV>
    __device__ static Pk<V, NV> cvt(const Raw<NV>& w)
    {
        Pk<V, NV> r;
#pragma unroll
        for (int e = 0; e < NV; ++e)
            r.v[e] = __builtin_bit_cast(float, w.v[e]);
        return r;
    }
    template <int NV>
    __device__ static Pk<V, NV> load(Buf b, uint32_t v, int32_t s)
    {
        return cvt<NV>(load_raw<NV>(b, v, s));
    }
    template <int NV>
    __device__ static void store_gx(Buf b, uint32_t v, int32_t s, const Pk<V, NV>& x)
    {
        Pk<uint32_t, NV> w;
#pragma unroll
        for (int e = 0; e < NV; ++e)
            w.v[e] = __builtin_bit_cast(uint32_t, x.v[e]);
        st_words<NV>(b, v, s, w);
    }
};

template <> struct IO<kBF16> {
    using V = float;
    using W = double;
    static constexpr int es = 2;
    static constexpr int gx_es = 2;
    // NV stored values packed two to a 32-bit word, widened only where they
    // are used
    template <int NV> using Raw = Halves<NV>;
    template <int NV>
    __device__ static Raw<NV> load_raw(Buf b, uint32_t v, int32_t s)
    {
        return ld_halves<NV>(b, v, s);
    }
    template <int NV>
    __device__ static Pk<V, NV> cvt(const Raw<NV>& w)
    {
        Pk<V, NV> r;
#pragma unroll
        for (int e = 0; e < NV; ++e)
            r.v[e] = __builtin_bit_cast(float, e % 2 == 0 ? (uint32_t)w.v[e / 2] << 16
                                                          : (uint32_t)w.v[e / 2] & 0xFFFF0000u);
        return r;
    }
    template <int NV>
    __device__ static Pk<V, NV> load(Buf b, uint32_t v, int32_t s)
    {
        return cvt<NV>(load_raw<NV>(b, v, s));
    }
    template <int NV>
    __device__ static void store_gx(Buf b, uint32_t v, int32_t s, const Pk<V, NV>& x)
    {
        // round to nearest even
        Pk<uint32_t, (NV + 1) / 2> w;
#pragma unroll
        for (int q = 0; q < (NV + 1) / 2; ++q) {
            const uint32_t h0 = __builtin_bit_cast(uint16_t, (__bf16)x.v[2 * q]);
            w.v[q] = h0;
            if (2 * q + 1 < NV)
                w.v[q] |= (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)x.v[2 * q + 1]) << 16;
        }
        st_halves<NV>(b, v, s, w);
    }
};

template <> struct IO<kQ88> {
    using V = int32_t;
    using W = int64_t;
    static constexpr int es = 2;
    static constexpr int gx_es = 4;
    template <int NV> using Raw = Halves<NV>;
    template <int NV>
    __device__ static Raw<NV> load_raw(Buf b, uint32_t v, int32_t s)
    {
        return ld_halves<NV>(b, v, s);
    }
    template <int NV>
    __device__ static Pk<V, NV> cvt(const Raw<NV>& w)
    {
        Pk<V, NV> r;
#pragma unroll
        for (int e = 0; e < NV; ++e)
            r.v[e] = e % 2 == 0 ? (int32_t)(int16_t)w.v[e / 2] : (int32_t)(uint32_t)w.v[e / 2] >> 16;
        return r;
    }
    template <int NV>
    __device__ static Pk<V, NV> load(Buf b, uint32_t v, int32_t s)
    {
        return cvt<NV>(load_raw<NV>(b, v, s));
    }
    template <int NV>
    __device__ static void store_gx(Buf b, uint32_t v, int32_t s, const Pk<V, NV>& x)
    {
        Pk<uint32_t, NV> w;
#pragma unroll
        for (int e = 0; e < NV; ++e)
            w.v[e] = (uint32_t)x.v[e];
        st_words<NV>(b, v, s, w);
    }
};

// ---------------------------------------------------------------------------
// taps: weight sign * 2^-shift.  Lane-channel mode holds one channel per lane
// (VGPRs); plane mode shares one channel across the block (SGPRs).
// ---------------------------------------------------------------------------
template <int K, int DT, int MODE> struct Taps;

template <int K, int MODE> struct TapsF {
    static constexpr bool kHasFast = true;
    // w[i] = sign_i * 2^-shift_i (shift in -126..126: a normal float).  The
    // product v * w[i] is the exponent move of the tap: exact when v is zero
    // or normal with a normal result, otherwise rounded once, as the move
    // itself (ldexp) rounds.
    float w[K];
    __device__ void load(const int8_t* sign, const int8_t* shift, int c, int lo, int hi)
    {
#pragma unroll
        for (int i = 0; i < K; ++i) {
            int s = shift[c * K + i];
            s = s < lo ? lo : (s > hi ? hi : s);
            uint32_t v = ((uint32_t)(127 - s) << 23) | (sign[c * K + i] < 0 ? 0x80000000u : 0u);
            w[i] = __builtin_bit_cast(float, MODE == kPlane ? uniform_u(v) : v);
        }
    }
    // the tap's term sign * 2^-shift * v, for any float v
    __device__ __forceinline__ float apply(float v, int i) const { return v * w[i]; }
    // acc + the tap's term in one rounding: the sum acc + apply(v, i) itself
    // whenever the term is exact (v zero or in the range where it is)
    __device__ __forceinline__ float fma(float v, int i, float acc) const { return __builtin_fmaf(v, w[i], acc); }
};
template <int K, int MODE> struct Taps<K, kF32, MODE> : TapsF<K, MODE> {};
template <int K, int MODE> struct Taps<K, kBF16, MODE> : TapsF<K, MODE> {};

template <int K, int MODE> struct Taps<K, kQ88, MODE> {
    static constexpr bool kHasFast = false;
    int sh[K];         // shift, 0..31
    int m[K];          // 0 (positive tap) or -1 (negative tap)
    int cneg;          // number of negative taps
    uint32_t negmask;  // bit i set for a negative tap i
    __device__ void load(const int8_t* sign, const int8_t* shift, int c, int lo, int hi)
    {
        cneg = 0;
        negmask = 0;
#pragma unroll
        for (int i = 0; i < K; ++i) {
            int s = shift[c * K + i];
            s = s < lo ? lo : (s > hi ? hi : s);
            const bool neg = sign[c * K + i] < 0;
            sh[i] = MODE == kPlane ? uniform(s) : s;
            m[i] = MODE == kPlane ? uniform(neg ? -1 : 0) : (neg ? -1 : 0);
            cneg += neg ? 1 : 0;
            negmask |= neg ? (1u << i) : 0u;
        }
    }
    // (v >> s) ^ m equals +(v >> s) or -(v >> s) - 1; the -1s are cancelled by
    // starting the sum at the number of negative taps it contains.
    __device__ __forceinline__ int apply(int v, int i) const { return (v >> sh[i]) ^ m[i]; }
};

// Q8.8 factors come from a table: u = H - v_th_q is an integer and L(u) is
// even in u (the float sequence sees |u|, or u only through u*u), so each
// block evaluates L(0 .. kQTable-1) once into LDS with the same sequence and
// looks factors up; |u| beyond the table takes the sequence directly.
constexpr int kQTable = 4096;

struct QTable {
    int32_t* tab;
    __device__ void fill(const Surrogate& sg) const
    {
        for (int j = threadIdx.x; j < kQTable; j += kThreads)
            tab[j] = sg_factor_q(sg, j);
    }
    __device__ __forceinline__ int32_t operator()(const Surrogate& sg, int32_t h, int v_th_q) const
    {
        const int32_t u = (int32_t)((uint32_t)h - (uint32_t)v_th_q);
        const uint32_t au = u < 0 ? 0u - (uint32_t)u : (uint32_t)u;
        int32_t L = tab[min(au, (uint32_t)(kQTable - 1))];
        if (__builtin_expect(au >= (uint32_t)kQTable, 0))
            L = sg_factor_q(sg, u);
        return L;
    }
};
// The taps of v are exact products (summed with one fused rounding each):
// v is zero, or normal far enough from the exponent limits.  (Bitwise
// operators: the short-circuit ones become a branch on the exec mask per
// operand.)
__device__ __forceinline__ bool tap_exact(float v, const Geom& g)
{
    const float m = __builtin_fabsf(v);
    return ((m >= g.fast_lo) & (m < g.fast_hi)) | (m == 0.0f);
}
// True (this lane) when one of its values has an inexact tap product.
template <int NV>
__device__ __forceinline__ bool lane_slow(const Pk<float, NV>& v, const Geom& g)
{
    bool out = false;
#pragma unroll
    for (int e = 0; e < NV; ++e)
        out = out | !tap_exact(v.v[e], g);
    return out;
}
template <int NV>
__device__ __forceinline__ bool lane_slow(const Pk<int32_t, NV>&, const Geom&)
{
    return false;
}
// True (wave-uniform) when some lane's value has an inexact tap product.
template <int NV>
__device__ __forceinline__ bool any_slow(const Pk<float, NV>& v, const Geom& g)
{
    return __builtin_amdgcn_ballot_w64(lane_slow(v, g)) != 0;
}
template <int NV>
__device__ __forceinline__ bool any_slow(const Pk<int32_t, NV>&, const Geom&)
{
    return false;
}
// The same for stored inputs, which are not checked where the storage type
// and shift range make every tap product exact.
template <typename PV>
__device__ __forceinline__ bool x_slow(const PV& v, const Geom& g)
{
    return !g.x_exact && any_slow(v, g);
}

// Q8.8 charge of one column: start + sum_i ((x_i >> s_i) ^ m_i), an exact
// integer sum, so it may be split into kQ88Sums independent partial sums
// (taps i, i + kQ88Sums, ...) that the hardware can issue interleaved; each
// partial sum is pinned, so it stays one shift and one xor-add per tap.
#ifndef MFPSN_Q88_SUMS
#define MFPSN_Q88_SUMS 1
#endif
constexpr int kQ88Sums = MFPSN_Q88_SUMS;
template <int K, typename TP, typename X>
__device__ __forceinline__ int32_t q88_charge(const TP& tp, int32_t start, X x)
{
    constexpr int NS = kQ88Sums < K ? kQ88Sums : K;
    int32_t part[NS];
#pragma unroll
    for (int p = 0; p < NS; ++p)
        part[p] = p == 0 ? start : 0;
#pragma unroll
    for (int i = 0; i < K; ++i) {
        part[i % NS] = part[i % NS] + tp.apply(x(i), i);
        pin(part[i % NS]);
    }
    int32_t acc = part[0];
#pragma unroll
    for (int p = 1; p < NS; ++p)
        acc += part[p];
    return acc;
}

// ---------------------------------------------------------------------------
// items.  Item q of a group: q = (tile * ncls + r) * nchunks + chunk, over
// the ncls = min(d, T) residue classes that hold a step.
// Lane -> column.  Lane-channel tiles: 64 consecutive channels of one sample.
// Plane tiles: 64 consecutive positions p = n*S + s of one channel's (n, s)
// plane.  A lane whose column does not exist reads and writes the column of
// the last existing lane of its wave: it computes that lane's values, so its
// stores duplicate that lane's.  Its grad_w / grad_b contribution is dropped.
// ---------------------------------------------------------------------------
// (every member is force-inlined: an out-of-line call puts the cursor on the
// stack, and the item loop then waits for every pending load to read it)
struct Cursor {
    int tile, r, chunk;
    __device__ __forceinline__ Cursor(const Geom& g, int64_t q) { set(g, q); }
    __device__ __forceinline__ void set(const Geom& g, int64_t q)
    {
        const uint32_t u = (uint32_t)q;  // items per group < 2^31 (planner)
        const uint32_t rc = u / (uint32_t)g.nchunks;
        chunk = (int)(u - rc * (uint32_t)g.nchunks);
        const uint32_t t = rc / (uint32_t)g.ncls;
        r = (int)(rc - t * (uint32_t)g.ncls);
        tile = (int)t;
    }
    __device__ __forceinline__ void next(const Geom& g)
    {
        if (++chunk == g.nchunks) {
            chunk = 0;
            if (++r == g.ncls) {
                r = 0;
                ++tile;
            }
        }
    }
    // to item q of a walk with item step `step` (1: the next item)
    __device__ __forceinline__ void advance(const Geom& g, int64_t q, int64_t step)
    {
        if (step == 1)
            next(g);
        else
            set(g, q);
    }
};

// The items of a wave: a contiguous range [q0, q1) (strided = 0), or every
// nw-th item from its wave index (strided = 1), so that the waves running
// at the same time walk neighbouring tiles and their accesses at each step
// fall into a few contiguous stretches of memory instead of being spread over
// the whole tensor.  Either way the waves' item counts differ by at most one.
struct ItemRange {
    int64_t q0, q1, step;
    __device__ __forceinline__ ItemRange(const Geom& g, int wid, int nw)
    {
        if (g.strided) {
            q0 = wid;
            q1 = g.items;
            step = nw;
        } else {
            q0 = g.items * wid / nw;
            q1 = g.items * (wid + 1) / nw;
            step = 1;
        }
    }
};

struct Cols {
    uint32_t col;  // the lane's first column, in [0, M)
    bool active;   // this lane's columns exist
    bool partial;  // plane tile with missing columns (wave-uniform)
};

template <int MODE, int NV>
__device__ __forceinline__ Cols tile_cols(const Geom& g, int tile, int grp, int lane)
{
    Cols t;
    if (MODE == kFlat) {
        // columns 64*NV*tile + NV*lane .. + NV-1 of the flattened row (M is a
        // multiple of NV)
        const uint32_t pos = (uint32_t)tile * (64u * NV) + (uint32_t)lane * NV;
        t.active = pos < g.M;
        t.partial = (uint64_t)tile * (64u * NV) + 64u * NV > g.M;
        t.col = min(pos, g.M - NV);
    } else if (MODE == kLaneChannel) {
        const int c = grp * 64 + lane;
        t.active = c < g.C;
        t.partial = false;
        t.col = (uint32_t)tile * (uint32_t)g.C + (uint32_t)min(c, g.C - 1);
    } else if (g.row_tiles > 0) {
        // tiles of one (n, c) row, starting on 128-byte lines: tile m covers
        // positions s0 .. s0 + 64*NV - 1 with s0 = m*64*NV - (elements of the
        // row's first line that precede it); lanes outside [0, S) are shadows
        const uint32_t S = (uint32_t)g.S;
        const uint32_t n = (uint32_t)tile / (uint32_t)g.row_tiles;
        const uint32_t m = (uint32_t)tile - n * (uint32_t)g.row_tiles;
        const uint32_t row = n * (uint32_t)g.C + (uint32_t)grp;
        const int lead = (int)((row * S) & (uint32_t)(g.line_elems - 1));
        const int s0 = (int)(m * (64u * NV)) - lead;
        const int sl = s0 + lane * NV;
        t.active = sl >= 0 && sl < (int)S;
        t.partial = s0 < 0 || s0 + 64 * NV > (int)S;
        t.col = row * S + (uint32_t)min(max(sl, 0), (int)S - NV);
    } else {
        // positions NV*lane .. NV*lane + NV-1 of the tile; with NV = 2, S is
        // even, so both lie in one (n, c) row of S adjacent columns
        const uint32_t NS = (uint32_t)g.N * (uint32_t)g.S;
        const uint32_t pos = (uint32_t)tile * (64u * NV) + (uint32_t)lane * NV;
        t.active = pos < NS;
        t.partial = (uint32_t)tile * (64u * NV) + 64u * NV > NS;
        const uint32_t pc = min(pos, NS - NV);
        const uint32_t n = pc / (uint32_t)g.S, s = pc - n * (uint32_t)g.S;
        t.col = (n * (uint32_t)g.C + (uint32_t)grp) * (uint32_t)g.S + s;
    }
    return t;
}

// steps of residue class r: T = tq*d + tr, so classes below tr hold one more
__device__ __forceinline__ int class_len(const Geom& g, int r) { return g.tq + (r < g.tr ? 1 : 0); }

// ---------------------------------------------------------------------------
// forward
// ---------------------------------------------------------------------------
template <int K, int DT, int MODE, int NV>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4))) void fwd_kernel(FwdArgs a)
{
    using V = typename IO<DT>::V;
    using PV = Pk<V, NV>;
    using TP = Taps<K, DT, MODE>;
    constexpr int es = IO<DT>::es;
    // 8 steps of x in flight, 2 for lanes holding two f32 columns (8 bytes
    // per access), 4 for 16-byte accesses: the depths measured fastest on
    // MI355X
    constexpr int P = prefetch_depth(K, NV * es >= 16               ? kFwdPrefetchWide
                                        : (NV == 2 && es == 4) ? kFwdPrefetchF32Pair
                                                               : kFwdPrefetch);
    constexpr bool kF = DT != kQ88;
    const Geom& g = a.g;
    const int lane = threadIdx.x & 63;
    const int grp = blockIdx.y;
    const int wid = (int)blockIdx.x * kWaves + uniform((int)threadIdx.x >> 6);
    const int nw = (int)gridDim.x * kWaves;
    const ItemRange range(g, wid, nw);
    const int64_t q0 = range.q0, q1 = range.q1, qstep = range.step;
    Surrogate sg;
    sg.init(g.sg, g.alpha);
    __shared__ int32_t qtab[kF ? 1 : kQTable];
    const QTable qt{qtab};
    if constexpr (!kF) {
        if (a.sg_out != nullptr) {
            qt.fill(sg);
            __syncthreads();
        }
    }
    if (q0 >= q1)
        return;

    // the lane's channel: taps, bias and threshold (Eq. mfdpsn_fire: V_th[c]
    // when given, else the one shared by every channel); flat tiles hold
    // columns of several channels, so they set it per tile
    TP tp;
    V bias, start;
    float vth = g.v_th;
    int vthq = g.v_th_q;
    auto set_channel = [&](int c) __attribute__((always_inline)) {
        tp.load(a.sign, a.shift, c, g.shift_lo, g.shift_hi);
        if constexpr (kF) {
            const float b = ((const float*)a.bias)[c];
            bias = b == 0.0f ? 0.0f : b;  // a zero bias is added as +0
            start = 0.0f;
        } else {
            bias = ((const int32_t*)a.bias)[c];
            start = bias + tp.cneg;
        }
        if (a.v_th_c != nullptr) {
            if constexpr (kF)
                vth = ((const float*)a.v_th_c)[c];
            else
                vthq = ((const int32_t*)a.v_th_c)[c];
        }
    };
    if constexpr (MODE != kFlat)
        set_channel((MODE == kLaneChannel) ? min(grp * 64 + lane, g.C - 1) : grp);
    const uint32_t M = g.M;
    const int d = g.d;
    const uint64_t xrow = (uint64_t)M * es;
    const uint64_t xbytes = (uint64_t)g.T * xrow, sbytes = (uint64_t)g.T * M;
    const int32_t xstep = (int32_t)((uint64_t)d * xrow), sstep = (int32_t)((uint64_t)d * M);
    const int want_h = a.h_out != nullptr ? 1 : 0;
    const int want_sg = a.sg_out != nullptr ? 1 : 0;
    // (4-byte rows only when they are written: the planner sizes chunks so
    // that the offsets of the streams a call moves fit 32 bits)
    const int32_t hstep = want_h | want_sg ? 4 * sstep : 0;

    Cursor cur(g, q0);
    int tile_cached = -1;
    Cols cols{};
    for (int64_t q = q0; q < q1; q += qstep, cur.advance(g, q, qstep)) {
        // item scalars, pinned to SGPRs; the consecutive chunks of this class
        // in the range are walked as one
        const int r = uniform(cur.r);
        const int Lr = uniform(class_len(g, r));
        const int j0 = uniform(cur.chunk * g.chunk);
        int more = 0;
        if (qstep == 1)
            more = (int)min(min(q1 - 1 - q, (int64_t)(g.nchunks - 1 - cur.chunk)), (int64_t)(g.run_max - 1));
        more = uniform(more);
        q += more;
        cur.chunk += more;
        const int j1 = uniform(min(Lr, j0 + (more + 1) * g.chunk));
        if (j0 >= j1)
            continue;
        if (cur.tile != tile_cached) {
            cols = tile_cols<MODE, NV>(g, cur.tile, grp, lane);
            tile_cached = cur.tile;
            if constexpr (MODE == kFlat)
                set_channel((int)((cols.col / (uint32_t)g.S) % (uint32_t)g.C));
        }
        // x rows from jb (the halo of a chunk) on; outputs from j0 on
        const int jb = j0 > 0 ? j0 - (K - 1) : 0;
        const Buf xs = make_buf(a.x, xbytes, ((uint64_t)r + (uint64_t)jb * d) * xrow);
        const uint64_t orow = (uint64_t)r + (uint64_t)j0 * d;
        const Buf ss = make_buf(a.spikes, sbytes, orow * M);
        const Buf hs = want_h ? make_buf(a.h_out, sbytes * 4, orow * M * 4) : ss;
        const Buf gs = want_sg ? make_buf(a.sg_out, sbytes * 4, orow * M * 4) : ss;
        const uint32_t vx = cols.col * es, vs = cols.col, vh = cols.col * 4u;
        const int32_t so_xlast = (Lr - 1 - jb) * xstep;

        PV ring[K];  // x[t] at slot t mod k
        int slow = 0;  // steps left with rounded products
#pragma unroll
        for (int i = 0; i < K; ++i)
#pragma unroll
            for (int e = 0; e < NV; ++e)
                ring[i].v[e] = V(0);
        // The halo x[j0-k+1 .. j0-1] (chunks after the first; j0 is a multiple
        // of k) and x[j0 .. j0+P-1] at prefetch slot j mod P, kept as loaded
        // (converted in the step that uses them, so no step waits for the
        // loads it issues itself).  Every load is issued before any value is
        // looked at: an item starts after one memory round trip.  A halo input
        // with an inexact tap product keeps the rounded products on for the steps
        // whose window holds it.
        if (j0 > 0) {
#pragma unroll
            for (int m = 0; m < K - 1; ++m)
                ring[(m + 1) % K] = IO<DT>::template load<NV>(xs, vx, m * xstep);
        }
        typename IO<DT>::template Raw<NV> pf[P];
#pragma unroll
        for (int p = 0; p < P; ++p)
            pf[p] = IO<DT>::template load_raw<NV>(xs, vx, min((j0 + p - jb) * xstep, so_xlast));
        if constexpr (TP::kHasFast) {
            if (j0 > 0) {
#pragma unroll
                for (int m = 0; m < K - 1; ++m) {
                    const bool bad = x_slow(ring[(m + 1) % K], g);
                    slow = bad ? m + 1 : slow;
                }
            }
        }
        int32_t so_xp = (j0 + P - jb) * xstep;  // prefetch of step j + P
        int32_t so_s = 0, so_h = 0;

        // one step (u: position in the block, j = bK + u); KIND with kEdge is
        // the block at the start of the sequence, which leaves out the float
        // taps that would read before time 0 (Q8.8 keeps them: the ring holds
        // zeros there, whose xor-terms the starting value cancels)
        auto step = [&](auto uc, auto kc_, int j) __attribute__((always_inline)) {
            constexpr int u = decltype(uc)::value;
            constexpr int kind = decltype(kc_)::value;
            constexpr int imin = (kF && (kind & kEdge) == kEdge) ? K - 1 - u : 0;
            (void)j;
            const PV xv = IO<DT>::template cvt<NV>(pf[u % P]);
            pf[u % P] = IO<DT>::template load_raw<NV>(xs, vx, kind == kFull ? so_xp : min(so_xp, so_xlast));
            advance(so_xp, xstep);
            ring[u] = xv;
            PV h;
            uint32_t spk[(NV + 3) / 4] = {};  // spike of column e in byte e mod 4 of word e / 4
            if constexpr (kF) {
                if (x_slow(xv, g))
                    slow = K;
                if (__builtin_expect(slow > 0, 0)) {
#pragma unroll
                    for (int e = 0; e < NV; ++e) {
                        V acc = tp.apply(ring[(u + 1 + imin) % K].v[e], imin);
#pragma unroll
                        for (int i = imin + 1; i < K; ++i)
                            acc = acc + tp.apply(ring[(u + 1 + i) % K].v[e], i);
                        h.v[e] = acc + bias;
                    }
                    --slow;
                } else {
#pragma unroll
                    for (int e = 0; e < NV; ++e) {
                        V acc = tp.apply(ring[(u + 1 + imin) % K].v[e], imin);
#pragma unroll
                        for (int i = imin + 1; i < K; ++i)
                            acc = tp.fma(ring[(u + 1 + i) % K].v[e], i, acc);
                        h.v[e] = acc + bias;
                    }
                }
#pragma unroll
                for (int e = 0; e < NV; ++e)
                    spk[e / 4] |= (h.v[e] >= vth ? 1u : 0u) << (8 * (e % 4));
            } else {
#pragma unroll
                for (int e = 0; e < NV; ++e) {
                    // (pinned partial sums: one shift and one xor-add per tap,
                    // instead of the reassociated shift, xor, add3 sequence)
                    h.v[e] = q88_charge<K>(tp, start, [&](int i) { return ring[(u + 1 + i) % K].v[e]; });
                    spk[e / 4] |= (h.v[e] >= vthq ? 1u : 0u) << (8 * (e % 4));
                }
            }
            st_bytes<NV>(ss, vs, so_s, spk);
            if (want_h != 0) {
                Pk<uint32_t, NV> w;
#pragma unroll
                for (int e = 0; e < NV; ++e)
                    w.v[e] = __builtin_bit_cast(uint32_t, h.v[e]);
                st_words<NV>(hs, vh, so_h, w);
            }
            if (want_sg != 0) {
                Pk<uint32_t, NV> w;
#pragma unroll
                for (int e = 0; e < NV; ++e)
                    if constexpr (kF)
                        w.v[e] = __builtin_bit_cast(uint32_t, sg_factor<false>(sg, h.v[e], vth, vthq));
                    else
                        w.v[e] = (uint32_t)qt(sg, h.v[e], vthq);
                st_words<NV>(gs, vh, so_h, w);
            }
            advance(so_s, sstep);
            advance(so_h, hstep);
            __builtin_amdgcn_sched_barrier(MFPSN_FWD_STEP_BARRIER);
        };
        auto block = [&](int jb0, auto kc_) __attribute__((always_inline)) {
            constexpr int kind = decltype(kc_)::value;
            [&]<int... U>(std::integer_sequence<int, U...>) __attribute__((always_inline)) {
                (void)(((kind == kFull || jb0 + U < j1) ? (step(ic<U>{}, kc_, jb0 + U), true) : false) && ...);
            }(std::make_integer_sequence<int, K>{});
        };
        int b = j0 / K;
        const int bend = (j1 + K - 1) / K;
        if (b == 0) {
            block(0, ic<kEdge>{});
            ++b;
        }
        if constexpr (K <= kFullBlockMaxK) {
            // full blocks: every step below j1, every prefetch inside the class
            const int bfull = min(j1 / K, (Lr - P) / K);
            for (; b < bfull; ++b)
                block(b * K, ic<kFull>{});
        }
        for (; b < bend; ++b)
            block(b * K, ic<kChecked>{});
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
__device__ __forceinline__ int64_t wave_sum(int64_t v)
{
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1)
        v += __shfl_xor(v, m, 64);
    return v;
}

// What the backward reads besides x and grad_spikes: nothing (H and the
// surrogate factor are recomputed from the x ring), the forward's saved
// surrogate factor, or the forward's saved potentials H.
enum SavedKind : int { kRecompute = 0, kSavedFactor = 1, kSavedH = 2 };

template <int K, int DT, int MODE, int HS, int NV>
__global__ __launch_bounds__(kThreads) void bwd_kernel(BwdArgs a)
{
    using V = typename IO<DT>::V;
    using W = typename IO<DT>::W;
    using PV = Pk<V, NV>;
    using TP = Taps<K, DT, MODE>;
    constexpr int es = IO<DT>::es;
    // Lane-channel waves at orders up to 16 run 4 per SIMD and stream three
    // 256-byte rows per step: a short queue is best.  Plane waves (narrower
    // rows) want a longer one, and high orders 8 steps (which keeps the Q8.8
    // order-32 saved-factor kernel at two waves per SIMD).
    // Lanes holding two columns do best with about 16 bytes per stream in
    // flight (2 steps of f32 pairs, 4 of bf16 or Q8.8 pairs).
    constexpr int P = prefetch_depth(
        K, K >= 24 ? kBwdPrefetchHighK
                   : (MODE == kLaneChannel ? kBwdPrefetch
                                           : (NV == 2 ? kBwdPairBytes / (es * NV) : 2 * kBwdPrefetch)));
    constexpr int gxs = IO<DT>::gx_es;
    constexpr bool kF = DT != kQ88;
    constexpr bool kRe = HS == kRecompute;  // recompute H from the x ring
    // x rings: double copies for the exact grad_w products of float data;
    // the stored value itself for the recompute of float data and for Q8.8
    // (whose products are exact 32x32 -> 64-bit integer products)
    constexpr bool kXD = kF;
    constexpr bool kXV = kRe || !kF;
    const Geom& g = a.g;
    const int lane = threadIdx.x & 63;
    const int wave = uniform((int)threadIdx.x >> 6);
    const int grp = blockIdx.y;
    const int wid = (int)blockIdx.x * kWaves + wave;
    const int nw = (int)gridDim.x * kWaves;
    const ItemRange range(g, wid, nw);
    const int64_t q0 = range.q0, q1 = range.q1, qstep = range.step;
    const int c = (MODE == kLaneChannel) ? min(grp * 64 + lane, g.C - 1) : grp;

    TP tp;
    tp.load(a.sign, a.shift, c, g.shift_lo, g.shift_hi);
    V bias = V(0), start = V(0), reset = V(0);
    if constexpr (kF) {
        const float b = ((const float*)a.bias)[c];
        bias = b == 0.0f ? 0.0f : b;
    } else {
        bias = ((const int32_t*)a.bias)[c];
        start = bias + tp.cneg;
        reset = tp.cneg;
    }
    float vth = g.v_th;  // the channel's threshold, as in the forward
    int vthq = g.v_th_q;
    if (a.v_th_c != nullptr) {
        if constexpr (kF)
            vth = ((const float*)a.v_th_c)[c];
        else
            vthq = ((const int32_t*)a.v_th_c)[c];
    }
    Surrogate sg;
    sg.init(g.sg, g.alpha);
    constexpr bool kQT = !kF && HS != kSavedFactor;  // Q8.8 factors from the table
    __shared__ int32_t qtab[kQT ? kQTable : 1];
    const QTable qt{qtab};
    if constexpr (kQT) {
        qt.fill(sg);
        __syncthreads();
    }
    auto factor = [&](V h) __attribute__((always_inline)) {
        if constexpr (kQT)
            return qt(sg, h, vthq);
        else
            return sg_factor(sg, h, vth, vthq);
    };

    const uint32_t M = g.M;
    const int d = g.d;
    const uint64_t xrow = (uint64_t)M * es, hrow = (uint64_t)M * 4, gxrow = (uint64_t)M * gxs;
    const uint64_t xbytes = (uint64_t)g.T * xrow, hbytes = (uint64_t)g.T * hrow, gxbytes = (uint64_t)g.T * gxrow;
    const int32_t xstep = (int32_t)((uint64_t)d * xrow), hstep = (int32_t)((uint64_t)d * hrow);
    const int32_t gxstep = (int32_t)((uint64_t)d * gxrow);

    W gw[K];
#pragma unroll
    for (int i = 0; i < K; ++i)
        gw[i] = W(0);
    W gb = W(0);

    Cursor cur(g, q0);
    int tile_cached = -1;
    Cols cols{};
    for (int64_t q = q0; q < q1; q += qstep, cur.advance(g, q, qstep)) {
        // item scalars, pinned to SGPRs; the consecutive chunks of this class
        // in the range are walked as one
        const int r = uniform(cur.r);
        const int Lr = uniform(class_len(g, r));
        const int j0 = uniform(cur.chunk * g.chunk);
        int more = 0;
        if (qstep == 1)
            more = (int)min(min(q1 - 1 - q, (int64_t)(g.nchunks - 1 - cur.chunk)), (int64_t)(g.run_max - 1));
        more = uniform(more);
        q += more;
        cur.chunk += more;
        const int j1 = uniform(min(Lr, j0 + (more + 1) * g.chunk));
        if (j0 >= j1)
            continue;
        if (cur.tile != tile_cached) {
            cols = tile_cols<MODE, NV>(g, cur.tile, grp, lane);
            tile_cached = cur.tile;
        }
        const bool partial = cols.partial;
        const bool active = cols.active;
        // steps j1..jtop are the halo of a lower chunk: their dH feeds outputs
        // below j1.  The walk runs down from jtop in blocks of k steps: step u
        // of block b is j = jtop - bk - u, and every value of time t sits in
        // ring slot (jtop - t) mod k, a compile-time index in every step.
        const int jtop = uniform(min(j1 + K - 1, Lr) - 1);
        const int jb = uniform(max(0, j0 - (K - 1) - P));  // lowest row any stream touches
        const uint64_t brow = (uint64_t)r + (uint64_t)jb * d;
        const Buf xs = make_buf(a.x, xbytes, brow * xrow);
        const Buf gsb = make_buf(a.gs, xbytes, brow * xrow);
        const Buf hsb = HS ? make_buf(HS == kSavedFactor ? a.sg : a.h, hbytes, brow * hrow) : xs;
        const Buf gxb = make_buf(a.grad_x, gxbytes, brow * gxrow);
        const uint32_t vx = cols.col * es, vh = cols.col * 4u, vgx = cols.col * gxs;
        const int32_t so_last = (Lr - 1 - jb) * xstep, so_hlast = (Lr - 1 - jb) * hstep;

        // grad_x accumulators: output t at slot (jtop - t) mod k, opened with
        // the start of its sum (Q8.8: the number of negative taps that reach it)
        PV gxa[K];
#pragma unroll
        for (int s = 0; s < K; ++s) {
            V v0;
            if constexpr (kF) {
                v0 = 0.0f;
            } else {
                const int t = jtop - s;               // output of slot s
                const int skip = max(0, t + K - Lr);  // taps whose source lies past the end
                v0 = __builtin_popcount(tp.negmask >> skip);
            }
#pragma unroll
            for (int e = 0; e < NV; ++e)
                gxa[s].v[e] = v0;
        }
        // x ring: x[t] at slot (jtop - t) mod k, for t in the window of the
        // step; zeros for times before 0
        Pk<double, NV> xd[kXD ? K : 1];
        PV xf[kXV ? K : 1];
        int slow_x = 0;  // live steps left on the exact recompute path
        // prefetch: step j's g[j], h[j], x[j-k+1] at slot (jtop - j) mod P, as
        // loaded (converted in the step that uses them)
        typename IO<DT>::template Raw<NV> pg[P], px[P];
        PV ph[HS ? P : 1];
        auto load_h = [&](int32_t so) __attribute__((always_inline)) {
            const Pk<uint32_t, NV> w = ld_words<NV>(hsb, vh, so);
            PV v;
#pragma unroll
            for (int e = 0; e < NV; ++e)
                v.v[e] = __builtin_bit_cast(V, w.v[e]);
            return v;
        };
        // Preload: the ring's inputs x[jtop-k+2 .. jtop] (slot jtop - t) and
        // the first P steps' streams.  Every load is issued before any value
        // is looked at, so an item starts after one memory round trip, not
        // one per ring slot.  Rows below jb (times before 0 of a short class,
        // or steps below the walk) are clamped; their ring values are zeros.
        {
            typename IO<DT>::template Raw<NV> rr[K - 1 > 0 ? K - 1 : 1];
#pragma unroll
            for (int m = 0; m < K - 1; ++m)
                rr[m] = IO<DT>::template load_raw<NV>(xs, vx, (max(jtop - m, jb) - jb) * xstep);
#pragma unroll
            for (int p = 0; p < P; ++p) {
                const int rowg = max(jtop - p, jb);
                pg[p] = IO<DT>::template load_raw<NV>(gsb, vx, (rowg - jb) * xstep);
                if constexpr (HS)
                    ph[p] = load_h((rowg - jb) * hstep);
                px[p] = IO<DT>::template load_raw<NV>(xs, vx, (max(jtop - p - K + 1, jb) - jb) * xstep);
            }
            bool out = false;  // some input of this lane with an inexact tap product
#pragma unroll
            for (int m = 0; m < K - 1; ++m) {
                PV v = IO<DT>::template cvt<NV>(rr[m]);
                const bool live = jtop - m >= 0;
#pragma unroll
                for (int e = 0; e < NV; ++e)
                    v.v[e] = live ? v.v[e] : V(0);
                if constexpr (kXD)
#pragma unroll
                    for (int e = 0; e < NV; ++e)
                        xd[m].v[e] = (double)v.v[e];
                if constexpr (kXV)
                    xf[m] = v;
                // x[t] (0 <= t <= jtop) is in the window of at most k live steps
                if constexpr (kRe && TP::kHasFast)
                    if (live)
                        out = out | lane_slow(v, g);
            }
            if (kRe && TP::kHasFast && !g.x_exact && __builtin_amdgcn_ballot_w64(out) != 0)
                slow_x = K;
        }
        int32_t so_gp = (jtop - P - jb) * xstep;           // g of step j - P
        int32_t so_hp = HS ? (jtop - P - jb) * hstep : 0;  // factor or H of step j - P
        int32_t so_xp = (jtop - P - K + 1 - jb) * xstep;   // x of step j - P
        int32_t so_gx = (jtop - jb) * gxstep;              // grad_x of step j

        // one step (u: position in the block, j = jtop - bk - u).  Time j - k +
        // 1 + i, the source of tap i and the output that tap i of dH[j]
        // reaches, sits in slot (u + k - 1 - i) mod k.  Steps j < k - 1 (only
        // in checked blocks) have sources before time 0: the ring holds zeros
        // there, whose exact zero terms change no bit of H once the bias is
        // added (they only lead the sum), and their outputs before time 0
        // are never stored.
        auto step = [&](auto uc, auto kc_, int j) __attribute__((always_inline)) {
            constexpr int u = decltype(uc)::value;
            constexpr int kind = decltype(kc_)::value;
            constexpr bool full = kind == kFull;
            constexpr int sp = u % P;  // prefetch slot
            auto sl = [](int i) constexpr { return (u + K - 1 - i) % K; };  // slot of time j-k+1+i
            const bool edge = !full && j < K - 1;  // some source before time 0 (wave-uniform)
            const PV gv = IO<DT>::template cvt<NV>(pg[sp]);
            PV xv = IO<DT>::template cvt<NV>(px[sp]);
            PV hv;
            if constexpr (HS)
                hv = ph[sp];
            pg[sp] = IO<DT>::template load_raw<NV>(gsb, vx, full ? so_gp : min(max(so_gp, 0), so_last));
            if constexpr (HS)
                ph[sp] = load_h(full ? so_hp : min(max(so_hp, 0), so_hlast));
            px[sp] = IO<DT>::template load_raw<NV>(xs, vx, full ? so_xp : min(max(so_xp, 0), so_last));
            advance(so_gp, -xstep);
            if constexpr (HS)
                advance(so_hp, -hstep);
            advance(so_xp, -xstep);
            // x[j-k+1] enters the ring (slot sl(0)); zeros before time 0
            if (edge) {
#pragma unroll
                for (int e = 0; e < NV; ++e)
                    xv.v[e] = j - K + 1 >= 0 ? xv.v[e] : V(0);
            }
            if constexpr (kXD)
#pragma unroll
                for (int e = 0; e < NV; ++e)
                    xd[sl(0)].v[e] = (double)xv.v[e];
            if constexpr (kXV)
                xf[sl(0)] = xv;
            if (kRe && TP::kHasFast && (full || j - K + 1 >= 0) && x_slow(xv, g))
                slow_x = K;
            {
                PV dh;
                if constexpr (HS == kSavedFactor) {
#pragma unroll
                    for (int e = 0; e < NV; ++e)
                        dh.v[e] = delta_h(gv.v[e], hv.v[e]);
                } else if constexpr (HS == kSavedH) {
#pragma unroll
                    for (int e = 0; e < NV; ++e)
                        dh.v[e] = delta_h(gv.v[e], factor(hv.v[e]));
                } else {
                    PV h;
                    if constexpr (kF) {
                        if (__builtin_expect(slow_x > 0, 0)) {
#pragma unroll
                            for (int e = 0; e < NV; ++e) {
                                V acc = tp.apply(xf[sl(0)].v[e], 0);
#pragma unroll
                                for (int i = 1; i < K; ++i)
                                    acc = acc + tp.apply(xf[sl(i)].v[e], i);
                                h.v[e] = acc + bias;
                            }
                        } else {
#pragma unroll
                            for (int e = 0; e < NV; ++e) {
                                V acc = tp.apply(xf[sl(0)].v[e], 0);
#pragma unroll
                                for (int i = 1; i < K; ++i)
                                    acc = tp.fma(xf[sl(i)].v[e], i, acc);
                                h.v[e] = acc + bias;
                            }
                        }
                    } else {
#pragma unroll
                        for (int e = 0; e < NV; ++e) {
                            h.v[e] = q88_charge<K>(tp, start, [&](int i) { return xf[sl(i)].v[e]; });
                        }
                    }
#pragma unroll
                    for (int e = 0; e < NV; ++e)
                        dh.v[e] = delta_h(gv.v[e], factor(h.v[e]));
                }
                const bool own = full || j < j1;
                if (own) {
#pragma unroll
                    for (int e = 0; e < NV; ++e) {
                        if constexpr (kF) {
                            V de = dh.v[e];
                            if (MODE == kPlane && partial)
                                de = active ? de : V(0);  // no contribution from shadow lanes
                            const double dd = (double)de;
#pragma unroll
                            for (int i = 0; i < K; ++i) {
                                gw[i] = __builtin_fma(xd[sl(i)].v[e], dd, gw[i]);
                                pin(gw[i]);
                            }
                            gb += dd;
                            pin(gb);
                        } else {
                            int32_t dq = dh.v[e];
                            if (MODE == kPlane && partial)
                                dq = active ? dq : 0;
#pragma unroll
                            for (int i = 0; i < K; ++i) {
                                gw[i] += (int64_t)xf[sl(i)].v[e] * (int64_t)dq;
                                pin(gw[i]);
                            }
                            gb += dq;
                            pin(gb);
                        }
                    }
                }
                // scatter dH[j] into outputs j-k+1+i (slot sl(i)).  Lanes whose
                // dH has exact tap products add them with one fused rounding;
                // the others (dH whose scaled terms leave the normal range:
                // tiny, huge, infinite or NaN) round each term, then add.
#pragma unroll
                for (int e = 0; e < NV; ++e) {
                    if constexpr (kF) {
                        const bool fast = tap_exact(dh.v[e], g);
                        if (fast) {
#pragma unroll
                            for (int i = 0; i < K; ++i)
                                gxa[sl(i)].v[e] = tp.fma(dh.v[e], i, gxa[sl(i)].v[e]);
                        }
                        if (__builtin_expect(!fast, 0)) {
#pragma unroll
                            for (int i = 0; i < K; ++i)
                                gxa[sl(i)].v[e] = gxa[sl(i)].v[e] + tp.apply(dh.v[e], i);
                        }
                    } else {
                        // (integer sums: pinned so they are not reassociated across
                        // steps, which would keep many steps' terms live)
#pragma unroll
                        for (int i = 0; i < K; ++i) {
                            gxa[sl(i)].v[e] = gxa[sl(i)].v[e] + tp.apply(dh.v[e], i);
                            pin(gxa[sl(i)].v[e]);
                        }
                    }
                }
                // output j is complete: the k-1 steps above it have scattered
                // into slot sl(k-1) = u already
                if (own)
                    IO<DT>::template store_gx<NV>(gxb, vgx, so_gx, gxa[u]);
#pragma unroll
                for (int e = 0; e < NV; ++e)
                    gxa[u].v[e] = reset;  // slot now holds output j - k
                if constexpr (kRe && kF)
                    if (slow_x > 0)
                        --slow_x;
            }
            advance(so_gx, -gxstep);
            // keep the scheduler from hoisting later steps' loads above this
            // step (which would hold them in registers for a whole block)
            __builtin_amdgcn_sched_barrier(MFPSN_BWD_STEP_BARRIER);
        };
        auto block = [&](int b, auto kc_) __attribute__((always_inline)) {
            constexpr int kind = decltype(kc_)::value;
            const int jhi = jtop - b * K;
            [&]<int... U>(std::integer_sequence<int, U...>) __attribute__((always_inline)) {
                (void)((((kind & kLast) != kLast || jhi - U >= j0) ? (step(ic<U>{}, kc_, jhi - U), true) : false) &&
                       ...);
            }(std::make_integer_sequence<int, K>{});
        };
        // Blocks b = 0 .. nb-1 cover the steps jtop down to j0.  Full blocks:
        // every step owned (below j1) with all its sources at or after time
        // 0, and every prefetch row at or above jb; the others check each step.
        // every block before the last runs all its steps
        const int blast = (jtop - j0) / K;
        int b = 0;
        if constexpr (K <= kFullBlockMaxK) {
            const int bf_lo = (jtop - j1 + K) / K;  // first block below j1
            const int lmin = max(max(j0, K - 1), jb + P + K - 1);
            const int span = jtop - (K - 1) - lmin;  // lowest step of block b: jtop - bk - (k-1)
            const int bf_hi = min(span >= 0 ? span / K : -1, blast - 1);
            for (; b < bf_lo && b < blast; ++b)
                block(b, ic<kChecked>{});
            for (; b <= bf_hi; ++b)
                block(b, ic<kFull>{});
        }
        for (; b < blast; ++b)
            block(b, ic<kChecked>{});
        block(blast, ic<kLast>{});
    }
    // block reduction in a fixed order, then one partial row per block
    const int C = g.C;
    if constexpr (MODE == kLaneChannel) {
        __shared__ W red[K + 1][64];
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
                ((W*)a.partial)[((size_t)blockIdx.x * (K + 1) + i) * C + cc] = red[i][l];
        }
    } else {
        __shared__ W red[kWaves][K + 1];
#pragma unroll
        for (int i = 0; i < K; ++i) {
            const W v = wave_sum(gw[i]);
            if (lane == 0)
                red[wave][i] = v;
        }
        {
            const W v = wave_sum(gb);
            if (lane == 0)
                red[wave][K] = v;
        }
        __syncthreads();
        if (threadIdx.x < K + 1) {
            W s = red[0][threadIdx.x];
            for (int w = 1; w < kWaves; ++w)
                s += red[w][threadIdx.x];
            ((W*)a.partial)[((size_t)blockIdx.x * (K + 1) + threadIdx.x) * C + grp] = s;
        }
    }
}

// ---------------------------------------------------------------------------
// finalize: grad_w[c,i] = sum_b partial[b][i][c], grad_b[c] = sum_b partial[b][k][c]
// ---------------------------------------------------------------------------
// One block of 16 waves per 64 outputs: wave w adds the partial rows of a
// fixed contiguous range of blocks, then wave 0 adds the 16 sums in order,
// so the result does not depend on scheduling.  Partials are double (float
// data) or int64 (Q8.8).
constexpr int kFinWaves = 16;

template <typename W>
__device__ __forceinline__ void fin_body(const FinArgs& a)
{
    const W* partial = (const W*)a.partial;
    const int lane = threadIdx.x & 63;
    const int w = threadIdx.x >> 6;
    const int n_out = (a.k + 1) * a.C;
    const int e = blockIdx.x * 64 + lane;
    const bool ok = e < n_out;
    const int ec = ok ? e : n_out - 1;  // loads stay inside the workspace
    const int per = (a.blocks + kFinWaves - 1) / kFinWaves;
    const int b0 = min(w * per, a.blocks);
    const int b1 = min(b0 + per, a.blocks);
    W s = W(0);
    int b = b0;
    for (; b + 8 <= b1; b += 8) {
        W v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            v[u] = partial[(size_t)(b + u) * n_out + ec];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            s += v[u];
    }
    for (; b < b1; ++b)
        s += partial[(size_t)b * n_out + ec];
    __shared__ W red[kFinWaves][64];
    red[w][lane] = s;
    __syncthreads();
    if (w != 0 || !ok)
        return;
    W t = red[0][lane];
    for (int q = 1; q < kFinWaves; ++q)
        t += red[q][lane];
    const int i = e / a.C, c = e % a.C;
    // grad_vth = -grad_b: V_th[c] enters the surrogate as H - V_th[c]
    if constexpr (std::is_same_v<W, int64_t>) {
        if (i < a.k) {
            ((int64_t*)a.grad_w)[c * a.k + i] = t;
        } else {
            ((int64_t*)a.grad_b)[c] = t;
            if (a.grad_vth != nullptr)
                ((int64_t*)a.grad_vth)[c] = -t;
        }
    } else {
        const float v = (float)t;
        if (i < a.k) {
            ((float*)a.grad_w)[c * a.k + i] = v;
        } else {
            ((float*)a.grad_b)[c] = v;
            if (a.grad_vth != nullptr)
                ((float*)a.grad_vth)[c] = -v;
        }
    }
}

__global__ __launch_bounds__(64 * kFinWaves) void fin_kernel(FinArgs a)
{
    if (a.dtype == kQ88)
        fin_body<int64_t>(a);
    else
        fin_body<double>(a);
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

// Persistent grid, never more blocks than the planner's bound; waves own
// contiguous ranges of items that differ by at most one.
//   fill = false (forward): equal shares, the fewest rounds of items the
//     resident waves allow, then the fewest blocks that still finish in that
//     many rounds (fewer waves streaming at once measured faster there);
//   fill = true (backward): every resident wave slot of the group's share of
//     the GPU (up to one wave per item).  That never raises the largest
//     share, and a SIMD with more waves issues faster: one wave alone issues
//     at most one VALU instruction every few cycles and cannot cover its own
//     dependency latencies (order-32 Q8.8 backward: 384 -> 304 us).
// Resident waves of one group (the planner's block bound included).
inline int64_t group_waves(const Geom& g, int resident)
{
    int64_t per_group = resident / g.groups;
    if (per_group < 1)
        per_group = 1;
    if (per_group > g.blocks)
        per_group = g.blocks;
    return per_group * kWaves;
}

inline int persistent_blocks(const Geom& g, int resident, bool fill)
{
    int64_t per_group = resident / g.groups;
    if (per_group < 1)
        per_group = 1;
    if (per_group > g.blocks)
        per_group = g.blocks;
    int64_t blocks;
    if (fill) {
        blocks = (g.items + kWaves - 1) / kWaves;
    } else {
        const int64_t waves_max = per_group * kWaves;
        const int64_t rounds = (g.items + waves_max - 1) / waves_max;
        blocks = (g.items + rounds * kWaves - 1) / (rounds * kWaves);
    }
    if (blocks > per_group)
        blocks = per_group;
    return (int)(blocks > 0 ? blocks : 1);
}

template <int K, int DT>
hipError_t fwd_k(FwdArgs& a, hipStream_t st)
{
    static int cache[3][16];
    static int cache_flat[16];
    void (*kern)(FwdArgs) = fwd_kernel<K, DT, kLaneChannel, 1>;
    int slot = 0;
    if (a.g.mode == kFlat) {
        constexpr int nv = flat_nv(K, DT);
        if constexpr (nv > 0) {
            if (a.g.nv != nv)
                return hipErrorInvalidValue;
            kern = fwd_kernel<K, DT, kFlat, nv>;
            a.g.blocks = persistent_blocks(a.g, resident_blocks(kern, cache_flat), false);
            hipLaunchKernelGGL(kern, dim3(a.g.blocks, a.g.groups), dim3(kThreads), 0, st, a);
            return hipGetLastError();
        } else {
            return hipErrorInvalidValue;
        }
    }
    if (a.g.mode == kPlane) {
        if (a.g.nv == 2) {
            if constexpr (K <= kPairMaxK) {
                kern = fwd_kernel<K, DT, kPlane, 2>;
                slot = 2;
            } else {
                return hipErrorInvalidValue;
            }
        } else {
            kern = fwd_kernel<K, DT, kPlane, 1>;
            slot = 1;
        }
    }
    a.g.blocks = persistent_blocks(a.g, resident_blocks(kern, cache[slot]), false);
    hipLaunchKernelGGL(kern, dim3(a.g.blocks, a.g.groups), dim3(kThreads), 0, st, a);
    return hipGetLastError();
}

template <int K, int DT, int HS>
void (*bwd_kernel_for(const Geom& g, int& slot))(BwdArgs)
{
    if (g.mode == kLaneChannel) {
        slot = 0;
        return bwd_kernel<K, DT, kLaneChannel, HS, 1>;
    }
    if (g.nv == 2) {
        if constexpr (K <= kPairMaxK) {
            slot = 2;
            return bwd_kernel<K, DT, kPlane, HS, 2>;
        } else {
            return nullptr;
        }
    }
    slot = 1;
    return bwd_kernel<K, DT, kPlane, HS, 1>;
}

template <int K, int DT>
hipError_t bwd_k(BwdArgs& a, hipStream_t st)
{
    static int cache[3][3][16];
    const int hs = a.sg != nullptr ? kSavedFactor : (a.h != nullptr ? kSavedH : kRecompute);
    int slot = 0;
    void (*kern)(BwdArgs) = hs == kSavedFactor ? bwd_kernel_for<K, DT, kSavedFactor>(a.g, slot)
                            : hs == kSavedH    ? bwd_kernel_for<K, DT, kSavedH>(a.g, slot)
                                               : bwd_kernel_for<K, DT, kRecompute>(a.g, slot);
    if (kern == nullptr)
        return hipErrorInvalidValue;
    const int res = resident_blocks(kern, cache[hs][slot]);
    balance_chunks(a.g, group_waves(a.g, res));
    a.g.blocks = persistent_blocks(a.g, res, true);
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
