// gfx950 kernels of the mul-free channel-wise neuron (arXiv 2501.14490,
// Eqs. mfdpsn_charge, mfdpsn_fire; App. A.3 Eqs. backward_X, backward_W,
// backward_b) for the time-last layout [N][C][S][T] (time innermost, the
// paper's second layout).
//
// Short columns (T <= 64): one wave per group of 64 columns, lane = column,
// the group transposed through LDS (tl_cols_kernel, tl_cols_bwd_kernel).
// Long columns: a wave per segment of consecutive time steps of one column,
// lane = time step, so the channel and its k taps are the same on every lane;
// the segment's inputs and the history its taps read are staged in the
// wave's LDS window with coalesced loads (tl_seg_fwd_kernel,
// tl_seg_bwd_kernel; tl_fwd_kernel for histories above 1024 steps, with the
// next segment's loads in flight while it computes and the taps read from
// global memory past 2048 steps).
//
// The arithmetic is the definition's, as in the time-first kernels: taps in
// ascending order starting from the first one whose input exists (time >= 0),
// bias last, every add rounded; a float tap is x * 2^-shift with the sign
// applied after the scaling, as a fused multiply-add by sign 2^-shift when
// every staged input of the wave has an exact product (tl_fwd_kernel: an
// integer add to the bit pattern), else as a rounded product (v_ldexp_f32 and
// a sign flip in tl_fwd_kernel) and an add; a Q8.8 tap is an arithmetic right
// shift and a negation after it (integer sums: any order gives the same
// value).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

#include "mfpsn.h"
#include "mfpsn_surrogate.h"
#include "mfpsn_tl.h"

namespace mfpsn {
namespace {

template <int DT> struct TlIO;
template <> struct TlIO<MFPSN_F32> {
    using V = float;
    static __device__ __forceinline__ V ld(const void* p, int64_t e) { return ((const float*)p)[e]; }
};
template <> struct TlIO<MFPSN_BF16> {
    using V = float;
    static __device__ __forceinline__ V ld(const void* p, int64_t e)
    {
        return __builtin_bit_cast(float, (uint32_t)((const uint16_t*)p)[e] << 16);
    }
};
template <> struct TlIO<MFPSN_Q8_8> {
    using V = int32_t;
    static __device__ __forceinline__ V ld(const void* p, int64_t e) { return (int32_t)((const int16_t*)p)[e]; }
};

__device__ __forceinline__ int uniform_i(int v) { return __builtin_amdgcn_readfirstlane(v); }

// LDS writes of every lane of the wave before any lane reads (a wave's LDS
// operations run in order; this keeps the compiler from moving them)
__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// One segment: steps [t0, t0 + 64 NS) of one column; its window of staged
// inputs [ws, we) is the segment and the (K-1) d steps before it
struct TlUnit {
    int64_t cbase;  // flat offset of the column's time 0
    int t0, ws, we, c;
};

// Forward for histories above kTlBwdMaxSpan steps (and T > kTlColsMaxT).
// Persistent waves: wave w takes segments w, w + W, ... (W waves in the
// grid) of 64 NS consecutive time steps of one column, lane l taking steps
// t0 + l + 64 v; the taps are wave-uniform and sit in scalar registers.
// LDS: the segment and the (k-1) d steps before it in the wave's window
// (every tap then reads its input at t - (k-1-i) d: consecutive lanes,
// consecutive addresses), the first NS+2 loads of the next segment's window
// in flight while the current one computes; without LDS (histories above
// kTlMaxHalo) the taps read global memory.
template <int DT, int K, int NS, bool LDS>
__global__ __launch_bounds__(kTlWaves * 64) void tl_fwd_kernel(TlArgs a)
{
    using V = typename TlIO<DT>::V;
    constexpr bool kF = DT != MFPSN_Q8_8;
    constexpr int kW = 64 * NS, kStage = NS + 2;
    extern __shared__ uint32_t tl_lds[];
    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6), lane = (int)threadIdx.x & 63;
    const int64_t units = a.M * a.nseg, stride = (int64_t)gridDim.x * kTlWaves;
    const int span = (K - 1) * a.d;
    V* win = reinterpret_cast<V*>(tl_lds) + (size_t)wave * (kW + a.halo);
    auto unit_of = [&](int64_t u) {
        TlUnit q;
        const int64_t col = u / a.nseg;
        q.t0 = (int)(u - col * a.nseg) * kW;
        q.c = (int)((col / a.S) % a.C);
        q.cbase = col * (int64_t)a.T;
        q.ws = q.t0 - span > 0 ? q.t0 - span : 0;
        q.we = q.t0 + kW < a.T ? q.t0 + kW : a.T;
        return q;
    };
    V buf[kStage];
    auto issue = [&](const TlUnit& q) {
#pragma unroll
        for (int j = 0; j < kStage; ++j) {
            const int t = q.ws + lane + 64 * j;
            buf[j] = TlIO<DT>::ld(a.x, q.cbase + (t < q.we ? t : q.we - 1));
        }
    };
    int64_t u = (int64_t)blockIdx.x * kTlWaves + wave;  // wave-uniform
    if (u >= units)
        return;  // no block-wide barrier in this kernel
    TlUnit cur = unit_of(u);
    if constexpr (LDS)
        issue(cur);
    for (; u < units; u += stride) {
        // taps of the segment's channel (wave-uniform): float bit-pattern
        // addend of x * 2^-s with the sign, or the Q8.8 shift and negation
        int sh[K], neg[K];
        uint32_t kc[K];
#pragma unroll
        for (int i = 0; i < K; ++i) {
            int sv = a.shift[cur.c * K + i];
            sv = sv < a.shift_lo ? a.shift_lo : (sv > a.shift_hi ? a.shift_hi : sv);
            const bool n = a.sign[cur.c * K + i] < 0;
            sh[i] = uniform_i(sv);
            neg[i] = uniform_i(n ? -1 : 0);
            kc[i] = (uint32_t)uniform_i((int)(((uint32_t)(-sv) << 23) ^ (n ? 0x80000000u : 0u)));
        }
        V bias;
        if constexpr (kF)
            bias = ((const float*)a.bias)[cur.c];
        else
            bias = ((const int32_t*)a.bias)[cur.c];

        bool slow = !LDS;  // the global-memory variant always takes the exact taps
        TlUnit nxt = cur;
        if constexpr (LDS) {
            bool out = false;
#pragma unroll
            for (int j = 0; j < kStage; ++j) {
                const int t = cur.ws + lane + 64 * j;
                if (t < cur.we) {
                    win[t - cur.ws] = buf[j];
                    if constexpr (kF) {
                        const float m = __builtin_fabsf(buf[j]);
                        out = out || !(m >= a.fast_lo && m < a.fast_hi);
                    }
                }
            }
            for (int t = cur.ws + lane + 64 * kStage; t < cur.we; t += 64) {  // longer histories
                const V v = TlIO<DT>::ld(a.x, cur.cbase + t);
                win[t - cur.ws] = v;
                if constexpr (kF) {
                    const float m = __builtin_fabsf(v);
                    out = out || !(m >= a.fast_lo && m < a.fast_hi);
                }
            }
            slow = __builtin_amdgcn_ballot_w64(out) != 0;
            wave_lds_sync();
            if (u + stride < units) {  // the next segment's loads, in flight during this one
                nxt = unit_of(u + stride);
                issue(nxt);
            }
        }

        // the tap input of output t: time t - (K-1-i) d; EXACT: v_ldexp_f32
        // and a sign flip, else the bit-pattern add (float); Q8.8 shift and
        // negation
        auto tap = [&](V in, int i, auto exact) -> V {
            if constexpr (kF) {
                if constexpr (decltype(exact)::value) {
                    const float y = ldexpf(in, -sh[i]);
                    return neg[i] ? -y : y;
                } else {
                    return __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, in) + kc[i]);
                }
            } else {
                const int32_t y = in >> sh[i];
                return (y ^ neg[i]) - neg[i];
            }
        };
        auto input = [&](int tt) -> V {
            if constexpr (LDS)
                return win[tt - cur.ws];
            else
                return TlIO<DT>::ld(a.x, cur.cbase + tt);
        };
        auto outputs = [&](auto exact) {
#pragma unroll
            for (int v = 0; v < NS; ++v) {
                const int t = cur.t0 + lane + 64 * v;
                if (cur.t0 + 64 * v >= a.T)
                    break;
                // lanes past the column's end compute on its last time step
                // (every address stays inside the window and the column) and
                // store nothing
                const int tc = t < a.T ? t : a.T - 1;
                V in[K];  // all inputs first: the reads issue back to back
#pragma unroll
                for (int i = 0; i < K; ++i) {
                    const int tt = tc - (K - 1 - i) * a.d;
                    in[i] = input(tt > 0 ? tt : 0);
                }
                V acc;
                if (cur.t0 + 64 * v >= span) {
                    // every tap of every lane reads a time >= 0 (wave-uniform)
                    acc = tap(in[0], 0, exact);
#pragma unroll
                    for (int i = 1; i < K; ++i)
                        acc = acc + tap(in[i], i, exact);
                } else {
                    // from the first tap whose input exists
                    const int back = tc / a.d;
                    const int imin = K - 1 - back > 0 ? K - 1 - back : 0;
                    acc = V(0);
#pragma unroll
                    for (int i = 0; i < K; ++i) {
                        const V term = tap(in[i], i, exact);
                        if constexpr (kF)
                            acc = i < imin ? acc : (i == imin ? term : acc + term);
                        else
                            acc = i < imin ? acc : acc + term;
                    }
                }
                if (t >= a.T)
                    continue;
                const V h = acc + bias;
                const int64_t e = cur.cbase + t;
                bool fire;
                if constexpr (kF)
                    fire = h >= a.v_th;
                else
                    fire = h >= a.v_th_q;
                a.spikes[e] = fire ? 1 : 0;
                if (a.h_out != nullptr)
                    reinterpret_cast<V*>(a.h_out)[e] = h;
            }
        };
        if (kF && slow)
            outputs(std::true_type{});
        else
            outputs(std::false_type{});
        if constexpr (LDS) {
            wave_lds_sync();  // every read of the window before the next segment's writes
            cur = nxt;
        } else if (u + stride < units) {
            cur = unit_of(u + stride);
        }
    }
}

typedef uint32_t U32x4 __attribute__((ext_vector_type(4)));

// Four consecutive stored elements (one vector load)
template <int DT> struct TlVec4;
template <> struct TlVec4<MFPSN_F32> {
    static __device__ __forceinline__ float4 ldraw(const void* p, int64_t e)
    {
        return *reinterpret_cast<const float4*>((const float*)p + e);
    }
    static __device__ __forceinline__ void cvt(const float4& w, float (&v)[4])
    {
        v[0] = w.x, v[1] = w.y, v[2] = w.z, v[3] = w.w;
    }
    static __device__ __forceinline__ void ld(const void* p, int64_t e, float (&v)[4]) { cvt(ldraw(p, e), v); }
};
template <> struct TlVec4<MFPSN_BF16> {
    static __device__ __forceinline__ uint2 ldraw(const void* p, int64_t e)
    {
        return *reinterpret_cast<const uint2*>((const uint16_t*)p + e);
    }
    static __device__ __forceinline__ void cvt(const uint2& w, float (&v)[4])
    {
        v[0] = __builtin_bit_cast(float, w.x << 16), v[1] = __builtin_bit_cast(float, w.x & 0xffff0000u);
        v[2] = __builtin_bit_cast(float, w.y << 16), v[3] = __builtin_bit_cast(float, w.y & 0xffff0000u);
    }
    static __device__ __forceinline__ void ld(const void* p, int64_t e, float (&v)[4]) { cvt(ldraw(p, e), v); }
};
template <> struct TlVec4<MFPSN_Q8_8> {
    static __device__ __forceinline__ uint2 ldraw(const void* p, int64_t e)
    {
        return *reinterpret_cast<const uint2*>((const int16_t*)p + e);
    }
    static __device__ __forceinline__ void cvt(const uint2& w, int32_t (&v)[4])
    {
        v[0] = (int32_t)(w.x << 16) >> 16, v[1] = (int32_t)w.x >> 16;
        v[2] = (int32_t)(w.y << 16) >> 16, v[3] = (int32_t)w.y >> 16;
    }
    static __device__ __forceinline__ void ld(const void* p, int64_t e, int32_t (&v)[4]) { cvt(ldraw(p, e), v); }
};

// The k taps of one lane's channel: for float data w = sign 2^-s, a normal
// float, whose product with an input is the tap's exponent move (exact, or
// rounded once where the move rounds); for Q8.8 the shift and the negation
// mask.
template <int DT, int K> struct TlLaneTaps {
    static constexpr bool kF = DT != MFPSN_Q8_8;
    using V = typename TlIO<DT>::V;
    float w[kF ? K : 1];
    int sh[kF ? 1 : K], neg[kF ? 1 : K];
    int nneg;          // Q8.8: number of negative taps
    uint32_t negmask;  // Q8.8: bit i set for a negative tap i
    __device__ __forceinline__ void load(const int8_t* sign, const int8_t* shift, int c, int lo, int hi)
    {
        nneg = 0;
        negmask = 0;
#pragma unroll
        for (int i = 0; i < K; ++i) {
            int sv = shift[c * K + i];
            sv = sv < lo ? lo : (sv > hi ? hi : sv);
            const bool n = sign[c * K + i] < 0;
            if constexpr (kF) {
                w[i] = __builtin_bit_cast(float, ((uint32_t)(127 - sv) << 23) | (n ? 0x80000000u : 0u));
            } else {
                sh[i] = sv, neg[i] = n ? -1 : 0;
                nneg += n ? 1 : 0;
                negmask |= n ? (1u << i) : 0u;
            }
        }
    }
    // A sum over all k taps (every input exists, or is a zero) as start()
    // followed by accumulate() per tap in ascending order.  Float: +0, then
    // each term added with one rounding; EXACT rounds the term first (any
    // input), else one fused rounding (inputs whose terms are exact: zero,
    // or in the exponent-add range).  Q8.8: ((v >> s) ^ m) is +(v >> s) or
    // -(v >> s) - 1, so the sum starts at the number of negative taps
    // (integers: any order, the same value).
    __device__ __forceinline__ V start() const
    {
        if constexpr (kF)
            return V(0);
        else
            return nneg;
    }
    template <bool EXACT> __device__ __forceinline__ V accumulate(V acc, V in, int i) const
    {
        if constexpr (kF) {
            if constexpr (EXACT)
                return acc + in * w[i];
            else
                return __builtin_fmaf(in, w[i], acc);
        } else {
            return ((in >> sh[i]) ^ neg[i]) + acc;
        }
    }
    // sign * in * 2^-s (float: rounded once, as the exponent move); Q8.8
    // floor shift and negation
    template <bool EXACT> __device__ __forceinline__ V apply(V in, int i) const
    {
        if constexpr (kF)
            return in * w[i];
        else
            return ((in >> sh[i]) ^ neg[i]) - neg[i];
    }
};

// The tap products of v are exact (v zero, or normal far enough from the
// exponent limits).  Bitwise logic: no branch per operand.
__device__ __forceinline__ bool tl_tap_exact(float v, float lo, float hi)
{
    const float m = __builtin_fabsf(v);
    return ((m >= lo) & (m < hi)) | (m == 0.0f);
}

constexpr int kTlRow = 65;                             // words per time row of a transposed tile
// The transposed LDS tiles of the short-column kernels hold bf16 data as its
// 16-bit values (half the LDS per wave, so twice the waves fit on a CU) and
// other data as the 32-bit values the registers hold.  Rows of 65 words (66
// halves): a row read by the 64 lanes touches every bank once.
template <int DT> struct TlTile {
    using V = typename TlIO<DT>::V;
    using E = V;
    static constexpr int kRow = kTlRow;
    static __device__ __forceinline__ E put(V v) { return v; }
    static __device__ __forceinline__ V get(E e) { return e; }
};
template <> struct TlTile<MFPSN_BF16> {
    using E = uint16_t;
    static constexpr int kRow = 2 * kTlRow - 64;
    static __device__ __forceinline__ E put(float v) { return (uint16_t)(__builtin_bit_cast(uint32_t, v) >> 16); }
    static __device__ __forceinline__ float get(E e) { return __builtin_bit_cast(float, (uint32_t)e << 16); }
};
template <int DT> constexpr size_t tl_tile_bytes(int T)
{
    return (size_t)T * TlTile<DT>::kRow * sizeof(typename TlTile<DT>::E);
}
constexpr int kTlMaxChunks = 16 * kTlColsMaxT / 64;     // 4-element chunks per lane and group

// Column of the e-th element of a group of columns of length T (e < 64 T)
__device__ __forceinline__ int tl_col_of(int e, int T, uint32_t tdiv)
{
    return T == 1 ? e : (int)__umulhi((uint32_t)e, tdiv);
}

// Stages a group's ncols * T contiguous elements of src (from element gbase)
// into the transposed tile tile[tau * kRow + col], with 4-element vector
// loads for a whole group when vec is set.  Returns (wave-uniform) whether
// some staged float lies outside [lo, hi); always false for Q8.8.
template <int DT>
__device__ __forceinline__ bool tl_stage(const void* src, int64_t gbase, int ncols, int T, uint32_t tdiv, bool vec,
                                         typename TlTile<DT>::E* tile, float lo, float hi)
{
    using V = typename TlIO<DT>::V;
    constexpr bool kF = DT != MFPSN_Q8_8;
    const int lane = (int)threadIdx.x & 63;
    bool out = false;
    auto put = [&](int e, V v) {
        const int c = tl_col_of(e, T, tdiv);
        tile[(e - c * T) * TlTile<DT>::kRow + c] = TlTile<DT>::put(v);
        if constexpr (kF)
            out = out | !tl_tap_exact(v, lo, hi);
    };
    if (ncols == 64 && vec && DT == MFPSN_F32) {
        const int nch = 16 * T;  // 4-element chunks of the group
        V v[kTlMaxChunks][4];
#pragma unroll
        for (int j = 0; j < kTlMaxChunks; ++j)
            if (lane + 64 * j < nch)
                TlVec4<DT>::ld(src, gbase + 4 * (lane + 64 * j), v[j]);
#pragma unroll
        for (int j = 0; j < kTlMaxChunks; ++j)
            if (lane + 64 * j < nch) {
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    put(4 * (lane + 64 * j) + q, v[j][q]);
            }
    } else if (ncols == 64 && vec) {
        if constexpr (DT != MFPSN_F32) {
            // 2-byte types: the chunks stay as loaded (two registers each)
            // and are widened where they are written
            const int nch = 16 * T;
            uint2 w[kTlMaxChunks];
#pragma unroll
            for (int j = 0; j < kTlMaxChunks; ++j)
                if (lane + 64 * j < nch)
                    w[j] = TlVec4<DT>::ldraw(src, gbase + 4 * (lane + 64 * j));
#pragma unroll
            for (int j = 0; j < kTlMaxChunks; ++j)
                if (lane + 64 * j < nch) {
                    V v[4];
                    TlVec4<DT>::cvt(w[j], v);
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        put(4 * (lane + 64 * j) + q, v[q]);
                }
        }
    } else {
        for (int e = lane; e < ncols * T; e += 64)
            put(e, TlIO<DT>::ld(src, gbase + e));
    }
    return kF && __builtin_amdgcn_ballot_w64(out) != 0;
}

// Stages x and grad_spikes of a group (as tl_stage does each) with every
// load of both issued before the first LDS write, so the two wait for one
// memory round trip together.  The pending vector loads take two registers
// per lane and chunk for 2-byte types and four for f32, which the callers
// afford only up to NCH chunks per lane (T <= 4 NCH).  Returns tl_stage's
// flag for x.
template <int DT, int NCH>
__device__ __forceinline__ bool tl_stage_pair(const void* x, const void* gsrc, int64_t gbase, int ncols, int T,
                                              uint32_t tdiv, bool vec, typename TlTile<DT>::E* xt,
                                              typename TlTile<DT>::E* gt, float lo, float hi)
{
    using V = typename TlIO<DT>::V;
    using R = decltype(TlVec4<DT>::ldraw(nullptr, 0));
    constexpr bool kF = DT != MFPSN_Q8_8;
    if (!(ncols == 64 && vec) || T > 4 * NCH) {
        const bool out = tl_stage<DT>(x, gbase, ncols, T, tdiv, vec, xt, lo, hi);
        (void)tl_stage<DT>(gsrc, gbase, ncols, T, tdiv, vec, gt, 0.0f, 0.0f);
        return out;
    }
    const int lane = (int)threadIdx.x & 63;
    const int nch = 16 * T;  // 4-element chunks of the group
    R rx[NCH], rg[NCH];  // as loaded, widened where written
#pragma unroll
    for (int j = 0; j < NCH; ++j)
        if (lane + 64 * j < nch)
            rx[j] = TlVec4<DT>::ldraw(x, gbase + 4 * (lane + 64 * j));
#pragma unroll
    for (int j = 0; j < NCH; ++j)
        if (lane + 64 * j < nch)
            rg[j] = TlVec4<DT>::ldraw(gsrc, gbase + 4 * (lane + 64 * j));
    bool out = false;
#pragma unroll
    for (int j = 0; j < NCH; ++j)
        if (lane + 64 * j < nch) {
            V v[4];
            TlVec4<DT>::cvt(rx[j], v);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int e = 4 * (lane + 64 * j) + q;
                const int c = tl_col_of(e, T, tdiv);
                xt[(e - c * T) * TlTile<DT>::kRow + c] = TlTile<DT>::put(v[q]);
                if constexpr (kF)
                    out = out | !tl_tap_exact(v[q], lo, hi);
            }
        }
#pragma unroll
    for (int j = 0; j < NCH; ++j)
        if (lane + 64 * j < nch) {
            V v[4];
            TlVec4<DT>::cvt(rg[j], v);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int e = 4 * (lane + 64 * j) + q;
                const int c = tl_col_of(e, T, tdiv);
                gt[(e - c * T) * TlTile<DT>::kRow + c] = TlTile<DT>::put(v[q]);
            }
        }
    return kF && __builtin_amdgcn_ballot_w64(out) != 0;
}

// Short columns (T <= kTlColsMaxT): one wave per group of 64 columns,
// lane = column.  The group's inputs, 64 T contiguous elements, are read with
// coalesced loads and written transposed into LDS, one row of 64 columns per
// time step (row stride 65 words: a row read by the 64 lanes touches every
// bank once).  Each lane then walks its column one residue class r of the
// dilation at a time (times r, r + d, ...: the taps of a step read the k
// latest steps of its class), reading one input per step from its LDS column
// into a k-slot register ring (slot j mod k, a compile-time index inside
// blocks of k unrolled steps), with the taps of its own channel in
// registers, and puts its spikes into a [column][time] byte tile that is
// written back with 16-byte stores.
template <int DT, int K>
__global__ __launch_bounds__(64) void tl_cols_kernel(TlArgs a)
{
    using V = typename TlIO<DT>::V;
    using Tile = TlTile<DT>;
    constexpr bool kF = DT != MFPSN_Q8_8;
    constexpr int kRow = Tile::kRow;
    extern __shared__ uint32_t tl_lds[];
    const int lane = (int)threadIdx.x;
    const int T = a.T;
    const int64_t col0 = (int64_t)blockIdx.x * 64;
    const int ncols = a.M - col0 < 64 ? (int)(a.M - col0) : 64;
    const int64_t gbase = col0 * T;
    typename Tile::E* xt = reinterpret_cast<typename Tile::E*>(tl_lds);
    uint8_t* st = reinterpret_cast<uint8_t*>(tl_lds) + ((tl_tile_bytes<DT>(T) + 15) & ~(size_t)15);
    // the lane's taps and bias first: their loads then wait with the
    // staging's instead of after it
    const int64_t col = col0 + (lane < ncols ? lane : 0);
    const int c = (int)((col / a.S) % a.C);
    TlLaneTaps<DT, K> taps;
    taps.load(a.sign, a.shift, c, a.shift_lo, a.shift_hi);
    V bias;
    if constexpr (kF) {
        const float b = ((const float*)a.bias)[c];
        bias = b == 0.0f ? 0.0f : b;  // a zero bias is added as +0
    } else {
        bias = ((const int32_t*)a.bias)[c];
    }
    const bool slow = tl_stage<DT>(a.x, gbase, ncols, T, a.tdiv, a.vec_x, xt, a.fast_lo, a.fast_hi);
    wave_lds_sync();

    const int d = a.d;
    const int ncls = d < T ? d : T;  // residue classes that hold a step
    V* hrow = a.h_out != nullptr ? reinterpret_cast<V*>(a.h_out) + gbase + (int64_t)lane * T : nullptr;
    auto walk = [&](auto exact) {
        constexpr bool EX = decltype(exact)::value;
        for (int r = 0; r < ncls; ++r) {
            const int Lr = (T - r + d - 1) / d;
            V ring[K];  // x of class step j at slot j mod k; zeros before time 0
#pragma unroll
            for (int i = 0; i < K; ++i)
                ring[i] = V(0);
            // one step (u: its slot; EDGE: the first block, whose float taps
            // before time 0 are left out -- Q8.8 keeps them: their zeros'
            // xor-terms are cancelled by the starting value)
            auto step = [&](auto uc, auto edge_c, int j) __attribute__((always_inline)) {
                constexpr int u = decltype(uc)::value;
                constexpr bool EDGE = decltype(edge_c)::value;
                constexpr int imin = (kF && EDGE) ? K - 1 - u : 0;
                const int t = r + j * d;
                ring[u] = Tile::get(xt[t * kRow + lane]);
                V acc;
                if constexpr (kF) {
                    acc = taps.template apply<EX>(ring[(u + 1 + imin) % K], imin);
#pragma unroll
                    for (int i = imin + 1; i < K; ++i)
                        acc = taps.template accumulate<EX>(acc, ring[(u + 1 + i) % K], i);
                } else {
                    acc = taps.start();
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        acc = taps.template accumulate<EX>(acc, ring[(u + 1 + i) % K], i);
                }
                const V h = acc + bias;
                bool fire;
                if constexpr (kF)
                    fire = h >= a.v_th;
                else
                    fire = h >= a.v_th_q;
                st[lane * T + t] = fire ? 1 : 0;
                if (hrow != nullptr && lane < ncols)
                    hrow[t] = h;
            };
            auto block = [&](int b, auto edge_c) __attribute__((always_inline)) {
                [&]<int... U>(std::integer_sequence<int, U...>) __attribute__((always_inline)) {
                    (void)((b * K + U < Lr ? (step(std::integral_constant<int, U>{}, edge_c, b * K + U), true)
                                           : false) &&
                           ...);
                }(std::make_integer_sequence<int, K>{});
            };
            block(0, std::true_type{});
            for (int b = 1; b * K < Lr; ++b)
                block(b, std::false_type{});
        }
    };
    if (slow)
        walk(std::true_type{});
    else
        walk(std::false_type{});
    wave_lds_sync();

    if (ncols == 64 && a.vec_s) {
        for (int q = lane; q < 4 * T; q += 64)
            __builtin_nontemporal_store(reinterpret_cast<const U32x4*>(st)[q],
                                        reinterpret_cast<U32x4*>(a.spikes + gbase) + q);
    } else {
        for (int e = lane; e < ncols * T; e += 64)
            a.spikes[gbase + e] = st[e];
    }
}

// 64-bit values across lanes (two 32-bit shuffles)
__device__ __forceinline__ double tl_shfl_up(double v, int off)
{
    return __shfl_up(v, (unsigned)off, 64);
}
__device__ __forceinline__ int64_t tl_shfl_up(int64_t v, int off)
{
    const int lo = __shfl_up((int)(uint32_t)v, (unsigned)off, 64);
    const int hi = __shfl_up((int)(uint32_t)((uint64_t)v >> 32), (unsigned)off, 64);
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// bfloat16 bits of a float, round to nearest even (NaN stays NaN)
__device__ __forceinline__ uint16_t tl_bf16_rne(float v)
{
    const uint32_t b = __builtin_bit_cast(uint32_t, v);
    if ((b & 0x7fffffffu) > 0x7f800000u)
        return (uint16_t)((b >> 16) | 0x40u);
    return (uint16_t)((b + 0x7fffu + ((b >> 16) & 1u)) >> 16);
}

// Backward (App. A.3: Eqs. backward_X, backward_W, backward_b, generalized
// to dilation d) for short columns in the time-last layout, lane = column
// as in tl_cols_kernel.  The group's x and grad_spikes are staged transposed
// in LDS.  Each lane walks every residue class of its column backwards in
// time, as the time-first backward walks one: a k-slot ring holds the inputs
// of the step's taps (zeros before time 0), H is recomputed from them, dH =
// grad_spikes * sigma'(H - V_th), the exact products x dH and dH are added
// to the lane's grad_w / grad_b sums (double, or int64 for Q8.8), and dH is
// scattered tap by tap into k grad_x accumulators; an output is complete
// when the walk reaches its own step, and is written over its grad_spikes in
// the tile, which is stored with coalesced writes at the end.  The 64
// lanes' sums are reduced per (n, c) row (lanes of one row are consecutive)
// and stored to the row's slot of this block, part[block + n C + c][k+1].
template <int DT, int K>
__global__ __launch_bounds__(64) void tl_cols_bwd_kernel(TlBwdArgs a)
{
    using V = typename TlIO<DT>::V;
    using Tile = TlTile<DT>;
    using E = typename Tile::E;
    constexpr bool kF = DT != MFPSN_Q8_8;
    using W = std::conditional_t<kF, double, int64_t>;
    constexpr int kRow = Tile::kRow;
    extern __shared__ uint32_t tl_lds[];
    const int lane = (int)threadIdx.x;
    const int T = a.T;
    const int64_t col0 = (int64_t)blockIdx.x * 64;
    const int ncols = a.M - col0 < 64 ? (int)(a.M - col0) : 64;
    const int64_t gbase = col0 * T;
    E* xt = reinterpret_cast<E*>(tl_lds);  // x
    E* gt = xt + T * kRow;                 // grad_spikes, then grad_x (bf16: its rounded bits)
    // the lane's taps and bias first: their loads then wait with the
    // staging's instead of after it
    const int64_t col = col0 + (lane < ncols ? lane : 0);
    const int c = (int)((col / a.S) % a.C);
    TlLaneTaps<DT, K> taps;
    taps.load(a.sign, a.shift, c, a.shift_lo, a.shift_hi);
    V bias;
    if constexpr (kF) {
        const float b = ((const float*)a.bias)[c];
        bias = b == 0.0f ? 0.0f : b;  // a zero bias is added as +0
    } else {
        bias = ((const int32_t*)a.bias)[c];
    }
    // (f32 pairs up to T = 32: eight chunks per lane and array)
    const bool slow_x = tl_stage_pair<DT, DT == MFPSN_F32 ? kTlMaxChunks / 2 : kTlMaxChunks>(
        a.x, a.g, gbase, ncols, T, a.tdiv, a.vec_x, xt, gt, a.fast_lo, a.fast_hi);
    Surrogate sg;
    sg.init(a.sg, a.alpha);
    wave_lds_sync();

    W gw[K], gb = W(0);
#pragma unroll
    for (int i = 0; i < K; ++i)
        gw[i] = W(0);
    const int d = a.d;
    const int ncls = d < T ? d : T;  // residue classes that hold a step
    const bool live = lane < ncols;  // lanes past the last column add nothing
    // the zero of the grad_x accumulators (Q8.8: one for each negative tap
    // that reaches the output)
    const V reset = kF ? V(0) : V(taps.nneg);
    auto walk = [&](auto exact) {
        constexpr bool EX = decltype(exact)::value;
        for (int r = 0; r < ncls; ++r) {
            const int jtop = (T - r + d - 1) / d - 1;  // last step of the class
            // time of class step j' sits in slot (jtop - j') mod k
            V xf[K];
            W xd[kF ? K : 1];
            V gxa[K];
#pragma unroll
            for (int m = 0; m < K - 1; ++m) {
                const int jm = jtop - m;
                xf[m] = jm >= 0 ? Tile::get(xt[(r + jm * d) * kRow + lane]) : V(0);
                if constexpr (kF)
                    xd[m] = (double)xf[m];
            }
#pragma unroll
            for (int s2 = 0; s2 < K; ++s2) {
                if constexpr (kF) {
                    gxa[s2] = V(0);
                } else {
                    const int skip = max(0, (jtop - s2) + K - (jtop + 1));  // taps whose source lies past the end
                    gxa[s2] = __builtin_popcount(taps.negmask >> skip);
                }
            }
            // one step (u: its position in the block, j = jtop - bk - u); time
            // j - k + 1 + i, the source of tap i and the output tap i of dH[j]
            // reaches, sits in slot (u + k - 1 - i) mod k
            auto step = [&](auto uc, int j) __attribute__((always_inline)) {
                constexpr int u = decltype(uc)::value;
                auto sl = [](int i) constexpr { return (u + K - 1 - i) % K; };
                const int t = r + j * d;
                const int jn = j - (K - 1);
                const V xn = jn >= 0 ? Tile::get(xt[(r + jn * d) * kRow + lane]) : V(0);
                const V gv = Tile::get(gt[t * kRow + lane]);
                xf[sl(0)] = xn;
                if constexpr (kF)
                    xd[sl(0)] = (double)xn;
                V acc;
                if constexpr (kF) {
                    acc = taps.template apply<EX>(xf[sl(0)], 0);
#pragma unroll
                    for (int i = 1; i < K; ++i)
                        acc = taps.template accumulate<EX>(acc, xf[sl(i)], i);
                } else {
                    acc = taps.start();
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        acc = taps.template accumulate<EX>(acc, xf[sl(i)], i);
                }
                const V h = acc + bias;
                const V dh = delta_h(gv, sg_factor(sg, h, a.v_th, a.v_th_q));
                if constexpr (kF) {
                    const double dd = live ? (double)dh : 0.0;
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        gw[i] = __builtin_fma(xd[sl(i)], dd, gw[i]);  // exact product, one rounding
                    gb += dd;
                    if (tl_tap_exact(dh, a.fast_lo, a.fast_hi)) {
#pragma unroll
                        for (int i = 0; i < K; ++i)
                            gxa[sl(i)] = __builtin_fmaf(dh, taps.w[i], gxa[sl(i)]);
                    } else {
#pragma unroll
                        for (int i = 0; i < K; ++i)
                            gxa[sl(i)] = gxa[sl(i)] + dh * taps.w[i];
                    }
                } else {
                    const int32_t dq = live ? dh : 0;
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        gw[i] += (int64_t)xf[sl(i)] * (int64_t)dq;
                    gb += dq;
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        gxa[sl(i)] = taps.template accumulate<true>(gxa[sl(i)], dh, i);
                }
                // output j is complete (the k-1 steps above it have scattered
                // into its slot, sl(k-1) = u): over its grad_spikes
                if constexpr (DT == MFPSN_BF16)
                    gt[t * kRow + lane] = tl_bf16_rne(gxa[u]);
                else
                    gt[t * kRow + lane] = gxa[u];
                gxa[u] = reset;  // the slot now holds output j - k
            };
            auto block = [&](int b, auto last_c) __attribute__((always_inline)) {
                constexpr bool LAST = decltype(last_c)::value;
                const int jhi = jtop - b * K;
                [&]<int... U>(std::integer_sequence<int, U...>) __attribute__((always_inline)) {
                    (void)(((!LAST || jhi - U >= 0) ? (step(std::integral_constant<int, U>{}, jhi - U), true)
                                                    : false) &&
                           ...);
                }(std::make_integer_sequence<int, K>{});
            };
            const int blast = jtop / K;
            for (int b = 0; b < blast; ++b)
                block(b, std::false_type{});
            block(blast, std::true_type{});
        }
    };
    if (slow_x)
        walk(std::true_type{});
    else
        walk(std::false_type{});
    wave_lds_sync();

    for (int e = lane; e < ncols * T; e += 64) {
        const int cc = tl_col_of(e, T, a.tdiv);
        reinterpret_cast<E*>(a.grad_x)[gbase + e] = gt[(e - cc * T) * kRow + cc];
    }

    // per-channel sums: segments of consecutive lanes with one channel
    // (lanes past the last column form their own and add nothing)
    const int cl = lane < ncols ? c : -1;
    const int cprev = __shfl_up(cl, 1u, 64);
    const uint64_t heads = __builtin_amdgcn_ballot_w64(lane == 0 || cprev != cl);
    const int seg = __popcll(heads & (lane == 63 ? ~0ull : ((2ull << lane) - 1))) - 1;
    const int seg_next = __shfl_down(seg, 1u, 64);
    const bool last = cl >= 0 && (lane == 63 || seg_next != seg);
    // same[j]: the lane 2^j below is in this lane's segment.  The shuffle
    // runs on every lane: a lane that sat out of it would hand 0 to the
    // lane reading it.
    bool same[6];
#pragma unroll
    for (int j = 0; j < 6; ++j) {
        const int below = __shfl_up(seg, (unsigned)(1 << j), 64);
        same[j] = (lane >= (1 << j)) & (below == seg);
    }
    auto seg_sum = [&](W v) {
#pragma unroll
        for (int j = 0; j < 6; ++j) {
            const W u = tl_shfl_up(v, 1 << j);
            v = same[j] ? v + u : v;
        }
        return v;
    };
    W* slot = reinterpret_cast<W*>(a.part) + ((int64_t)blockIdx.x + col / a.S) * (K + 1);
#pragma unroll
    for (int i = 0; i < K; ++i) {
        const W v = seg_sum(gw[i]);
        if (last)
            slot[i] = v;
    }
    const W v = seg_sum(gb);
    if (last)
        slot[K] = v;
}

// dst[j] = src[cbase + t_first + j] for j in [0, n), 0 where the time
// t_first + j lies outside [0, T); the loads go in batches of eight per lane,
// all issued before their LDS writes.  With CHECK, returns (wave-uniform)
// whether some staged float lies outside [lo, hi).
template <int DT, bool CHECK>
__device__ __forceinline__ bool tl_stage_window(const void* src, int64_t cbase, int t_first, int n, int T,
                                                typename TlIO<DT>::V* dst, float lo, float hi)
{
    using V = typename TlIO<DT>::V;
    constexpr int B = 8;
    const int lane = (int)threadIdx.x & 63;
    bool out = false;
    for (int base = 0; base < n; base += 64 * B) {
        V v[B];
#pragma unroll
        for (int q = 0; q < B; ++q) {
            const int j = base + lane + 64 * q;
            const int t = t_first + j;
            v[q] = j < n && t >= 0 && t < T ? TlIO<DT>::ld(src, cbase + t) : V(0);
        }
#pragma unroll
        for (int q = 0; q < B; ++q) {
            const int j = base + lane + 64 * q;
            if (j < n) {
                dst[j] = v[q];
                if constexpr (CHECK && DT != MFPSN_Q8_8) {
                    const int t = t_first + j;
                    out = out | ((t >= 0) & (t < T) & !tl_tap_exact(v[q], lo, hi));
                }
            }
        }
    }
    return CHECK && DT != MFPSN_Q8_8 && __builtin_amdgcn_ballot_w64(out) != 0;
}

// Sum over the 64 lanes, every lane gets it
template <typename W> __device__ __forceinline__ W tl_wave_sum(W v)
{
#pragma unroll
    for (int j = 1; j < 64; j <<= 1) {
        if constexpr (std::is_same_v<W, double>) {
            v += __shfl_xor(v, j, 64);
        } else {
            const int lo = __shfl_xor((int)(uint32_t)v, j, 64);
            const int hi = __shfl_xor((int)(uint32_t)((uint64_t)v >> 32), j, 64);
            v += (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
        }
    }
    return v;
}

// Backward for long columns (T > kTlColsMaxT) in the time-last layout:
// persistent waves over segments of L = a.seg time steps of one column, lane
// = time step, so the taps are the same on every lane.  With P = (k-1) d,
// a segment [t0, t0 + L) stages x over [t0 - P, t0 + L + P) and grad_spikes
// over [t0, t0 + L + P) in the wave's LDS windows (zeros outside [0, T)),
// recomputes H and dH over [t0, t0 + L + P) (the dH its grad_x needs), adds
// the exact products and dH of its own steps to grad_w / grad_b sums, forms
// grad_x over its own steps from the dH window.  A wave takes a contiguous
// run of a.chunk segments in channel-major order and stores its sums to
// its slot of the channel, part[wave + c][k+1], when the channel changes
// and at the end.  The dH of the P steps after a segment is recomputed by
// the next one.
template <int DT, int K>
__global__ __launch_bounds__(kTlWaves * 64) void tl_seg_bwd_kernel(TlBwdArgs a)
{
    using V = typename TlIO<DT>::V;
    constexpr bool kF = DT != MFPSN_Q8_8;
    using W = std::conditional_t<kF, double, int64_t>;
    extern __shared__ uint32_t tl_lds[];
    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6), lane = (int)threadIdx.x & 63;
    const int T = a.T, d = a.d, span = (K - 1) * d, L = a.seg;
    const int xw = L + 2 * span, dw = L + span;
    V* xs = reinterpret_cast<V*>(tl_lds) + (size_t)wave * (xw + dw);
    V* ds = xs + xw;
    // units in channel-major order (c, n, s, segment); wave w takes the
    // contiguous run [w chunk, (w+1) chunk), so its sums stay in registers
    // while the channel stays the same
    const int64_t units = a.M * a.nseg, per_c = units / a.C;
    const int64_t chunk = a.chunk;
    const int64_t wg = (int64_t)blockIdx.x * kTlWaves + wave;
    const int64_t v0 = wg * chunk;
    const int64_t v1 = v0 + chunk < units ? v0 + chunk : units;
    Surrogate sg;
    sg.init(a.sg, a.alpha);
    W* part = reinterpret_cast<W*>(a.part);
    W gw[K], gb = W(0);
#pragma unroll
    for (int i = 0; i < K; ++i)
        gw[i] = W(0);
    TlLaneTaps<DT, K> taps;
    V bias = V(0);
    int cur = -1;  // channel of the sums (wave-uniform)
    auto flush = [&]() {
        if (cur < 0)
            return;
        W* slot = part + (wg + cur) * (K + 1);
#pragma unroll
        for (int i = 0; i < K; ++i) {
            const W v = tl_wave_sum(gw[i]);
            gw[i] = W(0);
            if (lane == 0)
                slot[i] = v;
        }
        const W v = tl_wave_sum(gb);
        gb = W(0);
        if (lane == 0)
            slot[K] = v;
    };
    for (int64_t u = v0; u < v1; ++u) {
        const int c = (int)(u / per_c);
        const int64_t r = u - (int64_t)c * per_c;
        const int64_t ns = r / a.nseg;  // n S + s
        const int t0 = (int)(r - ns * a.nseg) * L;
        const int64_t n = ns / a.S;
        const int64_t col = (n * a.C + c) * a.S + (ns - n * a.S);
        const int64_t cbase = col * (int64_t)T;
        if (c != cur) {
            flush();
            cur = c;
            taps.load(a.sign, a.shift, c, a.shift_lo, a.shift_hi);
            if constexpr (kF)
                bias = ((const float*)a.bias)[c];
            else
                bias = ((const int32_t*)a.bias)[c];
        }
        const bool slow_x = tl_stage_window<DT, true>(a.x, cbase, t0 - span, xw, T, xs, a.fast_lo, a.fast_hi);
        (void)tl_stage_window<DT, false>(a.g, cbase, t0, dw, T, ds, 0.0f, 0.0f);
        wave_lds_sync();

        // H and dH over [t0, t0 + L + P); x of time t - (k-1-i) d is xs[j + i d]
        bool out_dh = false;
        const bool head = t0 < span;  // some tap input before time 0 (zeros in the window)
        auto walk1 = [&](auto exact) {
            constexpr bool EX = decltype(exact)::value;
            for (int j = lane; j < dw; j += 64) {
                const int t = t0 + j;
                if (t >= T)
                    break;
                V acc = V(0);
                if (!EX && head) {
#pragma unroll
                    for (int i = 0; i < K; ++i) {
                        const V sum = acc + taps.template apply<EX>(xs[j + i * d], i);
                        acc = t - (K - 1 - i) * d >= 0 ? sum : acc;
                    }
                } else {
                    acc = taps.start();
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        acc = taps.template accumulate<EX>(acc, xs[j + i * d], i);
                }
                const V h = acc + bias;
                const V dh = delta_h(ds[j], sg_factor(sg, h, a.v_th, a.v_th_q));
                ds[j] = dh;
                if constexpr (kF) {
                    out_dh = out_dh | !tl_tap_exact(dh, a.fast_lo, a.fast_hi);
                }
                if (j < L) {  // this segment's own step
                    gb += (W)dh;
#pragma unroll
                    for (int i = 0; i < K; ++i) {
                        if constexpr (kF)
                            gw[i] = __builtin_fma((double)xs[j + i * d], (double)dh, gw[i]);
                        else
                            gw[i] += (int64_t)xs[j + i * d] * (int64_t)dh;
                    }
                }
            }
        };
        if (slow_x)
            walk1(std::true_type{});
        else
            walk1(std::false_type{});
        const bool slow_dh = kF && __builtin_amdgcn_ballot_w64(out_dh) != 0;
        wave_lds_sync();

        // grad_x over [t0, t0 + L): dH of time t + (k-1-i) d is ds[j + (k-1-i) d]
        const bool tail = t0 + L + span > T;  // some tap input past the end (zeros)
        auto walk2 = [&](auto exact) {
            constexpr bool EX = decltype(exact)::value;
            for (int j = lane; j < L; j += 64) {
                const int t = t0 + j;
                if (t >= T)
                    break;
                V acc = V(0);
                if (!EX && tail) {
#pragma unroll
                    for (int i = 0; i < K; ++i) {
                        const V sum = acc + taps.template apply<EX>(ds[j + (K - 1 - i) * d], i);
                        acc = t + (K - 1 - i) * d < T ? sum : acc;
                    }
                } else {
                    acc = taps.start();
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        acc = taps.template accumulate<EX>(acc, ds[j + (K - 1 - i) * d], i);
                }
                if constexpr (DT == MFPSN_BF16)
                    reinterpret_cast<uint16_t*>(a.grad_x)[cbase + t] = tl_bf16_rne(acc);
                else
                    reinterpret_cast<V*>(a.grad_x)[cbase + t] = acc;
            }
        };
        if (slow_dh)
            walk2(std::true_type{});
        else
            walk2(std::false_type{});
        wave_lds_sync();  // every read of the windows before the next segment's writes
    }
    flush();
}

__global__ void tl_zero_kernel(uint64_t* p, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0;
}

// acc[i][c] = the sum of channel c's slots of sum i, in a fixed order.  The
// channel's groups are g = n C + c, n < ng, each of z consecutive units of
// a sequence cut into pieces of b units (blocks or waves); group g meets
// the pieces first = g z / b .. last = (g z + z - 1) / b, whose slots are
// piece + g.  One wave per (c, i): lane l adds the (n, piece) pairs
// l + 64 j in four interleaved sums, which are added pairwise, then across
// the lanes in a fixed tree.
template <typename W>
__global__ __launch_bounds__(64) void tl_bwd_reduce_kernel(const W* part, W* acc, int32_t C, int32_t k1, int64_t ng,
                                                           int64_t z, int64_t b)
{
    const int c = blockIdx.x, i = blockIdx.y, lane = threadIdx.x;
    const int64_t span = (z + b - 1) / b + 1;  // pieces one group can meet, at most
    const int64_t total = ng * span;
    auto term = [&](int64_t q) -> W {
        if (q >= total)
            return W(0);
        const int64_t n = q / span, j = q - n * span;
        const int64_t g = n * C + c;
        const int64_t first = g * z / b, last = (g * z + z - 1) / b;
        return first + j <= last ? part[(first + j + g) * k1 + i] : W(0);
    };
    W s[4] = {W(0), W(0), W(0), W(0)};
    for (int64_t q = lane; q < total; q += 256) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
            s[u] += term(q + 64 * u);
    }
    const W v = tl_wave_sum((s[0] + s[1]) + (s[2] + s[3]));
    if (lane == 0)
        acc[(int64_t)i * C + c] = v;
}

// Forward for long columns (T > kTlColsMaxT) with histories P = (k-1) d of
// at most kTlBwdMaxSpan steps: persistent waves over segments [t0, t0 + L)
// of one column (L = a.seg), lane = time step, in channel-major runs as in
// tl_seg_bwd_kernel (the taps are loaded again only when the channel
// changes).  A segment stages x over [t0 - P, t0 + L) in the wave's LDS
// window (zeros before time 0), so the input of tap i for step t0 + j is
// xs[j + i d]; only the first segment of a column, whose taps reach before
// time 0, selects the exponent-add terms of those zeros away.
template <int DT, int K>
__global__ __launch_bounds__(kTlWaves * 64) void tl_seg_fwd_kernel(TlArgs a)
{
    using V = typename TlIO<DT>::V;
    constexpr bool kF = DT != MFPSN_Q8_8;
    extern __shared__ uint32_t tl_lds[];
    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6), lane = (int)threadIdx.x & 63;
    const int T = a.T, d = a.d, span = (K - 1) * d, L = a.seg;
    const int xw = L + span;
    V* xs = reinterpret_cast<V*>(tl_lds) + (size_t)wave * xw;
    const int64_t units = a.M * a.nseg, per_c = units / a.C;
    const int64_t nwaves = (int64_t)gridDim.x * kTlWaves;
    const int64_t chunk = (units + nwaves - 1) / nwaves;
    const int64_t v0 = ((int64_t)blockIdx.x * kTlWaves + wave) * chunk;
    const int64_t v1 = v0 + chunk < units ? v0 + chunk : units;
    TlLaneTaps<DT, K> taps;
    V bias = V(0);
    int cur = -1;
    for (int64_t u = v0; u < v1; ++u) {
        const int c = (int)(u / per_c);
        const int64_t r = u - (int64_t)c * per_c;
        const int64_t ns = r / a.nseg;  // n S + s
        const int t0 = (int)(r - ns * a.nseg) * L;
        const int64_t n = ns / a.S;
        const int64_t cbase = ((n * a.C + c) * a.S + (ns - n * a.S)) * (int64_t)T;
        if (c != cur) {
            cur = c;
            taps.load(a.sign, a.shift, c, a.shift_lo, a.shift_hi);
            if constexpr (kF)
                bias = ((const float*)a.bias)[c];
            else
                bias = ((const int32_t*)a.bias)[c];
        }
        const bool slow = tl_stage_window<DT, true>(a.x, cbase, t0 - span, xw, T, xs, a.fast_lo, a.fast_hi);
        wave_lds_sync();
        const bool head = t0 < span;
        auto walk = [&](auto exact) {
            constexpr bool EX = decltype(exact)::value;
            for (int j = lane; j < L; j += 64) {
                const int t = t0 + j;
                if (t >= T)
                    break;
                V acc = V(0);
                if (!EX && head) {
#pragma unroll
                    for (int i = 0; i < K; ++i) {
                        const V sum = acc + taps.template apply<EX>(xs[j + i * d], i);
                        acc = t - (K - 1 - i) * d >= 0 ? sum : acc;
                    }
                } else {
                    acc = taps.start();
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        acc = taps.template accumulate<EX>(acc, xs[j + i * d], i);
                }
                const V h = acc + bias;
                bool fire;
                if constexpr (kF)
                    fire = h >= a.v_th;
                else
                    fire = h >= a.v_th_q;
                a.spikes[cbase + t] = fire ? 1 : 0;
                if (a.h_out != nullptr)
                    reinterpret_cast<V*>(a.h_out)[cbase + t] = h;
            }
        };
        if (slow)
            walk(std::true_type{});
        else
            walk(std::false_type{});
        wave_lds_sync();  // every read of the window before the next segment's writes
    }
}

template <int DT, int K, int NS, bool LDS>
void launch_variant(const TlArgs& a, hipStream_t st)
{
    constexpr int kW = 64 * NS;
    auto kern = tl_fwd_kernel<DT, K, NS, LDS>;
    const size_t lds = LDS ? (size_t)kTlWaves * (kW + a.halo) * 4 : 0;
    // persistent grid: every resident block slot of the device, at most one
    // segment per wave
    static int resident = 0, cus = 0;
    static size_t resident_lds = (size_t)-1;
    if (resident == 0 || resident_lds != lds) {
        int dev = 0, nb = 0;
        (void)hipGetDevice(&dev);
        (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kern, kTlWaves * 64, lds);
        resident = nb > 0 ? nb : 1;
        resident_lds = lds;
    }
    const int64_t units = a.M * a.nseg;
    int64_t blocks = (units + kTlWaves - 1) / kTlWaves;
    const int64_t cap = (int64_t)resident * (cus > 0 ? cus : 1);
    blocks = blocks < cap ? blocks : cap;
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kTlWaves * 64), lds, st, a);
}

template <int DT, int K>
void launch_k(const TlArgs& a, hipStream_t st)
{
    if (a.T <= kTlColsMaxT) {
        const size_t lds = (tl_tile_bytes<DT>(a.T) + 15) / 16 * 16 + (size_t)64 * a.T;
        const int64_t blocks = (a.M + 63) / 64;
        auto kern = tl_cols_kernel<DT, K>;
        hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(64), lds, st, a);
        return;
    }
    if (a.seg > 0) {  // histories of at most kTlBwdMaxSpan steps
        const size_t lds = (size_t)kTlWaves * ((size_t)a.seg + (size_t)(K - 1) * a.d) * 4;
        auto kern = tl_seg_fwd_kernel<DT, K>;
        int dev = 0, nb = 0, cus = 0;
        (void)hipGetDevice(&dev);
        (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kern, kTlWaves * 64, lds);
        const int64_t units = a.M * a.nseg;
        int64_t blocks = (units + kTlWaves - 1) / kTlWaves;
        const int64_t cap = (int64_t)(nb > 0 ? nb : 1) * (cus > 0 ? cus : 1);
        blocks = blocks < cap ? blocks : cap;
        hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kTlWaves * 64), lds, st, a);
        return;
    }
    const bool lds = a.halo > 0 || (K - 1) * a.d == 0;
    const bool short_steps = a.steps_per_lane == 1;
    if (lds)
        short_steps ? launch_variant<DT, K, 1, true>(a, st) : launch_variant<DT, K, 4, true>(a, st);
    else
        short_steps ? launch_variant<DT, K, 1, false>(a, st) : launch_variant<DT, K, 4, false>(a, st);
}
template <int DT, int... Ks>
void dispatch_k(const TlArgs& a, hipStream_t st, std::integer_sequence<int, Ks...>)
{
    (void)((a.k == Ks + 1 ? (launch_k<DT, Ks + 1>(a, st), true) : false) || ...);
}

template <int DT, int K>
int64_t launch_bwd_k(const TlBwdArgs& a, hipStream_t st)
{
    if (a.T <= kTlColsMaxT) {
        const size_t lds = 2 * tl_tile_bytes<DT>(a.T);
        const int64_t blocks = (a.M + 63) / 64;
        auto kern = tl_cols_bwd_kernel<DT, K>;
        hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(64), lds, st, a);
        return 64;
    }
    // persistent grid: every resident block slot (at most kTlSegMaxBlocks,
    // which bounds the slots), at most one segment per wave
    const int span = (K - 1) * a.d;
    const size_t lds = (size_t)kTlWaves * (2 * (size_t)a.seg + 3 * (size_t)span) * 4;
    auto kern = tl_seg_bwd_kernel<DT, K>;
    int dev = 0, nb = 0, cus = 0;
    (void)hipGetDevice(&dev);
    (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kern, kTlWaves * 64, lds);
    const int64_t units = a.M * a.nseg;
    int64_t blocks = (units + kTlWaves - 1) / kTlWaves;
    const int64_t cap = (int64_t)(nb > 0 ? nb : 1) * (cus > 0 ? cus : 1);
    blocks = blocks < cap ? blocks : cap;
    blocks = blocks < kTlSegMaxBlocks ? blocks : kTlSegMaxBlocks;
    TlBwdArgs b = a;
    const int64_t nwaves = blocks * kTlWaves;
    b.chunk = (units + nwaves - 1) / nwaves;
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kTlWaves * 64), lds, st, b);
    return b.chunk;
}
template <int DT, int... Ks>
int64_t dispatch_bwd_k(const TlBwdArgs& a, hipStream_t st, std::integer_sequence<int, Ks...>)
{
    int64_t piece = 0;
    (void)((a.k == Ks + 1 ? (piece = launch_bwd_k<DT, Ks + 1>(a, st), true) : false) || ...);
    return piece;
}

}  // namespace

// Every storage type's kernels are compiled in a translation unit of their
// own (MFPSN_TL_DTYPE = 0, 1, 2); the unit without it holds the dispatch.
#if defined(MFPSN_TL_DTYPE)
using TlKs = std::make_integer_sequence<int, MFPSN_MAX_K>;
#if MFPSN_TL_DTYPE == 0
void tl_forward_f32(const TlArgs& a, hipStream_t st) { dispatch_k<MFPSN_F32>(a, st, TlKs{}); }
int64_t tl_backward_f32(const TlBwdArgs& a, hipStream_t st) { return dispatch_bwd_k<MFPSN_F32>(a, st, TlKs{}); }
#elif MFPSN_TL_DTYPE == 1
void tl_forward_bf16(const TlArgs& a, hipStream_t st) { dispatch_k<MFPSN_BF16>(a, st, TlKs{}); }
int64_t tl_backward_bf16(const TlBwdArgs& a, hipStream_t st) { return dispatch_bwd_k<MFPSN_BF16>(a, st, TlKs{}); }
#else
void tl_forward_q88(const TlArgs& a, hipStream_t st) { dispatch_k<MFPSN_Q8_8>(a, st, TlKs{}); }
int64_t tl_backward_q88(const TlBwdArgs& a, hipStream_t st) { return dispatch_bwd_k<MFPSN_Q8_8>(a, st, TlKs{}); }
#endif
#else
hipError_t launch_forward_time_last(const TlArgs& a, int dtype, hipStream_t st)
{
    if (a.M == 0 || a.T == 0)
        return hipSuccess;
    switch (dtype) {
    case MFPSN_F32: tl_forward_f32(a, st); break;
    case MFPSN_BF16: tl_forward_bf16(a, st); break;
    default: tl_forward_q88(a, st); break;
    }
    return hipGetLastError();
}

hipError_t launch_backward_time_last(const TlBwdArgs& a, int dtype, hipStream_t st)
{
    const int64_t n = (int64_t)(a.k + 1) * a.C;
    if (n == 0)
        return hipSuccess;
    if (a.M == 0 || a.T == 0) {
        const int64_t blocks = (n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024;
        hipLaunchKernelGGL(tl_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, st, (uint64_t*)a.acc, n);
        return hipGetLastError();
    }
    int64_t piece = 0;
    switch (dtype) {
    case MFPSN_F32: piece = tl_backward_f32(a, st); break;
    case MFPSN_BF16: piece = tl_backward_bf16(a, st); break;
    default: piece = tl_backward_q88(a, st); break;
    }
    // groups: the (n, c) rows of S columns, or the channels' runs of segments
    const bool cols = a.T <= kTlColsMaxT;
    const int64_t ng = cols ? a.M / ((int64_t)a.C * a.S) : 1;
    const int64_t z = cols ? (int64_t)a.S : a.M / a.C * a.nseg;
    const dim3 grid((unsigned)a.C, (unsigned)(a.k + 1));
    if (dtype == MFPSN_Q8_8)
        hipLaunchKernelGGL(tl_bwd_reduce_kernel<int64_t>, grid, dim3(64), 0, st, (const int64_t*)a.part,
                           (int64_t*)a.acc, a.C, a.k + 1, ng, z, piece);
    else
        hipLaunchKernelGGL(tl_bwd_reduce_kernel<double>, grid, dim3(64), 0, st, (const double*)a.part,
                           (double*)a.acc, a.C, a.k + 1, ng, z, piece);
    return hipGetLastError();
}
#endif

}  // namespace mfpsn
