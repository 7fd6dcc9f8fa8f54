"""Oracle for the mul-free channel-wise PSN training step (arXiv 2501.14490).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It wraps the
plain single-threaded C implementation in ``mfpsn_oracle.c`` (which shares no
code with the HIP library) and adds numpy marshalling.  Every function states
the passage of the paper it follows in the C source.

Functions whose results are pinned, and by what (see ``tests/test_oracle_pins.py``
and ``tests/test_golden.py``):
  quantize        exact rational arithmetic (Fraction) around 2^(m+1/2)
  quantizer_grad  Eq. ste_q's factor times |W| is |Wq| (exact rational check),
                  power-of-two weights are fixed points, evenness in W
  forward_*       k=1 closed form, np.convolve (sliding PSN), dense Toeplitz
                  matrix of App. A.2, causality, time-shift, zero input,
                  power-of-two scaling, Fraction brute force, the op counts of
                  Table "params and shape" / Table "energy"; per-channel
                  thresholds: equal values reproduce the shared threshold bit
                  for bit, each channel equals its own scalar run, firing at
                  equality
  backward_*      transposed Toeplitz, adjoint identity, finite differences
                  of the smoothed loss (also in the per-channel thresholds:
                  grad_vth = -sum dH), exact big-integer sums (Q8.8)
  surrogate, exp  closed forms at 0, symmetry, unit integral, 2-ulp bound
                  against double exp
  sawtooth        the printed sequence and receptive-field example of Sec. 4.1
  bn_forward_stats, bn_backward
                  numpy mean / biased variance of the latent convolution; the
                  fusion identity s*(W*x) + (beta - s*mu) = BN(W*x); central
                  finite differences of a smooth version of the whole fused
                  step (quantizer taken as identity, Heaviside as a sigmoid)
  stream_forward  the (pinned) whole-sequence forward, bit for bit, from a
                  history ring that starts as garbage; the exact receptive
                  field (k-1)d+1 that sizes the ring
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mfpsn_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liborc.so")
_lock = threading.Lock()
_lib = None

SG_SIGMOID, SG_ATAN, SG_RATIONAL = 0, 1, 2
SURROGATES = {"sigmoid": SG_SIGMOID, "atan": SG_ATAN, "arctan": SG_ATAN, "rational": SG_RATIONAL}

GCC_FLAGS = ["-O2", "-ffp-contract=off", "-fno-fast-math", "-fno-builtin", "-std=c11",
             "-Wall", "-Wextra", "-shared", "-fPIC"]


def build(force: bool = False) -> str:
    """Compile the oracle with gcc into ``oracle/liborc.so`` (IEEE single and
    double arithmetic, no FMA contraction)."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", *GCC_FLAGS, "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is None:
            lib = ctypes.CDLL(build())
            P = ctypes.c_void_p
            i32, i64, f32 = ctypes.c_int, ctypes.c_int64, ctypes.c_float
            lib.orc_exp.argtypes = [f32]
            lib.orc_exp.restype = f32
            lib.orc_surrogate.argtypes = [i32, f32, f32]
            lib.orc_surrogate.restype = f32
            lib.orc_surrogate_q15.argtypes = [i32, f32, ctypes.c_int32]
            lib.orc_surrogate_q15.restype = ctypes.c_int32
            lib.orc_f32_to_bf16.argtypes = [f32]
            lib.orc_f32_to_bf16.restype = ctypes.c_uint16
            lib.orc_quantize.argtypes = [P, i64, i32, i32, P, P]
            lib.orc_quantize.restype = None
            geo = [i32] * 6  # T N C S k d
            lib.orc_forward_f32.argtypes = [P, *geo, P, P, i32, i32, P, f32, P, P, P, P]
            lib.orc_forward_f32.restype = None
            lib.orc_forward_q88.argtypes = [P, *geo, P, P, i32, i32, P, ctypes.c_int32, P, P, P, P]
            lib.orc_forward_q88.restype = None
            lib.orc_backward_f32.argtypes = [P, P, *geo, P, P, i32, i32, P, f32, P, i32, f32, P, P, P, P, P, P]
            lib.orc_backward_f32.restype = None
            lib.orc_backward_q88.argtypes = [P, P, *geo, P, P, i32, i32, P, ctypes.c_int32, P, i32, f32,
                                             P, P, P, P, P, P]
            lib.orc_backward_q88.restype = None
            lib.orc_bn_forward_stats.argtypes = [P, *geo, P, P, P, f32, P, P, P, P]
            lib.orc_bn_forward_stats.restype = None
            lib.orc_bn_backward.argtypes = [P, *geo, P, P, f32, P, P, P, P, P, P, P, P]
            lib.orc_bn_backward.restype = None
            lib.orc_quantizer_grad.argtypes = [P, P, i32, i32, P, i64, i32, P]
            lib.orc_quantizer_grad.restype = None
            lib.orc_stream_step_f32.argtypes = [P, i32, i32, i32, i32, i32, i64, P, P, P, i32, i32, P, f32,
                                                P, P]
            lib.orc_stream_step_f32.restype = None
            lib.orc_stream_step_q88.argtypes = [P, i32, i32, i32, i32, i32, i64, P, P, P, i32, i32, P,
                                                ctypes.c_int32, P, P]
            lib.orc_stream_step_q88.restype = None
            lib.orc_sawtooth_dilation.argtypes = [i32, i32]
            lib.orc_sawtooth_dilation.restype = i32
            _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a


def _geometry(x: np.ndarray):
    """x is [T, N, C, *spatial]; returns T, N, C, S."""
    if x.ndim < 3:
        raise ValueError("x must be [T, N, C, ...]")
    T, N, C = x.shape[:3]
    S = int(np.prod(x.shape[3:], dtype=np.int64)) if x.ndim > 3 else 1
    return int(T), int(N), int(C), S


def _sg(kind) -> int:
    return SURROGATES[kind] if isinstance(kind, str) else int(kind)


# ---------------------------------------------------------------------------
# scalar helpers
# ---------------------------------------------------------------------------
def exp_f32(y: float) -> np.float32:
    return np.float32(_load().orc_exp(float(y)))


def surrogate(kind, alpha: float, u) -> np.ndarray:
    lib = _load()
    k = _sg(kind)
    u = np.asarray(u, dtype=np.float32)
    out = np.array([lib.orc_surrogate(k, float(alpha), float(v)) for v in u.ravel()], dtype=np.float32)
    return out.reshape(u.shape)


def surrogate_q15(kind, alpha: float, u) -> np.ndarray:
    lib = _load()
    k = _sg(kind)
    u = np.asarray(u, dtype=np.int64)
    out = np.array([lib.orc_surrogate_q15(k, float(alpha), int(v)) for v in u.ravel()], dtype=np.int32)
    return out.reshape(u.shape)


def f32_to_bf16_bits(a) -> np.ndarray:
    lib = _load()
    a = np.asarray(a, dtype=np.float32)
    out = np.array([lib.orc_f32_to_bf16(float(v)) for v in a.ravel()], dtype=np.uint16)
    return out.reshape(a.shape)


def bf16_bits_to_f32(b) -> np.ndarray:
    b = np.asarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def sawtooth_dilation(layer: int, period: int) -> int:
    return int(_load().orc_sawtooth_dilation(int(layer), int(period)))


# ---------------------------------------------------------------------------
# quantizer
# ---------------------------------------------------------------------------
def quantize(w, shift_lo: int, shift_hi: int):
    """Q(W) = sign(W) 2^round(log2|W|) (Eq. round_w) -> (sign int8, shift int8)."""
    w = _c(w, np.float32)
    sign = np.empty(w.shape, np.int8)
    shift = np.empty(w.shape, np.int8)
    _load().orc_quantize(_ptr(w), w.size, int(shift_lo), int(shift_hi), _ptr(sign), _ptr(shift))
    return sign, shift


def bn_forward_stats(x, w, gamma, beta, eps: float, k: int, d: int):
    """App. C, training mode: statistics of the latent-weight convolution and
    the fused weight and bias.  Returns dict w_f, b_f (float32), aux [C, 4]
    (mu, var, s, 1/sqrt(var+eps), float64), stats [C, 2] (sum, sum of squares)."""
    x = _c(x, np.float32)
    T, N, C, S = _geometry(x)
    w = _c(w, np.float32).reshape(C, k)
    gamma = _c(gamma, np.float32).reshape(C)
    beta = _c(beta, np.float32).reshape(C)
    w_f = np.empty((C, k), np.float32)
    b_f = np.empty(C, np.float32)
    aux = np.empty((C, 4), np.float64)
    stats = np.empty((C, 2), np.float64)
    _load().orc_bn_forward_stats(_ptr(x), T, N, C, S, int(k), int(d), _ptr(w), _ptr(gamma), _ptr(beta),
                                 float(eps), _ptr(w_f), _ptr(b_f), _ptr(aux), _ptr(stats))
    return {"w_f": w_f, "b_f": b_f, "aux": aux, "stats": stats}


def bn_backward(x, w, gamma, eps: float, aux, grad_wf, grad_bf, grad_xq, k: int, d: int):
    """Backward of the fusion and the batch statistics (App. C): returns dict
    grad_x (grad_xq plus the statistics path), grad_w, grad_gamma, grad_beta,
    all float64."""
    x = _c(x, np.float32)
    T, N, C, S = _geometry(x)
    w = _c(w, np.float32).reshape(C, k)
    gamma = _c(gamma, np.float32).reshape(C)
    aux = _c(aux, np.float64).reshape(C, 4)
    gwf = _c(grad_wf, np.float64).reshape(C, k)
    gbf = _c(grad_bf, np.float64).reshape(C)
    gxq = _c(grad_xq, np.float64).reshape(x.shape)
    gx = np.empty(x.shape, np.float64)
    gw = np.empty((C, k), np.float64)
    gg = np.empty(C, np.float64)
    gb = np.empty(C, np.float64)
    _load().orc_bn_backward(_ptr(x), T, N, C, S, int(k), int(d), _ptr(w), _ptr(gamma), float(eps), _ptr(aux),
                            _ptr(gwf), _ptr(gbf), _ptr(gxq), _ptr(gx), _ptr(gw), _ptr(gg), _ptr(gb))
    return {"grad_x": gx, "grad_w": gw, "grad_gamma": gg, "grad_beta": gb}


def quantizer_grad(w, shift, grad_wq, mode: int, shift_lo: int, shift_hi: int) -> np.ndarray:
    """grad of the latent weight: mode 0 whole-quantizer STE (identity),
    mode 1 round-only STE (grad_wq * 2^-shift / |w|, Eq. ste_q)."""
    w = _c(w, np.float32)
    shift = _c(shift, np.int8).reshape(w.shape)
    g = _c(grad_wq, np.float32).reshape(w.shape)
    out = np.empty(w.shape, np.float32)
    _load().orc_quantizer_grad(_ptr(w), _ptr(shift), int(shift_lo), int(shift_hi), _ptr(g), int(w.size),
                               int(mode), _ptr(out))
    return out


# ---------------------------------------------------------------------------
# forward
# ---------------------------------------------------------------------------
def _thresholds(v_th_c, C, dtype):
    """Per-channel thresholds [C] as a contiguous array, or None (the scalar
    threshold applies to every channel)."""
    if v_th_c is None:
        return None
    return _c(v_th_c, dtype).reshape(C)


def forward_f32(x, sign, shift, bias, k: int, d: int, v_th: float, shift_lo: int = -127,
                shift_hi: int = 127, with_tap_count: bool = False, v_th_c=None):
    """Float potentials H and spikes for x [T, N, C, ...] float32.  v_th_c:
    optional per-channel thresholds [C] (then v_th is not used)."""
    x = _c(x, np.float32)
    T, N, C, S = _geometry(x)
    sign = _c(sign, np.int8).reshape(C, k)
    shift = _c(shift, np.int8).reshape(C, k)
    bias = _c(bias, np.float32).reshape(C)
    vc = _thresholds(v_th_c, C, np.float32)
    H = np.empty(x.shape, np.float32)
    spk = np.empty(x.shape, np.uint8)
    taps = ctypes.c_int64(0)
    _load().orc_forward_f32(_ptr(x), T, N, C, S, int(k), int(d), _ptr(sign), _ptr(shift),
                            int(shift_lo), int(shift_hi), _ptr(bias), float(v_th),
                            None if vc is None else _ptr(vc), _ptr(H), _ptr(spk), ctypes.byref(taps))
    if with_tap_count:
        return H, spk, int(taps.value)
    return H, spk


def forward_q88(x, sign, shift, bias, k: int, d: int, v_th: int, shift_lo: int = 0,
                shift_hi: int = 31, with_tap_count: bool = False, v_th_c=None):
    """Q8.8 potentials H (int32) and spikes for x [T, N, C, ...] int16.
    v_th_c: optional per-channel Q8.8 thresholds [C] (int32)."""
    x = _c(x, np.int16)
    T, N, C, S = _geometry(x)
    sign = _c(sign, np.int8).reshape(C, k)
    shift = _c(shift, np.int8).reshape(C, k)
    bias = _c(bias, np.int32).reshape(C)
    vc = _thresholds(v_th_c, C, np.int32)
    H = np.empty(x.shape, np.int32)
    spk = np.empty(x.shape, np.uint8)
    taps = ctypes.c_int64(0)
    _load().orc_forward_q88(_ptr(x), T, N, C, S, int(k), int(d), _ptr(sign), _ptr(shift),
                            int(shift_lo), int(shift_hi), _ptr(bias), int(v_th),
                            None if vc is None else _ptr(vc), _ptr(H), _ptr(spk), ctypes.byref(taps))
    if with_tap_count:
        return H, spk, int(taps.value)
    return H, spk


def stream_ring_steps(k: int, d: int) -> int:
    """History slots of the step-by-step neuron: its receptive field (k-1)d+1."""
    return (int(k) - 1) * int(d) + 1


def stream_forward(x, sign, shift, bias, k: int, d: int, v_th, dtype: str = "f32", shift_lo: int = -127,
                   shift_hi: int = 127):
    """Runs the step-by-step neuron (orc_stream_step_*) over x [T, N, C, ...]
    one time step per call, with a history ring of stream_ring_steps(k, d)
    slots; returns H and spikes stacked over time.  dtype "f32" (float32 x),
    "bf16" (uint16 bit patterns, arithmetic in float) or "q8_8" (int16 x)."""
    lib = _load()
    if dtype == "bf16":
        x = bf16_bits_to_f32(x)
        dtype = "f32"
    q = dtype == "q8_8"
    x = _c(x, np.int16 if q else np.float32)
    T, N, C, S = _geometry(x)
    sign = _c(sign, np.int8).reshape(C, k)
    shift = _c(shift, np.int8).reshape(C, k)
    bias = _c(bias, np.int32 if q else np.float32).reshape(C)
    R = stream_ring_steps(k, d)
    # the ring starts with garbage: no step may read a slot before writing it
    hist = np.full((R,) + x.shape[1:], 0x5A5A if q else np.nan, dtype=np.int16 if q else np.float32)
    H = np.empty(x.shape, np.int32 if q else np.float32)
    spk = np.empty(x.shape, np.uint8)
    for t in range(T):
        xt = np.ascontiguousarray(x[t])
        Ht = np.empty(x.shape[1:], H.dtype)
        st = np.empty(x.shape[1:], np.uint8)
        if q:
            lib.orc_stream_step_q88(_ptr(xt), N, C, S, int(k), int(d), t, _ptr(hist), _ptr(sign), _ptr(shift),
                                    int(shift_lo), int(shift_hi), _ptr(bias), int(v_th), _ptr(Ht), _ptr(st))
        else:
            lib.orc_stream_step_f32(_ptr(xt), N, C, S, int(k), int(d), t, _ptr(hist), _ptr(sign), _ptr(shift),
                                    int(shift_lo), int(shift_hi), _ptr(bias), float(v_th), _ptr(Ht), _ptr(st))
        H[t] = Ht
        spk[t] = st
    return H, spk


# ---------------------------------------------------------------------------
# backward
# ---------------------------------------------------------------------------
def backward_f32(x, g, sign, shift, bias, k: int, d: int, v_th: float, surrogate_kind="sigmoid",
                 alpha: float = 4.0, shift_lo: int = -127, shift_hi: int = 127, v_th_c=None):
    """Returns dict with H, dH, grad_x (float32), grad_w, grad_b, grad_vth
    (float64 sums).  v_th_c: optional per-channel thresholds [C]."""
    x = _c(x, np.float32)
    g = _c(g, np.float32)
    T, N, C, S = _geometry(x)
    assert g.shape == x.shape
    sign = _c(sign, np.int8).reshape(C, k)
    shift = _c(shift, np.int8).reshape(C, k)
    bias = _c(bias, np.float32).reshape(C)
    vc = _thresholds(v_th_c, C, np.float32)
    H = np.empty(x.shape, np.float32)
    dH = np.empty(x.shape, np.float32)
    gx = np.empty(x.shape, np.float32)
    gw = np.empty((C, k), np.float64)
    gb = np.empty((C,), np.float64)
    gv = np.empty((C,), np.float64)
    _load().orc_backward_f32(_ptr(x), _ptr(g), T, N, C, S, int(k), int(d), _ptr(sign), _ptr(shift),
                             int(shift_lo), int(shift_hi), _ptr(bias), float(v_th),
                             None if vc is None else _ptr(vc), _sg(surrogate_kind), float(alpha), _ptr(H),
                             _ptr(dH), _ptr(gx), _ptr(gw), _ptr(gb), _ptr(gv))
    return {"H": H, "dH": dH, "grad_x": gx, "grad_w": gw, "grad_b": gb, "grad_vth": gv}


def backward_q88(x, g, sign, shift, bias, k: int, d: int, v_th: int, surrogate_kind="sigmoid",
                 alpha: float = 4.0, shift_lo: int = 0, shift_hi: int = 31, v_th_c=None):
    """Returns dict with H, dH, grad_x (int32), grad_w, grad_b, grad_vth
    (int64).  v_th_c: optional per-channel Q8.8 thresholds [C] (int32)."""
    x = _c(x, np.int16)
    g = _c(g, np.int16)
    T, N, C, S = _geometry(x)
    assert g.shape == x.shape
    sign = _c(sign, np.int8).reshape(C, k)
    shift = _c(shift, np.int8).reshape(C, k)
    bias = _c(bias, np.int32).reshape(C)
    vc = _thresholds(v_th_c, C, np.int32)
    H = np.empty(x.shape, np.int32)
    dH = np.empty(x.shape, np.int32)
    gx = np.empty(x.shape, np.int32)
    gw = np.empty((C, k), np.int64)
    gb = np.empty((C,), np.int64)
    gv = np.empty((C,), np.int64)
    _load().orc_backward_q88(_ptr(x), _ptr(g), T, N, C, S, int(k), int(d), _ptr(sign), _ptr(shift),
                             int(shift_lo), int(shift_hi), _ptr(bias), int(v_th),
                             None if vc is None else _ptr(vc), _sg(surrogate_kind), float(alpha), _ptr(H),
                             _ptr(dH), _ptr(gx), _ptr(gw), _ptr(gb), _ptr(gv))
    return {"H": H, "dH": dH, "grad_x": gx, "grad_w": gw, "grad_b": gb, "grad_vth": gv}


# bf16 storage: inputs are bfloat16 bit patterns (uint16); they widen exactly
# to float32 and follow the float path; grad_x is rounded to bfloat16 (RNE).
def forward_bf16(x_bits, sign, shift, bias, k, d, v_th, **kw):
    return forward_f32(bf16_bits_to_f32(x_bits), sign, shift, bias, k, d, v_th, **kw)


def backward_bf16(x_bits, g_bits, sign, shift, bias, k, d, v_th, **kw):
    out = backward_f32(bf16_bits_to_f32(x_bits), bf16_bits_to_f32(g_bits), sign, shift, bias, k, d,
                       v_th, **kw)
    out["grad_x_bits"] = f32_to_bf16_bits_vec(out["grad_x"])
    return out


def f32_to_bf16_bits_vec(a) -> np.ndarray:
    """Vectorised round-to-nearest-even float32 -> bfloat16 bits; the scalar
    C routine orc_f32_to_bf16 pins it in the tests."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    b = a.view(np.uint32).astype(np.uint64)
    nan = ((b & 0x7F800000) == 0x7F800000) & ((b & 0x007FFFFF) != 0)
    r = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)
    r[nan] = ((b[nan] >> 16) | 0x40).astype(np.uint16)
    return r.reshape(a.shape)
