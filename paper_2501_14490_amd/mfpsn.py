"""Python binding of libmfpsn.so (declared in include/mfpsn.h).

Argument marshalling only: every step of the neuron's training step runs in
the library's HIP kernels.  PyTorch supplies device memory and the stream.
Importing this module loads the library and raises if it is missing (build
it with ``python -m paper_2501_14490_amd.build``); there is no fallback.

The functions named like the C entry points take tensors for the C
pointers; ``forward``/``backward``/``quantize`` additionally allocate their
outputs, and ``MfPSNFunction`` wires quantize -> forward -> backward into
autograd with the straight-through estimator of the quantizer (Sec. 4.2).
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmfpsn.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2501_14490_amd.build`")

_lib = ctypes.CDLL(LIB_PATH)

MFPSN_OK = 0
MFPSN_F32, MFPSN_BF16, MFPSN_Q8_8 = 0, 1, 2
MFPSN_SG_SIGMOID, MFPSN_SG_ATAN, MFPSN_SG_RATIONAL = 0, 1, 2
MFPSN_STE_WHOLE, MFPSN_STE_ROUND = 0, 1
STE = {"whole": MFPSN_STE_WHOLE, "round": MFPSN_STE_ROUND}
MFPSN_MAX_K = 32

DTYPES = {"f32": MFPSN_F32, "bf16": MFPSN_BF16, "q8_8": MFPSN_Q8_8}
SURROGATES = {"sigmoid": MFPSN_SG_SIGMOID, "atan": MFPSN_SG_ATAN, "arctan": MFPSN_SG_ATAN,
              "rational": MFPSN_SG_RATIONAL}
STORAGE = {MFPSN_F32: torch.float32, MFPSN_BF16: torch.bfloat16, MFPSN_Q8_8: torch.int16}
GRAD_X = {MFPSN_F32: torch.float32, MFPSN_BF16: torch.bfloat16, MFPSN_Q8_8: torch.int32}
H_OUT = {MFPSN_F32: torch.float32, MFPSN_BF16: torch.float32, MFPSN_Q8_8: torch.int32}
SG_OUT = H_OUT
BIAS = {MFPSN_F32: torch.float32, MFPSN_BF16: torch.float32, MFPSN_Q8_8: torch.int32}
GRAD_WB = {MFPSN_F32: torch.float32, MFPSN_BF16: torch.float32, MFPSN_Q8_8: torch.int64}


class MfpsnDesc(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("N", ctypes.c_int32), ("C", ctypes.c_int32),
                ("S", ctypes.c_int32), ("k", ctypes.c_int32), ("dilation", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("surrogate", ctypes.c_int32), ("alpha", ctypes.c_float),
                ("v_th", ctypes.c_float), ("v_th_q", ctypes.c_int32), ("shift_lo", ctypes.c_int32),
                ("shift_hi", ctypes.c_int32)]


_P = ctypes.c_void_p
_DP = ctypes.POINTER(MfpsnDesc)
_lib.mfpsn_forward.argtypes = [_DP, _P, _P, _P, _P, _P, _P, _P, _P, _P]
_lib.mfpsn_forward.restype = ctypes.c_int
_lib.mfpsn_backward_workspace_size.argtypes = [_DP, ctypes.POINTER(ctypes.c_size_t)]
_lib.mfpsn_backward_workspace_size.restype = ctypes.c_int
_lib.mfpsn_backward.argtypes = [_DP, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]
_lib.mfpsn_backward.restype = ctypes.c_int
_lib.mfpsn_backward_no_alloc.argtypes = [_DP, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]
_lib.mfpsn_backward_no_alloc.restype = ctypes.c_int
_lib.mfpsn_quantize_weights.argtypes = [_P, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, _P, _P, _P]
_lib.mfpsn_quantize_weights.restype = ctypes.c_int
_lib.mfpsn_bn_workspace_size.argtypes = [_DP, ctypes.POINTER(ctypes.c_size_t)]
_lib.mfpsn_bn_workspace_size.restype = ctypes.c_int
_lib.mfpsn_bn_forward_stats.argtypes = [_DP, _P, _P, _P, _P, ctypes.c_float, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]
_lib.mfpsn_bn_forward_stats.restype = ctypes.c_int
_lib.mfpsn_bn_backward.argtypes = [_DP, _P, _P, _P, ctypes.c_float, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]
_lib.mfpsn_bn_backward.restype = ctypes.c_int
_lib.mfpsn_quantizer_grad.argtypes = [_P, _P, ctypes.c_int32, ctypes.c_int32, _P, ctypes.c_int64, ctypes.c_int32, _P,
                                      _P]
_lib.mfpsn_quantizer_grad.restype = ctypes.c_int
_lib.mfpsn_stream_ring_bytes.argtypes = [_DP, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_size_t)]
_lib.mfpsn_stream_ring_bytes.restype = ctypes.c_int
_lib.mfpsn_stream_step.argtypes = [_DP, ctypes.c_int64, _P, _P, _P, _P, _P, _P, _P, _P]
_lib.mfpsn_stream_step.restype = ctypes.c_int
_lib.mfpsn_forward_time_last.argtypes = [_DP, _P, _P, _P, _P, _P, _P, _P]
_lib.mfpsn_forward_time_last.restype = ctypes.c_int
_lib.mfpsn_backward_time_last_workspace_size.argtypes = [_DP, ctypes.POINTER(ctypes.c_size_t)]
_lib.mfpsn_backward_time_last_workspace_size.restype = ctypes.c_int
_lib.mfpsn_backward_time_last.argtypes = [_DP, _P, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]
_lib.mfpsn_backward_time_last.restype = ctypes.c_int
_lib.mfpsn_spikes_to_input.argtypes = [_P, ctypes.c_int64, ctypes.c_int32, _P, _P]
_lib.mfpsn_spikes_to_input.restype = ctypes.c_int
_lib.mfpsn_sawtooth_dilation.argtypes = [ctypes.c_int32, ctypes.c_int32]
_lib.mfpsn_sawtooth_dilation.restype = ctypes.c_int32
_lib.mfpsn_status_string.argtypes = [ctypes.c_int]
_lib.mfpsn_status_string.restype = ctypes.c_char_p
_lib.mfpsn_abi_version.argtypes = []
_lib.mfpsn_abi_version.restype = ctypes.c_int32


class MfpsnError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {mfpsn_status_string(status)} (status {status})")
        self.status = status


def _check(status: int, where: str):
    if status != MFPSN_OK:
        raise MfpsnError(status, where)


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else None
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def make_desc(shape, k: int, dilation: int, dtype="f32", surrogate="sigmoid", alpha: float = 4.0,
              v_th: float = 1.0, v_th_q: int = 256, shift_lo: int = 0, shift_hi: int = 7) -> MfpsnDesc:
    """Descriptor for x of shape [T, N, C, *spatial]."""
    T, N, C = (int(v) for v in shape[:3])
    S = 1
    for v in shape[3:]:
        S *= int(v)
    dt = DTYPES[dtype] if isinstance(dtype, str) else int(dtype)
    sg = SURROGATES[surrogate] if isinstance(surrogate, str) else int(surrogate)
    return MfpsnDesc(T, N, C, S, int(k), int(dilation), dt, sg, float(alpha), float(v_th), int(v_th_q),
                     int(shift_lo), int(shift_hi))


# ---------------------------------------------------------------------------
# the C entry points
# ---------------------------------------------------------------------------
def mfpsn_abi_version() -> int:
    return int(_lib.mfpsn_abi_version())


def mfpsn_status_string(status: int) -> str:
    return _lib.mfpsn_status_string(int(status)).decode()


def mfpsn_sawtooth_dilation(layer: int, period: int) -> int:
    return int(_lib.mfpsn_sawtooth_dilation(int(layer), int(period)))


def mfpsn_forward(desc: MfpsnDesc, x, sign, shift, bias, v_th_c, spikes, h_out=None, sg_out=None,
                  stream=None) -> None:
    _check(_lib.mfpsn_forward(ctypes.byref(desc), _ptr(x), _ptr(sign), _ptr(shift), _ptr(bias), _ptr(v_th_c),
                              _ptr(spikes), _ptr(h_out), _ptr(sg_out), _stream(stream)), "mfpsn_forward")


def mfpsn_backward_workspace_size(desc: MfpsnDesc) -> int:
    n = ctypes.c_size_t(0)
    _check(_lib.mfpsn_backward_workspace_size(ctypes.byref(desc), ctypes.byref(n)),
           "mfpsn_backward_workspace_size")
    return int(n.value)


def mfpsn_backward(desc: MfpsnDesc, x, grad_spikes, h, sg, sign, shift, bias, v_th_c, grad_x, grad_w, grad_b,
                   grad_vth, workspace, workspace_bytes=None, stream=None) -> None:
    if workspace_bytes is None:
        workspace_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(_lib.mfpsn_backward(ctypes.byref(desc), _ptr(x), _ptr(grad_spikes), _ptr(h), _ptr(sg), _ptr(sign),
                               _ptr(shift), _ptr(bias), _ptr(v_th_c), _ptr(grad_x), _ptr(grad_w), _ptr(grad_b),
                               _ptr(grad_vth), _ptr(workspace), int(workspace_bytes), _stream(stream)),
           "mfpsn_backward")


def mfpsn_backward_no_alloc(desc: MfpsnDesc, x, grad_spikes, h, sg, sign, shift, bias, v_th_c, grad_x, grad_w,
                            grad_b, grad_vth, stream=None) -> None:
    _check(_lib.mfpsn_backward_no_alloc(ctypes.byref(desc), _ptr(x), _ptr(grad_spikes), _ptr(h), _ptr(sg),
                                        _ptr(sign), _ptr(shift), _ptr(bias), _ptr(v_th_c), _ptr(grad_x),
                                        _ptr(grad_w), _ptr(grad_b), _ptr(grad_vth), _stream(stream)),
           "mfpsn_backward_no_alloc")


def mfpsn_quantize_weights(w, shift_lo: int, shift_hi: int, sign, shift, stream=None) -> None:
    _check(_lib.mfpsn_quantize_weights(_ptr(w), int(w.numel()), int(shift_lo), int(shift_hi), _ptr(sign),
                                       _ptr(shift), _stream(stream)), "mfpsn_quantize_weights")


def mfpsn_quantizer_grad(w, shift, shift_lo: int, shift_hi: int, grad_wq, mode: int, grad_w, stream=None) -> None:
    _check(_lib.mfpsn_quantizer_grad(_ptr(w), _ptr(shift), int(shift_lo), int(shift_hi), _ptr(grad_wq),
                                     int(grad_wq.numel()), int(mode), _ptr(grad_w), _stream(stream)),
           "mfpsn_quantizer_grad")


def mfpsn_forward_time_last(desc: MfpsnDesc, x, sign, shift, bias, spikes, h_out=None, stream=None) -> None:
    _check(_lib.mfpsn_forward_time_last(ctypes.byref(desc), _ptr(x), _ptr(sign), _ptr(shift), _ptr(bias),
                                        _ptr(spikes), _ptr(h_out), _stream(stream)), "mfpsn_forward_time_last")


def mfpsn_backward_time_last_workspace_size(desc: MfpsnDesc) -> int:
    n = ctypes.c_size_t(0)
    _check(_lib.mfpsn_backward_time_last_workspace_size(ctypes.byref(desc), ctypes.byref(n)),
           "mfpsn_backward_time_last_workspace_size")
    return int(n.value)


def mfpsn_backward_time_last(desc: MfpsnDesc, x, grad_spikes, sign, shift, bias, grad_x, grad_w, grad_b, workspace,
                             stream=None) -> None:
    nbytes = workspace.numel() * workspace.element_size()
    _check(_lib.mfpsn_backward_time_last(ctypes.byref(desc), _ptr(x), _ptr(grad_spikes), _ptr(sign), _ptr(shift),
                                         _ptr(bias), _ptr(grad_x), _ptr(grad_w), _ptr(grad_b), _ptr(workspace),
                                         nbytes, _stream(stream)), "mfpsn_backward_time_last")


def mfpsn_spikes_to_input(spikes, dtype: int, x, stream=None) -> None:
    _check(_lib.mfpsn_spikes_to_input(_ptr(spikes), int(spikes.numel()), int(dtype), _ptr(x), _stream(stream)),
           "mfpsn_spikes_to_input")


def mfpsn_bn_workspace_size(desc: MfpsnDesc) -> int:
    n = ctypes.c_size_t(0)
    _check(_lib.mfpsn_bn_workspace_size(ctypes.byref(desc), ctypes.byref(n)), "mfpsn_bn_workspace_size")
    return int(n.value)


def mfpsn_bn_forward_stats(desc: MfpsnDesc, x, w, gamma, beta, eps: float, w_f, b_f, aux, stats, workspace,
                           stream=None) -> None:
    nbytes = workspace.numel() * workspace.element_size()
    _check(_lib.mfpsn_bn_forward_stats(ctypes.byref(desc), _ptr(x), _ptr(w), _ptr(gamma), _ptr(beta), float(eps),
                                       _ptr(w_f), _ptr(b_f), _ptr(aux), _ptr(stats), _ptr(workspace), nbytes,
                                       _stream(stream)), "mfpsn_bn_forward_stats")


def mfpsn_bn_backward(desc: MfpsnDesc, x, w, aux, eps: float, grad_wf, grad_bf, grad_x, grad_w, grad_gamma,
                      grad_beta, workspace, stream=None) -> None:
    nbytes = workspace.numel() * workspace.element_size()
    _check(_lib.mfpsn_bn_backward(ctypes.byref(desc), _ptr(x), _ptr(w), _ptr(aux), float(eps), _ptr(grad_wf),
                                  _ptr(grad_bf), _ptr(grad_x), _ptr(grad_w), _ptr(grad_gamma), _ptr(grad_beta),
                                  _ptr(workspace), nbytes, _stream(stream)), "mfpsn_bn_backward")


def mfpsn_stream_ring_bytes(desc: MfpsnDesc):
    """(ring slots R = (k-1)*dilation + 1, ring size in bytes)."""
    steps = ctypes.c_int32(0)
    n = ctypes.c_size_t(0)
    _check(_lib.mfpsn_stream_ring_bytes(ctypes.byref(desc), ctypes.byref(steps), ctypes.byref(n)),
           "mfpsn_stream_ring_bytes")
    return int(steps.value), int(n.value)


def mfpsn_stream_step(desc: MfpsnDesc, t: int, x_t, ring, sign, shift, bias, spikes_t, h_t=None,
                      stream=None) -> None:
    _check(_lib.mfpsn_stream_step(ctypes.byref(desc), int(t), _ptr(x_t), _ptr(ring), _ptr(sign), _ptr(shift),
                                  _ptr(bias), _ptr(spikes_t), _ptr(h_t), _stream(stream)), "mfpsn_stream_step")


# ---------------------------------------------------------------------------
# allocating wrappers
# ---------------------------------------------------------------------------
def _expect(t, dtype, device, name):
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.device != device:
        raise ValueError(f"{name} must be on {device}, got {t.device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def forward(desc: MfpsnDesc, x, sign, shift, bias, want_h: bool = False, want_sg: bool = False, stream=None,
            v_th_c=None):
    """spikes, plus H (want_h) and the surrogate factor (want_sg) in that order.
    v_th_c: optional per-channel thresholds [C] (float, int32 for Q8.8)."""
    dev = x.device
    _expect(x, STORAGE[desc.dtype], dev, "x")
    _expect(bias, BIAS[desc.dtype], dev, "bias")
    if v_th_c is not None:
        _expect(v_th_c, BIAS[desc.dtype], dev, "v_th_c")
    spikes = torch.empty(x.shape, dtype=torch.uint8, device=dev)
    h = torch.empty(x.shape, dtype=H_OUT[desc.dtype], device=dev) if want_h else None
    sg = torch.empty(x.shape, dtype=SG_OUT[desc.dtype], device=dev) if want_sg else None
    mfpsn_forward(desc, x, sign, shift, bias, v_th_c, spikes, h, sg, stream)
    out = (spikes,) + ((h,) if want_h else ()) + ((sg,) if want_sg else ())
    return out if len(out) > 1 else spikes


def backward(desc: MfpsnDesc, x, grad_spikes, sign, shift, bias, workspace=None, stream=None, sg=None, h=None,
             v_th_c=None, want_vth: bool = False):
    """sg: optional surrogate factor saved by forward(..., want_sg=True); h:
    optional potentials saved by forward(..., want_h=True).  sg is used if
    given, else h, else both are recomputed from x.  v_th_c: the per-channel
    thresholds the forward used; want_vth: also return the threshold gradient.
    Returns grad_x, grad_w, grad_b (and grad_vth)."""
    dev = x.device
    if v_th_c is not None:
        _expect(v_th_c, BIAS[desc.dtype], dev, "v_th_c")
    _expect(x, STORAGE[desc.dtype], dev, "x")
    _expect(grad_spikes, STORAGE[desc.dtype], dev, "grad_spikes")
    if sg is not None:
        _expect(sg, SG_OUT[desc.dtype], dev, "sg")
    if h is not None:
        _expect(h, H_OUT[desc.dtype], dev, "h")
    grad_x = torch.empty(x.shape, dtype=GRAD_X[desc.dtype], device=dev)
    grad_w = torch.empty((desc.C, desc.k), dtype=GRAD_WB[desc.dtype], device=dev)
    grad_b = torch.empty((desc.C,), dtype=GRAD_WB[desc.dtype], device=dev)
    grad_vth = torch.empty((desc.C,), dtype=GRAD_WB[desc.dtype], device=dev) if want_vth else None
    need = mfpsn_backward_workspace_size(desc)
    if workspace is None or workspace.numel() * workspace.element_size() < need:
        workspace = torch.empty(max(need, 8), dtype=torch.uint8, device=dev)
    mfpsn_backward(desc, x, grad_spikes, h, sg, sign, shift, bias, v_th_c, grad_x, grad_w, grad_b, grad_vth,
                   workspace, stream=stream)
    return (grad_x, grad_w, grad_b, grad_vth) if want_vth else (grad_x, grad_w, grad_b)


def quantize(w, shift_lo: int, shift_hi: int, stream=None):
    _expect(w, torch.float32, w.device, "w")
    sign = torch.empty(w.shape, dtype=torch.int8, device=w.device)
    shift = torch.empty(w.shape, dtype=torch.int8, device=w.device)
    mfpsn_quantize_weights(w, shift_lo, shift_hi, sign, shift, stream)
    return sign, shift


def quantizer_grad(w, shift, grad_wq, ste="whole", shift_lo: int = 0, shift_hi: int = 7, stream=None):
    """Latent-weight gradient: "whole" (the paper's whole-quantizer STE:
    grad_wq unchanged) or "round" (Eq. ste_q: grad_wq * 2^-shift / |w|)."""
    _expect(grad_wq, torch.float32, grad_wq.device, "grad_wq")
    out = torch.empty_like(grad_wq)
    mfpsn_quantizer_grad(w, shift, shift_lo, shift_hi, grad_wq, STE[ste], out, stream)
    return out


def forward_time_last(desc: MfpsnDesc, x, sign, shift, bias, want_h: bool = False, stream=None):
    """Forward for x in the time-last layout [N, C, *spatial, T]: spikes (and
    H with want_h) in the same layout.  desc is the one of the time-first
    shape [T, N, C, *spatial] (make_desc)."""
    dev = x.device
    _expect(x, STORAGE[desc.dtype], dev, "x")
    _expect(bias, BIAS[desc.dtype], dev, "bias")
    if x.shape[-1] != desc.T or x.numel() != desc.T * desc.N * desc.C * desc.S:
        raise ValueError(f"x of shape {tuple(x.shape)} does not match the descriptor (time last)")
    spikes = torch.empty(x.shape, dtype=torch.uint8, device=dev)
    h = torch.empty(x.shape, dtype=H_OUT[desc.dtype], device=dev) if want_h else None
    mfpsn_forward_time_last(desc, x, sign, shift, bias, spikes, h, stream)
    return (spikes, h) if want_h else spikes


def backward_time_last(desc: MfpsnDesc, x, grad_spikes, sign, shift, bias, workspace=None, stream=None):
    """Backward for x and grad_spikes in the time-last layout [N, C, *spatial,
    T] (T <= 64): grad_x in the same layout, grad_w [C, k], grad_b [C]."""
    dev = x.device
    _expect(x, STORAGE[desc.dtype], dev, "x")
    _expect(grad_spikes, STORAGE[desc.dtype], dev, "grad_spikes")
    if x.shape[-1] != desc.T or x.numel() != desc.T * desc.N * desc.C * desc.S or grad_spikes.shape != x.shape:
        raise ValueError(f"x of shape {tuple(x.shape)} does not match the descriptor (time last)")
    grad_x = torch.empty(x.shape, dtype=GRAD_X[desc.dtype], device=dev)
    grad_w = torch.empty((desc.C, desc.k), dtype=GRAD_WB[desc.dtype], device=dev)
    grad_b = torch.empty((desc.C,), dtype=GRAD_WB[desc.dtype], device=dev)
    need = mfpsn_backward_time_last_workspace_size(desc)
    if workspace is None or workspace.numel() * workspace.element_size() < need:
        workspace = torch.empty(max(need, 8), dtype=torch.uint8, device=dev)
    mfpsn_backward_time_last(desc, x, grad_spikes, sign, shift, bias, grad_x, grad_w, grad_b, workspace, stream)
    return grad_x, grad_w, grad_b


def spikes_to_input(spikes, dtype: str = "f32", stream=None):
    """One layer's spikes (uint8) as the next layer's input in storage type
    `dtype` ("f32", "bf16": returned as torch.bfloat16, "q8_8": int16 256)."""
    _expect(spikes, torch.uint8, spikes.device, "spikes")
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "q8_8": torch.int16}[dtype]
    x = torch.empty(spikes.shape, dtype=tdt, device=spikes.device)
    mfpsn_spikes_to_input(spikes, DTYPES[dtype], x, stream)
    return x


def bn_workspace(desc: MfpsnDesc, device):
    return torch.empty(max(mfpsn_bn_workspace_size(desc), 8), dtype=torch.uint8, device=device)


def bn_forward_stats(desc: MfpsnDesc, x, w, gamma, beta, eps: float = 1e-5, workspace=None, stream=None,
                     want_stats: bool = False):
    """Fused weight and bias of App. C from the batch statistics of the
    latent-weight convolution: (w_f, b_f, aux[, stats])."""
    dev = x.device
    _expect(x, torch.float32, dev, "x")
    w_f = torch.empty((desc.C, desc.k), dtype=torch.float32, device=dev)
    b_f = torch.empty((desc.C,), dtype=torch.float32, device=dev)
    aux = torch.empty((desc.C, 4), dtype=torch.float64, device=dev)
    stats = torch.empty((desc.C, 2), dtype=torch.float64, device=dev) if want_stats else None
    ws = workspace if workspace is not None else bn_workspace(desc, dev)
    mfpsn_bn_forward_stats(desc, x, w, gamma, beta, eps, w_f, b_f, aux, stats, ws, stream)
    return (w_f, b_f, aux, stats) if want_stats else (w_f, b_f, aux)


def bn_backward(desc: MfpsnDesc, x, w, aux, grad_wf, grad_bf, grad_x, eps: float = 1e-5, workspace=None,
                stream=None):
    """Adds the batch-statistics path to grad_x (in place) and returns
    (grad_w, grad_gamma, grad_beta) of the latent weight and the BN affine
    parameters."""
    dev = x.device
    grad_w = torch.empty((desc.C, desc.k), dtype=torch.float32, device=dev)
    grad_gamma = torch.empty((desc.C,), dtype=torch.float32, device=dev)
    grad_beta = torch.empty((desc.C,), dtype=torch.float32, device=dev)
    ws = workspace if workspace is not None else bn_workspace(desc, dev)
    mfpsn_bn_backward(desc, x, w, aux, eps, grad_wf, grad_bf, grad_x, grad_w, grad_gamma, grad_beta, ws, stream)
    return grad_w, grad_gamma, grad_beta


class StreamState:
    """Step-by-step inference of one neuron layer: owns the history ring of
    the last (k-1)*dilation + 1 inputs ([R, N, C, *spatial], the storage type
    of the layer) and the time index.  ``step(x_t)`` consumes the inputs of
    the next time step ([N, C, *spatial]) and returns its spikes (and H with
    want_h); over a sequence this equals ``forward`` bit for bit.  The ring
    needs no initialization: no slot is read before it is written."""

    def __init__(self, desc: MfpsnDesc, spatial_shape, sign, shift, bias, device=None):
        self.desc = desc
        self.shape = tuple(int(v) for v in spatial_shape)  # (N, C, *spatial)
        self.steps, nbytes = mfpsn_stream_ring_bytes(desc)
        dev = torch.device(device) if device is not None else bias.device
        self.ring = torch.empty((self.steps,) + self.shape, dtype=STORAGE[desc.dtype], device=dev)
        assert self.ring.numel() * self.ring.element_size() == nbytes
        self.sign, self.shift, self.bias = sign, shift, bias
        self.t = 0

    def step(self, x_t, want_h: bool = False, stream=None, out=None):
        _expect(x_t, STORAGE[self.desc.dtype], self.ring.device, "x_t")
        if tuple(x_t.shape) != self.shape:
            raise ValueError(f"x_t must have shape {self.shape}, got {tuple(x_t.shape)}")
        spikes, h = out if out is not None else (
            torch.empty(self.shape, dtype=torch.uint8, device=x_t.device),
            torch.empty(self.shape, dtype=H_OUT[self.desc.dtype], device=x_t.device) if want_h else None)
        mfpsn_stream_step(self.desc, self.t, x_t, self.ring, self.sign, self.shift, self.bias, spikes, h, stream)
        self.t += 1
        return (spikes, h) if want_h else spikes


class MfPSNFunction(torch.autograd.Function):
    """spikes = Theta(conv_{Q(W)}(x) + b - V_th) with the surrogate-gradient
    backward (Sec. 4.2, App. A.3).  Float storage paths (f32, bf16).

    ste="whole" (default): the gradient of W is the gradient of Q(W) (the
    whole-quantizer straight-through estimator the paper trains with);
    ste="round": only round()'s derivative is replaced by 1, so the gradient
    of W is that of Q(W) times |Q(W)|/|W| (Eq. ste_q).
    v_th: a float, or a per-channel tensor [C] (the learnable channel-wise
    threshold of Eq. mfdpsn_fire), passed to the library as is; its gradient
    comes from the library's backward."""

    @staticmethod
    def forward(ctx, x, w, b, k, dilation, v_th, surrogate, alpha, shift_lo, shift_hi, ste="whole"):
        dtype = "bf16" if x.dtype == torch.bfloat16 else "f32"
        per_channel = torch.is_tensor(v_th)
        bc = b.detach().float().contiguous()
        vc = v_th.detach().float().reshape(bc.shape).contiguous() if per_channel else None
        desc = make_desc(x.shape, k, dilation, dtype, surrogate, alpha, 0.0 if per_channel else v_th, 0,
                         shift_lo, shift_hi)
        wc = w.detach().contiguous()
        sign, shift = quantize(wc, shift_lo, shift_hi)
        xc = x.detach().contiguous()
        spikes, sg = forward(desc, xc, sign, shift, bc, want_sg=True, v_th_c=vc)
        ctx.save_for_backward(xc, wc, sign, shift, bc, sg, vc)
        ctx.desc, ctx.per_channel, ctx.ste = desc, per_channel, ste
        ctx.shift_range = (shift_lo, shift_hi)
        return spikes.to(x.dtype)

    @staticmethod
    def backward(ctx, grad_spikes):
        xc, wc, sign, shift, bc, sg, vc = ctx.saved_tensors
        g = grad_spikes.to(xc.dtype).contiguous()
        out = backward(ctx.desc, xc, g, sign, shift, bc, sg=sg, v_th_c=vc, want_vth=ctx.per_channel)
        grad_x, grad_wq, grad_b = out[:3]
        grad_vth = out[3] if ctx.per_channel else None
        grad_w = grad_wq if ctx.ste == "whole" else quantizer_grad(wc, shift, grad_wq, ctx.ste, *ctx.shift_range)
        return grad_x, grad_w, grad_b, None, None, grad_vth, None, None, None, None, None


class MfPSNBNFunction(torch.autograd.Function):
    """The training step of App. C: spikes = Theta(BN(W * x)) with the batch
    statistics of the latent-weight convolution, run as
    Theta(Q(W_f) * x + b_f) with the fused weight W_f = gamma W/sqrt(var+eps)
    and bias b_f = beta - gamma mu/sqrt(var+eps) (Eqs. weight fuse, bias
    fuse; the quantizer's whole straight-through estimator passes the
    gradient of Q(W_f) to W_f).  Float x only."""

    @staticmethod
    def forward(ctx, x, w, gamma, beta, k, dilation, eps, surrogate, alpha, shift_lo, shift_hi):
        xc = x.detach().contiguous()
        wc = w.detach().contiguous()
        desc = make_desc(x.shape, k, dilation, "f32", surrogate, alpha, 0.0, 0, shift_lo, shift_hi)
        ws = bn_workspace(desc, x.device)
        w_f, b_f, aux = bn_forward_stats(desc, xc, wc, gamma.detach().contiguous(), beta.detach().contiguous(),
                                         eps, ws)
        sign, shift = quantize(w_f, shift_lo, shift_hi)
        spikes, sg = forward(desc, xc, sign, shift, b_f, want_sg=True)
        ctx.save_for_backward(xc, wc, sign, shift, b_f, sg, aux)
        ctx.desc, ctx.eps, ctx.ws = desc, eps, ws
        return spikes.to(x.dtype)

    @staticmethod
    def backward(ctx, grad_spikes):
        xc, wc, sign, shift, b_f, sg, aux = ctx.saved_tensors
        g = grad_spikes.to(torch.float32).contiguous()
        grad_x, grad_wf, grad_bf = backward(ctx.desc, xc, g, sign, shift, b_f, sg=sg)
        grad_w, grad_gamma, grad_beta = bn_backward(ctx.desc, xc, wc, aux, grad_wf, grad_bf, grad_x, ctx.eps,
                                                    ctx.ws)
        return grad_x, grad_w, grad_gamma, grad_beta, None, None, None, None, None, None, None
