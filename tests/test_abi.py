"""The C ABI on the CPU: the library loads, exports every declared symbol, and
rejects invalid arguments on the host before touching the GPU."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mfpsn.h")
LIB = os.path.join(ROOT, "paper_2501_14490_amd", "libmfpsn.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libmfpsn.so not built (run __graft_entry__.build())")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mfpsn_[a-z_0-9]+)\s*\(", text)))


class Desc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("T", "N", "C", "S", "k", "dilation", "dtype", "surrogate")] + [
        ("alpha", ctypes.c_float), ("v_th", ctypes.c_float), ("v_th_q", ctypes.c_int32),
        ("shift_lo", ctypes.c_int32), ("shift_hi", ctypes.c_int32)]


def good_desc(**kw):
    d = dict(T=16, N=2, C=64, S=1, k=4, dilation=2, dtype=0, surrogate=0, alpha=4.0, v_th=1.0, v_th_q=256,
             shift_lo=0, shift_hi=7)
    d.update(kw)
    return Desc(**d)


@pytest.fixture(scope="module")
def lib():
    L = ctypes.CDLL(LIB)
    P = ctypes.c_void_p
    DP = ctypes.POINTER(Desc)
    L.mfpsn_forward.argtypes = [DP, P, P, P, P, P, P, P, P, P]
    L.mfpsn_backward.argtypes = [DP, P, P, P, P, P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P]
    L.mfpsn_backward_workspace_size.argtypes = [DP, ctypes.POINTER(ctypes.c_size_t)]
    L.mfpsn_quantize_weights.argtypes = [P, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, P, P, P]
    L.mfpsn_bn_workspace_size.argtypes = [DP, ctypes.POINTER(ctypes.c_size_t)]
    L.mfpsn_bn_forward_stats.argtypes = [DP, P, P, P, P, ctypes.c_float, P, P, P, P, P, ctypes.c_size_t, P]
    L.mfpsn_bn_backward.argtypes = [DP, P, P, P, ctypes.c_float, P, P, P, P, P, P, P, ctypes.c_size_t, P]
    L.mfpsn_quantizer_grad.argtypes = [P, P, ctypes.c_int32, ctypes.c_int32, P, ctypes.c_int64, ctypes.c_int32, P, P]
    L.mfpsn_stream_ring_bytes.argtypes = [DP, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_size_t)]
    L.mfpsn_stream_step.argtypes = [DP, ctypes.c_int64, P, P, P, P, P, P, P, P]
    L.mfpsn_status_string.restype = ctypes.c_char_p
    return L


def test_header_declares_the_three_entry_points():
    fns = declared_functions()
    for name in ("mfpsn_forward", "mfpsn_backward", "mfpsn_quantize_weights"):
        assert name in fns


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_struct_layout_matches_header():
    # 13 four-byte fields, no padding
    assert ctypes.sizeof(Desc) == 52
    text = open(HEADER).read()
    body = text[text.index("typedef struct mfpsn_desc"):text.index("} mfpsn_desc;")]
    names = re.findall(r"\b(?:int32_t|float)\s+([A-Za-z_, 0-9]+);", body)
    flat = [n.strip() for group in names for n in group.split(",")]
    assert flat == [f[0] for f in Desc._fields_]


def test_version_and_status_strings(lib):
    assert lib.mfpsn_abi_version() == 10
    for s in range(-7, 1):
        assert lib.mfpsn_status_string(s)
    assert lib.mfpsn_status_string(-99) == b"unknown status"


def test_sawtooth_matches_schedule(lib):
    assert [lib.mfpsn_sawtooth_dilation(l, 3) for l in range(7)] == [1, 2, 3, 1, 2, 3, 1]
    assert lib.mfpsn_sawtooth_dilation(-1, 3) == 0 and lib.mfpsn_sawtooth_dilation(2, 0) == 0


FAKE = 0x100000  # never dereferenced: validation fails first


@pytest.mark.parametrize("kw,status", [
    (dict(k=0), -3), (dict(k=33), -3), (dict(dilation=0), -3), (dict(T=-1), -2), (dict(C=-5), -2),
    (dict(dtype=7), -4), (dict(surrogate=3), -4), (dict(shift_lo=3, shift_hi=2), -3),
    (dict(dtype=2, shift_lo=-1), -3), (dict(dtype=2, shift_hi=32), -3), (dict(shift_hi=127), -3),
    (dict(alpha=-1.0), -3), (dict(alpha=float("nan")), -3), (dict(v_th=float("inf")), -3),
    (dict(N=1 << 20, C=1 << 10), -2),
])
def test_forward_rejects_bad_descriptors(lib, kw, status):
    d = good_desc(**kw)
    assert lib.mfpsn_forward(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, None, FAKE, None, None, None) == status


def test_forward_rejects_null_and_misaligned(lib):
    assert lib.mfpsn_forward(None, FAKE, FAKE, FAKE, FAKE, None, FAKE, None, None, None) == -1
    d = good_desc()
    assert lib.mfpsn_forward(ctypes.byref(d), None, FAKE, FAKE, FAKE, None, FAKE, None, None, None) == -1
    assert lib.mfpsn_forward(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, None, None, None, None, None) == -1
    assert lib.mfpsn_forward(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, None, FAKE, None, FAKE + 2, None) == -6
    assert lib.mfpsn_forward(ctypes.byref(d), FAKE + 2, FAKE, FAKE, FAKE, None, FAKE, None, None, None) == -6
    assert lib.mfpsn_forward(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE + 1, None, FAKE, None, None, None) == -6
    d16 = good_desc(dtype=1)
    assert lib.mfpsn_forward(ctypes.byref(d16), FAKE + 1, FAKE, FAKE, FAKE, None, FAKE, None, None, None) == -6


def test_forward_rejects_misaligned_thresholds_and_bad_q88_threshold(lib):
    d = good_desc()
    assert lib.mfpsn_forward(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE + 2, FAKE, None, None, None) == -6
    q = good_desc(dtype=2, v_th_q=(1 << 30) + 1)
    assert lib.mfpsn_forward(ctypes.byref(q), FAKE, FAKE, FAKE, FAKE, None, FAKE, None, None, None) == -3
    q = good_desc(dtype=2, v_th_q=-(1 << 30) - 1)
    assert lib.mfpsn_forward(ctypes.byref(q), FAKE, FAKE, FAKE, FAKE, None, FAKE, None, None, None) == -3


def test_empty_forward_is_a_no_op(lib):
    d = good_desc(T=0)
    assert lib.mfpsn_forward(ctypes.byref(d), None, FAKE, FAKE, FAKE, None, None, None, None, None) == 0


def test_backward_workspace_and_validation(lib):
    d = good_desc()
    n = ctypes.c_size_t(0)
    assert lib.mfpsn_backward_workspace_size(ctypes.byref(d), ctypes.byref(n)) == 0
    assert n.value > 0 and n.value % 8 == 0
    assert lib.mfpsn_backward_workspace_size(ctypes.byref(d), None) == -1
    e = good_desc(T=0)
    assert lib.mfpsn_backward_workspace_size(ctypes.byref(e), ctypes.byref(n)) == 0 and n.value == 0
    # too small / misaligned / missing workspace
    need = ctypes.c_size_t(0)
    lib.mfpsn_backward_workspace_size(ctypes.byref(d), ctypes.byref(need))
    # x, grad_spikes, h, sg, sign, shift, bias, v_th_c, grad_x, grad_w, grad_b, grad_vth
    args = [FAKE] * 12
    assert lib.mfpsn_backward(ctypes.byref(d), *args, FAKE, need.value - 8, None) == -5
    assert lib.mfpsn_backward(ctypes.byref(d), *args, FAKE + 4, need.value, None) == -5
    assert lib.mfpsn_backward(ctypes.byref(d), *args, None, need.value, None) == -5
    # null tensors (h and sg may be NULL; grad_w may not)
    bad = list(args)
    bad[9] = None  # grad_w
    assert lib.mfpsn_backward(ctypes.byref(d), *bad, FAKE, need.value, None) == -1
    for i in (2, 3, 7, 11):  # misaligned h, sg, v_th_c, grad_vth
        bad = list(args)
        bad[i] = FAKE + 2
        assert lib.mfpsn_backward(ctypes.byref(d), *bad, FAKE, need.value, None) == -6
    # Q8.8 bound on the int64 grad_w sums
    q = good_desc(dtype=2, T=1 << 16, N=1 << 16, C=1, S=1)
    assert lib.mfpsn_backward(ctypes.byref(q), *args, FAKE, 1 << 40, None) == -2


def test_quantize_validation(lib):
    assert lib.mfpsn_quantize_weights(FAKE, -1, 0, 7, FAKE, FAKE, None) == -2
    assert lib.mfpsn_quantize_weights(FAKE, 10, 5, 4, FAKE, FAKE, None) == -3
    assert lib.mfpsn_quantize_weights(None, 10, 0, 7, FAKE, FAKE, None) == -1
    assert lib.mfpsn_quantize_weights(FAKE + 2, 10, 0, 7, FAKE, FAKE, None) == -6
    assert lib.mfpsn_quantize_weights(None, 0, 0, 7, None, None, None) == 0


def test_workspace_grows_with_problem(lib):
    sizes = []
    for N in (16, 64, 256):
        d = good_desc(T=250, N=N, C=512, k=16, dilation=4)
        n = ctypes.c_size_t(0)
        assert lib.mfpsn_backward_workspace_size(ctypes.byref(d), ctypes.byref(n)) == 0
        sizes.append(n.value)
    assert sizes == sorted(sizes)
    # bounded by the resident-grid limit, not by the problem: per-block
    # partial rows stay well below the size of x
    assert sizes[-1] < 250 * 256 * 512 * 4 // 4


@pytest.mark.parametrize("k,d,dtype,es", [(4, 2, 0, 4), (16, 4, 0, 4), (8, 3, 1, 2), (32, 8, 2, 2), (1, 5, 0, 4)])
def test_stream_ring_size(lib, k, d, dtype, es):
    """The ring holds the receptive field, (k-1)d + 1 steps of N*C*S inputs."""
    desc = good_desc(T=-7 if k == 1 else 0, k=k, dilation=d, dtype=dtype, N=3, C=5, S=7)  # T is ignored
    steps, n = ctypes.c_int32(0), ctypes.c_size_t(0)
    assert lib.mfpsn_stream_ring_bytes(ctypes.byref(desc), ctypes.byref(steps), ctypes.byref(n)) == 0
    assert steps.value == (k - 1) * d + 1
    assert n.value == steps.value * 3 * 5 * 7 * es
    assert lib.mfpsn_stream_ring_bytes(ctypes.byref(desc), None, None) == -1


def test_stream_step_validation(lib):
    d = good_desc()
    args = [FAKE] * 7  # x_t, ring, sign, shift, bias, spikes_t, h_t
    assert lib.mfpsn_stream_step(None, 0, *args, None) == -1
    assert lib.mfpsn_stream_step(ctypes.byref(d), -1, *args, None) == -3
    for i in (0, 1, 5):  # x_t, ring, spikes_t
        bad = list(args)
        bad[i] = None
        assert lib.mfpsn_stream_step(ctypes.byref(d), 3, *bad, None) == -1
    bad = list(args)
    bad[1] = FAKE + 2  # misaligned float ring
    assert lib.mfpsn_stream_step(ctypes.byref(d), 3, *bad, None) == -6
    bad = list(args)
    bad[6] = FAKE + 1  # misaligned h_t
    assert lib.mfpsn_stream_step(ctypes.byref(d), 3, *bad, None) == -6
    e = good_desc(k=40)
    assert lib.mfpsn_stream_step(ctypes.byref(e), 3, *args, None) == -3
    z = good_desc(N=0)
    assert lib.mfpsn_stream_step(ctypes.byref(z), 3, None, None, FAKE, FAKE, FAKE, None, None, None) == 0


def test_quantizer_grad_validation(lib):
    q = lib.mfpsn_quantizer_grad
    assert q(FAKE, FAKE, 0, 7, FAKE, -1, 0, FAKE, None) == -2
    assert q(FAKE, FAKE, 0, 7, FAKE, 10, 2, FAKE, None) == -3      # unknown mode
    assert q(FAKE, FAKE, 5, 4, FAKE, 10, 1, FAKE, None) == -3
    assert q(None, FAKE, 0, 7, FAKE, 10, 1, FAKE, None) == -1      # round-only needs w
    assert q(FAKE, None, 0, 7, FAKE, 10, 1, FAKE, None) == -1      # ... and shift
    assert q(FAKE, FAKE, 0, 7, None, 10, 0, FAKE, None) == -1
    assert q(FAKE, FAKE, 0, 7, FAKE + 2, 10, 0, FAKE, None) == -6
    assert q(None, None, 0, 7, None, 0, 1, None, None) == 0         # nothing to do


def test_bn_validation(lib):
    d = good_desc()
    n = ctypes.c_size_t(0)
    assert lib.mfpsn_bn_workspace_size(ctypes.byref(d), ctypes.byref(n)) == 0 and n.value > 0
    need = n.value
    f = lib.mfpsn_bn_forward_stats
    args = [FAKE] * 4  # x, w, gamma, beta
    outs = [FAKE] * 4  # w_f, b_f, aux, stats
    assert f(ctypes.byref(good_desc(dtype=1)), *args, 1e-5, *outs, FAKE, need, None) == -4
    assert f(ctypes.byref(d), *args, 0.0, *outs, FAKE, need, None) == -3
    assert f(ctypes.byref(d), *args, float("nan"), *outs, FAKE, need, None) == -3
    assert f(ctypes.byref(good_desc(T=0)), *args, 1e-5, *outs, FAKE, need, None) == -2
    assert f(ctypes.byref(d), None, FAKE, FAKE, FAKE, 1e-5, *outs, FAKE, need, None) == -1
    assert f(ctypes.byref(d), *args, 1e-5, FAKE, FAKE, FAKE + 4, FAKE, FAKE, need, None) == -6
    assert f(ctypes.byref(d), *args, 1e-5, *outs, FAKE, need - 8, None) == -5
    b = lib.mfpsn_bn_backward
    bargs = [FAKE] * 3  # x, w, aux
    grads = [FAKE] * 6  # grad_wf, grad_bf, grad_x, grad_w, grad_gamma, grad_beta
    assert b(ctypes.byref(good_desc(dtype=2)), *bargs, 1e-5, *grads, FAKE, need, None) == -4
    assert b(ctypes.byref(d), *bargs, -1.0, *grads, FAKE, need, None) == -3
    assert b(ctypes.byref(d), FAKE, FAKE, None, 1e-5, *grads, FAKE, need, None) == -1
    assert b(ctypes.byref(d), *bargs, 1e-5, *grads, None, need, None) == -5


def test_spikes_to_input_validation(lib):
    f = lib.mfpsn_spikes_to_input
    f.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    assert f(FAKE, -1, 0, FAKE, None) == -2                 # negative count
    assert f(FAKE, 10, 3, FAKE, None) == -4                 # unknown storage type
    assert f(None, 10, 0, FAKE, None) == -1
    assert f(FAKE, 10, 0, None, None) == -1
    assert f(FAKE, 10, 0, FAKE + 2, None) == -6             # float output 4-byte aligned
    assert f(FAKE, 10, 1, FAKE + 1, None) == -6             # bfloat16 output 2-byte aligned
    assert f(None, 0, 2, None, None) == 0                   # nothing to do


def test_forward_time_last_validation(lib):
    f = lib.mfpsn_forward_time_last
    f.argtypes = [ctypes.POINTER(Desc)] + [ctypes.c_void_p] * 7
    d = good_desc()
    assert f(None, FAKE, FAKE, FAKE, FAKE, FAKE, None, None) == -1
    assert f(ctypes.byref(good_desc(dtype=7)), FAKE, FAKE, FAKE, FAKE, FAKE, None, None) == -4
    assert f(ctypes.byref(good_desc(k=0)), FAKE, FAKE, FAKE, FAKE, FAKE, None, None) == -3
    assert f(ctypes.byref(d), None, FAKE, FAKE, FAKE, FAKE, None, None) == -1
    assert f(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, None, None, None) == -1
    assert f(ctypes.byref(d), FAKE + 2, FAKE, FAKE, FAKE, FAKE, None, None) == -6
    assert f(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE + 2, None) == -6
    assert f(ctypes.byref(good_desc(T=0)), None, None, None, None, None, None, None) == 0


def test_backward_time_last_validation(lib):
    f = lib.mfpsn_backward_time_last
    f.argtypes = [ctypes.POINTER(Desc)] + [ctypes.c_void_p] * 9 + [ctypes.c_size_t, ctypes.c_void_p]
    ws = lib.mfpsn_backward_time_last_workspace_size
    ws.argtypes = [ctypes.POINTER(Desc), ctypes.POINTER(ctypes.c_size_t)]
    n = ctypes.c_size_t(0)
    d = good_desc()
    assert ws(ctypes.byref(d), ctypes.byref(n)) == 0 and n.value == _tl_ws_bytes(d)
    assert ws(ctypes.byref(d), None) == -1
    # the size of every kernel's slots: short columns (one slot per block
    # and (n, c) row it meets), long columns (the segment kernel's waves)
    for kw in (dict(T=64, N=3, C=5, S=100), dict(T=65, N=3, C=5, S=100), dict(T=4096, N=16, C=1024, S=1, k=32),
               dict(T=3000, N=1, C=7, S=1, k=3, dilation=40), dict(T=0), dict(N=0)):
        e = good_desc(**kw)
        assert ws(ctypes.byref(e), ctypes.byref(n)) == 0 and n.value == _tl_ws_bytes(e), kw
    need = n.value
    assert f(None, *_bwd_tl_args(), need, None) == -1
    assert f(ctypes.byref(good_desc(T=65, k=32, dilation=34)), *_bwd_tl_args(), need, None) == -2  # history > 1024
    assert f(ctypes.byref(good_desc(k=0)), *_bwd_tl_args(), need, None) == -3
    assert f(ctypes.byref(good_desc(dtype=7)), *_bwd_tl_args(), need, None) == -4
    assert f(ctypes.byref(d), *_bwd_tl_args(x=None), need, None) == -1
    assert f(ctypes.byref(d), *_bwd_tl_args(gw=None), need, None) == -1
    assert f(ctypes.byref(d), *_bwd_tl_args(x=FAKE + 2), need, None) == -6
    assert f(ctypes.byref(d), *_bwd_tl_args(gx=FAKE + 2), need, None) == -6
    assert f(ctypes.byref(good_desc(dtype=2)), *_bwd_tl_args(gw=FAKE + 4), need, None) == -6  # int64 grad_w
    assert f(ctypes.byref(d), *_bwd_tl_args(), need - 8, None) == -5
    assert f(ctypes.byref(d), *_bwd_tl_args(ws=None), need, None) == -5
    assert f(ctypes.byref(d), *_bwd_tl_args(ws=FAKE + 4), need, None) == -5


def _tl_ws_bytes(d):
    """Workspace of the time-last backward as the header states it: (k+1)
    sums per channel and per partial-sum slot."""
    M = d.N * d.C * d.S
    if M == 0 or d.T == 0:
        slots = 0
    elif d.T <= 64:
        slots = -(-M // 64) + d.N * d.C
    else:
        L = 1024 if (d.k - 1) * d.dilation > 64 else 256
        units = M * -(-d.T // L)
        slots = 4 * min(-(-units // 4), 8192) + d.C
    return (d.k + 1) * (d.C + slots) * 8


def _bwd_tl_args(**kw):
    a = dict(x=FAKE, g=FAKE, sign=FAKE, shift=FAKE, bias=FAKE, gx=FAKE, gw=FAKE, gb=FAKE, ws=FAKE)
    a.update(kw)
    return [a[k] for k in ("x", "g", "sign", "shift", "bias", "gx", "gw", "gb", "ws")]
