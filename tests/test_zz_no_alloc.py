"""mfpsn_backward_no_alloc (the backward for callers that cannot allocate,
with its workspace in a fixed device array of the library) against
mfpsn_backward with a caller-provided workspace, through the C ABI: the same
kernels on the same inputs, so every output must be identical, on two calls
in a row (the second with a smaller input, on the same scratch array)."""
import ctypes

import numpy as np
import pytest

from paper_2501_14490_amd import workloads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2501_14490_amd import mfpsn  # noqa: E402  (loads libmfpsn.so or raises)

DEV = torch.device("cuda:0")
LIMIT = 64 << 20

_lib = mfpsn._lib
_lib.mfpsn_backward_no_alloc.argtypes = [ctypes.POINTER(mfpsn.MfpsnDesc)] + [ctypes.c_void_p] * 13
_lib.mfpsn_backward_no_alloc.restype = ctypes.c_int


def dev(a, dtype):
    if dtype == "bf16" and a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(DEV).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def both(shape, k, d, dtype, saved, seed):
    c = workloads.make_small(*shape[:3], shape[3:], k=k, dtype=dtype, seed=seed)
    x, g = dev(c["x"], dtype), dev(c["grad_spikes"], dtype)
    sign, shift, bias = (dev(c[n], None) for n in ("sign", "shift", "bias"))
    desc = mfpsn.make_desc(c["x"].shape, k, d, dtype, "sigmoid", 4.0, 0.3, 77, 0, 7)
    spikes, h, sg = mfpsn.forward(desc, x, sign, shift, bias, want_h=True, want_sg=True)
    hh = h if saved == "h" else None
    ss = sg if saved == "sg" else None
    ref = mfpsn.backward(desc, x, g, sign, shift, bias, h=hh, sg=ss, want_vth=True)
    out = [torch.full_like(t, 7) for t in ref]
    st = _lib.mfpsn_backward_no_alloc(ctypes.byref(desc), x.data_ptr(), g.data_ptr(),
                                      hh.data_ptr() if hh is not None else None,
                                      ss.data_ptr() if ss is not None else None, sign.data_ptr(),
                                      shift.data_ptr(), bias.data_ptr(), None, out[0].data_ptr(),
                                      out[1].data_ptr(), out[2].data_ptr(), out[3].data_ptr(),
                                      torch.cuda.current_stream().cuda_stream)
    assert st == 0, mfpsn.mfpsn_status_string(st)
    torch.cuda.synchronize()
    for a, b, name in zip(out, ref, ("grad_x", "grad_w", "grad_b", "grad_vth")):
        ia = a.view(torch.int16) if a.element_size() == 2 else (a.view(torch.int32) if a.element_size() == 4
                                                                  else a.view(torch.int64))
        ib = b.view(torch.int16) if b.element_size() == 2 else (b.view(torch.int32) if b.element_size() == 4
                                                                  else b.view(torch.int64))
        assert torch.equal(ia, ib), f"{name} differs ({shape}, k={k}, d={d}, {dtype}, saved={saved})"


@pytest.mark.parametrize("dtype,saved", [("f32", None), ("bf16", "sg"), ("q8_8", "h"), ("q8_8", None)])
def test_no_alloc_matches_backward_twice(dtype, saved):
    # a large lane-channel problem, then a smaller plane-mode one on the same
    # scratch array: the second call must not see the first call's partials
    both((120, 40, 300), 16, 3, dtype, saved, seed=1)
    both((33, 5, 3, 10), 5, 2, dtype, saved, seed=2)


def test_no_alloc_rejects_workspace_beyond_its_array():
    # 2^20 channels, k = 32: the per-block partial sums need more than the
    # fixed array holds, so the call fails before launching anything
    desc = mfpsn.make_desc((4, 1, 1 << 20), 32, 1, "f32")
    need = mfpsn.mfpsn_backward_workspace_size(desc)
    assert need > LIMIT
    p = 0x100000
    st = _lib.mfpsn_backward_no_alloc(ctypes.byref(desc), *([p] * 12), None)
    assert st == -5  # MFPSN_ERR_WORKSPACE


def test_no_alloc_empty_problem():
    desc = mfpsn.make_desc((0, 2, 64), 4, 1, "f32")
    grad_w = torch.full((64, 4), 3.0, device=DEV)
    grad_b = torch.full((64,), 3.0, device=DEV)
    one = torch.zeros(64 * 4, dtype=torch.int8, device=DEV)
    bias = torch.zeros(64, device=DEV)
    st = _lib.mfpsn_backward_no_alloc(ctypes.byref(desc), None, None, None, None, one.data_ptr(), one.data_ptr(),
                                      bias.data_ptr(), None, None, grad_w.data_ptr(), grad_b.data_ptr(), None,
                                      torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert st == 0 and torch.all(grad_w == 0) and torch.all(grad_b == 0)
