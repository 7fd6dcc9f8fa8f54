"""The training-step variants on the GPU, through the C ABI and the autograd
function: the quantizer's gradient (whole-quantizer and round-only
straight-through estimators, Sec. 4.2, Eq. ste_q) and the learnable
channel-wise threshold (Eq. mfdpsn_fire), against the oracle.

Bar: mfpsn_quantizer_grad bit-exact (one rounded quotient, one rounded
product); spikes and grad_x bit-exact; grad_w, grad_b, grad_vth within 1e-6
absolute + 1e-5 relative of the oracle's double sums (the oracle states the
per-channel threshold itself: spike iff fl(acc + b) >= V_th[c]).
"""
import numpy as np
import pytest

from paper_2501_14490_amd import workloads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2501_14490_amd import mfpsn  # noqa: E402  (loads libmfpsn.so or raises)

DEV = torch.device("cuda:0")
ABS, REL = 1e-6, 1e-5


def close(got, want):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert np.all(np.abs(got - want) <= ABS + REL * np.abs(want)), float(np.max(np.abs(got - want)))


@pytest.mark.parametrize("mode", ["whole", "round"])
@pytest.mark.parametrize("lo,hi", [(0, 7), (-12, 12)])
def test_quantizer_grad_matches_oracle(orc, mode, lo, hi):
    rng = np.random.default_rng(21 + lo)
    n = 4096 + 37
    w = (rng.normal(0, 1, n) * np.exp2(rng.integers(-9, 9, n))).astype(np.float32)
    w[:8] = [0.0, -0.0, np.inf, -np.inf, np.nan, 1e-45, 3.0, -0.7071067]
    g = rng.normal(0, 1, n).astype(np.float32)
    _, shift = orc.quantize(w, lo, hi)
    want = orc.quantizer_grad(w, shift, g, {"whole": 0, "round": 1}[mode], lo, hi)
    wt, st, gt = (torch.from_numpy(a).to(DEV) for a in (w, shift, g))
    got = mfpsn.quantizer_grad(wt, st, gt, mode, lo, hi)
    torch.cuda.synchronize()
    assert np.array_equal(got.cpu().numpy().view(np.uint32), want.view(np.uint32))


def run_function(case, w, v_th, ste, k, d, lo=0, hi=7, seed=3):
    x = torch.from_numpy(case["x"]).to(DEV).requires_grad_(True)
    wt = torch.from_numpy(w).to(DEV).requires_grad_(True)
    bt = torch.from_numpy(case["bias"]).to(DEV).requires_grad_(True)
    vt = torch.from_numpy(v_th).to(DEV).requires_grad_(True) if isinstance(v_th, np.ndarray) else v_th
    spikes = mfpsn.MfPSNFunction.apply(x, wt, bt, k, d, vt, "sigmoid", 4.0, lo, hi, ste)
    g = torch.from_numpy(case["grad_spikes"]).to(DEV)
    spikes.backward(g)
    torch.cuda.synchronize()
    out = {"spikes": spikes.detach().cpu().numpy(), "gx": x.grad.cpu().numpy(), "gw": wt.grad.cpu().numpy(),
           "gb": bt.grad.cpu().numpy()}
    if isinstance(v_th, np.ndarray):
        out["gv"] = vt.grad.cpu().numpy()
    return out


@pytest.mark.parametrize("ste", ["whole", "round"])
@pytest.mark.parametrize("per_channel", [False, True])
def test_autograd_function_variants(orc, ste, per_channel):
    k, d = 5, 2
    case = workloads.make_small(23, 3, 70, (), k=k, seed=31)  # lane-channel layout with a ragged group
    rng = np.random.default_rng(32)
    w = (rng.normal(0, 0.5, (70, k))).astype(np.float32)
    v_th = (rng.normal(0.3, 0.2, 70)).astype(np.float32) if per_channel else 0.3
    got = run_function(case, w, v_th, ste, k, d)
    sign, shift = orc.quantize(w, 0, 7)
    # the oracle compares H with V_th[c] itself (no fold into the bias)
    vc = v_th if per_channel else None
    vth = 0.0 if per_channel else v_th
    H, S = orc.forward_f32(case["x"], sign, shift, case["bias"], k, d, vth, 0, 7, v_th_c=vc)
    ref = orc.backward_f32(case["x"], case["grad_spikes"], sign, shift, case["bias"], k, d, vth, "sigmoid", 4.0,
                           0, 7, v_th_c=vc)
    assert np.array_equal(got["spikes"], S.astype(np.float32))
    assert np.array_equal(got["gx"].view(np.uint32), ref["grad_x"].view(np.uint32))
    gwq = ref["grad_w"].astype(np.float32)
    want_gw = gwq if ste == "whole" else orc.quantizer_grad(w, shift, gwq, 1, 0, 7)
    close(got["gw"], want_gw)
    close(got["gb"], ref["grad_b"])
    if per_channel:
        close(got["gv"], ref["grad_vth"])
