"""A stack of neuron layers joined by identity stateless layers (the sawtooth
stack of Sec. 4.1: dilations 1..P, one layer after the other), on the GPU
through the C ABI.

mfpsn_spikes_to_input makes one layer's spikes the next layer's input (1 in
the storage type, bit-exact); in the backward the next layer's grad_x is this
layer's grad_spikes.  Each layer of the chain is checked against the oracle
on the inputs the chain gave it, to the bars of the single-layer parity
tests (spikes and grad_x bit-exact except the documented tiny-dH outputs,
grad_w and grad_b within 1e-6 absolute + 1e-5 relative).
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2501_14490_amd import mfpsn  # noqa: E402  (loads libmfpsn.so or raises)
from tests.test_parity_gpu import check_grad_x  # noqa: E402

DEV = torch.device("cuda:0")
ONE = {"f32": np.float32(1.0).view(np.uint32), "bf16": np.uint16(0x3F80), "q8_8": np.int16(256)}
VIEW = {"f32": np.uint32, "bf16": np.uint16, "q8_8": np.int16}


@pytest.mark.parametrize("dtype", ["f32", "bf16", "q8_8"])
@pytest.mark.parametrize("count,offset", [(0, 0), (1, 0), (15, 0), (16, 0), (17, 0), (1000003, 0), (1000003, 3),
                                          (4097, 1), (4099, 4)])
def test_spikes_to_input_is_one_in_the_storage_type(dtype, count, offset):
    rng = np.random.default_rng(count + offset)
    s = (rng.random(count) < 0.3).astype(np.uint8)
    s[rng.random(count) < 0.01] = 7  # any nonzero byte counts as a spike
    buf = torch.zeros(count + offset, dtype=torch.uint8, device=DEV)
    buf[offset:] = torch.from_numpy(s).to(DEV)
    spikes = buf[offset:]
    x = mfpsn.spikes_to_input(spikes, dtype)
    torch.cuda.synchronize()
    got = x.view({"f32": torch.int32, "bf16": torch.int16, "q8_8": torch.int16}[dtype]).cpu().numpy().view(VIEW[dtype])
    want = np.where(s != 0, ONE[dtype], 0).astype(VIEW[dtype])
    assert np.array_equal(got, want)


def layer_params(rng, C, k):
    w = rng.normal(0, 0.7, (C, k)).astype(np.float32)
    bias = rng.normal(0.0, 0.3, C).astype(np.float32)
    return w, bias


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("T,N,C,S,k,P", [(40, 3, 16, 5, 4, 3), (33, 2, 70, 1, 8, 3)])
def test_chained_stack_matches_the_oracle_layer_by_layer(orc, dtype, T, N, C, S, k, P):
    rng = np.random.default_rng(T * P + k)
    shape = (T, N, C) + ((S,) if S > 1 else ())
    x0 = rng.normal(0.5, 1.0, shape).astype(np.float32)
    g_top = rng.normal(0, 1.0, shape).astype(np.float32)
    if dtype == "bf16":
        x0 = orc.bf16_bits_to_f32(orc.f32_to_bf16_bits_vec(x0))
        g_top = orc.bf16_bits_to_f32(orc.f32_to_bf16_bits_vec(g_top))
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    lo, hi = 0, 7
    layers = []
    x = torch.from_numpy(x0).to(DEV).to(tdt)
    for layer in range(P):
        d = orc.sawtooth_dilation(layer, P)
        w, bias = layer_params(rng, C, k)
        sign, shift = mfpsn.quantize(torch.from_numpy(w).to(DEV), lo, hi)
        b = torch.from_numpy(bias).to(DEV)
        desc = mfpsn.make_desc(shape, k, d, dtype, "sigmoid", 4.0, 0.5, 0, lo, hi)
        spikes, sg = mfpsn.forward(desc, x, sign, shift, b, want_sg=True)
        layers.append({"d": d, "desc": desc, "x": x, "sign": sign, "shift": shift, "b": b, "bias": bias,
                       "spikes": spikes, "sg": sg})
        x = mfpsn.spikes_to_input(spikes, dtype)
    g = torch.from_numpy(g_top).to(DEV).to(tdt)
    for L in reversed(layers):
        L["g"] = g
        L["gx"], L["gw"], L["gb"] = mfpsn.backward(L["desc"], L["x"], g, L["sign"], L["shift"], L["b"], sg=L["sg"])
        g = L["gx"]
    torch.cuda.synchronize()
    for i, L in enumerate(layers):
        label = f"{dtype} layer {i} d={L['d']}"
        xl = L["x"].float().cpu().numpy()
        if i > 0:
            assert np.array_equal(xl, layers[i - 1]["spikes"].cpu().numpy().astype(np.float32)), label
        sgn, sh = L["sign"].cpu().numpy(), L["shift"].cpu().numpy()
        _, s_ref = orc.forward_f32(xl, sgn, sh, L["bias"], k, L["d"], 0.5, lo, hi)
        assert np.array_equal(L["spikes"].cpu().numpy(), s_ref), label + ": spikes differ"
        gl = L["g"].float().cpu().numpy()
        r = orc.backward_f32(xl, gl, sgn, sh, L["bias"], k, L["d"], 0.5, "sigmoid", 4.0, lo, hi)
        if dtype == "bf16":
            got = (L["gx"].view(torch.int16).cpu().numpy().view(np.uint16).astype(np.uint32) << 16).view(np.float32)
            want = (orc.f32_to_bf16_bits_vec(r["grad_x"]).astype(np.uint32) << 16).view(np.float32)
            check_grad_x(got, want, label)
        else:
            check_grad_x(L["gx"].cpu().numpy(), r["grad_x"], label)
        for name, ref in (("gw", r["grad_w"]), ("gb", r["grad_b"])):
            got = L[name].cpu().numpy().astype(np.float64)
            assert np.all(np.abs(got - ref) <= 1e-6 + 1e-5 * np.abs(ref)), f"{label}: {name} differs"
