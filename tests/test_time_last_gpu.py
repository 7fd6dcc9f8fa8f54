"""The forward in the time-last layout [N][C][S][T] on the GPU, through the C
ABI, against the oracle (which takes the time-first layout: the test moves
the time axis) and against the library's own time-first forward.

Bar: spikes and H bit-exact (float: the definition's operation sequence;
Q8.8: integers).  Cases cover one and several wave segments per column
(T above 256 and ragged), T below a wave, k = 1 and k = 32, histories staged
in LDS and one too long for it (taps read from global memory), and inputs
with zeros and subnormals (the exact ldexp taps).
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2501_14490_amd import mfpsn  # noqa: E402  (loads libmfpsn.so or raises)

DEV = torch.device("cuda:0")


def to_time_last(a):
    return np.ascontiguousarray(np.moveaxis(a, 0, -1))


def make(T, N, C, S, k, dtype, seed, special=False):
    rng = np.random.default_rng(seed)
    shape = (T, N, C) + ((S,) if S > 1 else ())
    x = rng.normal(0.3, 1.0, shape).astype(np.float32)
    if special:
        m = rng.random(shape)
        x[m < 0.2] = 0.0
        x[(m >= 0.2) & (m < 0.25)] = np.float32(3e-39)  # subnormal
        x[(m >= 0.25) & (m < 0.27)] = -0.0
    w = rng.normal(0, 0.7, (C, k)).astype(np.float32)
    bias = rng.normal(0.0, 0.3, C).astype(np.float32)
    if dtype == "q8_8":
        xq = np.clip(np.round(x * 256), -32768, 32767).astype(np.int16)
        return shape, xq, w, np.round(bias * 256).astype(np.int32)
    if dtype == "bf16":
        return shape, x, w, bias  # rounded to bfloat16 below
    return shape, x, w, bias


CASES = [
    (40, 3, 5, 7, 4, 2, "f32", False),
    (300, 2, 9, 1, 16, 3, "f32", False),
    (300, 2, 9, 1, 16, 3, "f32", True),
    (33, 2, 70, 1, 8, 1, "bf16", False),
    (520, 1, 3, 2, 5, 4, "bf16", True),
    (600, 1, 4, 3, 32, 1, "q8_8", False),
    (257, 1, 3, 2, 1, 1, "q8_8", False),
    (2100, 2, 3, 1, 3, 1100, "f32", False),   # history (k-1)d = 2200: taps from global memory
    (17, 2, 6, 3, 32, 1, "f32", False),
]


@pytest.mark.parametrize("T,N,C,S,k,d,dtype,special", CASES)
def test_time_last_forward_matches_oracle(orc, T, N, C, S, k, d, dtype, special):
    shape, x, w, bias = make(T, N, C, S, k, dtype, seed=T + 7 * k + d, special=special)
    lo, hi = (0, 7) if dtype != "f32" or not special else (-3, 9)
    sign, shift = orc.quantize(w, lo, hi)
    v_th, v_th_q = 0.4, 100
    desc = mfpsn.make_desc(shape, k, d, dtype, "sigmoid", 4.0, v_th, v_th_q, lo, hi)
    if dtype == "q8_8":
        H_ref, s_ref = orc.forward_q88(x, sign, shift, bias, k, d, v_th_q, lo, hi)
        xt = torch.from_numpy(to_time_last(x)).to(DEV)
        x_tf = torch.from_numpy(x).to(DEV)
    elif dtype == "bf16":
        bits = orc.f32_to_bf16_bits_vec(x)
        H_ref, s_ref = orc.forward_bf16(bits, sign, shift, bias, k, d, v_th, shift_lo=lo, shift_hi=hi)
        xt = torch.from_numpy(to_time_last(bits).view(np.int16)).to(DEV).view(torch.bfloat16)
        x_tf = torch.from_numpy(bits.view(np.int16)).to(DEV).view(torch.bfloat16)
    else:
        H_ref, s_ref = orc.forward_f32(x, sign, shift, bias, k, d, v_th, lo, hi)
        xt = torch.from_numpy(to_time_last(x)).to(DEV)
        x_tf = torch.from_numpy(x).to(DEV)
    sg, sh, b = (torch.from_numpy(a).to(DEV) for a in (sign, shift, bias))
    spikes, h = mfpsn.forward_time_last(desc, xt, sg, sh, b, want_h=True)
    spikes_tf, h_tf = mfpsn.forward(desc, x_tf, sg, sh, b, want_h=True)
    torch.cuda.synchronize()
    got_s, got_h = spikes.cpu().numpy(), h.cpu().numpy()
    assert np.array_equal(got_s, to_time_last(s_ref)), "spikes differ from the oracle"
    view = np.int32 if dtype == "q8_8" else np.uint32
    assert np.array_equal(got_h.view(view), to_time_last(H_ref).view(view)), "H differs from the oracle"
    assert np.array_equal(got_s, to_time_last(spikes_tf.cpu().numpy()))
    assert np.array_equal(got_h.view(view), to_time_last(h_tf.cpu().numpy()).view(view))


def test_time_last_without_h(orc):
    T, N, C, S, k, d = 70, 2, 64, 1, 6, 2
    shape, x, w, bias = make(T, N, C, S, k, "f32", seed=5)
    sign, shift = orc.quantize(w, 0, 7)
    desc = mfpsn.make_desc(shape, k, d, "f32", "sigmoid", 4.0, 0.4, 0, 0, 7)
    _, s_ref = orc.forward_f32(x, sign, shift, bias, k, d, 0.4, 0, 7)
    spikes = mfpsn.forward_time_last(desc, torch.from_numpy(to_time_last(x)).to(DEV),
                                     *(torch.from_numpy(a).to(DEV) for a in (sign, shift, bias)))
    torch.cuda.synchronize()
    assert np.array_equal(spikes.cpu().numpy(), to_time_last(s_ref))
