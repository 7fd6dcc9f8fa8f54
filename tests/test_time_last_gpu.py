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
    # lane-per-column kernel (T <= 64): full groups of 64 columns (vector
    # loads and stores), T a multiple of 4 or not, a history longer than T
    (32, 4, 16, 2, 8, 2, "f32", False),
    (30, 2, 64, 3, 8, 3, "bf16", True),
    (64, 1, 64, 1, 8, 4, "q8_8", False),
    (2, 1, 64, 1, 3, 1, "f32", True),
    (31, 3, 64, 1, 32, 2, "f32", False),
    # long columns: 1024-step segments (history above 64), a history longer
    # than T, and a history of 1200 steps (the LDS-window segment kernel)
    (2500, 1, 3, 1, 16, 6, "q8_8", False),
    (65, 3, 5, 1, 8, 20, "bf16", True),
    (1500, 1, 2, 1, 3, 600, "f32", True),
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


@pytest.mark.parametrize("dtype", ["f32", "bf16", "q8_8"])
def test_time_last_unaligned_views(orc, dtype):
    """x one element past a 16-byte boundary and spikes 3 bytes past one:
    element loads and byte stores instead of the vector forms."""
    T, N, C, S, k, d = 30, 2, 64, 1, 8, 3
    shape, x, w, bias = make(T, N, C, S, k, dtype, seed=11)
    sign, shift = orc.quantize(w, 0, 7)
    desc = mfpsn.make_desc(shape, k, d, dtype, "sigmoid", 4.0, 0.4, 100, 0, 7)
    if dtype == "q8_8":
        _, s_ref = orc.forward_q88(x, sign, shift, bias, k, d, 100, 0, 7)
        flat = to_time_last(x).reshape(-1)
    elif dtype == "bf16":
        bits = orc.f32_to_bf16_bits_vec(x)
        _, s_ref = orc.forward_bf16(bits, sign, shift, bias, k, d, 0.4, shift_lo=0, shift_hi=7)
        flat = to_time_last(bits).view(np.int16).reshape(-1)
    else:
        _, s_ref = orc.forward_f32(x, sign, shift, bias, k, d, 0.4, 0, 7)
        flat = to_time_last(x).reshape(-1)
    buf = torch.zeros(flat.size + 1, dtype=torch.from_numpy(flat[:1]).dtype, device=DEV)
    buf[1:] = torch.from_numpy(flat).to(DEV)
    xt = buf[1:].view(to_time_last(x).shape)
    if dtype == "bf16":
        xt = xt.view(torch.bfloat16)
    sbuf = torch.zeros(flat.size + 3, dtype=torch.uint8, device=DEV)
    spikes = sbuf[3:].view(xt.shape)
    sg, sh, b = (torch.from_numpy(a).to(DEV) for a in (sign, shift, bias))
    mfpsn.mfpsn_forward_time_last(desc, xt, sg, sh, b, spikes, None, torch.cuda.current_stream())
    torch.cuda.synchronize()
    assert np.array_equal(spikes.cpu().numpy(), to_time_last(s_ref))


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


# (T, N, C, S, k, d, dtype, special, surrogate, alpha)
BWD_CASES = [
    (40, 3, 5, 7, 4, 2, "f32", False, "sigmoid", 4.0),     # ragged last group
    (32, 4, 16, 2, 8, 2, "f32", False, "atan", 2.0),       # whole groups, vector loads
    (30, 2, 64, 3, 8, 3, "bf16", True, "sigmoid", 4.0),    # zeros and subnormals: exact taps
    (64, 1, 64, 1, 8, 4, "q8_8", False, "sigmoid", 4.0),
    (31, 3, 64, 1, 32, 2, "q8_8", False, "atan", 5.0),
    (17, 2, 6, 3, 32, 1, "f32", False, "rational", 10.0),  # history longer than T
    (1, 3, 64, 1, 3, 1, "f32", False, "sigmoid", 4.0),     # one step
    (20, 8, 3, 1, 5, 1, "f32", True, "sigmoid", 4.0),      # channels alternate across lanes
    (16, 2, 2, 200, 4, 1, "bf16", False, "sigmoid", 4.0),  # one channel per wave
    (12, 2, 20, 5, 3, 1, "f32", False, "sigmoid", 4.0),    # a one-lane channel run at lane 0, then five lanes
    # long columns (T > 64): segments of 256 steps, one channel per wave
    (300, 2, 9, 1, 16, 3, "f32", False, "sigmoid", 4.0),   # two segments, the second ragged
    (300, 2, 9, 1, 16, 3, "f32", True, "atan", 2.0),       # zeros and subnormals: exact taps
    (520, 1, 3, 2, 5, 4, "bf16", True, "sigmoid", 4.0),
    (600, 1, 4, 3, 32, 8, "q8_8", False, "sigmoid", 4.0),  # history of 248 steps
    (257, 1, 3, 2, 1, 1, "q8_8", False, "rational", 10.0),
    (65, 3, 5, 1, 8, 20, "f32", False, "sigmoid", 4.0),    # history 140 > T: every step in the head
    (1100, 1, 2, 1, 32, 33, "f32", False, "sigmoid", 4.0), # history 1023 (the longest), several segments
    (2500, 1, 2, 1, 16, 6, "q8_8", False, "sigmoid", 4.0), # 1024-step segments, the last one ragged
]


@pytest.mark.parametrize("T,N,C,S,k,d,dtype,special,sg,alpha", BWD_CASES)
def test_time_last_backward_matches_oracle(orc, T, N, C, S, k, d, dtype, special, sg, alpha):
    """grad_x bit for bit (every term of the definition, the surrogate's
    fixed sequence); grad_w, grad_b within 1e-6 absolute + 1e-5 relative of
    the oracle's double sums (Q8.8: exact integers)."""
    shape, x, w, bias = make(T, N, C, S, k, dtype, seed=3 * T + k + d, special=special)
    rng = np.random.default_rng(T * 31 + k)
    g = rng.normal(0.0, 1.0, x.shape).astype(np.float32)
    lo, hi = (0, 7) if dtype != "f32" or not special else (-3, 9)
    sign, shift = orc.quantize(w, lo, hi)
    v_th, v_th_q = 0.4, 100
    desc = mfpsn.make_desc(shape, k, d, dtype, sg, alpha, v_th, v_th_q, lo, hi)
    if dtype == "q8_8":
        gq = np.clip(np.round(g * 256), -32768, 32767).astype(np.int16)
        ref = orc.backward_q88(x, gq, sign, shift, bias, k, d, v_th_q, sg, alpha, lo, hi)
        xt, gt = (torch.from_numpy(to_time_last(a)).to(DEV) for a in (x, gq))
    elif dtype == "bf16":
        xb, gb_ = orc.f32_to_bf16_bits_vec(x), orc.f32_to_bf16_bits_vec(g)
        ref = orc.backward_bf16(xb, gb_, sign, shift, bias, k, d, v_th, surrogate_kind=sg, alpha=alpha,
                                shift_lo=lo, shift_hi=hi)
        xt, gt = (torch.from_numpy(to_time_last(a).view(np.int16)).to(DEV).view(torch.bfloat16) for a in (xb, gb_))
    else:
        ref = orc.backward_f32(x, g, sign, shift, bias, k, d, v_th, sg, alpha, lo, hi)
        xt, gt = (torch.from_numpy(to_time_last(a)).to(DEV) for a in (x, g))
    sg_t, sh_t, b_t = (torch.from_numpy(a).to(DEV) for a in (sign, shift, bias))
    gx, gw, gb = mfpsn.backward_time_last(desc, xt, gt, sg_t, sh_t, b_t)
    torch.cuda.synchronize()
    if dtype == "bf16":
        got = gx.view(torch.int16).cpu().numpy().view(np.uint16)
        assert np.array_equal(got, to_time_last(ref["grad_x_bits"])), "grad_x differs from the oracle"
    elif dtype == "q8_8":
        assert np.array_equal(gx.cpu().numpy(), to_time_last(ref["grad_x"])), "grad_x differs from the oracle"
    else:
        assert np.array_equal(gx.cpu().numpy().view(np.uint32), to_time_last(ref["grad_x"]).view(np.uint32)), \
            "grad_x differs from the oracle"
    if dtype == "q8_8":
        assert np.array_equal(gw.cpu().numpy(), ref["grad_w"])
        assert np.array_equal(gb.cpu().numpy(), ref["grad_b"])
    else:
        for got, want in ((gw, ref["grad_w"]), (gb, ref["grad_b"])):
            got = got.cpu().numpy().astype(np.float64)
            assert np.all(np.abs(got - want) <= 1e-6 + 1e-5 * np.abs(want)), np.max(np.abs(got - want))


@pytest.mark.parametrize("T,N,C,S,k,d", [(24, 2, 64, 2, 6, 2), (30, 8, 6, 500, 8, 3), (700, 9, 5, 3, 5, 7)])
def test_time_last_backward_repeated_calls_and_empty(orc, T, N, C, S, k, d):
    """The workspace's contents on entry do not matter and the sums are
    added in a fixed order: a second call over a garbage-filled workspace
    gives the same gradients bit for bit (short columns whose (n, c) rows
    span several blocks, and long columns whose channels span several
    waves), and N = 0 gives zero gradients."""
    shape, x, w, bias = make(T, N, C, S, k, "f32", seed=21)
    g = np.random.default_rng(22).normal(0, 1, x.shape).astype(np.float32)
    sign, shift = orc.quantize(w, 0, 7)
    desc = mfpsn.make_desc(shape, k, d, "f32", "sigmoid", 4.0, 0.4, 0, 0, 7)
    args = [torch.from_numpy(to_time_last(a)).to(DEV) for a in (x, g)]
    args += [torch.from_numpy(a).to(DEV) for a in (sign, shift, bias)]
    ws = torch.empty(mfpsn.mfpsn_backward_time_last_workspace_size(desc), dtype=torch.uint8, device=DEV)
    ws.fill_(0x5A)
    first = [t.clone() for t in mfpsn.backward_time_last(desc, *args, workspace=ws)]
    ws.fill_(0xA7)
    second = mfpsn.backward_time_last(desc, *args, workspace=ws)
    ref = orc.backward_f32(x, g, sign, shift, bias, k, d, 0.4, "sigmoid", 4.0, 0, 7)
    for a, b in zip(first, second):
        assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    got = second[1].cpu().numpy().astype(np.float64)
    assert np.all(np.abs(got - ref["grad_w"]) <= 1e-6 + 1e-5 * np.abs(ref["grad_w"]))
    empty = mfpsn.make_desc((T, 0, C, S), k, d, "f32", "sigmoid", 4.0, 0.4, 0, 0, 7)
    z = torch.empty((0, C, S, T), dtype=torch.float32, device=DEV)
    gx, gw, gb = mfpsn.backward_time_last(empty, z, z, *args[2:], workspace=ws)
    torch.cuda.synchronize()
    assert gx.numel() == 0 and not gw.any() and not gb.any()
