"""Parity of the step-by-step (streaming) inference kernel with the oracle, on
the GPU, through the C ABI (mfpsn_stream_step).

Bar: one call per time step through a history ring of (k-1)d+1 slots gives
the oracle's whole-sequence potentials H and spikes bit for bit, for float,
bf16 and Q8.8 storage; ragged column counts, orders 1..32, dilations longer
than the sequence and rings that wrap many times are covered.  A HIP graph
that captures a whole sequence replays to the eager result every time.
"""
import dataclasses

import numpy as np
import pytest

from paper_2501_14490_amd import workloads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2501_14490_amd import mfpsn  # noqa: E402  (loads libmfpsn.so or raises)

DEV = torch.device("cuda:0")


def to_dev(a, dtype=None):
    if dtype == "bf16" and a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(DEV).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def oracle_forward(orc, case, k, d, dtype, v_th, v_th_q, lo, hi):
    if dtype == "q8_8":
        return orc.forward_q88(case["x"], case["sign"], case["shift"], case["bias"], k, d, v_th_q, lo, hi)
    if dtype == "bf16":
        return orc.forward_bf16(case["x"], case["sign"], case["shift"], case["bias"], k, d, v_th,
                                shift_lo=lo, shift_hi=hi)
    return orc.forward_f32(case["x"], case["sign"], case["shift"], case["bias"], k, d, v_th, lo, hi)


def stream_gpu(case, k, d, dtype, v_th, v_th_q, lo, hi, ring_fill=True):
    """Runs the sequence one step per call; returns stacked H and spikes."""
    x = to_dev(case["x"], dtype)
    desc = mfpsn.make_desc(case["x"].shape, k, d, dtype, "sigmoid", 4.0, v_th, v_th_q, lo, hi)
    st = mfpsn.StreamState(desc, x.shape[1:], to_dev(case["sign"]), to_dev(case["shift"]),
                           to_dev(case["bias"]))
    assert st.steps == (k - 1) * d + 1
    if ring_fill:  # garbage in the ring: no slot may be read before it is written
        st.ring.view(torch.int16).fill_(0x7FC1)
    H = torch.empty(x.shape, dtype=mfpsn.H_OUT[desc.dtype], device=DEV)
    spikes = torch.empty(x.shape, dtype=torch.uint8, device=DEV)
    for t in range(x.shape[0]):
        st.step(x[t], out=(spikes[t], H[t]))
    torch.cuda.synchronize()
    return H.cpu().numpy(), spikes.cpu().numpy()


def check(orc, case, k, d, dtype, v_th=0.3, v_th_q=80, lo=0, hi=7):
    Hr, Sr = oracle_forward(orc, case, k, d, dtype, v_th, v_th_q, lo, hi)
    Hg, Sg = stream_gpu(case, k, d, dtype, v_th, v_th_q, lo, hi)
    if dtype == "q8_8":
        assert np.array_equal(Hg, Hr)
    else:
        assert np.array_equal(Hg.view(np.uint32), Hr.view(np.uint32))
    assert np.array_equal(Sg, Sr)


@pytest.mark.parametrize("dtype", ["f32", "bf16", "q8_8"])
@pytest.mark.parametrize("k,d,T", [(1, 1, 5), (3, 1, 17), (4, 3, 29), (8, 2, 40), (5, 9, 12), (16, 4, 70),
                                   (32, 1, 45)])
def test_stream_matches_oracle(orc, dtype, k, d, T):
    case = workloads.make_small(T, 3, 5, (7,), k=k, dtype=dtype, seed=100 + k * 7 + d)  # 105 columns
    check(orc, case, k, d, dtype)


@pytest.mark.parametrize("dtype", ["f32", "q8_8"])
def test_stream_lane_aligned_and_wide_rows(orc, dtype):
    case = workloads.make_small(24, 4, 128, (), k=6, dtype=dtype, seed=5)  # 512 columns, two full blocks
    check(orc, case, 6, 2, dtype)
    case = workloads.make_small(9, 1, 3, (1000,), k=3, dtype=dtype, seed=6)  # 3000 columns, ragged block
    check(orc, case, 3, 3, dtype)


def test_stream_special_values(orc):
    """Zeros, subnormals, infinities and NaN take the same exact taps as the
    whole-sequence forward (the streaming kernel has no fast path)."""
    case = workloads.make_small(20, 2, 3, (5,), k=4, seed=9)
    x = case["x"]
    x.reshape(-1)[::7] = 0.0
    x.reshape(-1)[1::11] = np.float32(1e-40)
    x.reshape(-1)[2::13] = -np.float32(3e-39)
    x.reshape(-1)[3::17] = np.inf
    x.reshape(-1)[4::19] = np.nan
    check(orc, case, 4, 2, "f32", lo=-3, hi=9)


@pytest.mark.parametrize("wid,T", [(2, 72), (5, 300)])
def test_stream_workload_shapes(orc, wid, T):
    """The audio-spike shape (N=256, C=512, k=16, d=4: a 61-step ring) and
    the long fixed-point shape (N=16, C=1024, k=32, d=8: 249 steps), run long
    enough that the ring wraps."""
    wl = workloads.WORKLOADS[wid]
    wl_t = dataclasses.replace(wl, T=T)
    case = workloads.make_inputs(wl_t)
    check(orc, case, wl.k, wl.period, wl.dtype, wl.v_th, wl.v_th_q, 0, wl.s_max)


def test_stream_graph_replays_match_eager(orc):
    """A whole sequence (t = 0..T-1 on a fresh ring) captured in a HIP graph:
    every replay recomputes it, and each replay, with eager work and
    synchronizations in between, equals the eager run."""
    k, d, T = 8, 3, 40
    case = workloads.make_small(T, 4, 64, (3,), k=k, seed=12)
    x = to_dev(case["x"])
    desc = mfpsn.make_desc(case["x"].shape, k, d, "f32", "sigmoid", 4.0, 0.2, 0, 0, 7)
    sign, shift, bias = to_dev(case["sign"]), to_dev(case["shift"]), to_dev(case["bias"])
    H = torch.empty(x.shape, dtype=torch.float32, device=DEV)
    spikes = torch.empty(x.shape, dtype=torch.uint8, device=DEV)

    def run_sequence(state, stream=None):
        for t in range(T):
            state.step(x[t], stream=stream, out=(spikes[t], H[t]))

    eager = mfpsn.StreamState(desc, x.shape[1:], sign, shift, bias)
    run_sequence(eager)
    torch.cuda.synchronize()
    H_ref, S_ref = H.clone(), spikes.clone()
    Hr, Sr = oracle_forward(orc, case, k, d, "f32", 0.2, 0, 0, 7)
    assert np.array_equal(H_ref.cpu().numpy().view(np.uint32), Hr.view(np.uint32))
    assert np.array_equal(S_ref.cpu().numpy(), Sr)

    graphed = mfpsn.StreamState(desc, x.shape[1:], sign, shift, bias)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            run_sequence(graphed, stream=side)
    torch.cuda.current_stream().wait_stream(side)
    for rep in range(4):
        H.fill_(-1.0)
        spikes.fill_(7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(H.view(torch.int32), H_ref.view(torch.int32)), rep
        assert torch.equal(spikes, S_ref), rep
        _ = (x * 2).sum().item()  # unrelated eager work between replays
