"""The batch-normalized threshold with fused-weight quantization (App. C) on
the GPU, through the C ABI, stage by stage against the oracle.

Stages and bars:
  statistics and fusion: mu, the sums within 1e-12 relative, var within 1e-9
    relative (the GPU takes sum Tv^2/n - mu^2, the oracle two passes), s and
    1/sqrt(var+eps) within 1e-9, w_f and b_f within 1e-6 relative;
  quantizing w_f and the charge/fire with bias b_f, threshold 0: bit-exact
    against the oracle run on the GPU's w_f and b_f (the float decisions are
    taken on the same values);
  backward of the fusion and the statistics, fed the GPU's aux, grad_wf,
    grad_bf and quantized-path grad_x: grad_x bit-exact (same double
    operations in the same order), grad_gamma and grad_beta within 1e-12
    relative, grad_w within 1e-6 absolute + 1e-5 relative (sums over the
    batch in another order).
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
EPS = 1e-5


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def rel_close(got, want, rel, abs_=0.0):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    err = np.abs(got - want)
    assert np.all(err <= abs_ + rel * np.abs(want)), float(np.max(err))


def make_case(T, N, C, S, k, seed):
    rng = np.random.default_rng(seed)
    spatial = (S,) if S > 1 else ()
    x = rng.normal(0.3, 1.0, (T, N, C) + spatial).astype(np.float32)
    w = rng.normal(0, 0.5, (C, k)).astype(np.float32)
    gamma = rng.uniform(0.5, 1.5, C).astype(np.float32)
    beta = rng.normal(-1.0, 0.3, C).astype(np.float32)
    g = rng.normal(0, 1, x.shape).astype(np.float32)
    return x, w, gamma, beta, g


def run_case(orc, T, N, C, S, k, d, seed, lo=0, hi=7):
    x, w, gamma, beta, g = make_case(T, N, C, S, k, seed)
    desc = mfpsn.make_desc(x.shape, k, d, "f32", "sigmoid", 4.0, 0.0, 0, lo, hi)
    xt, wt = dev(x), dev(w)
    ws = mfpsn.bn_workspace(desc, DEV)
    w_f, b_f, aux, stats = mfpsn.bn_forward_stats(desc, xt, wt, dev(gamma), dev(beta), EPS, ws, want_stats=True)
    # statistics and fusion
    ref = orc.bn_forward_stats(x, w, gamma, beta, EPS, k, d)
    a = aux.cpu().numpy()
    rel_close(stats.cpu().numpy(), ref["stats"], 1e-12, 1e-9)
    rel_close(a[:, 0], ref["aux"][:, 0], 1e-12, 1e-12)
    rel_close(a[:, 1], ref["aux"][:, 1], 1e-9, 1e-12)
    rel_close(a[:, 2:], ref["aux"][:, 2:], 1e-9)
    rel_close(w_f.cpu().numpy(), ref["w_f"], 1e-6)
    rel_close(b_f.cpu().numpy(), ref["b_f"], 1e-6, 1e-7)
    # quantize the GPU's fused weight, charge and fire with its fused bias
    sign, shift = mfpsn.quantize(w_f, lo, hi)
    wf_np, bf_np = w_f.cpu().numpy(), b_f.cpu().numpy()
    s_ref, sh_ref = orc.quantize(wf_np, lo, hi)
    assert np.array_equal(sign.cpu().numpy(), s_ref) and np.array_equal(shift.cpu().numpy(), sh_ref)
    spikes, sg = mfpsn.forward(desc, xt, sign, shift, b_f, want_sg=True)
    H, S_ref = orc.forward_f32(x, s_ref, sh_ref, bf_np, k, d, 0.0, lo, hi)
    assert np.array_equal(spikes.cpu().numpy(), S_ref)
    # quantized-path backward, then the statistics path
    gx, gwf, gbf = mfpsn.backward(desc, xt, dev(g), sign, shift, b_f, sg=sg)
    gxq = gx.clone()
    grad_w, grad_gamma, grad_beta = mfpsn.bn_backward(desc, xt, wt, aux, gwf, gbf, gx, EPS, ws)
    torch.cuda.synchronize()
    rb = orc.bn_backward(x, w, gamma, EPS, a, gwf.cpu().numpy().astype(np.float64),
                         gbf.cpu().numpy().astype(np.float64), gxq.cpu().numpy().astype(np.float64), k, d)
    want_gx = rb["grad_x"].astype(np.float32)
    assert np.array_equal(gx.cpu().numpy().view(np.uint32), want_gx.view(np.uint32))
    rel_close(grad_gamma.cpu().numpy(), rb["grad_gamma"].astype(np.float32), 1e-6, 1e-12)
    rel_close(grad_beta.cpu().numpy(), rb["grad_beta"].astype(np.float32), 0.0)
    rel_close(grad_w.cpu().numpy(), rb["grad_w"], 1e-5, 1e-6)
    return {"spikes": spikes, "grad_x": gx, "grad_w": grad_w, "grad_gamma": grad_gamma, "grad_beta": grad_beta,
            "case": (x, w, gamma, beta, g)}


@pytest.mark.parametrize("T,N,C,S,k,d", [(13, 3, 5, 7, 3, 1), (20, 2, 70, 1, 5, 2), (17, 4, 9, 3, 1, 1),
                                         (40, 2, 64, 1, 8, 3), (9, 3, 4, 5, 4, 4)])
def test_bn_stages_match_oracle(orc, T, N, C, S, k, d):
    run_case(orc, T, N, C, S, k, d, seed=T * 7 + k)


@pytest.mark.parametrize("T,N,C,S,k,d", [(25, 96, 64, 16, 3, 2), (50, 48, 128, 16, 8, 1)])
def test_bn_threads_with_several_items(orc, T, N, C, S, k, d):
    """Shapes with more than 2^17 (chunk, class, column) items, so that each
    thread of the walks sums two items of its channel and the partials span
    several row groups of the reduction; classes of unequal length (T not a
    multiple of d) and chunks that are not a multiple of k steps."""
    run_case(orc, T, N, C, S, k, d, seed=T + k)


def test_bn_audio_spike_shape(orc):
    """The audio-spike layer's channels and order (C=512, k=16, d=4) on a
    shorter batch, so that the oracle finishes in seconds."""
    run_case(orc, 40, 16, 512, 1, 16, 4, seed=2)


@pytest.mark.parametrize("d", [1, 4])
def test_bn_full_audio_spike_layer_sampled_channels(orc, d):
    """The whole audio-spike layer (T=250, N=256, C=512, k=16), in the launch
    configuration the bench times, checked on a sample of channels: every
    stage of the step is independent per channel, so the oracle run on the
    sampled channels' slices of x, W, gamma, beta and of the GPU's gradients
    must give the GPU's values on those channels, to the bars above."""
    T, N, C, S, k = 250, 256, 512, 1, 16
    x, w, gamma, beta, g = make_case(T, N, C, S, k, seed=400 + d)
    desc = mfpsn.make_desc(x.shape, k, d, "f32", "sigmoid", 4.0, 0.0, 0, 0, 7)
    xt, wt = dev(x), dev(w)
    ws = mfpsn.bn_workspace(desc, DEV)
    w_f, b_f, aux, stats = mfpsn.bn_forward_stats(desc, xt, wt, dev(gamma), dev(beta), EPS, ws, want_stats=True)
    sign, shift = mfpsn.quantize(w_f, 0, 7)
    spikes, sg = mfpsn.forward(desc, xt, sign, shift, b_f, want_sg=True)
    gx, gwf, gbf = mfpsn.backward(desc, xt, dev(g), sign, shift, b_f, sg=sg)
    gxq = gx.clone()
    grad_w, grad_gamma, grad_beta = mfpsn.bn_backward(desc, xt, wt, aux, gwf, gbf, gx, EPS, ws)
    torch.cuda.synchronize()
    ch = np.array([0, 1, 77, 255, 256, 300, 510, 511])
    xs = np.ascontiguousarray(x[:, :, ch])
    ref = orc.bn_forward_stats(xs, w[ch], gamma[ch], beta[ch], EPS, k, d)
    a = aux.cpu().numpy()[ch]
    rel_close(stats.cpu().numpy()[ch], ref["stats"], 1e-12, 1e-9)
    rel_close(a[:, 0], ref["aux"][:, 0], 1e-12, 1e-12)
    rel_close(a[:, 1], ref["aux"][:, 1], 1e-9, 1e-12)
    rel_close(a[:, 2:], ref["aux"][:, 2:], 1e-9)
    wf_np, bf_np = w_f.cpu().numpy()[ch], b_f.cpu().numpy()[ch]
    rel_close(wf_np, ref["w_f"], 1e-6)
    rel_close(bf_np, ref["b_f"], 1e-6, 1e-7)
    s_ref, sh_ref = orc.quantize(wf_np, 0, 7)
    assert np.array_equal(sign.cpu().numpy()[ch], s_ref) and np.array_equal(shift.cpu().numpy()[ch], sh_ref)
    _, S_ref = orc.forward_f32(xs, s_ref, sh_ref, bf_np, k, d, 0.0, 0, 7)
    assert np.array_equal(spikes.cpu().numpy()[:, :, ch], S_ref)
    rb = orc.bn_backward(xs, w[ch], gamma[ch], EPS, a, gwf.cpu().numpy()[ch].astype(np.float64),
                         gbf.cpu().numpy()[ch].astype(np.float64),
                         np.ascontiguousarray(gxq.cpu().numpy()[:, :, ch]).astype(np.float64), k, d)
    want_gx = rb["grad_x"].astype(np.float32)
    got_gx = np.ascontiguousarray(gx.cpu().numpy()[:, :, ch])
    assert np.array_equal(got_gx.view(np.uint32), want_gx.view(np.uint32))
    rel_close(grad_gamma.cpu().numpy()[ch], rb["grad_gamma"].astype(np.float32), 1e-6, 1e-12)
    rel_close(grad_beta.cpu().numpy()[ch], rb["grad_beta"].astype(np.float32), 0.0)
    rel_close(grad_w.cpu().numpy()[ch], rb["grad_w"], 1e-5, 1e-6)


def test_bn_autograd_function_equals_the_stages(orc):
    T, N, C, S, k, d = 15, 3, 6, 4, 3, 2
    staged = run_case(orc, T, N, C, S, k, d, seed=77)
    x, w, gamma, beta, g = staged["case"]
    xt = dev(x).requires_grad_(True)
    wt, gt, bt = dev(w).requires_grad_(True), dev(gamma).requires_grad_(True), dev(beta).requires_grad_(True)
    spikes = mfpsn.MfPSNBNFunction.apply(xt, wt, gt, bt, k, d, EPS, "sigmoid", 4.0, 0, 7)
    spikes.backward(dev(g))
    torch.cuda.synchronize()
    assert torch.equal(spikes.to(torch.uint8), staged["spikes"])
    for got, want in ((xt.grad, staged["grad_x"]), (wt.grad, staged["grad_w"]), (gt.grad, staged["grad_gamma"]),
                      (bt.grad, staged["grad_beta"])):
        assert torch.equal(got, want)


@pytest.mark.parametrize("d", [1, 4])
def test_bn_variance_when_the_mean_dwarfs_the_spread(orc, d):
    """The whole audio-spike layer with inputs around 3000 and a dominant
    "now" tap, so that every channel's |mu|/sigma of Tv is at least 10^3: the
    variance (and s, W_f, b_f after it) must still match the oracle's
    two-pass variance within 1e-9 relative."""
    T, N, C, S, k = 250, 256, 512, 1, 16
    rng = np.random.default_rng(500 + d)
    x = (3000.0 + rng.normal(0.0, 1.0, (T, N, C))).astype(np.float32)
    w = rng.normal(0.0, 1e-4, (C, k)).astype(np.float32)
    w[:, k - 1] = rng.uniform(0.5, 1.5, C).astype(np.float32)
    gamma = rng.uniform(0.5, 1.5, C).astype(np.float32)
    beta = rng.normal(-1.0, 0.3, C).astype(np.float32)
    desc = mfpsn.make_desc(x.shape, k, d, "f32", "sigmoid", 4.0, 0.0, 0, 0, 7)
    ws = mfpsn.bn_workspace(desc, DEV)
    w_f, b_f, aux, stats = mfpsn.bn_forward_stats(desc, dev(x), dev(w), dev(gamma), dev(beta), EPS, ws,
                                                  want_stats=True)
    torch.cuda.synchronize()
    ch = np.array([0, 1, 63, 64, 200, 383, 384, 511])
    ref = orc.bn_forward_stats(np.ascontiguousarray(x[:, :, ch]), w[ch], gamma[ch], beta[ch], EPS, k, d)
    ratio = np.abs(ref["aux"][:, 0]) / np.sqrt(ref["aux"][:, 1])
    assert np.all(ratio >= 1e3), ratio
    a = aux.cpu().numpy()[ch]
    rel_close(a[:, 0], ref["aux"][:, 0], 1e-12)
    rel_close(a[:, 1], ref["aux"][:, 1], 1e-9)
    rel_close(a[:, 2:], ref["aux"][:, 2:], 1e-9)
    rel_close(stats.cpu().numpy()[ch], ref["stats"], 1e-12)
    rel_close(w_f.cpu().numpy()[ch], ref["w_f"], 1e-6)
    rel_close(b_f.cpu().numpy()[ch], ref["b_f"], 1e-6, 1e-5)


def test_bn_step_from_raw_inputs_on_both_sides(orc):
    """The whole fused step from the same raw x, W, gamma, beta and
    grad_spikes on both sides (each side quantizes its own W_f and fires on
    its own b_f): spikes equal except where the oracle's potential lies
    within 1e-5 of the threshold, gradients within the float tolerance."""
    T, N, C, S, k, d = 24, 4, 70, 1, 5, 2
    x, w, gamma, beta, g = make_case(T, N, C, S, k, seed=901)
    desc = mfpsn.make_desc(x.shape, k, d, "f32", "sigmoid", 4.0, 0.0, 0, 0, 7)
    xt = dev(x)
    ws = mfpsn.bn_workspace(desc, DEV)
    w_f, b_f, aux = mfpsn.bn_forward_stats(desc, xt, dev(w), dev(gamma), dev(beta), EPS, ws)
    sign, shift = mfpsn.quantize(w_f, 0, 7)
    spikes, sg = mfpsn.forward(desc, xt, sign, shift, b_f, want_sg=True)
    gx, gwf, gbf = mfpsn.backward(desc, xt, dev(g), sign, shift, b_f, sg=sg)
    grad_w, grad_gamma, grad_beta = mfpsn.bn_backward(desc, xt, dev(w), aux, gwf, gbf, gx, EPS, ws)
    torch.cuda.synchronize()
    # the oracle, from the raw inputs only
    ref = orc.bn_forward_stats(x, w, gamma, beta, EPS, k, d)
    s_o, sh_o = orc.quantize(ref["w_f"], 0, 7)
    H, S_o = orc.forward_f32(x, s_o, sh_o, ref["b_f"], k, d, 0.0, 0, 7)
    b = orc.backward_f32(x, g, s_o, sh_o, ref["b_f"], k, d, 0.0, "sigmoid", 4.0, 0, 7)
    gwf_o = b["grad_w"].astype(np.float32).astype(np.float64)
    gbf_o = b["grad_b"].astype(np.float32).astype(np.float64)
    rb = orc.bn_backward(x, w, gamma, EPS, ref["aux"], gwf_o, gbf_o, b["grad_x"].astype(np.float64), k, d)
    assert np.array_equal(sign.cpu().numpy(), s_o) and np.array_equal(shift.cpu().numpy(), sh_o)
    near = np.abs(H) < 1e-5
    got_s = spikes.cpu().numpy()
    assert np.array_equal(got_s[~near], S_o[~near])
    rel_close(gx.cpu().numpy(), rb["grad_x"], 1e-5, 1e-6)
    rel_close(grad_w.cpu().numpy(), rb["grad_w"], 1e-5, 1e-6)
    rel_close(grad_gamma.cpu().numpy(), rb["grad_gamma"], 1e-5, 1e-6)
    rel_close(grad_beta.cpu().numpy(), rb["grad_beta"], 1e-5, 1e-6)
