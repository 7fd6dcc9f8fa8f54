"""Pins of the oracle against what the paper and the mathematics fix.

Nothing here calls the HIP library.  Each test names the passage or the
mathematical fact it checks; together they are chosen so that a plausible
mistake in the oracle (a flipped tap index, a wrong sign, a dropped term, a
missing dilation factor, a transposed operand, a truncating instead of a
flooring shift) fails at least one of them.
"""
import math
import struct
from fractions import Fraction

import numpy as np
import pytest

from paper_2501_14490_amd import workloads

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def f32_bits(v):
    return struct.unpack("<I", struct.pack("<f", float(v)))[0]


def ulp_diff(a, b):
    ia, ib = f32_bits(a), f32_bits(b)
    if ia >> 31:
        ia = 0x80000000 - (ia & 0x7FFFFFFF)
    else:
        ia = ia + 0x80000000
    if ib >> 31:
        ib = 0x80000000 - (ib & 0x7FFFFFFF)
    else:
        ib = ib + 0x80000000
    return abs(ia - ib)


def small_case(T=11, N=2, C=3, S=2, k=3, seed=0, s_lo=0, s_hi=4, bias_std=0.1):
    spatial = (S,) if S > 1 else ()
    return workloads.make_small(T, N, C, spatial, k=k, s_lo=s_lo, s_hi=s_hi, seed=seed,
                                bias_std=bias_std)


def tap_weights(sign, shift):
    """Real-valued quantized weights W_q = sign * 2^-shift (double)."""
    return sign.astype(np.float64) * np.ldexp(1.0, -shift.astype(np.int64))


def dense_toeplitz(wq_c, T, k, d):
    """App. A.2, time-first: A[i][j] = W_q[k-1-(i-j)/d] when
    i - d(k-1) <= j <= i and (i-j) % d == 0, else 0."""
    A = np.zeros((T, T))
    for i in range(T):
        for j in range(T):
            if i - d * (k - 1) <= j <= i and (i - j) % d == 0:
                A[i, j] = wq_c[k - 1 - (i - j) // d]
    return A


# ---------------------------------------------------------------------------
# exp and surrogates (closed forms)
# ---------------------------------------------------------------------------
def test_exp_within_two_ulp_of_double_exp(orc):
    ys = np.concatenate([np.linspace(-86.0, 88.0, 20001), -np.logspace(-8, 1.9, 2001),
                         np.logspace(-8, 1.9, 2001), [0.0, -0.0, -1.0, 1.0, math.log(2), -math.log(2)]])
    worst = 0
    for y in ys.astype(np.float32):
        got = orc.exp_f32(float(y))
        ref = np.float32(math.exp(float(y)))
        worst = max(worst, ulp_diff(got, ref))
    assert worst <= 2, worst
    assert orc.exp_f32(0.0) == np.float32(1.0)


def test_exp_limits(orc):
    assert orc.exp_f32(-86.5) == 0.0
    assert orc.exp_f32(float("nan")) == 0.0
    assert orc.exp_f32(-86.0) > 0.0 and np.isfinite(orc.exp_f32(88.0))
    assert orc.exp_f32(1000.0) == orc.exp_f32(88.0)


@pytest.mark.parametrize("kind,alpha,peak", [("sigmoid", 4.0, 1.0), ("sigmoid", 2.0, 0.5),
                                             ("atan", 2.0, 1.0), ("atan", 5.0, 2.5),
                                             ("rational", 10.0, 1.0)])
def test_surrogate_peak_and_symmetry(orc, kind, alpha, peak):
    # sigma'(0) = alpha/4 (sigmoid), alpha/2 (arctan), 1 (rational) exactly.
    assert orc.surrogate(kind, alpha, 0.0) == np.float32(peak)
    u = np.linspace(-9, 9, 1801).astype(np.float32)
    a = orc.surrogate(kind, alpha, u)
    b = orc.surrogate(kind, alpha, -u)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))  # even, bitwise
    assert np.all(np.diff(a[900:]) <= 0)  # non-increasing in |u|


@pytest.mark.parametrize("kind,alpha", [("sigmoid", 4.0), ("atan", 2.0), ("atan", 5.0), ("rational", 10.0)])
def test_surrogate_matches_closed_form_in_double(orc, kind, alpha):
    u = np.linspace(-6, 6, 2401).astype(np.float32)
    got = orc.surrogate(kind, alpha, u).astype(np.float64)
    ud = u.astype(np.float64)
    if kind == "sigmoid":
        # alpha s(1-s) with s = sigmoid(alpha u), in the cancellation-free form
        e = np.exp(-alpha * np.abs(ud))
        ref = alpha * e / (1.0 + e) ** 2
    elif kind == "atan":
        ref = alpha / (2.0 * (1.0 + (math.pi / 2 * alpha * ud) ** 2))
    else:
        ref = 1.0 / (1.0 + alpha * ud * ud)
    rel = np.abs(got - ref) / np.maximum(np.abs(ref), 1e-30)
    assert rel.max() < 1e-6, rel.max()


@pytest.mark.parametrize("kind,alpha,L,closed", [
    ("sigmoid", 4.0, 6.0, lambda a, L: 1 - 2 / (1 + math.exp(a * L))),
    ("atan", 2.0, 6.0, lambda a, L: 2 / math.pi * math.atan(math.pi / 2 * a * L)),
])
def test_surrogate_integral(orc, kind, alpha, L, closed):
    # the surrogate is the derivative of a smooth step: its integral over
    # [-L, L] is the closed form and tends to 1.
    u = np.linspace(-L, L, 120001)
    v = orc.surrogate(kind, alpha, u.astype(np.float32)).astype(np.float64)
    integral = np.trapezoid(v, u)
    assert abs(integral - closed(alpha, L)) < 1e-5
    assert closed(alpha, L) > 0.9


# ---------------------------------------------------------------------------
# quantizer (Eq. round_w) against exact rational arithmetic
# ---------------------------------------------------------------------------
def exact_round_log2(v: float) -> int:
    q = abs(Fraction(v))
    m = 0
    while q >= 2:
        q /= 2
        m += 1
    while q < 1:
        q *= 2
        m -= 1
    # q in [1, 2): round(log2 q) is 1 iff q^2 >= 2
    return m + (1 if q * q >= 2 else 0)


def test_quantizer_matches_fraction(orc):
    rng = np.random.default_rng(7)
    w = np.concatenate([rng.standard_normal(4000) * 0.3, rng.standard_normal(500) * 1e-3,
                        rng.standard_normal(500) * 50]).astype(np.float32)
    sign, shift = orc.quantize(w, -20, 40)
    for v, sg, sh in zip(w, sign, shift):
        assert sg == (-1 if v < 0 else 1)
        e = exact_round_log2(float(v))
        assert sh == min(max(-e, -20), 40), (v, sh, e)


def test_quantizer_boundaries_near_sqrt2(orc):
    # the floats adjacent to sqrt(2) * 2^m round to m (below) and m+1 (above);
    # exact powers of two are fixed points; zero and clamps follow the reading.
    for m in range(-10, 6):
        t = np.float32(math.sqrt(2) * 2.0 ** m)
        below = np.nextafter(t, np.float32(0)) if float(t) > math.sqrt(2) * 2.0 ** m else t
        above = np.nextafter(below, np.float32(np.inf))
        assert float(below) < math.sqrt(2) * 2.0 ** m < float(above)
        s, sh = orc.quantize(np.array([below, above, -above, np.float32(2.0 ** m)]), -64, 64)
        assert list(sh) == [-m, -(m + 1), -(m + 1), -m]
        assert list(s) == [1, 1, -1, 1]
    s, sh = orc.quantize(np.array([0.0, -0.0, 1e-30, 100.0, np.inf, np.nan], np.float32), 0, 7)
    assert list(s) == [1, 1, 1, 1, 1, 1]
    assert list(sh) == [7, 7, 7, 0, 0, 7]


def test_log2f_rounding_would_be_wrong(orc):
    # the reading of round(log2|W|) is the exact one: the float log2 of the
    # float just below 2*sqrt(2) rounds to 1.5 and then to 2, the exact answer is 1.
    v = np.float32(2.8284270763)
    assert float(v) < 2 * math.sqrt(2)
    _, sh = orc.quantize(np.array([v]), -8, 8)
    assert sh[0] == -1


# ---------------------------------------------------------------------------
# forward: closed forms, textbook routines, dense Toeplitz, invariants
# ---------------------------------------------------------------------------
def test_order_one_is_per_channel_scaling(orc):
    c = small_case(k=1, s_lo=-3, s_hi=6)
    H, spk = orc.forward_f32(c["x"], c["sign"], c["shift"], c["bias"], 1, 3, 0.25)
    C = c["x"].shape[2]
    w = (c["sign"].reshape(C).astype(np.float32) *
         np.ldexp(np.float32(1), -c["shift"].reshape(C).astype(np.int32)).astype(np.float32))
    wb = w.reshape(1, 1, C, 1)
    ref = (c["x"] * wb).astype(np.float32) + c["bias"].reshape(1, 1, C, 1)
    assert np.array_equal(H, ref.astype(np.float32))
    assert np.array_equal(spk, (ref >= np.float32(0.25)).astype(np.uint8))


def test_shared_taps_undilated_is_sliding_psn_convolution(orc):
    # Eq. SlidingPSN-charge: H[t] = sum_i W[i] X[t-k+1+i] (X[j<0] = 0) with the
    # same taps in every channel and d = 1; textbook routine np.convolve.
    T, N, C, k = 40, 3, 4, 6
    rng = np.random.default_rng(3)
    x = rng.standard_normal((T, N, C)).astype(np.float32)
    sign1 = np.where(rng.integers(0, 2, k) == 0, -1, 1).astype(np.int8)
    shift1 = rng.integers(0, 6, k).astype(np.int8)
    sign = np.tile(sign1, (C, 1))
    shift = np.tile(shift1, (C, 1))
    H, _ = orc.forward_f32(x, sign, shift, np.zeros(C, np.float32), k, 1, 1.0)
    w = tap_weights(sign1, shift1)
    for n in range(N):
        for c in range(C):
            ref = np.convolve(x[:, n, c].astype(np.float64), w[::-1])[:T]
            bound = k * 2.0 ** -24 * np.convolve(np.abs(x[:, n, c]).astype(np.float64), np.abs(w[::-1]))[:T]
            assert np.all(np.abs(H[:, n, c] - ref) <= bound + 1e-30)


@pytest.mark.parametrize("d", [1, 2, 3])
def test_dense_toeplitz_forward_and_transposed_backward(orc, d):
    # App. A.2: H[c] = A[c] X[c] (time-first) and, being linear, grad_x = A^T dH.
    k = 4
    c = small_case(T=17, N=2, C=3, S=2, k=k, seed=11)
    x, sign, shift, bias = c["x"], c["sign"], c["shift"], c["bias"]
    T, N, C, S = x.shape
    H, _ = orc.forward_f32(x, sign, shift, bias, k, d, 0.5)
    out = orc.backward_f32(x, c["grad_spikes"], sign, shift, bias, k, d, 0.5, "sigmoid", 4.0)
    assert np.array_equal(out["H"], H)
    for ch in range(C):
        A = dense_toeplitz(tap_weights(sign[ch], shift[ch]), T, k, d)
        Aabs = np.abs(A)
        for n in range(N):
            for s in range(S):
                xv = x[:, n, ch, s].astype(np.float64)
                ref = A @ xv + float(bias[ch])
                bound = (k + 1) * 2.0 ** -24 * (Aabs @ np.abs(xv) + abs(float(bias[ch])))
                assert np.all(np.abs(H[:, n, ch, s] - ref) <= bound)
                dh = out["dH"][:, n, ch, s].astype(np.float64)
                gref = A.T @ dh
                gbound = k * 2.0 ** -24 * (Aabs.T @ np.abs(dh))
                assert np.all(np.abs(out["grad_x"][:, n, ch, s] - gref) <= gbound + 1e-30)


def test_forward_bruteforce_fraction_exact_sum(orc):
    # exact rational sum of the taps bounds the float result; each term is
    # exactly sign * x * 2^-shift.
    k, d = 5, 2
    c = small_case(T=9, N=1, C=2, S=1, k=k, seed=5, s_lo=-2, s_hi=9)
    x, sign, shift, bias = c["x"], c["sign"], c["shift"], c["bias"]
    H, _ = orc.forward_f32(x, sign, shift, bias, k, d, 0.0)
    T, N, C = x.shape
    for t in range(T):
        for ch in range(C):
            exact = Fraction(0)
            absum = Fraction(0)
            for i in range(k):
                tau = t - (k - 1 - i) * d
                if tau < 0:
                    continue
                term = Fraction(float(x[tau, 0, ch])) * Fraction(2) ** (-int(shift[ch, i]))
                term = -term if sign[ch, i] < 0 else term
                exact += term
                absum += abs(term)
            exact += Fraction(float(bias[ch]))
            absum += abs(Fraction(float(bias[ch])))
            err = abs(Fraction(float(H[t, 0, ch])) - exact)
            assert err <= (k + 1) * Fraction(1, 2 ** 24) * absum


def test_causality_bitwise(orc):
    c = small_case(T=20, k=4, seed=2)
    x = c["x"].copy()
    H0, S0 = orc.forward_f32(x, c["sign"], c["shift"], c["bias"], 4, 2, 0.3)
    t0 = 9
    x[t0 + 1:] = np.random.default_rng(1).standard_normal(x[t0 + 1:].shape).astype(np.float32) * 5
    H1, S1 = orc.forward_f32(x, c["sign"], c["shift"], c["bias"], 4, 2, 0.3)
    assert np.array_equal(H0[:t0 + 1].view(np.uint32), H1[:t0 + 1].view(np.uint32))
    assert np.array_equal(S0[:t0 + 1], S1[:t0 + 1])
    assert not np.array_equal(H0[t0 + 1:], H1[t0 + 1:])


@pytest.mark.parametrize("m", [1, 3, 7])
def test_time_shift_equivariance(orc, m):
    c = small_case(T=15, k=3, seed=4)
    x = c["x"]
    H0, S0 = orc.forward_f32(x, c["sign"], c["shift"], c["bias"], 3, 2, 0.2)
    xs = np.concatenate([np.zeros((m,) + x.shape[1:], np.float32), x])
    H1, S1 = orc.forward_f32(xs, c["sign"], c["shift"], c["bias"], 3, 2, 0.2)
    assert np.array_equal(H1[m:], H0)
    assert np.array_equal(S1[m:], S0)
    assert np.array_equal(H1[:m], np.broadcast_to(c["bias"].reshape(1, 1, -1, 1), H1[:m].shape))


def test_zero_input_and_zero_gradient(orc):
    c = small_case(T=10, k=3, seed=6)
    z = np.zeros_like(c["x"])
    H, _ = orc.forward_f32(z, c["sign"], c["shift"], c["bias"], 3, 2, 0.5)
    assert np.array_equal(H, np.broadcast_to(c["bias"].reshape(1, 1, -1, 1), H.shape))
    out = orc.backward_f32(z, c["grad_spikes"], c["sign"], c["shift"], c["bias"], 3, 2, 0.5)
    assert np.all(out["grad_w"] == 0)
    out = orc.backward_f32(c["x"], np.zeros_like(c["x"]), c["sign"], c["shift"], c["bias"], 3, 2, 0.5)
    assert np.all(out["grad_x"] == 0) and np.all(out["grad_w"] == 0) and np.all(out["grad_b"] == 0)


@pytest.mark.parametrize("p", [-3, 1, 5])
def test_power_of_two_scaling_bitwise(orc, p):
    c = small_case(T=13, k=4, seed=8)
    b0 = np.zeros_like(c["bias"])
    H0, _ = orc.forward_f32(c["x"], c["sign"], c["shift"], b0, 4, 3, 1.0)
    H1, _ = orc.forward_f32(np.ldexp(c["x"], p).astype(np.float32), c["sign"], c["shift"], b0, 4, 3, 1.0)
    assert np.array_equal(H1, np.ldexp(H0, p).astype(np.float32))


def test_op_count_matches_table_formula(orc):
    # Table "params and shape": ((T + (1-k)/2) k) SHIFT per neuron at d = 1;
    # with dilation the omitted (negative-time) taps are sum_i max(0, (k-1-i) d) ... counted directly.
    for T, k, d in [(32, 16, 1), (20, 5, 1), (9, 9, 1), (30, 4, 3), (7, 3, 4)]:
        x = np.ones((T, 1, 1), np.float32)
        _, _, taps = orc.forward_f32(x, np.ones((1, k), np.int8), np.zeros((1, k), np.int8),
                                     np.zeros(1, np.float32), k, d, 1.0, with_tap_count=True)
        assert taps == sum(max(0, T - (k - 1 - i) * d) for i in range(k))
        if d == 1:
            assert Fraction(taps) == (Fraction(T) + Fraction(1 - k, 2)) * k


# ---------------------------------------------------------------------------
# backward: finite differences of the smoothed loss, adjoint identity
# ---------------------------------------------------------------------------
def primitive(kind, alpha, u):
    """A primitive of the surrogate derivative (a smooth step), in double."""
    if kind == "sigmoid":
        return 1.0 / (1.0 + np.exp(-alpha * u))
    if kind == "atan":
        return np.arctan(math.pi / 2 * alpha * u) / math.pi + 0.5
    return np.arctan(math.sqrt(alpha) * u) / math.sqrt(alpha)


def smooth_loss(x, g, wq, bias, k, d, v_th, kind, alpha):
    """L = sum g * sigma(H - v_th) with H the exact (double) charge; its
    derivative is the surrogate-gradient backward of the neuron."""
    T = x.shape[0]
    H = np.zeros(x.shape)
    for i in range(k):
        lag = (k - 1 - i) * d
        if lag >= T:
            continue
        w = wq[:, i].reshape(1, 1, -1, 1)
        H[lag:] += w * x[:T - lag]
    H += bias.reshape(1, 1, -1, 1)
    return float(np.sum(g * primitive(kind, alpha, H - v_th)))


@pytest.mark.parametrize("kind,alpha,d", [("sigmoid", 4.0, 2), ("atan", 2.0, 3), ("rational", 10.0, 1)])
def test_backward_matches_finite_differences(orc, kind, alpha, d):
    k = 3
    c = small_case(T=12, N=2, C=3, S=2, k=k, seed=21)
    x = c["x"].astype(np.float64)
    g = c["grad_spikes"].astype(np.float64)
    wq = tap_weights(c["sign"], c["shift"])
    b = c["bias"].astype(np.float64)
    v_th = 0.3
    out = orc.backward_f32(c["x"], c["grad_spikes"], c["sign"], c["shift"], c["bias"], k, d, v_th, kind, alpha)
    h = 1e-6

    def L(xx=x, ww=wq, bb=b):
        return smooth_loss(xx, g, ww, bb, k, d, v_th, kind, alpha)

    scale_w = np.abs(out["grad_w"]).max()
    for ch in range(wq.shape[0]):
        for i in range(k):
            wp, wm = wq.copy(), wq.copy()
            wp[ch, i] += h
            wm[ch, i] -= h
            fd = (L(ww=wp) - L(ww=wm)) / (2 * h)
            assert abs(fd - out["grad_w"][ch, i]) <= 2e-4 * scale_w + 1e-6, (ch, i, fd, out["grad_w"][ch, i])
        bp, bm = b.copy(), b.copy()
        bp[ch] += h
        bm[ch] -= h
        fd = (L(bb=bp) - L(bb=bm)) / (2 * h)
        assert abs(fd - out["grad_b"][ch]) <= 2e-4 * np.abs(out["grad_b"]).max() + 1e-6
    rng = np.random.default_rng(0)
    scale_x = np.abs(out["grad_x"]).max()
    for _ in range(40):
        idx = tuple(int(rng.integers(0, s)) for s in x.shape)
        xp, xm = x.copy(), x.copy()
        xp[idx] += h
        xm[idx] -= h
        fd = (L(xx=xp) - L(xx=xm)) / (2 * h)
        assert abs(fd - out["grad_x"][idx]) <= 2e-4 * scale_x + 1e-6, (idx, fd, out["grad_x"][idx])


# ---------------------------------------------------------------------------
# learnable channel-wise threshold V_th[c] (Sec. 4.2, Eq. mfdpsn_fire)
# ---------------------------------------------------------------------------
def test_per_channel_threshold_equal_to_scalar_is_the_scalar_path(orc):
    # one value in every channel: the same neuron as the shared threshold,
    # bit for bit (float and Q8.8, forward and backward)
    k, d = 4, 2
    c = small_case(T=17, N=3, C=5, S=3, k=k, seed=41)
    v = 0.37
    vc = np.full(5, v, np.float32)
    H0, S0 = orc.forward_f32(c["x"], c["sign"], c["shift"], c["bias"], k, d, v)
    H1, S1 = orc.forward_f32(c["x"], c["sign"], c["shift"], c["bias"], k, d, -99.0, v_th_c=vc)
    assert np.array_equal(H0.view(np.uint32), H1.view(np.uint32)) and np.array_equal(S0, S1)
    b0 = orc.backward_f32(c["x"], c["grad_spikes"], c["sign"], c["shift"], c["bias"], k, d, v)
    b1 = orc.backward_f32(c["x"], c["grad_spikes"], c["sign"], c["shift"], c["bias"], k, d, -99.0, v_th_c=vc)
    for name in ("dH", "grad_x"):
        assert np.array_equal(b0[name].view(np.uint32), b1[name].view(np.uint32)), name
    for name in ("grad_w", "grad_b"):
        assert np.array_equal(b0[name], b1[name]), name
    q = workloads.make_small(17, 3, 5, (3,), k=k, dtype="q8_8", seed=42)
    H0, S0 = orc.forward_q88(q["x"], q["sign"], q["shift"], q["bias"], k, d, 95, 0, 7)
    H1, S1 = orc.forward_q88(q["x"], q["sign"], q["shift"], q["bias"], k, d, -7, 0, 7,
                             v_th_c=np.full(5, 95, np.int32))
    assert np.array_equal(H0, H1) and np.array_equal(S0, S1)
    b0 = orc.backward_q88(q["x"], q["grad_spikes"], q["sign"], q["shift"], q["bias"], k, d, 95, "sigmoid", 4.0, 0, 7)
    b1 = orc.backward_q88(q["x"], q["grad_spikes"], q["sign"], q["shift"], q["bias"], k, d, -7, "sigmoid", 4.0, 0, 7,
                          v_th_c=np.full(5, 95, np.int32))
    for name in ("dH", "grad_x", "grad_w", "grad_b"):
        assert np.array_equal(b0[name], b1[name]), name


@pytest.mark.parametrize("dtype", ["f32", "q8_8"])
def test_per_channel_threshold_is_each_channel_with_its_own_scalar(orc, dtype):
    # channels are independent neurons: channel c with thresholds V_th[c] is
    # the shared-threshold neuron run on that channel alone with V_th[c]
    k, d, C = 5, 3, 6
    c = workloads.make_small(23, 2, C, (4,), k=k, dtype=dtype, seed=43)
    rng = np.random.default_rng(44)
    if dtype == "q8_8":
        vc = rng.integers(-300, 300, C).astype(np.int32)
        fw, bw, extra = orc.forward_q88, orc.backward_q88, (0, 7)
        bargs = ("sigmoid", 4.0, 0, 7)
    else:
        vc = rng.normal(0.2, 0.5, C).astype(np.float32)
        fw, bw, extra = orc.forward_f32, orc.backward_f32, ()
        bargs = ()
    H, S = fw(c["x"], c["sign"], c["shift"], c["bias"], k, d, 0, *extra, v_th_c=vc)
    b = bw(c["x"], c["grad_spikes"], c["sign"], c["shift"], c["bias"], k, d, 0, *bargs, v_th_c=vc)
    for ch in range(C):
        one = {n: (np.ascontiguousarray(v[:, :, ch:ch + 1]) if n in ("x", "grad_spikes") else v[ch:ch + 1])
               for n, v in c.items()}
        v = vc[ch].item()
        H1, S1 = fw(one["x"], one["sign"], one["shift"], one["bias"], k, d, v, *extra)
        b1 = bw(one["x"], one["grad_spikes"], one["sign"], one["shift"], one["bias"], k, d, v, *bargs)
        assert np.array_equal(H[:, :, ch:ch + 1], H1) and np.array_equal(S[:, :, ch:ch + 1], S1), ch
        for name in ("dH", "grad_x"):
            assert np.array_equal(b[name][:, :, ch:ch + 1], b1[name]), (ch, name)
        for name in ("grad_w", "grad_b"):
            assert np.array_equal(b[name][ch], b1[name][0]), (ch, name)
        assert b["grad_vth"][ch] == -b1["grad_b"][0], ch


def test_per_channel_threshold_fires_at_equality(orc):
    # Theta(0) = 1: a channel whose threshold equals one of its potentials
    # exactly fires there, and one just above it does not
    k, d = 3, 1
    c = small_case(T=9, N=1, C=2, S=1, k=k, seed=45)
    H, _ = orc.forward_f32(c["x"], c["sign"], c["shift"], c["bias"], k, d, 0.0)
    h = H[4, 0, 1]
    vc = np.array([np.inf, h], np.float32)
    _, S = orc.forward_f32(c["x"], c["sign"], c["shift"], c["bias"], k, d, 0.0, v_th_c=vc)
    assert S[4, 0, 1] == 1 and not S[:, :, 0].any()
    vc[1] = np.nextafter(h, np.float32(np.inf))
    _, S = orc.forward_f32(c["x"], c["sign"], c["shift"], c["bias"], k, d, 0.0, v_th_c=vc)
    assert S[4, 0, 1] == 0


@pytest.mark.parametrize("kind,alpha", [("sigmoid", 4.0), ("atan", 2.0)])
def test_per_channel_threshold_gradient_matches_finite_differences(orc, kind, alpha):
    # L = sum g * step(H - V_th[c]) with a smooth step whose derivative is the
    # surrogate: dL/dV_th[c] = -sum dH over the channel
    k, d = 3, 2
    c = small_case(T=12, N=2, C=3, S=2, k=k, seed=46)
    x = c["x"].astype(np.float64)
    g = c["grad_spikes"].astype(np.float64)
    wq = tap_weights(c["sign"], c["shift"])
    b = c["bias"].astype(np.float64)
    vc = np.array([0.1, 0.45, -0.2], np.float32)
    out = orc.backward_f32(c["x"], c["grad_spikes"], c["sign"], c["shift"], c["bias"], k, d, 0.0, kind, alpha,
                           v_th_c=vc)

    def L(v):
        T = x.shape[0]
        H = np.zeros(x.shape)
        for i in range(k):
            lag = (k - 1 - i) * d
            if lag < T:
                H[lag:] += wq[:, i].reshape(1, 1, -1, 1) * x[:T - lag]
        H += b.reshape(1, 1, -1, 1)
        return float(np.sum(g * primitive(kind, alpha, H - v.reshape(1, 1, -1, 1))))

    h = 1e-6
    scale = np.abs(out["grad_vth"]).max()
    for ch in range(3):
        vp, vm = vc.astype(np.float64), vc.astype(np.float64)
        vp[ch] += h
        vm[ch] -= h
        fd = (L(vp) - L(vm)) / (2 * h)
        assert abs(fd - out["grad_vth"][ch]) <= 2e-4 * scale + 1e-6, (ch, fd, out["grad_vth"][ch])
        assert out["grad_vth"][ch] == -out["grad_b"][ch]


def test_grad_w_exact_in_double_against_fraction(orc):
    # grad_w sums products of two floats, each exact in double; the double sum
    # of a few hundred terms is within n*eps of the exact rational sum.
    k, d = 3, 2
    c = small_case(T=10, N=2, C=2, S=3, k=k, seed=9)
    out = orc.backward_f32(c["x"], c["grad_spikes"], c["sign"], c["shift"], c["bias"], k, d, 0.4)
    x, dH = c["x"], out["dH"]
    T = x.shape[0]
    for ch in range(2):
        for i in range(k):
            lag = (k - 1 - i) * d
            exact = Fraction(0)
            ab = Fraction(0)
            for t in range(lag, T):
                for n in range(2):
                    for s in range(3):
                        p = Fraction(float(x[t - lag, n, ch, s])) * Fraction(float(dH[t, n, ch, s]))
                        exact += p
                        ab += abs(p)
            assert abs(Fraction(out["grad_w"][ch, i]) - exact) <= 64 * Fraction(1, 2 ** 53) * ab
        gb = sum(Fraction(float(v)) for v in dH[:, :, ch, :].ravel())
        assert abs(Fraction(out["grad_b"][ch]) - gb) <= Fraction(1, 2 ** 40)


def test_adjoint_identity(orc):
    # <A x, y> = <x, A^T y> for the charge operator without bias, in double.
    k, d = 4, 2
    c = small_case(T=16, k=k, seed=13)
    zero_b = np.zeros_like(c["bias"])
    y = np.random.default_rng(5).standard_normal(c["x"].shape).astype(np.float32)
    H, _ = orc.forward_f32(c["x"], c["sign"], c["shift"], zero_b, k, d, 0.0)
    # grad_x of the rational surrogate with alpha = 0 has sigma' = 1, so dH = g
    out = orc.backward_f32(c["x"], y, c["sign"], c["shift"], zero_b, k, d, 0.0, "rational", 0.0)
    assert np.array_equal(out["dH"], y)
    lhs = float(np.sum(H.astype(np.float64) * y))
    rhs = float(np.sum(c["x"].astype(np.float64) * out["grad_x"]))
    assert abs(lhs - rhs) <= 1e-5 * (np.abs(H).sum() * np.abs(y).max())


# ---------------------------------------------------------------------------
# Q8.8 fixed point
# ---------------------------------------------------------------------------
def test_q88_forward_bruteforce_python_ints(orc):
    # Python's >> on ints is the arithmetic (flooring) shift.
    k, d = 4, 3
    c = workloads.make_small(14, 2, 3, (2,), k=k, s_lo=0, s_hi=9, dtype="q8_8", seed=17)
    x, sign, shift, bias = c["x"], c["sign"], c["shift"], c["bias"]
    H, spk = orc.forward_q88(x, sign, shift, bias, k, d, 256)
    T, N, C, S = x.shape
    for t in range(T):
        for n in range(N):
            for ch in range(C):
                for s in range(S):
                    acc = int(bias[ch])
                    for i in range(k):
                        tau = t - (k - 1 - i) * d
                        if tau >= 0:
                            y = int(x[tau, n, ch, s]) >> int(shift[ch, i])
                            acc += -y if sign[ch, i] < 0 else y
                    assert H[t, n, ch, s] == acc
                    assert spk[t, n, ch, s] == (1 if acc >= 256 else 0)


def test_q88_backward_bruteforce_python_ints(orc):
    k, d = 3, 2
    c = workloads.make_small(12, 2, 2, (3,), k=k, s_lo=0, s_hi=7, dtype="q8_8", seed=19)
    x, g, sign, shift, bias = c["x"], c["grad_spikes"], c["sign"], c["shift"], c["bias"]
    out = orc.backward_q88(x, g, sign, shift, bias, k, d, 256, "sigmoid", 4.0)
    H, dH = out["H"], out["dH"]
    T, N, C, S = x.shape
    L = orc.surrogate_q15("sigmoid", 4.0, (H - 256).ravel()).reshape(H.shape)
    ref_dH = (g.astype(object) * L.astype(object))
    ref_dH = np.vectorize(lambda v: int(v) >> 15)(ref_dH)
    assert np.array_equal(dH, ref_dH.astype(np.int32))
    for ch in range(C):
        for i in range(k):
            lag = (k - 1 - i) * d
            s = sum(int(x[t - lag, n, ch, sp]) * int(dH[t, n, ch, sp])
                    for t in range(lag, T) for n in range(N) for sp in range(S))
            assert out["grad_w"][ch, i] == s
        assert out["grad_b"][ch] == int(dH[:, :, ch, :].astype(np.int64).sum())
    for t in range(T):
        for n in range(N):
            for ch in range(C):
                for sp in range(S):
                    acc = 0
                    for i in range(k):
                        tau = t + (k - 1 - i) * d
                        if tau < T:
                            y = int(dH[tau, n, ch, sp]) >> int(shift[ch, i])
                            acc += -y if sign[ch, i] < 0 else y
                    assert out["grad_x"][t, n, ch, sp] == acc


def test_q88_surrogate_factor(orc):
    # L(0) = 2^15 * alpha/4 for the sigmoid, symmetric, and the float value it rounds.
    assert orc.surrogate_q15("sigmoid", 4.0, 0) == 32768
    u = np.arange(-3000, 3001)
    Lq = orc.surrogate_q15("sigmoid", 4.0, u)
    assert np.array_equal(Lq, Lq[::-1])
    ref = np.rint(orc.surrogate("sigmoid", 4.0, (u / 256.0).astype(np.float32)) * 32768.0)
    assert np.array_equal(Lq, ref.astype(np.int32))


def test_q88_matches_float_path_when_shifts_are_exact(orc):
    # for inputs that are multiples of 2^s_max the floor shift is exact, so the
    # Q8.8 potential equals 256 times the float potential (cross-path invariant).
    k, d, s_hi = 4, 2, 5
    c = workloads.make_small(16, 2, 3, (), k=k, s_lo=0, s_hi=s_hi, dtype="q8_8", seed=23)
    xq = ((c["x"].astype(np.int32) >> s_hi) << s_hi).astype(np.int16)
    bq = (c["bias"] >> 0).astype(np.int32)
    Hq, _ = orc.forward_q88(xq, c["sign"], c["shift"], bq, k, d, 256)
    xf = (xq.astype(np.float32) / np.float32(256))
    Hf, _ = orc.forward_f32(xf, c["sign"], c["shift"], (bq / 256).astype(np.float32), k, d, 1.0)
    assert np.array_equal(Hq.astype(np.float64), Hf.astype(np.float64) * 256)


# ---------------------------------------------------------------------------
# bf16 storage
# ---------------------------------------------------------------------------
def test_bf16_rounding_matches_torch(orc):
    import torch
    rng = np.random.default_rng(1)
    a = np.concatenate([rng.standard_normal(3000).astype(np.float32),
                        np.array([0.0, -0.0, 1e-40, 3.4e38, -3.4e38, np.inf, -np.inf], np.float32)])
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(orc.f32_to_bf16_bits(a), ref)
    assert np.array_equal(orc.f32_to_bf16_bits_vec(a), ref)
    assert np.array_equal(orc.bf16_bits_to_f32(ref), torch.from_numpy(ref.view(np.int16)).view(
        torch.bfloat16).float().numpy())


# ---------------------------------------------------------------------------
# step-by-step inference (Sec. 3.2: H[t] is available at step t; Sec. 5,
# Table "inference memory": the neuron stores an input history whose length
# grows with its order)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("k,d,T", [(1, 1, 7), (3, 1, 12), (4, 3, 20), (5, 2, 6), (2, 9, 12), (8, 4, 40)])
def test_stream_steps_reproduce_the_parallel_forward(orc, k, d, T):
    """Feeding one time step per call through a ring of (k-1)d+1 slots gives
    the potentials and spikes of the whole-sequence forward bit for bit (the
    ring starts as NaN / a garbage pattern, so a slot read before it was
    written would show)."""
    c = small_case(T=T, N=2, C=3, S=2, k=k, seed=40 + k * d)
    H, S = orc.forward_f32(c["x"], c["sign"], c["shift"], c["bias"], k, d, 0.3, 0, 4)
    Hs, Ss = orc.stream_forward(c["x"], c["sign"], c["shift"], c["bias"], k, d, 0.3, "f32", 0, 4)
    assert np.array_equal(H.view(np.uint32), Hs.view(np.uint32))
    assert np.array_equal(S, Ss)


def test_stream_steps_bf16_and_q88(orc):
    k, d, T = 4, 2, 15
    cb = workloads.make_small(T, 2, 5, (3,), k=k, dtype="bf16", seed=7)
    H, S = orc.forward_bf16(cb["x"], cb["sign"], cb["shift"], cb["bias"], k, d, 0.2, shift_lo=0, shift_hi=7)
    Hs, Ss = orc.stream_forward(cb["x"], cb["sign"], cb["shift"], cb["bias"], k, d, 0.2, "bf16", 0, 7)
    assert np.array_equal(H.view(np.uint32), Hs.view(np.uint32)) and np.array_equal(S, Ss)
    cq = workloads.make_small(T, 2, 5, (3,), k=k, dtype="q8_8", seed=8)
    H, S = orc.forward_q88(cq["x"], cq["sign"], cq["shift"], cq["bias"], k, d, 100, 0, 7)
    Hs, Ss = orc.stream_forward(cq["x"], cq["sign"], cq["shift"], cq["bias"], k, d, 100, "q8_8", 0, 7)
    assert np.array_equal(H, Hs) and np.array_equal(S, Ss)


@pytest.mark.parametrize("k,d", [(4, 3), (2, 5), (6, 1)])
def test_receptive_field_is_exactly_the_ring_length(orc, k, d):
    """H[t] depends on x[t - (k-1)d] and on nothing older (every tap is a
    nonzero power of two), so (k-1)d + 1 inputs are the smallest history a
    step-by-step neuron can keep."""
    R = orc.stream_ring_steps(k, d)
    assert R == (k - 1) * d + 1
    T = R + 6
    c = small_case(T=T, N=1, C=2, S=1, k=k, seed=3)
    x = c["x"].astype(np.float32)
    H0, _ = orc.forward_f32(x, c["sign"], c["shift"], c["bias"], k, d, 0.0, 0, 4)
    t = T - 1
    for age, changes in ((R - 1, True), (R, False), (R + 3, False)):
        x1 = x.copy()
        x1[t - age] += np.float32(64.0)
        H1, _ = orc.forward_f32(x1, c["sign"], c["shift"], c["bias"], k, d, 0.0, 0, 4)
        assert bool(np.any(H1[t] != H0[t])) == changes, (age, changes)


# ---------------------------------------------------------------------------
# gradients of the quantizer (Sec. 4.2: Eq. ste, Eq. ste_q, and the
# whole-quantizer straight-through estimator the paper trains with)
# ---------------------------------------------------------------------------
def test_quantizer_grad_whole_ste_is_identity(orc):
    rng = np.random.default_rng(4)
    w = rng.normal(0, 1, 200).astype(np.float32)
    g = rng.normal(0, 1, 200).astype(np.float32)
    _, shift = orc.quantize(w, -10, 10)
    assert np.array_equal(orc.quantizer_grad(w, shift, g, 0, -10, 10), g)


def test_quantizer_grad_round_only_factor_is_wq_over_w(orc):
    """Eq. ste_q: Q'(W) = 2^round(log2|W|)/|W|.  The factor is one rounded
    division, so factor*|W| lies within half an ulp of the factor (times |W|)
    of |Wq| = 2^round(log2|W|), the exactly rounded power of two (checked
    with rational arithmetic); it is even in W; powers of two inside the
    shift range are fixed points (factor 1)."""
    rng = np.random.default_rng(5)
    w = (rng.normal(0, 1, 400) * np.exp2(rng.integers(-6, 6, 400))).astype(np.float32)
    w[:10] = np.ldexp(1.0, -np.arange(10)).astype(np.float32)
    ones = np.ones_like(w)
    lo, hi = -20, 20
    _, shift = orc.quantize(w, lo, hi)
    fac = orc.quantizer_grad(w, shift, ones, 1, lo, hi)
    for wi, f in zip(w, fac):
        m = math.frexp(abs(float(wi)))[1] - 1        # |w| = f 2^m, f in [1, 2)
        e = m + (1 if Fraction(abs(float(wi))) ** 2 >= Fraction(2) ** (2 * m + 1) else 0)
        exact = Fraction(2) ** e / Fraction(abs(float(wi)))
        ulp = Fraction(2) ** (math.frexp(float(f))[1] - 24)
        assert abs(Fraction(float(f)) - exact) <= ulp / 2, (wi, f)
    assert np.all(fac[:10] == 1.0)
    assert np.array_equal(orc.quantizer_grad(-w, shift, ones, 1, lo, hi), fac)
    g = rng.normal(0, 1, 400).astype(np.float32)
    assert np.array_equal(orc.quantizer_grad(w, shift, g, 1, lo, hi), (g * fac).astype(np.float32))


def test_quantizer_grad_round_only_special_values(orc):
    w = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 1e-45, 3.0], np.float32)
    _, shift = orc.quantize(w, 0, 7)
    out = orc.quantizer_grad(w, shift, np.ones_like(w), 1, 0, 7)
    assert np.all(out[:5] == 0.0)
    # 1e-45 is far below 2^-7: the clamped |Wq| = 2^-7 over |W| overflows -> 0
    assert out[5] == 0.0
    # Q(3) rounds to 4 (shift -2), clamped into [0, 7] to shift 0: |Wq| = 1, factor 1/3
    assert out[6] == np.float32(1.0) / np.float32(3.0)


# ---------------------------------------------------------------------------
# batch-normalized threshold with fused-weight quantization (App. C)
# ---------------------------------------------------------------------------
def latent_conv(x, w, k, d):
    """W * x in float64 with the causal, dilated taps (independent numpy form)."""
    x = x.astype(np.float64)
    T = x.shape[0]
    out = np.zeros_like(x)
    C = x.shape[2]
    sh = (1, 1, C) + (1,) * (x.ndim - 3)
    for i in range(k):
        off = (k - 1 - i) * d
        if off < T:
            out[off:] += w[:, i].astype(np.float64).reshape(sh) * x[:T - off]
    return out


def bn_case(seed=60, T=13, N=3, C=4, S=2, k=3):
    rng = np.random.default_rng(seed)
    x = rng.normal(0.4, 1.0, (T, N, C, S)).astype(np.float32)
    w = rng.normal(0, 0.6, (C, k)).astype(np.float32)
    gamma = rng.uniform(0.5, 1.5, C).astype(np.float32)
    beta = rng.normal(-1.0, 0.2, C).astype(np.float32)
    return x, w, gamma, beta


@pytest.mark.parametrize("d", [1, 3])
def test_bn_statistics_are_mean_and_biased_variance(orc, d):
    x, w, gamma, beta = bn_case()
    k, eps = 3, 1e-5
    r = orc.bn_forward_stats(x, w, gamma, beta, eps, k, d)
    tv = latent_conv(x, w, k, d)
    axes = (0, 1, 3)
    mu, var = tv.mean(axis=axes), tv.var(axis=axes)
    assert np.allclose(r["aux"][:, 0], mu, rtol=1e-12, atol=1e-13)
    assert np.allclose(r["aux"][:, 1], var, rtol=1e-12, atol=1e-13)
    assert np.allclose(r["stats"][:, 0], tv.sum(axis=axes), rtol=1e-12, atol=1e-12)
    assert np.allclose(r["stats"][:, 1], (tv * tv).sum(axis=axes), rtol=1e-12, atol=1e-12)


def test_bn_fusion_identity(orc):
    """Eqs. weight fuse, bias fuse: the fused convolution plus the fused bias
    is the batch-normalized latent convolution, gamma (Tv - mu)/sqrt(var +
    eps) + beta; W_f and b_f are those values rounded to float."""
    x, w, gamma, beta = bn_case(61)
    k, d, eps = 3, 2, 1e-5
    r = orc.bn_forward_stats(x, w, gamma, beta, eps, k, d)
    mu, var, sc, inv = r["aux"].T
    tv = latent_conv(x, w, k, d)
    sh = (1, 1, 4, 1)
    bn = gamma.astype(np.float64).reshape(sh) * (tv - mu.reshape(sh)) * inv.reshape(sh) + beta.reshape(sh)
    fused = latent_conv(x, (sc[:, None] * w.astype(np.float64)), k, d) + (beta - sc * mu).reshape(sh)
    assert np.allclose(fused, bn, rtol=1e-12, atol=1e-12)
    assert np.allclose(inv, 1.0 / np.sqrt(var + eps), rtol=1e-15)
    assert np.array_equal(r["w_f"], (sc[:, None] * w.astype(np.float64)).astype(np.float32))
    assert np.array_equal(r["b_f"], (beta.astype(np.float64) - sc * mu).astype(np.float32))


@pytest.mark.parametrize("d", [1, 2])
def test_bn_backward_matches_finite_differences(orc, d):
    """With the quantizer taken as identity (its straight-through gradient)
    and the Heaviside replaced by a sigmoid of slope alpha, the fused step is
    a smooth function of x, W, gamma and beta; the oracle's backward of the
    fusion and the statistics, fed with that function's gradients of W_f,
    b_f and the quantized-path input gradient, must equal its central finite
    differences."""
    x, w, gamma, beta = bn_case(62 + d)
    k, eps, alpha = 3, 1e-5, 2.0
    rng = np.random.default_rng(70 + d)
    g = rng.normal(0, 1, x.shape)
    sh = (1, 1, x.shape[2], 1)

    def loss(xv, wv, gv, bv):
        tv = latent_conv(xv, wv, k, d)
        mu = tv.mean(axis=(0, 1, 3))
        var = tv.var(axis=(0, 1, 3))
        sc = gv / np.sqrt(var + eps)
        hf = latent_conv(xv, sc[:, None] * wv, k, d) + (bv - sc * mu).reshape(sh)
        return float(np.sum(g / (1.0 + np.exp(-alpha * hf))))

    r = orc.bn_forward_stats(x, w, gamma, beta, eps, k, d)
    mu, var, sc, inv = r["aux"].T
    wf = sc[:, None] * w.astype(np.float64)
    hf = latent_conv(x, wf, k, d) + (beta - sc * mu).reshape(sh)
    sg = 1.0 / (1.0 + np.exp(-alpha * hf))
    dh = g * alpha * sg * (1.0 - sg)
    T = x.shape[0]
    xd = x.astype(np.float64)
    gwf = np.zeros((x.shape[2], k))
    gxq = np.zeros_like(xd)
    for i in range(k):
        off = (k - 1 - i) * d
        if off < T:
            gwf[:, i] = np.sum(dh[off:] * xd[:T - off], axis=(0, 1, 3))
            gxq[:T - off] += wf[:, i].reshape(sh) * dh[off:]
    gbf = dh.sum(axis=(0, 1, 3))
    b = orc.bn_backward(x, w, gamma, eps, r["aux"], gwf, gbf, gxq, k, d)
    h = 1e-6
    for idx in [(0, 0, 0, 0), (5, 1, 2, 1), (T - 1, 2, 3, 0), (T - 4, 0, 1, 1)]:
        xp, xm = xd.copy(), xd.copy()
        xp[idx] += h
        xm[idx] -= h
        fd = (loss(xp, w.astype(np.float64), gamma.astype(np.float64), beta.astype(np.float64)) -
              loss(xm, w.astype(np.float64), gamma.astype(np.float64), beta.astype(np.float64))) / (2 * h)
        assert abs(fd - b["grad_x"][idx]) <= 1e-6 + 1e-5 * abs(fd), ("x", idx, fd, b["grad_x"][idx])
    for c, i in [(0, 0), (2, 2), (3, 1)]:
        wp, wm = w.astype(np.float64), w.astype(np.float64)
        wp[c, i] += h
        wm[c, i] -= h
        fd = (loss(xd, wp, gamma.astype(np.float64), beta.astype(np.float64)) -
              loss(xd, wm, gamma.astype(np.float64), beta.astype(np.float64))) / (2 * h)
        assert abs(fd - b["grad_w"][c, i]) <= 1e-6 + 1e-5 * abs(fd), ("w", c, i, fd, b["grad_w"][c, i])
    for c in range(x.shape[2]):
        for name, which in (("gamma", 0), ("beta", 1)):
            gp, gm = gamma.astype(np.float64), gamma.astype(np.float64)
            bp, bm = beta.astype(np.float64), beta.astype(np.float64)
            if which == 0:
                gp[c] += h
                gm[c] -= h
            else:
                bp[c] += h
                bm[c] -= h
            fd = (loss(xd, w.astype(np.float64), gp, bp) - loss(xd, w.astype(np.float64), gm, bm)) / (2 * h)
            got = b["grad_gamma" if which == 0 else "grad_beta"][c]
            assert abs(fd - got) <= 1e-6 + 1e-5 * abs(fd), (name, c, fd, got)
