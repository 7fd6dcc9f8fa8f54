"""Seeded synthetic workloads for the mul-free channel-wise PSN training step.

This module only draws random inputs; it holds none of the neuron's
arithmetic, so both the HIP path and the oracle can consume what it produces.

The five workloads mirror the shapes of the paper's experiments (no dataset
is read or needed):
  1 tiny             x[64,4,128]          f32  k=8  period 4
  2 audio_spike      x[250,256,512]       f32  k=16 period 4  (SHD-shaped, Sec. 5.1)
  3 seq_image        x[32,128,256,32]     f32  k=8  period 2  (sequential CIFAR-shaped)
  4 event_vision     x[30,32,64,44,44]    bf16 k=8  period 3  (DVS-Lip-shaped)
  5 long_fixed_point x[4096,16,1024]      Q8.8 k=32 period 8  (pixel-CIFAR-length)

Generator: numpy PCG64 seeded with SeedSequence(10_000 + workload id), split
into six child streams used in the order x, sign, shift, bias, grad_spikes,
spare.  Taps are w = sign * 2^-shift with sign uniform in {-1, +1} and shift
uniform in {0..s_max}.  Each workload runs at every dilation d = 1..period,
the per-layer values of the sawtooth schedule with that period.
"""
from __future__ import annotations

import dataclasses

import numpy as np


@dataclasses.dataclass(frozen=True)
class Workload:
    wid: int
    name: str
    T: int
    N: int
    C: int
    spatial: tuple
    k: int
    period: int
    dtype: str          # "f32" | "bf16" | "q8_8"
    s_max: int
    bias: str           # "zero" | "normal0.1"
    v_th: float         # float paths; Q8.8 threshold is round(256 * v_th)
    surrogate: str = "sigmoid"
    alpha: float = 4.0

    @property
    def S(self) -> int:
        return int(np.prod(self.spatial, dtype=np.int64)) if self.spatial else 1

    @property
    def shape(self) -> tuple:
        return (self.T, self.N, self.C, *self.spatial)

    @property
    def elements(self) -> int:
        return self.T * self.N * self.C * self.S

    @property
    def v_th_q(self) -> int:
        return int(round(self.v_th * 256))

    @property
    def dilations(self) -> list:
        return [(layer % self.period) + 1 for layer in range(self.period)]

    def describe(self) -> str:
        dims = ",".join(str(v) for v in self.shape)
        return f"{self.name} x[{dims}] {self.dtype} k={self.k} period={self.period}"


WORKLOADS = {
    1: Workload(1, "tiny", 64, 4, 128, (), 8, 4, "f32", 7, "zero", 1.0),
    2: Workload(2, "audio_spike", 250, 256, 512, (), 16, 4, "f32", 7, "normal0.1", 1.0),
    3: Workload(3, "seq_image", 32, 128, 256, (32,), 8, 2, "f32", 5, "zero", 1.0),
    4: Workload(4, "event_vision", 30, 32, 64, (44, 44), 8, 3, "bf16", 7, "normal0.1", 0.5),
    5: Workload(5, "long_fixed_point", 4096, 16, 1024, (), 32, 8, "q8_8", 7, "zero", 1.0),
}


def _streams(seed: int):
    ss = np.random.SeedSequence(seed)
    return [np.random.Generator(np.random.PCG64(c)) for c in ss.spawn(6)]


def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even.
    Used only to draw bf16-stored inputs."""
    b = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    return ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint16)


def _normal_q88(rng, shape) -> np.ndarray:
    v = np.rint(rng.standard_normal(shape, dtype=np.float64) * 256.0)
    return np.clip(v, -32768, 32767).astype(np.int16)


def _audio_currents(rng, T, N, C, n_in=700, p=0.05, mean=0.5, std=0.2) -> np.ndarray:
    """Synaptic currents: Bernoulli(p) spike counts of n_in inputs times
    N(mean, std^2) synaptic weights, summed over the inputs (float64 sum,
    rounded once to float32)."""
    wsyn = rng.normal(mean, std, size=(n_in, C))
    out = np.empty((T, N, C), np.float32)
    rows = T * N
    flat = out.reshape(rows, C)
    step = 4096
    for r0 in range(0, rows, step):
        r1 = min(rows, r0 + step)
        spikes = (rng.random((r1 - r0, n_in)) < p).astype(np.float64)
        flat[r0:r1] = (spikes @ wsyn).astype(np.float32)
    return out


def make_inputs(wl: Workload, seed: int | None = None) -> dict:
    """Draw x, grad_spikes, sign, shift, bias for a workload.

    Returns numpy arrays: x / grad_spikes are float32 (f32), uint16 bfloat16
    bit patterns (bf16) or int16 (q8_8); sign/shift int8 [C, k]; bias float32
    [C] (int32 [C] for q8_8)."""
    seed = 10_000 + wl.wid if seed is None else seed
    rx, rsign, rshift, rbias, rg, _ = _streams(seed)
    shape = wl.shape
    C, k = wl.C, wl.k
    sign = np.where(rsign.integers(0, 2, size=(C, k)) == 0, -1, 1).astype(np.int8)
    shift = rshift.integers(0, wl.s_max + 1, size=(C, k)).astype(np.int8)
    if wl.dtype == "q8_8":
        x = _normal_q88(rx, shape)
        g = _normal_q88(rg, shape)
        if wl.bias == "zero":
            bias = np.zeros(C, np.int32)
        else:
            bias = np.rint(rbias.normal(0.0, 0.1, size=C) * 256).astype(np.int32)
        return {"x": x, "grad_spikes": g, "sign": sign, "shift": shift, "bias": bias}
    if wl.name == "audio_spike":
        x32 = _audio_currents(rx, wl.T, wl.N, wl.C)
    else:
        x32 = rx.standard_normal(shape, dtype=np.float32)
    g32 = rg.standard_normal(shape, dtype=np.float32)
    if wl.bias == "zero":
        bias = np.zeros(C, np.float32)
    else:
        bias = rbias.normal(0.0, 0.1, size=C).astype(np.float32)
    if wl.dtype == "bf16":
        return {"x": to_bf16_bits(x32).reshape(shape), "grad_spikes": to_bf16_bits(g32).reshape(shape),
                "sign": sign, "shift": shift, "bias": bias}
    return {"x": x32, "grad_spikes": g32, "sign": sign, "shift": shift, "bias": bias}


def make_small(T, N, C, spatial=(), k=4, s_lo=0, s_hi=7, dtype="f32", seed=0, bias_std=0.1,
               x_scale=1.0) -> dict:
    """Small seeded case for parity sweeps (same distributions as above)."""
    rx, rsign, rshift, rbias, rg, _ = _streams(seed)
    shape = (T, N, C, *spatial)
    sign = np.where(rsign.integers(0, 2, size=(C, k)) == 0, -1, 1).astype(np.int8)
    shift = rshift.integers(s_lo, s_hi + 1, size=(C, k)).astype(np.int8)
    if dtype == "q8_8":
        x = _normal_q88(rx, shape)
        g = _normal_q88(rg, shape)
        bias = np.rint(rbias.normal(0.0, bias_std, size=C) * 256).astype(np.int32)
        return {"x": x, "grad_spikes": g, "sign": sign, "shift": shift, "bias": bias}
    x32 = (rx.standard_normal(shape, dtype=np.float32) * np.float32(x_scale)).astype(np.float32)
    g32 = rg.standard_normal(shape, dtype=np.float32)
    bias = rbias.normal(0.0, bias_std, size=C).astype(np.float32)
    if dtype == "bf16":
        return {"x": to_bf16_bits(x32).reshape(shape), "grad_spikes": to_bf16_bits(g32).reshape(shape),
                "sign": sign, "shift": shift, "bias": bias}
    return {"x": x32, "grad_spikes": g32, "sign": sign, "shift": shift, "bias": bias}
