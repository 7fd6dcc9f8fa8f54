#!/usr/bin/env python3
"""Benchmark of the mul-free channel-wise PSN training step on one MI355X.

A step is one training pass of a sawtooth stack of P neuron layers over one
batch: the forward of every layer (dilations d = 1..P in layer order), then
the backward of every layer in reverse order, as autograd would run them.
Each layer reads its own x and grad_spikes tensors (the batch rolled along N).
Inputs are resident in HBM, and the last-level cache is cold for every call:
before each forward and backward a 1 GiB scratch buffer is read on the same
stream, outside the HIP events that time the call.

The headline workload (default) is the event-vision shape x[30,32,64,44,44],
bf16 storage with f32 arithmetic, k = 8, sawtooth period 3 (the largest
single-GPU workload); the same run measures the audio-spike, sequential-image
and long fixed-point workloads under "configs".

Prints ONE JSON line on stdout (everything else goes to stderr):
  value      = P * T*N*C*S / step time, the step time being the sum of the
               per-call durations (HIP events on the launch stream, cold
               cache) of the P forwards and P backwards (elements/s)
  roofline   = the dominant kernel, mfpsn_backward (bwd_kernel + fin_kernel):
               algorithmic bytes per launch (read x, read grad_spikes, write
               grad_x) / its average event-timed duration, against 8 TB/s;
               traffic = HBM bytes per launch from the committed rocprofv3
               counter summary (null when it was taken on other kernel
               sources); fwd_bwd = the same for forward + backward together
  configs    = the other workloads, each with per-dilation call times and
               algorithmic-bandwidth fractions
  cpu_baseline = the oracle (single-threaded C) timed on this host on a
               channel slice of the headline workload
The events are created without the system-scope fence
(hipEventDisableSystemFence), so recording them does not write back and
invalidate the caches between launches.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0

BACKWARD_INPUTS = ("recompute", "h", "sg")
# what the forward saves for the backward in each workload (the fastest step
# measured on MI355X)
AUTO_BACKWARD_INPUT = {1: "recompute", 2: "recompute", 3: "recompute", 4: "recompute", 5: "sg"}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def alg_bytes(wl):
    """Algorithmic HBM bytes per element (forward, backward)."""
    es = {"f32": 4, "bf16": 2, "q8_8": 2}[wl.dtype]
    gxs = {"f32": 4, "bf16": 2, "q8_8": 4}[wl.dtype]
    return es + 1, es + es + gxs


KERNEL_SOURCES = ("mfpsn_kernels.hip", "mfpsn_api.cpp", "mfpsn_internal.h", "mfpsn_surrogate.h")
COUNTERS_FILE = os.path.join(ROOT, "profiles", "counters.json")
SIMDS, CLOCK_HZ = 1024, 2.4e9   # MI355X: 256 CUs x 4 SIMDs, peak engine clock
VALU_CYCLES = 2                 # cycles per plain wave64 VALU instruction on one SIMD


def kernel_source_hash():
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(os.path.join(ROOT, "paper_2501_14490_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def committed_counters(wl_name, mode):
    """The committed rocprofv3 counter summary of a workload (HBM bytes and
    VALU instructions per launch), if it was taken on the current kernel
    sources; else None."""
    try:
        rec = json.load(open(COUNTERS_FILE))
    except (OSError, ValueError):
        return None
    ent = rec.get(f"{wl_name}|{mode}")
    if not ent or ent.get("kernel_source") != kernel_source_hash():
        return None
    return ent


def cpu_model() -> str:
    """The host CPU's model name as lscpu reports it (else /proc/cpuinfo)."""
    import subprocess

    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.strip().startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


class HipEvents:
    """Timing events of the HIP runtime, recorded on a given stream, created
    without the system-scope release fence (which would add a cache write-back
    and invalidate between the kernels they separate)."""

    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self):
        import ctypes

        self.ct = ctypes
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def new(self):
        e = self.ct.c_void_p()
        rc = self.hip.hipEventCreateWithFlags(self.ct.byref(e), self.DISABLE_SYSTEM_FENCE)
        if rc != 0:
            raise RuntimeError(f"hipEventCreateWithFlags failed ({rc})")
        return e

    def record(self, e, stream):
        rc = self.hip.hipEventRecord(e, self.ct.c_void_p(stream.cuda_stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed ({rc})")

    def elapsed_ms(self, a, b) -> float:
        ms = self.ct.c_float()
        rc = self.hip.hipEventElapsedTime(self.ct.byref(ms), a, b)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return float(ms.value)


def cpu_baseline(wl, case, channels: int):
    import oracle

    oracle.build()
    sub = {n: (np.ascontiguousarray(v[:, :, :channels]) if n in ("x", "grad_spikes") else v[:channels])
           for n, v in case.items()}
    t0 = time.perf_counter()
    for d in wl.dilations:
        if wl.dtype == "q8_8":
            oracle.forward_q88(sub["x"], sub["sign"], sub["shift"], sub["bias"], wl.k, d, wl.v_th_q, 0, wl.s_max)
            oracle.backward_q88(sub["x"], sub["grad_spikes"], sub["sign"], sub["shift"], sub["bias"], wl.k, d,
                                wl.v_th_q, wl.surrogate, wl.alpha, 0, wl.s_max)
        elif wl.dtype == "bf16":
            oracle.forward_bf16(sub["x"], sub["sign"], sub["shift"], sub["bias"], wl.k, d, wl.v_th,
                                shift_lo=0, shift_hi=wl.s_max)
            oracle.backward_bf16(sub["x"], sub["grad_spikes"], sub["sign"], sub["shift"], sub["bias"], wl.k, d,
                                 wl.v_th, surrogate_kind=wl.surrogate, alpha=wl.alpha, shift_lo=0,
                                 shift_hi=wl.s_max)
        else:
            oracle.forward_f32(sub["x"], sub["sign"], sub["shift"], sub["bias"], wl.k, d, wl.v_th, 0, wl.s_max)
            oracle.backward_f32(sub["x"], sub["grad_spikes"], sub["sign"], sub["shift"], sub["bias"], wl.k, d,
                                wl.v_th, wl.surrogate, wl.alpha, 0, wl.s_max)
    dt = time.perf_counter() - t0
    elems = wl.T * wl.N * channels * wl.S * len(wl.dilations)
    return {"value": elems / dt, "unit": "elements/s", "cores": 1, "kind": "oracle",
            "cpu": cpu_model(), "nproc": os.cpu_count(),
            "sample": f"{channels} of {wl.C} channels ({elems} element-layers, every dilation), "
                      f"fwd+bwd in {dt:.1f} s, single thread"}


def memory_ceiling(torch, dev, wl):
    """Bandwidth of torch's own elementwise kernels on float32 tensors with the
    workload's element count: copy (8 B/el) and addcmul (3 reads + 1 write,
    16 B/el: the saved-factor backward's mix)."""
    n = wl.elements
    a, b, c, o = (torch.ones(n, dtype=torch.float32, device=dev) for _ in range(4))
    res = {}
    for name, fn, bpe in (("copy_1r1w", lambda: o.copy_(a), 8),
                          ("addcmul_3r1w", lambda: torch.addcmul(a, b, c, out=o), 16)):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        reps = 20
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / reps
        res[name] = {"us": round(us, 2), "GB/s": round(bpe * n / (us * 1e-6) / 1e9, 1)}
        log(f"{name}: {us:.1f} us  {res[name]['GB/s']:.0f} GB/s")
    print(json.dumps({"memory_ceiling": res, "elements": n, "workload": wl.name}), flush=True)


def stream_inference(torch, dev, wl, case, reps: int, warmup: int):
    """Step-by-step inference of the workload's layers (one per dilation, each
    with its own input sequence): for t = 0..T-1, one mfpsn_stream_step per
    layer, each layer on its own history ring of (k-1)d+1 steps.  The whole
    sequence is captured once in a HIP graph (no slot of a fresh ring is read
    before it is written, so every replay recomputes the sequence) and
    replayed; value = layers * T * N*C*S / replay time."""
    from paper_2501_14490_amd import mfpsn

    def dev_tensor(a, storage):
        if wl.dtype == "bf16" and storage:
            return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    x0 = dev_tensor(case["x"], True)
    sign, shift, bias = (dev_tensor(case[n], False) for n in ("sign", "shift", "bias"))
    es = {"f32": 4, "bf16": 2, "q8_8": 2}[wl.dtype]
    M = wl.N * wl.C * wl.S
    layers, alg_bytes, ring_bytes = [], 0, 0
    for li, d in enumerate(wl.dilations):
        desc = mfpsn.make_desc(wl.shape, wl.k, d, wl.dtype, wl.surrogate, wl.alpha, wl.v_th, wl.v_th_q, 0,
                               wl.s_max)
        x = torch.roll(x0, shifts=7 * li, dims=1).contiguous() if li else x0
        st = mfpsn.StreamState(desc, x.shape[1:], sign, shift, bias)
        ring_bytes += st.ring.numel() * st.ring.element_size()
        spikes = torch.empty(x.shape, dtype=torch.uint8, device=dev)
        layers.append((st, x, spikes))
        # per step: read x_t, store it in the ring, read the older inputs the
        # taps reach (fewer at the start), write the spike byte
        alg_bytes += sum(M * (2 * es + min(wl.k - 1, t // d) * es + 1) for t in range(wl.T))
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())

    def sequence():
        for st, _, _ in layers:
            st.t = 0
        for t in range(wl.T):
            for st, x, spikes in layers:
                st.step(x[t], stream=side, out=(spikes[t], None))

    with torch.cuda.stream(side):
        sequence()  # eager run (also loads the kernels)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            sequence()
    torch.cuda.synchronize()
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    hev = HipEvents()
    e0, e1 = hev.new(), hev.new()
    cur = torch.cuda.current_stream()
    hev.record(e0, cur)
    for _ in range(reps):
        g.replay()
    hev.record(e1, cur)
    torch.cuda.synchronize()
    ms = hev.elapsed_ms(e0, e1) / reps
    P = len(wl.dilations)
    calls = P * wl.T
    value = calls * M / (ms * 1e-3)
    achieved = alg_bytes / (ms * 1e-3) / 1e9
    log(f"stream inference: {ms * 1e3:.1f} us per sequence ({calls} steps, {ms * 1e3 / calls:.2f} us/step), "
        f"{value / 1e9:.2f} G elements/s, {achieved:.0f} GB/s of step traffic")
    print(json.dumps({
        "metric": "step-by-step inference elements/s (T*N*C*S per layer)",
        "value": value, "unit": "elements/s", "n_gpus": 1, "steps": reps, "warmup": warmup,
        "ms_per_sequence": ms, "higher_is_better": True, "dtype": {"f32": "f32", "bf16": "bf16",
                                                                   "q8_8": "int16 Q8.8 / int32"}[wl.dtype],
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: x[{','.join(map(str, wl.shape))}] {wl.dtype}, k={wl.k}, one layer "
                               f"per d={wl.dilations}, one mfpsn_stream_step per layer and time step, "
                               f"the sequence replayed from a HIP graph",
                   "calls_per_sequence": calls, "ring_bytes_all_layers": ring_bytes},
        "step_traffic": {"alg_bytes_per_sequence": alg_bytes, "achieved_GBs": achieved,
                         "us_per_step": ms * 1e3 / calls,
                         "note": "the rings are small enough to stay in the on-chip caches"},
    }), flush=True)


def bn_step(torch, dev, wl, case, steps: int, warmup: int):
    """The batch-normalized-threshold training step of App. C for the
    workload's layers (float storage): per layer, mfpsn_bn_forward_stats
    (statistics of the latent-weight convolution and the fusion),
    mfpsn_quantize_weights(W_f), mfpsn_forward (bias b_f, threshold 0, saving
    the surrogate factor); then per layer in reverse, mfpsn_backward and
    mfpsn_bn_backward.  value = layers * T*N*C*S / step time."""
    from paper_2501_14490_amd import mfpsn

    if wl.dtype != "f32":
        log("the batch-normalized step takes float x: choose an f32 workload")
        sys.exit(2)
    rng = np.random.default_rng(90)
    x0 = torch.from_numpy(np.ascontiguousarray(case["x"])).to(dev)
    g0 = torch.from_numpy(np.ascontiguousarray(case["grad_spikes"])).to(dev)
    P = len(wl.dilations)
    eps = 1e-5
    layers = []
    for li, d in enumerate(wl.dilations):
        desc = mfpsn.make_desc(wl.shape, wl.k, d, "f32", wl.surrogate, wl.alpha, 0.0, 0, 0, wl.s_max)
        C, k = wl.C, wl.k
        L = {"d": d, "desc": desc,
             "x": torch.roll(x0, shifts=7 * li, dims=1).contiguous() if li else x0,
             "g": torch.roll(g0, shifts=11 * li, dims=1).contiguous() if li else g0,
             "w": torch.from_numpy(rng.normal(0, 0.3, (C, k)).astype(np.float32)).to(dev),
             "gamma": torch.ones(C, dtype=torch.float32, device=dev),
             "beta": torch.full((C,), -1.0, dtype=torch.float32, device=dev),  # the paper's initialization
             "w_f": torch.empty((C, k), dtype=torch.float32, device=dev),
             "b_f": torch.empty(C, dtype=torch.float32, device=dev),
             "aux": torch.empty((C, 4), dtype=torch.float64, device=dev),
             "sign": torch.empty((C, k), dtype=torch.int8, device=dev),
             "shift": torch.empty((C, k), dtype=torch.int8, device=dev),
             "spikes": torch.empty(wl.shape, dtype=torch.uint8, device=dev),
             "sg": torch.empty(wl.shape, dtype=torch.float32, device=dev),
             "gx": torch.empty(wl.shape, dtype=torch.float32, device=dev),
             "gwf": torch.empty((C, k), dtype=torch.float32, device=dev),
             "gbf": torch.empty(C, dtype=torch.float32, device=dev),
             "gw": torch.empty((C, k), dtype=torch.float32, device=dev),
             "ggamma": torch.empty(C, dtype=torch.float32, device=dev),
             "gbeta": torch.empty(C, dtype=torch.float32, device=dev),
             "ws": torch.empty(max(mfpsn.mfpsn_backward_workspace_size(desc), 8), dtype=torch.uint8, device=dev),
             "bnws": mfpsn.bn_workspace(desc, dev)}
        layers.append(L)
    del x0, g0
    stream = torch.cuda.current_stream()
    hev = HipEvents()
    stages = ("stats", "quantize", "forward", "backward", "bn_backward")

    def step(ev=None):
        def mark(name, li, end):
            if ev is not None:
                hev.record(ev[(name, li)][end], stream)
        for li, L in enumerate(layers):
            mark("stats", li, 0)
            mfpsn.mfpsn_bn_forward_stats(L["desc"], L["x"], L["w"], L["gamma"], L["beta"], eps, L["w_f"], L["b_f"],
                                         L["aux"], None, L["bnws"], stream)
            mark("stats", li, 1)
            mark("quantize", li, 0)
            mfpsn.mfpsn_quantize_weights(L["w_f"], 0, wl.s_max, L["sign"], L["shift"], stream)
            mark("quantize", li, 1)
            mark("forward", li, 0)
            mfpsn.mfpsn_forward(L["desc"], L["x"], L["sign"], L["shift"], L["b_f"], None, L["spikes"], None, L["sg"],
                                stream)
            mark("forward", li, 1)
        for li in reversed(range(P)):
            L = layers[li]
            mark("backward", li, 0)
            mfpsn.mfpsn_backward(L["desc"], L["x"], L["g"], None, L["sg"], L["sign"], L["shift"], L["b_f"], None,
                                 L["gx"], L["gwf"], L["gbf"], None, L["ws"], stream=stream)
            mark("backward", li, 1)
            mark("bn_backward", li, 0)
            mfpsn.mfpsn_bn_backward(L["desc"], L["x"], L["w"], L["aux"], eps, L["gwf"], L["gbf"], L["gx"], L["gw"],
                                    L["ggamma"], L["gbeta"], L["bnws"], stream)
            mark("bn_backward", li, 1)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    evs = [{(n, li): [hev.new(), hev.new()] for n in stages for li in range(P)} for _ in range(steps)]
    t0 = time.perf_counter()
    for s_ in range(steps):
        step(evs[s_])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    per_stage = {n: round(float(np.mean([hev.elapsed_ms(*e[(n, li)]) for e in evs for li in range(P)])) * 1e3, 2)
                 for n in stages}
    value = P * wl.elements / (elapsed / steps)
    log(f"bn step {elapsed * 1e3 / steps:.3f} ms, {value / 1e9:.2f} G elements/s, per layer (us): {per_stage}")
    print(json.dumps({
        "metric": "batch-normalized-threshold training step elements/s (T*N*C*S per layer)",
        "value": value, "unit": "elements/s", "n_gpus": 1, "steps": steps, "warmup": warmup,
        "ms_per_step": elapsed * 1e3 / steps, "higher_is_better": True, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"{wl.name}: x[{','.join(map(str, wl.shape))}] f32, k={wl.k}, one layer per "
                               f"d={wl.dilations}; statistics + fusion, quantize, forward, backward, "
                               f"backward of the statistics",
                   "eps": eps, "gamma_init": 1.0, "beta_init": -1.0},
        "per_layer_us": per_stage,
    }), flush=True)


def stack_step(torch, dev, wl, case, mode: str, steps: int, warmup: int):
    """The sawtooth stack: the workload's layers (one per dilation) chained
    through identity stateless layers.  Forward: layer l's spikes become
    layer l+1's input (mfpsn_spikes_to_input); backward: layer l+1's grad_x is
    layer l's grad_spikes.  Float storage types only.  value = layers *
    T*N*C*S / step time, the casts included."""
    from paper_2501_14490_amd import mfpsn

    if wl.dtype == "q8_8":
        log("the chained stack takes float or bfloat16 storage: choose an f32 or bf16 workload")
        sys.exit(2)

    def dev_tensor(a, storage):
        if wl.dtype == "bf16" and storage:
            return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    x0 = dev_tensor(case["x"], True)
    g_top = dev_tensor(case["grad_spikes"], True)
    sign = dev_tensor(case["sign"], False)
    shift = dev_tensor(case["shift"], False)
    bias = dev_tensor(case["bias"], False)
    P = len(wl.dilations)
    layers = []
    for li, d in enumerate(wl.dilations):
        desc = mfpsn.make_desc(wl.shape, wl.k, d, wl.dtype, wl.surrogate, wl.alpha, wl.v_th, wl.v_th_q, 0,
                               wl.s_max)
        layers.append({
            "d": d, "desc": desc,
            "x": x0 if li == 0 else torch.empty(wl.shape, dtype=x0.dtype, device=dev),
            "ws": torch.empty(max(mfpsn.mfpsn_backward_workspace_size(desc), 8), dtype=torch.uint8, device=dev),
            "spikes": torch.empty(wl.shape, dtype=torch.uint8, device=dev),
            "gx": torch.empty(wl.shape, dtype=mfpsn.GRAD_X[desc.dtype], device=dev),
            "h": torch.empty(wl.shape, dtype=mfpsn.H_OUT[desc.dtype], device=dev) if mode == "h" else None,
            "sg": torch.empty(wl.shape, dtype=mfpsn.SG_OUT[desc.dtype], device=dev) if mode == "sg" else None,
            "gw": torch.empty((wl.C, wl.k), dtype=mfpsn.GRAD_WB[desc.dtype], device=dev),
            "gb": torch.empty((wl.C,), dtype=mfpsn.GRAD_WB[desc.dtype], device=dev),
        })
    stream = torch.cuda.current_stream()
    dt = mfpsn.DTYPES[wl.dtype]

    def step():
        for li, L in enumerate(layers):
            mfpsn.mfpsn_forward(L["desc"], L["x"], sign, shift, bias, None, L["spikes"], L["h"], L["sg"], stream)
            if li + 1 < P:
                mfpsn.mfpsn_spikes_to_input(L["spikes"], dt, layers[li + 1]["x"], stream)
        g = g_top
        for li in reversed(range(P)):
            L = layers[li]
            mfpsn.mfpsn_backward(L["desc"], L["x"], g, L["h"], L["sg"], sign, shift, bias, None, L["gx"], L["gw"],
                                 L["gb"], None, L["ws"], stream=stream)
            g = L["gx"]

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    value = P * wl.elements / (elapsed / steps)
    rate = float(torch.cat([L["spikes"].reshape(-1)[: 1 << 20].float().mean().reshape(1) for L in layers]).mean())
    log(f"stack step {elapsed * 1e3 / steps:.3f} ms, {value / 1e9:.2f} G elements/s, "
        f"mean firing rate of the layers {rate:.3f}")
    print(json.dumps({
        "metric": "chained sawtooth stack fwd+bwd elements/s (T*N*C*S per layer)",
        "value": value, "unit": "elements/s", "n_gpus": 1, "steps": steps, "warmup": warmup,
        "ms_per_step": elapsed * 1e3 / steps, "higher_is_better": True, "dtype": wl.dtype, "data": "synthetic",
        "config": {"workload": f"{wl.name}: x[{','.join(map(str, wl.shape))}] {wl.dtype}, k={wl.k}, layers "
                               f"d={wl.dilations} chained (spikes of one layer are the next layer's input); "
                               f"forward of every layer, then backward in reverse",
                   "backward_input": mode},
    }), flush=True)


def time_last(torch, dev, wl, case, steps: int, warmup: int):
    """The workload's layers in the time-last layout [N][C][S][T], timed beside
    the time-first entry points on the same inputs: the forward (charge and
    fire, spikes only; mfpsn_forward_time_last) and the backward
    (mfpsn_backward_time_last, H recomputed).
    value = layers * T*N*C*S / time of the time-last step; roofline: the
    dominant kernel's algorithmic bytes per launch (backward: x, grad_spikes
    read, grad_x written; forward: x read, spikes written) over its average
    duration."""
    from paper_2501_14490_amd import mfpsn

    es = {"f32": 4, "bf16": 2, "q8_8": 2}[wl.dtype]
    gxs = {"f32": 4, "bf16": 2, "q8_8": 4}[wl.dtype]
    with_bwd = (wl.k - 1) * max(wl.dilations) <= 1024 or wl.shape[0] <= 64
    raw = {}
    for name in ("x", "grad_spikes"):
        a = case[name]
        raw[name] = a.view(np.int16) if wl.dtype == "bf16" else a

    def up(a):
        t = torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        return t.view(torch.bfloat16) if wl.dtype == "bf16" else t

    xs = {"tf": up(raw["x"]), "tl": up(np.moveaxis(raw["x"], 0, -1))}
    gs = {"tf": up(raw["grad_spikes"]), "tl": up(np.moveaxis(raw["grad_spikes"], 0, -1))}
    tl_shape = tuple(xs["tl"].shape)
    sign, shift, bias = (torch.from_numpy(np.ascontiguousarray(case[n])).to(dev) for n in ("sign", "shift", "bias"))
    descs = [mfpsn.make_desc(wl.shape, wl.k, d, wl.dtype, wl.surrogate, wl.alpha, wl.v_th, wl.v_th_q, 0, wl.s_max)
             for d in wl.dilations]
    shapes = {"tl": tl_shape, "tf": tuple(wl.shape)}
    spk = {lay: torch.empty(shapes[lay], dtype=torch.uint8, device=dev) for lay in shapes}
    gx = {lay: torch.empty(shapes[lay], dtype=mfpsn.GRAD_X[descs[0].dtype], device=dev) for lay in shapes}
    gw = torch.empty((wl.C, wl.k), dtype=mfpsn.GRAD_WB[descs[0].dtype], device=dev)
    gb = torch.empty((wl.C,), dtype=mfpsn.GRAD_WB[descs[0].dtype], device=dev)
    ws_bytes = max(max(mfpsn.mfpsn_backward_workspace_size(d), mfpsn.mfpsn_backward_time_last_workspace_size(d))
                   for d in descs)
    ws = torch.empty(max(ws_bytes, 8), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    hev = HipEvents()

    def run(layout, ev=None):
        for li, desc in enumerate(descs):
            if ev is not None:
                hev.record(ev[li][0], stream)
            if layout == "tl":
                mfpsn.mfpsn_forward_time_last(desc, xs["tl"], sign, shift, bias, spk["tl"], None, stream)
            else:
                mfpsn.mfpsn_forward(desc, xs["tf"], sign, shift, bias, None, spk["tf"], None, None, stream)
            if ev is not None:
                hev.record(ev[li][1], stream)
        if not with_bwd:
            return
        for li in reversed(range(len(descs))):
            desc = descs[li]
            if ev is not None:
                hev.record(ev[li][2], stream)
            if layout == "tl":
                mfpsn.mfpsn_backward_time_last(desc, xs["tl"], gs["tl"], sign, shift, bias, gx["tl"], gw, gb, ws,
                                               stream)
            else:
                mfpsn.mfpsn_backward(desc, xs["tf"], gs["tf"], None, None, sign, shift, bias, None, gx["tf"], gw, gb, None,
                                     ws, stream=stream)
            if ev is not None:
                hev.record(ev[li][3], stream)

    out = {}
    for layout in ("tl", "tf"):
        for _ in range(warmup):
            run(layout)
        torch.cuda.synchronize()
        evs = [[[hev.new() for _ in range(4)] for _ in descs] for _ in range(steps)]
        t0 = time.perf_counter()
        for s_ in range(steps):
            run(layout, evs[s_])
        torch.cuda.synchronize()
        out[layout] = {"elapsed": (time.perf_counter() - t0) / steps,
                       "fwd_ms": float(np.mean([hev.elapsed_ms(e[0], e[1]) for st in evs for e in st]))}
        if with_bwd:
            out[layout]["bwd_ms"] = float(np.mean([hev.elapsed_ms(e[2], e[3]) for st in evs for e in st]))
    same = bool(torch.equal(spk["tl"].cpu(), torch.from_numpy(np.ascontiguousarray(
        np.moveaxis(spk["tf"].cpu().numpy(), 0, -1)))))
    P = len(descs)
    value = P * wl.elements / out["tl"]["elapsed"]
    if with_bwd:
        alg, ms, kern = wl.elements * (2 * es + gxs), out["tl"]["bwd_ms"], "backward"
    else:
        alg, ms, kern = wl.elements * (es + 1), out["tl"]["fwd_ms"], "forward"
    ach = alg / (ms * 1e-3) / 1e9
    line = (f"time-last forward {out['tl']['fwd_ms'] * 1e3:.1f} us per layer, time-first "
            f"{out['tf']['fwd_ms'] * 1e3:.1f} us")
    if with_bwd:
        line += (f"; backward {out['tl']['bwd_ms'] * 1e3:.1f} us per layer, time-first "
                 f"{out['tf']['bwd_ms'] * 1e3:.1f} us")
    log(f"{line}; {value / 1e9:.2f} G elements/s; {kern} {ach:.0f} GB/s alg; last layer's spikes equal: {same}")
    rec = {
        "metric": "time-last " + ("forward+backward" if with_bwd else "forward") + " elements/s (T*N*C*S per layer)",
        "value": value, "unit": "elements/s", "n_gpus": 1, "steps": steps, "warmup": warmup,
        "ms_per_step": out["tl"]["elapsed"] * 1e3, "higher_is_better": True, "dtype": wl.dtype, "data": "synthetic",
        "config": {"workload": f"{wl.name}: x[{','.join(map(str, tl_shape))}] {wl.dtype} time last, k={wl.k}, "
                               f"one layer per d={wl.dilations}; forward (spikes only)"
                               + (" and backward (H recomputed)" if with_bwd else "")},
        "roofline": {"bound": "hbm", "kernel": kern, "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": ach / HBM_PEAK_GBS},
        "time_first_forward_us_per_layer": out["tf"]["fwd_ms"] * 1e3,
        "time_last_forward_us_per_layer": out["tl"]["fwd_ms"] * 1e3,
        "spikes_equal_time_first": same,
    }
    if with_bwd:
        rec["time_first_backward_us_per_layer"] = out["tf"]["bwd_ms"] * 1e3
        rec["time_last_backward_us_per_layer"] = out["tl"]["bwd_ms"] * 1e3
    print(json.dumps(rec), flush=True)


class Flush:
    """A 1 GiB device buffer read before every timed call (on the call's
    stream, outside its events), so no call finds its inputs in the 256 MB
    last-level (memory-side) cache or the L2s: every timed byte comes from
    HBM.  The buffer is read, not written: a write would leave up to 256 MB
    of dirty lines that the timed kernel would then have to write back,
    charging it for the flush's own traffic; after a read every line is
    clean."""

    BYTES = 1 << 30

    def __init__(self, torch, dev):
        self.torch = torch
        self.buf = torch.ones(self.BYTES // 4, dtype=torch.float32, device=dev)
        self.acc = torch.zeros((), dtype=torch.float32, device=dev)

    def __call__(self):
        # a float sum reduces the buffer in place (an int32 sum into int64
        # first writes a converted 2 GiB copy, whose dirty lines the timed
        # call would then evict)
        self.acc += self.buf.sum()


def measure(torch, dev, wl, mode, steps: int, warmup: int, flush, hev):
    """Time `steps` training steps of the workload's sawtooth stack (P layers,
    forward of every layer then backward in reverse), every call cold.
    Returns the per-call averages and the derived rates."""
    from paper_2501_14490_amd import mfpsn, workloads

    t0 = time.time()
    case = workloads.make_inputs(wl)
    log(f"{wl.name}: inputs drawn in {time.time() - t0:.1f}s")

    def dev_tensor(a, storage):
        if wl.dtype == "bf16" and storage:
            return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    x0 = dev_tensor(case["x"], True)
    g0 = dev_tensor(case["grad_spikes"], True)
    sign = dev_tensor(case["sign"], False)
    shift = dev_tensor(case["shift"], False)
    bias = dev_tensor(case["bias"], False)
    del case
    P = len(wl.dilations)
    layers = []
    for li, d in enumerate(wl.dilations):
        x = torch.roll(x0, shifts=7 * li, dims=1).contiguous() if li else x0
        g = torch.roll(g0, shifts=11 * li, dims=1).contiguous() if li else g0
        desc = mfpsn.make_desc(wl.shape, wl.k, d, wl.dtype, wl.surrogate, wl.alpha, wl.v_th, wl.v_th_q, 0,
                               wl.s_max)
        ws = torch.empty(max(mfpsn.mfpsn_backward_workspace_size(desc), 8), dtype=torch.uint8, device=dev)
        layers.append({
            "d": d, "desc": desc, "x": x, "g": g, "ws": ws,
            "spikes": torch.empty(wl.shape, dtype=torch.uint8, device=dev),
            "gx": torch.empty(wl.shape, dtype=mfpsn.GRAD_X[desc.dtype], device=dev),
            "h": torch.empty(wl.shape, dtype=mfpsn.H_OUT[desc.dtype], device=dev) if mode == "h" else None,
            "sg": torch.empty(wl.shape, dtype=mfpsn.SG_OUT[desc.dtype], device=dev) if mode == "sg" else None,
            "gw": torch.empty((wl.C, wl.k), dtype=mfpsn.GRAD_WB[desc.dtype], device=dev),
            "gb": torch.empty((wl.C,), dtype=mfpsn.GRAD_WB[desc.dtype], device=dev),
        })
    del x0, g0
    stream = torch.cuda.current_stream()

    def step(events=None):
        for li, L in enumerate(layers):
            flush()
            if events is not None:
                hev.record(events[("fwd", li)][0], stream)
            mfpsn.mfpsn_forward(L["desc"], L["x"], sign, shift, bias, None, L["spikes"], L["h"], L["sg"], stream)
            if events is not None:
                hev.record(events[("fwd", li)][1], stream)
        for li in reversed(range(P)):
            L = layers[li]
            flush()
            if events is not None:
                hev.record(events[("bwd", li)][0], stream)
            mfpsn.mfpsn_backward(L["desc"], L["x"], L["g"], L["h"], L["sg"], sign, shift, bias, None, L["gx"],
                                 L["gw"], L["gb"], None, L["ws"], stream=stream)
            if events is not None:
                hev.record(events[("bwd", li)][1], stream)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    ev = {(kind, li): [[hev.new(), hev.new()] for _ in range(steps)]
          for kind in ("fwd", "bwd") for li in range(P)}
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for st in range(steps):
        step({key: ev[key][st] for key in ev})
        if st % 10 == 9:
            log(f"  {wl.name}: step {st + 1}/{steps}")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start

    def avg_us(kind, li):
        return 1e3 * float(np.mean([hev.elapsed_ms(a, b) for a, b in ev[(kind, li)]]))

    fb, bb = alg_bytes(wl)
    elems = wl.elements
    per_d = {}
    for li, L in enumerate(layers):
        f_us, b_us = avg_us("fwd", li), avg_us("bwd", li)
        per_d[f"d{L['d']}"] = {
            "fwd_us": round(f_us, 2), "bwd_us": round(b_us, 2),
            "fwd_frac": round(elems * fb / (f_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
            "bwd_frac": round(elems * bb / (b_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
            "fwd_bwd_frac": round(elems * (fb + bb) / ((f_us + b_us) * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}
    fwd_us = float(np.mean([v["fwd_us"] for v in per_d.values()]))
    bwd_us = float(np.mean([v["bwd_us"] for v in per_d.values()]))
    step_us = P * (fwd_us + bwd_us)
    for L in layers:
        L.clear()
    torch.cuda.empty_cache()
    return {
        "wl": wl, "mode": mode, "P": P, "per_d": per_d, "fwd_us": fwd_us, "bwd_us": bwd_us,
        "step_ms": step_us / 1e3, "wall_ms_per_step": wall * 1e3 / steps,
        "value": P * elems / (step_us * 1e-6),
        "fwd_bytes": elems * fb, "bwd_bytes": elems * bb,
        "fwd_GBs": elems * fb / (fwd_us * 1e-6) / 1e9, "bwd_GBs": elems * bb / (bwd_us * 1e-6) / 1e9,
        "fwd_bwd_GBs": elems * (fb + bb) / ((fwd_us + bwd_us) * 1e-6) / 1e9,
    }


def describe(wl, P):
    storage = {"f32": "f32", "bf16": "bf16 storage with f32 arithmetic",
               "q8_8": "int16 Q8.8 storage with int32 arithmetic"}[wl.dtype]
    return (f"{wl.name}: x[{','.join(map(str, wl.shape))}] {storage}, k={wl.k}, sawtooth period {P} "
            f"(one layer per d={wl.dilations}), forward of every layer then backward of every layer")


BACKWARD_INPUT_TEXT = {"recompute": "H and sigma'(H - v_th) recomputed from x", "h": "H saved by the forward",
                       "sg": "sigma'(H - v_th) saved by the forward"}


def roofline(r, counters):
    """Roofline of the dominant kernel (mfpsn_backward) and of forward +
    backward together, from the event-timed averages; traffic and VALU
    fraction from the committed counters (None when stale)."""
    out = {
        "kernel": "mfpsn_backward (bwd_kernel + fin_kernel)",
        "bound": "hbm",
        "achieved": r["bwd_GBs"],
        "peak": HBM_PEAK_GBS,
        "unit": "GB/s",
        "frac": r["bwd_GBs"] / HBM_PEAK_GBS,
        "traffic": None,
        "alg_bytes_per_launch": r["bwd_bytes"],
        "avg_launch_us": r["bwd_us"],
        "fwd_bwd": {"achieved": r["fwd_bwd_GBs"], "frac": r["fwd_bwd_GBs"] / HBM_PEAK_GBS,
                    "alg_bytes": r["fwd_bytes"] + r["bwd_bytes"], "us": r["fwd_us"] + r["bwd_us"]},
        "forward": {"achieved": r["fwd_GBs"], "frac": r["fwd_GBs"] / HBM_PEAK_GBS,
                    "alg_bytes_per_launch": r["fwd_bytes"], "avg_launch_us": r["fwd_us"]},
    }
    if counters is not None:
        out["traffic"] = counters["bwd_bytes_per_launch"]
        out["traffic_note"] = ("HBM bytes per mfpsn_backward launch: 2*FETCH_SIZE + WRITE_SIZE (KiB -> bytes; "
                               "FETCH_SIZE reads half of a 1 GiB copy's bytes on this part), averaged over "
                               f"{counters.get('dispatches_averaged')} dispatches; forward "
                               f"{counters['fwd_bytes_per_launch']} bytes per launch")
        if "bwd_valu_insts" in counters:
            ws = r["wl"].elements / 64
            out["valu_frac"] = counters["bwd_valu_insts"] * VALU_CYCLES / (SIMDS * CLOCK_HZ * r["bwd_us"] * 1e-6)
            out["valu_insts_per_wave_step"] = counters["bwd_valu_insts"] / ws
            out["fwd_valu_frac"] = counters["fwd_valu_insts"] * VALU_CYCLES / (SIMDS * CLOCK_HZ * r["fwd_us"] * 1e-6)
            out["fwd_valu_insts_per_wave_step"] = counters["fwd_valu_insts"] / ws
            out["valu_note"] = (f"SQ_INSTS_VALU (wave64 instructions) x {VALU_CYCLES} cycles / ({SIMDS} SIMDs x "
                                f"{CLOCK_HZ / 1e9:.1f} GHz x event-timed duration): the share of the chip's issue "
                                "capacity for plain VALU instructions")
    return out


def summarize_counters(out_dir):
    """Write profiles/counters.json from rocprofv3 --pmc CSV outputs under
    out_dir: <workload>_<mode>_fetch, _write and _valu runs of
    `bench.py --workload W --only --steps 2 --warmup 1 --no-cpu-baseline`,
    plus calibrate_fetch / calibrate_write runs of `bench.py
    --calibrate-copy` (the byte-counter scale of a plain 1 GiB copy)."""
    import csv
    import glob

    def rows(tag):
        files = glob.glob(os.path.join(out_dir, tag, "**", "*counter_collection.csv"), recursive=True)
        if not files:
            raise SystemExit(f"no counter_collection.csv under {os.path.join(out_dir, tag)}")
        out = []
        for f in files:
            out += list(csv.DictReader(open(f)))
        return out

    def per_dispatch(tag, counter, name_part):
        vals = {}
        for row in rows(tag):
            if name_part in row["Kernel_Name"] and row["Counter_Name"] == counter:
                key = row.get("Dispatch_Id") or row.get("Correlation_Id")
                vals[key] = vals.get(key, 0.0) + float(row["Counter_Value"])
        if not vals:
            raise SystemExit(f"{tag}: no {counter} rows for kernels named like {name_part}")
        return float(np.mean(list(vals.values()))), len(vals)

    def largest(tag, counter):
        # the 1 GiB copy is the dispatch with the largest count in its run
        vals = {}
        for row in rows(tag):
            if row["Counter_Name"] == counter:
                key = row.get("Dispatch_Id") or row.get("Correlation_Id")
                vals[key] = vals.get(key, 0.0) + float(row["Counter_Value"])
        return max(vals.values())

    copy = 1 << 30
    fetch_cal = largest("calibrate_fetch", "FETCH_SIZE")
    write_cal = largest("calibrate_write", "WRITE_SIZE")
    fscale, wscale = copy / (fetch_cal * 1024), copy / (write_cal * 1024)
    rec = {"_calibration": {"copy_bytes": copy, "FETCH_SIZE_kib": fetch_cal, "WRITE_SIZE_kib": write_cal,
                            "fetch_scale": fscale, "write_scale": wscale,
                            "command": "rocprofv3 --pmc FETCH_SIZE -f csv -d DIR/calibrate_fetch -o p -- python3 "
                                       "bench.py --calibrate-copy (then WRITE_SIZE into DIR/calibrate_write)"}}
    from paper_2501_14490_amd import workloads
    for wid, wl in workloads.WORKLOADS.items():
        mode = AUTO_BACKWARD_INPUT[wid]
        tag = f"{wl.name}_{mode}"
        if not os.path.isdir(os.path.join(out_dir, tag + "_fetch")):
            continue
        ent = {"kernel_source": kernel_source_hash(),
               "command": f"rocprofv3 --pmc FETCH_SIZE -f csv -d DIR/{tag}_fetch -o p -- python3 "
                          f"bench.py --workload {wid} --only --steps 2 --warmup 1 --no-cpu-baseline "
                          f"(then WRITE_SIZE into {tag}_write, SQ_INSTS_VALU into {tag}_valu)"}
        fb = {}
        for kern in ("bwd_kernel", "fin_kernel", "fwd_kernel"):
            f, n = per_dispatch(tag + "_fetch", "FETCH_SIZE", kern)
            w, _ = per_dispatch(tag + "_write", "WRITE_SIZE", kern)
            fb[kern] = f * 1024 * fscale + w * 1024 * wscale
            ent[f"{kern}_fetch_kib"] = f
            ent[f"{kern}_write_kib"] = w
            ent["dispatches_averaged"] = n
        ent["bwd_bytes_per_launch"] = fb["bwd_kernel"] + fb["fin_kernel"]
        ent["fwd_bytes_per_launch"] = fb["fwd_kernel"]
        fbytes, bbytes = alg_bytes(wl)
        ent["bwd_alg_bytes_per_launch"] = wl.elements * bbytes
        ent["fwd_alg_bytes_per_launch"] = wl.elements * fbytes
        if os.path.isdir(os.path.join(out_dir, tag + "_valu")):
            ent["bwd_valu_insts"], _ = per_dispatch(tag + "_valu", "SQ_INSTS_VALU", "bwd_kernel")
            ent["fwd_valu_insts"], _ = per_dispatch(tag + "_valu", "SQ_INSTS_VALU", "fwd_kernel")
        rec[f"{wl.name}|{mode}"] = ent
    with open(COUNTERS_FILE, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps({k: v.get("bwd_bytes_per_launch") for k, v in rec.items() if "|" in k}))


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=4,
                    help="headline workload 1..5 (default 4: event-vision-shaped, the largest)")
    ap.add_argument("--only", action="store_true", help="measure the headline workload only")
    ap.add_argument("--cpu-channels", type=int, default=None, help="channels in the oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-flush", action="store_true",
                    help="do not read the 1 GiB scratch buffer before each call (warm last-level cache)")
    ap.add_argument("--backward-input", choices=("auto",) + BACKWARD_INPUTS, default="auto",
                    help="what the forward saves for the backward: nothing (recompute: the backward "
                         "recomputes H and the surrogate factor from x), the potentials H (h), or the "
                         "surrogate factor sigma'(H - v_th) (sg); auto: the best one measured for the "
                         "workload")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device copy (reference for HBM byte counters)")
    ap.add_argument("--summarize-counters", metavar="DIR", default=None,
                    help="only write profiles/counters.json from the rocprofv3 --pmc outputs under DIR")
    ap.add_argument("--bn-step", action="store_true",
                    help="only time the batch-normalized-threshold training step of App. C (float workloads)")
    ap.add_argument("--time-last", action="store_true",
                    help="only time the forward in the time-last layout [N][C][S][T] beside the time-first one")
    ap.add_argument("--stack", action="store_true",
                    help="only time the workload's layers chained into one sawtooth stack (float workloads)")
    ap.add_argument("--stream-inference", action="store_true",
                    help="only time step-by-step inference (mfpsn_stream_step per layer and time step, "
                         "the sequence replayed from a HIP graph)")
    ap.add_argument("--memory-ceiling", action="store_true",
                    help="only time plain library streams of the workload's size (1 read + 1 write, "
                         "3 reads + 1 write): the bandwidth a kernel with that mix can reach")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported (the neuron layer "
              f"shards over the batch with one all-reduce of grad_w/grad_b per layer, not built here)",
              file=sys.stderr)
        sys.exit(2)
    if args.summarize_counters:
        summarize_counters(args.summarize_counters)
        return

    import torch

    from paper_2501_14490_amd import mfpsn, workloads  # noqa: F401  (loads libmfpsn.so or raises)

    if not torch.cuda.is_available():
        log("no GPU visible")
        sys.exit(1)
    dev = torch.device("cuda:0")
    if args.calibrate_copy:
        n = 1 << 28  # 2^28 floats = 1 GiB read + 1 GiB written per copy
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes_read": 4 * n, "calibrate_copy_bytes_written": 4 * n,
                          "copies": 5}), flush=True)
        return
    wl = workloads.WORKLOADS[args.workload]
    log(f"workload {wl.wid}: {wl.describe()}  dilations {wl.dilations}")
    if args.memory_ceiling:
        memory_ceiling(torch, dev, wl)
        return
    mode = args.backward_input if args.backward_input != "auto" else AUTO_BACKWARD_INPUT[wl.wid]
    if args.stream_inference or args.bn_step or args.stack or args.time_last:
        case = workloads.make_inputs(wl)
        if args.stream_inference:
            stream_inference(torch, dev, wl, case, args.steps, args.warmup)
        elif args.bn_step:
            bn_step(torch, dev, wl, case, args.steps, args.warmup)
        elif args.stack:
            stack_step(torch, dev, wl, case, mode, args.steps, args.warmup)
        else:
            time_last(torch, dev, wl, case, args.steps, args.warmup)
        return

    hev = HipEvents()
    flush = (lambda: None) if args.no_flush else Flush(torch, dev)
    head = measure(torch, dev, wl, mode, args.steps, args.warmup, flush, hev)
    log(f"{wl.name}: step {head['step_ms']:.3f} ms (cold calls; wall {head['wall_ms_per_step']:.3f} ms with the "
        f"flushes)  fwd {head['fwd_us']:.1f} us  bwd {head['bwd_us']:.1f} us  "
        f"{head['value'] / 1e9:.2f} G elements/s  fwd+bwd {head['fwd_bwd_GBs']:.0f} GB/s alg")
    log("per dilation:", head["per_d"])
    others = {}
    if not args.only:
        for wid in (2, 3, 4, 5):
            if wid == wl.wid:
                continue
            owl = workloads.WORKLOADS[wid]
            omode = AUTO_BACKWARD_INPUT[wid]
            r = measure(torch, dev, owl, omode, args.steps, args.warmup, flush, hev)
            log(f"{owl.name}: {r['value'] / 1e9:.2f} G elements/s  fwd {r['fwd_us']:.1f} us  bwd "
                f"{r['bwd_us']:.1f} us  fwd+bwd {r['fwd_bwd_GBs']:.0f} GB/s alg  {r['per_d']}")
            c = committed_counters(owl.name, omode)
            others[owl.name] = {
                "workload": describe(owl, r["P"]), "value": r["value"], "unit": "elements/s",
                "ms_per_step": r["step_ms"], "backward_input": BACKWARD_INPUT_TEXT[omode],
                "fwd_us": r["fwd_us"], "bwd_us": r["bwd_us"],
                "fwd_frac": r["fwd_GBs"] / HBM_PEAK_GBS, "bwd_frac": r["bwd_GBs"] / HBM_PEAK_GBS,
                "fwd_bwd_frac": r["fwd_bwd_GBs"] / HBM_PEAK_GBS, "per_d": r["per_d"],
                "traffic": None if c is None else c["bwd_bytes_per_launch"],
            }
    P = head["P"]
    result = {
        "metric": "neuron fwd+bwd elements/s (T*N*C*S) and achieved HBM GB/s vs MI355X peak",
        "value": head["value"],
        "unit": "elements/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["step_ms"],
        "wall_ms_per_step_with_flushes": head["wall_ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"f32": "f32", "bf16": "bf16", "q8_8": "int16 Q8.8 / int32"}[wl.dtype],
        "data": "synthetic",
        "config": {
            "workload": describe(wl, P),
            "elements_per_layer": wl.elements,
            "layers_per_step": P,
            "surrogate": f"{wl.surrogate} alpha={wl.alpha}",
            "backward_input": BACKWARD_INPUT_TEXT[mode],
            "v_th": wl.v_th,
            "cache": "cold: 1 GiB read before every call, outside its events" if not args.no_flush
                     else "warm (no flush)",
        },
        "roofline": roofline(head, committed_counters(wl.name, mode)),
        "per_d": head["per_d"],
        "configs": others,
    }
    if not args.no_cpu_baseline:
        channels = args.cpu_channels or {1: 128, 2: 320, 3: 64, 4: 48, 5: 48}[wl.wid]
        log(f"oracle baseline on {channels} channels ...")
        case = workloads.make_inputs(wl)
        result["cpu_baseline"] = cpu_baseline(wl, case, channels)
        log(f"oracle: {result['cpu_baseline']['value'] / 1e6:.2f} M elements/s")
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
