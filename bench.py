"""Benchmark of the W8A8 linear on one MI355X.

One step is one pass of the hot path over one batch of synthetic input. The
layer goes through the protection router: a W8A8 layer runs smoothing +
per-token quantization (w8a8_quant_act) and then the INT8 GEMM with its fused
epilogue (w8a8_linear). A protected layer runs bf16_linear. Weights are
prepared (quantized) once, outside the timed region, as in deployment.

Default workload: the DiT FFN up-projection of one branch, X [4608 x 4096] ->
Y [4608 x 16384]. Other workloads (--workload): ffn_down (W8A8 and protected
paths), dit_block (the four linears of a block, both CFG branches), backbone
(211 linears x 2 branches, 17 protected per branch).

Prints one JSON line. ``value`` is the step's throughput in TOPS
(2 M N K per step divided by the step time). ``roofline`` covers the dominant
kernel (the INT8 GEMM); its ``clock`` holds the XCD clocks read while that
kernel runs back to back, the fraction of the peak at that clock, and the
socket power over the same window. ``cpu_baseline`` is the CPU oracle timed
on a bounded sample of the same workload on this host. ``eager_torch`` times the dominant
layer run the way the paper runs it, as eager Torch ops with torch._int_mm for
the GEMM, on the same GPU. ``accuracy`` (FFN workloads) gives the W8A8 and
bf16 paths' error against X W^T + b in binary64.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402
from paper_2606_12280_amd import layer as L  # noqa: E402
from paper_2606_12280_amd import ops  # noqa: E402
from paper_2606_12280_amd._lib import MOMENTS_WORK_BYTES as _MOMENTS_WORK  # noqa: E402

METRIC = "W8A8 linear TOPS (% INT8 MFMA peak) + act-quant GB/s at DiT FFN shapes"
PEAK_INT8_TOPS = 5000.0    # MI355X dense INT8 MFMA
PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0      # MI355X HBM3E
PEAK_CLOCK_MHZ = 2400.0    # the engine clock the MFMA peaks are quoted at
GEMM_SOURCES = ["paper_2606_12280_amd/csrc/gemm.hip"]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def sources_sha(paths) -> str:
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def to_dev_bf16(bits: np.ndarray, dev) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)


# --------------------------------------------------------------------------
# workloads: lists of (prepared layer, input pool)
# --------------------------------------------------------------------------

class Linear:
    def __init__(self, name, lay: L.PreparedLinear, xs: list[torch.Tensor]):
        self.name = name
        self.lay = lay
        self.xs = xs
        self.M = xs[0].shape[0]
        self.Y = torch.empty(self.M, lay.N, dtype=torch.bfloat16, device=xs[0].device)
        self.mod = None   # (shift, scale) bf16 [K]: the input is adaLN-modulated first
        self.case = None  # the host case the layer and xs[0] were made from, if any

    def quant(self, X, Xq, xs):
        """The activation step of this layer (fused with adaLN if modulated)."""
        if self.mod is None:
            return ops.w8a8_quant_act(X, self.lay.inv_lambda, Xq=Xq, x_scale=xs)
        return ops.w8a8_adaln_quant_act(X, self.mod[0], self.mod[1], self.lay.inv_lambda,
                                        Xq=Xq, x_scale=xs)

    @property
    def ops(self) -> int:
        return 2 * self.M * self.lay.N * self.lay.K


def calibrated_layer(X: torch.Tensor, W: torch.Tensor, bias, protected: bool):
    """lambda from the activation absmax of X (calibration on the layer's
    own input) and the weight column absmax, alpha = 0.5; then prepare."""
    if protected:
        return L.prepare_linear(W, bias, None, True)
    s = torch.zeros(W.shape[1], dtype=torch.float32, device=W.device)
    ops.w8a8_act_absmax(X, s)
    lam = ops.w8a8_smooth_factors(s, W, 0.5)
    return L.prepare_linear(W, bias, lam, False)


def host_case_linear(name, case, dev, pool: int, protected: bool, seed_base) -> Linear:
    """A layer from the seeded host generator (the documented case) plus
    pool - 1 further inputs of the same distribution for rotation."""
    M, N, K = case["M"], case["N"], case["K"]
    X0 = to_dev_bf16(case["X"].reshape(M, K), dev)
    W = to_dev_bf16(case["W"].reshape(N, K), dev)
    b = to_dev_bf16(case["bias"], dev)
    lay = calibrated_layer(X0, W, b, protected)
    if not protected:
        del W
    xs = [X0]
    act = "gelu" if K == 16384 else "outlier"
    for i in range(1, pool):
        rng = np.random.default_rng([seed_base, 1000 + i])
        if act == "gelu":
            x = synth.gelu_lognormal_activations(rng, M, K)
        else:
            x = synth.outlier_activations(rng, M, K, int(round(0.01 * K)), 20.0)
        xs.append(to_dev_bf16(synth.to_bf16_bits(x), dev))
    lin = Linear(name, lay, xs)
    lin.case = case
    return lin


def device_linear(name, M, N, K, dev, gen: torch.Generator, protected: bool, x_pool) -> Linear:
    """A layer with device-generated N(0, 0.02) weights (the large sweeps;
    timing only), sharing an input pool with the layers of its shape."""
    W = (torch.randn(N, K, device=dev, generator=gen) * 0.02).bfloat16()
    b = (torch.randn(N, device=dev, generator=gen) * 0.01).bfloat16()
    lay = calibrated_layer(x_pool[0], W, b, protected)
    return Linear(name, lay, x_pool)


def device_inputs(M, K, dev, gen, n, gelu: bool):
    out = []
    for _ in range(n):
        if gelu:
            z = torch.randn(M, K, device=dev, generator=gen) * 1.5
            c = torch.exp(torch.randn(K, device=dev, generator=gen) * 1.5)
            out.append((torch.nn.functional.gelu(z) * c).bfloat16())
        else:
            x = torch.randn(M, K, device=dev, generator=gen)
            idx = torch.randperm(K, device=dev, generator=gen)[: int(round(0.01 * K))]
            x[:, idx] *= 20.0
            out.append(x.bfloat16())
    return out


def modulate(layers, dev, seed: int) -> None:
    """Give the QKV and FFN-up layers (the inputs a DiT block modulates with
    adaLN) a per-layer shift and scale, bf16 N(0, 0.05) and N(0, 0.1): their
    activation step becomes w8a8_adaln_quant_act."""
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    for lin in layers:
        if lin.lay.protected or not any(t in lin.name for t in ("qkv", "ffn_up")):
            continue
        K = lin.lay.K
        lin.mod = tuple((torch.randn(K, device=dev, generator=gen) * sd).bfloat16()
                        for sd in (0.05, 0.1))


def build_workload(name: str, dev, pool: int):
    if name in ("q8_0_ffn_up", "q4_k_ffn_up"):
        c = synth.ffn_up_case()
        lin = host_case_linear("ffn_up", c, dev, pool, True, 2)
        prep = L.prepare_q8_0 if name == "q8_0_ffn_up" else L.prepare_q4_k
        lin.lay = prep(lin.lay.W, lin.lay.bias)  # the bf16 copy is dropped
        return [lin]
    if name == "ffn_up":
        return [host_case_linear("ffn_up", synth.ffn_up_case(), dev, pool, False, 2)]
    if name == "adaln_ffn_up":
        c = synth.ffn_up_case()
        lin = host_case_linear("adaln_ffn_up", c, dev, pool, False, 2)
        rng = np.random.default_rng([2, 77])
        lin.mod = tuple(to_dev_bf16(synth.to_bf16_bits(rng.normal(0, sd, c["K"]).astype(np.float32)), dev)
                        for sd in (0.05, 0.1))
        return [lin]
    if name == "ffn_down":
        c = synth.ffn_down_case()
        return [host_case_linear("ffn_down_w8a8", c, dev, pool, False, 3),
                host_case_linear("ffn_down_bf16", c, dev, pool, True, 3)]
    gen = torch.Generator(device=dev)
    if name == "dit_block":
        out = []
        for br in range(2):
            for li in range(4):
                c = synth.block_case(br, li)
                out.append(host_case_linear(f"b{br}_{c['name']}", c, dev, 1,
                                            c["name"] == "ffn_down", 40 + 10 * br + li))
        return out
    if name == "backbone":
        gen.manual_seed(5)
        M = synth.TOKENS
        pools = {}
        for sname, N, K in synth.BLOCK_SHAPES:
            pools[sname] = device_inputs(M, K, dev, gen, 2, sname == "ffn_down")
        flags = L.protected_layers(211, 17)
        out = []
        for br in range(2):
            for i in range(211):
                sname, N, K = synth.BLOCK_SHAPES[i % 4]
                out.append(device_linear(f"b{br}_{i}_{sname}", M, N, K, dev, gen, flags[i],
                                         pools[sname]))
        return out
    raise SystemExit(f"unknown workload {name}")


# --------------------------------------------------------------------------
# timing
# --------------------------------------------------------------------------

def run_step(layers, it: int, ws: L.Workspace, events=None):
    """One pass over every layer. If events is given, records
    (start, after-quant, end) per layer."""
    for li, lin in enumerate(layers):
        X = lin.xs[it % len(lin.xs)]
        if lin.lay.protected:
            if events is not None:
                events[li][0].record()
                events[li][1].record()
            ops.bf16_linear(X, lin.lay.W, lin.lay.bias, out=lin.Y)
        elif lin.lay.weight_only:
            if events is not None:
                events[li][0].record()
            if lin.lay.q8_0:
                ops.q8_0_dequantize(lin.lay.q8_qs, lin.lay.q8_d, out=ws.weights(lin.lay.N, lin.lay.K))
            else:
                ops.q4_k_dequantize(lin.lay.q4k, out=ws.weights(lin.lay.N, lin.lay.K))
            if events is not None:
                events[li][1].record()
            ops.bf16_linear(X, ws.weights(lin.lay.N, lin.lay.K), lin.lay.bias, out=lin.Y)
        else:
            Xq, xs = ws.get(lin.M, lin.lay.K)
            if events is not None:
                events[li][0].record()
            lin.quant(X, Xq, xs)
            if events is not None:
                events[li][1].record()
            ops.w8a8_linear(Xq, xs, lin.lay.Wq, lin.lay.w_scale, lin.lay.bias, out=lin.Y)
        if events is not None:
            events[li][2].record()


class BranchStreams:
    """The two CFG branches of a step on two streams of default priority:
    their layers are independent (separate weights, separate inputs), so the
    kernels of one branch can fill the GPU where the other's leave it idle
    (the per-XCD tail of a GEMM, the ramp of a launch). Layer i of each
    branch is issued in turn; each stream has its own workspace."""

    def __init__(self, layers, dev):
        self.branches = [[lin for lin in layers if lin.name.startswith(f"b{b}_")] for b in (0, 1)]
        if len(self.branches[0]) + len(self.branches[1]) != len(layers) or \
                len(self.branches[0]) != len(self.branches[1]):
            raise SystemExit("--branch-streams needs the two branches' layers b0_* and b1_*")
        self.streams = [torch.cuda.Stream(device=dev) for _ in range(2)]
        self.ws = [L.Workspace(dev) for _ in range(2)]

    def step(self, it: int):
        cur = torch.cuda.current_stream()
        for st in self.streams:
            st.wait_stream(cur)
        for pair in zip(*self.branches):
            for b in (0, 1):
                with torch.cuda.stream(self.streams[b]):
                    run_step([pair[b]], it, self.ws[b])
        for st in self.streams:
            cur.wait_stream(st)


def captured_steps(step, layers, warmup: int):
    """The step as HIP graphs, one per input of the rotation (a graph holds
    fixed pointers): captured once each after an eager warm-up on the
    capture stream, then replayed. The kernels of the step allocate nothing
    and issue no memset, so a replay does what the eager step does."""
    n = max(len(lin.xs) for lin in layers)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for i in range(n):
            step(warmup + i)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graphs = {}
    for i in range(n):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step(warmup + i)
        graphs[(warmup + i) % n] = g
    torch.cuda.synchronize()
    return lambda it, e=None: graphs[it % n].replay()


def measure(layers, steps: int, warmup: int, dev, per_kernel: bool, warm_ms: float = 200.0,
            branch_streams: bool = False, graph: bool = False):
    ws = L.Workspace(dev)
    two = BranchStreams(layers, dev) if branch_streams and not per_kernel else None
    step = (lambda it, e=None: two.step(it)) if two else \
        (lambda it, e=None: run_step(layers, it, ws, e))
    if graph and not per_kernel:
        step = captured_steps(step, layers, warmup)
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    # keep the GPU busy long enough for its clocks to settle before timing
    t_end = time.perf_counter() + warm_ms * 1e-3
    i = warmup
    while time.perf_counter() < t_end:
        step(i)
        torch.cuda.synchronize()
        i += 1
    ev = None
    if per_kernel:
        ev = [[[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in layers]
              for _ in range(steps)]
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t0.record()
    for s in range(steps):
        step(warmup + s, ev[s] if ev else None)
    t1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = t0.elapsed_time(t1)
    quant_us = np.zeros(len(layers))
    gemm_us = np.zeros(len(layers))
    gemm_each = np.zeros((steps, len(layers)))
    if ev:
        for s in range(steps):
            for li in range(len(layers)):
                a, b, c = ev[s][li]
                quant_us[li] += a.elapsed_time(b) * 1e3
                gemm_each[s, li] = b.elapsed_time(c) * 1e3
        quant_us /= steps
        gemm_us = gemm_each.mean(axis=0)
    measure.gemm_each = gemm_each  # per-step GEMM times of the last call, us
    return total_ms / steps, wall / steps * 1e3, quant_us, gemm_us


def _settle(fn, seconds: float = 0.05):
    """Run fn back to back for a short while before a timed leg, so that the
    clock has moved from the state the previous leg left (the GEMM's steps
    hold the power-limited clock) to this kernel's own."""
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(10):
            fn()
        torch.cuda.synchronize()


def quant_isolated(lin: Linear, dev, reps: int = 60, rounds: int = 5):
    """Quant kernel alone, inputs rotating over buffers larger than the
    256 MB Infinity Cache so that X is read from HBM. Each round times `reps`
    back-to-back launches between one pair of events; an event pair around
    every launch would add several microseconds to a ~10 us kernel. Returns
    the median, min and max per-launch time over the rounds."""
    M, K = lin.M, lin.lay.K
    nbuf = max(3, int(np.ceil(700e6 / (3 * M * K))))
    xs = [lin.xs[i % len(lin.xs)].clone() for i in range(nbuf)]
    qs = [torch.empty(M, K, dtype=torch.int8, device=dev) for _ in range(nbuf)]
    sc = torch.empty(M, dtype=torch.float32, device=dev)
    for i in range(nbuf):
        lin.quant(xs[i], qs[i], sc)
    rot = {"i": 0}

    def one():
        rot["i"] = (rot["i"] + 1) % nbuf
        lin.quant(xs[rot["i"]], qs[rot["i"]], sc)
    _settle(one)
    per = []
    for _ in range(rounds):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        for r in range(reps):
            i = r % nbuf
            lin.quant(xs[i], qs[i], sc)
        b.record()
        torch.cuda.synchronize()
        per.append(a.elapsed_time(b) * 1e3 / reps)
    del xs, qs
    per = np.array(per)
    return float(np.median(per)), float(per.min()), float(per.max())


def moments_isolated(lin: Linear, dev, reps: int = 30, rounds: int = 5):
    """The fragility-statistics call (two passes over X) alone, inputs
    rotating over more than 700 MB so that X comes from HBM; back-to-back
    calls between one pair of events. Median, min, max per call."""
    M, K = lin.M, lin.lay.K
    nbuf = max(3, int(np.ceil(700e6 / (2 * M * K))))
    xs = [lin.xs[i % len(lin.xs)].clone() for i in range(nbuf)]
    work = torch.empty(_MOMENTS_WORK, dtype=torch.uint8, device=dev)
    out = torch.empty(4, dtype=torch.float64, device=dev)
    for i in range(nbuf):
        ops.w8a8_act_moments(xs[i], work, out=out)
    _settle(lambda: ops.w8a8_act_moments(xs[0], work, out=out))
    per = []
    for _ in range(rounds):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        for r in range(reps):
            ops.w8a8_act_moments(xs[r % nbuf], work, out=out)
        b.record()
        torch.cuda.synchronize()
        per.append(a.elapsed_time(b) * 1e3 / reps)
    del xs
    per = np.array(per)
    return float(np.median(per)), float(per.min()), float(per.max())


def absmax_isolated(lin: Linear, dev, reps: int = 30, rounds: int = 5):
    """The per-channel absmax (calibration) alone, inputs rotating over more
    than 700 MB; back-to-back calls between one pair of events."""
    M, K = lin.M, lin.lay.K
    nbuf = max(3, int(np.ceil(700e6 / (2 * M * K))))
    xs = [lin.xs[i % len(lin.xs)].clone() for i in range(nbuf)]
    s = torch.zeros(K, dtype=torch.float32, device=dev)
    for i in range(nbuf):
        ops.w8a8_act_absmax(xs[i], s)
    _settle(lambda: ops.w8a8_act_absmax(xs[0], s))
    per = []
    for _ in range(rounds):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        for r in range(reps):
            ops.w8a8_act_absmax(xs[r % nbuf], s)
        b.record()
        torch.cuda.synchronize()
        per.append(a.elapsed_time(b) * 1e3 / reps)
    del xs
    per = np.array(per)
    return float(np.median(per)), float(per.min()), float(per.max())


def eager_torch(lin: Linear, dev, reps: int = 20, rounds: int = 5):
    """The same layer as the paper runs it: eager Torch ops, one pass each
    (smoothing, per-token absmax, scale, round and clamp, INT8 GEMM by
    torch._int_mm, dequantization and bias), on this GPU. Timing context
    only; it is no part of the library. Returns (median us per layer, median
    us of the _int_mm alone, mean |difference| to the fused path's output
    over mean |output|)."""
    lay = lin.lay
    X = lin.xs[0]
    Wt = lay.Wq.t()
    inv = lay.inv_lambda
    ws_ = lay.w_scale
    b = lay.bias.float() if lay.bias is not None else None

    def step():
        xs_ = X.float() * inv
        s = xs_.abs().amax(dim=1, keepdim=True) / 127.0
        q = torch.clamp(torch.round(xs_ / s), -127, 127).to(torch.int8)
        y = torch._int_mm(q, Wt).float() * s * ws_
        if b is not None:
            y = y + b
        return y.bfloat16(), q

    def timed(fn):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        per = []
        for _ in range(rounds):
            a = torch.cuda.Event(enable_timing=True)
            e = torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(reps):
                fn()
            e.record()
            torch.cuda.synchronize()
            per.append(a.elapsed_time(e) * 1e3 / reps)
        return float(np.median(per))

    y, q = step()
    ours = torch.empty_like(y)
    Xq = torch.empty(lin.M, lay.K, dtype=torch.int8, device=dev)
    xsc = torch.empty(lin.M, dtype=torch.float32, device=dev)
    lin.quant(X, Xq, xsc)
    ops.w8a8_linear(Xq, xsc, lay.Wq, lay.w_scale, lay.bias, out=ours)
    torch.cuda.synchronize()
    diff = float((y.float() - ours.float()).abs().mean() / ours.float().abs().mean())
    us = timed(step)
    us_mm = timed(lambda: torch._int_mm(q, Wt))
    del y, q, ours, Xq
    return us, us_mm, diff


def accuracy_report(layers, dev):
    """Error of the W8A8 and bf16 paths of the workload's layer against
    X W^T + b in binary64 (numpy on the host, from the same seeded case):
    relative Frobenius norm and largest absolute difference of the bf16
    output. Where the workload has no protected copy, the bf16 path runs on
    the case's weights for comparison."""
    lin = next(l for l in layers if l.case is not None and not l.lay.protected)
    c = lin.case
    M, N, K = c["M"], c["N"], c["K"]
    X = synth.bf16_bits_to_f32(c["X"]).reshape(M, K).astype(np.float64)
    W = synth.bf16_bits_to_f32(c["W"]).reshape(N, K).astype(np.float64)
    b = synth.bf16_bits_to_f32(c["bias"]).astype(np.float64)
    ref = X @ W.T + b
    del X, W
    nref = float(np.linalg.norm(ref))

    def err(Y):
        d = Y.float().cpu().numpy().astype(np.float64) - ref
        return {"rel_frobenius": float(f"{np.linalg.norm(d) / nref:.4g}"),
                "max_abs": float(f"{np.abs(d).max():.4g}")}

    out = {"shape": [M, K, N], "reference": "X W^T + b in binary64 (numpy, host)",
           "max_abs_reference": float(f"{np.abs(ref).max():.4g}")}
    Xq = torch.empty(M, K, dtype=torch.int8, device=dev)
    xsc = torch.empty(M, dtype=torch.float32, device=dev)
    lin.quant(lin.xs[0], Xq, xsc)
    Y = ops.w8a8_linear(Xq, xsc, lin.lay.Wq, lin.lay.w_scale, lin.lay.bias)
    out["w8a8"] = err(Y)
    prot = next((l for l in layers if l.lay.protected and l.case is c), None)
    Wd = prot.lay.W if prot is not None else to_dev_bf16(c["W"].reshape(N, K), dev)
    Y = ops.bf16_linear(lin.xs[0], Wd, lin.lay.bias)
    out["bf16"] = err(Y)
    del Y, Xq, Wd
    return out


def _amdsmi_handle(amdsmi, dev):
    """The amdsmi handle of torch device `dev` (matched by PCI address)."""
    props = torch.cuda.get_device_properties(dev)
    want = (getattr(props, "pci_domain_id", None), getattr(props, "pci_bus_id", None),
            getattr(props, "pci_device_id", None))
    handles = amdsmi.amdsmi_get_processor_handles()
    for h in handles:
        try:
            bdf = amdsmi.amdsmi_get_gpu_device_bdf(h)  # "dddd:bb:dd.f"
            dom, bus, rest = bdf.split(":")
            if (int(dom, 16), int(bus, 16), int(rest.split(".")[0], 16)) == want:
                return h
        except Exception:
            continue
    return handles[0] if len(handles) == 1 else None


def clock_under_load(lin: Linear, dev, seconds: float = 3.0):
    """The graphics clock of each XCD while `lin`'s INT8 GEMM runs back to
    back, read in-process from the GPU metrics table through amdsmi (no
    child process). The first second is left out while the clock settles.
    None where amdsmi or the metric is missing.

    From the same table, over the sampled window: the share of the power
    manager's 1 ms intervals in which package power tracking (the socket
    power limit) held the clock down, the average socket power, and the
    energy per launch. On MI355X the energy accumulator counts 2^-16 J and
    the firmware timestamp 10 ns (under a sustained load the two give the
    1400 W power limit)."""
    try:
        import amdsmi
        amdsmi.amdsmi_init()
    except Exception:
        return None
    try:
        h = _amdsmi_handle(amdsmi, dev)
        if h is None:
            return None
        Xq = torch.empty(lin.M, lin.lay.K, dtype=torch.int8, device=dev)
        xsc = torch.empty(lin.M, dtype=torch.float32, device=dev)
        lin.quant(lin.xs[0], Xq, xsc)
        per = max(1, int(10e-3 / max(lin.ops / 2.5e15, 1e-6)))  # about 10 ms of launches
        samples = []
        uclk = []
        t0 = time.perf_counter()
        last = 0.0
        first = None      # metrics table at the start of the sampled window
        launches = 0      # launches since then
        t_first = 0.0
        while time.perf_counter() - t0 < seconds:
            for _ in range(per):
                ops.w8a8_linear(Xq, xsc, lin.lay.Wq, lin.lay.w_scale, lin.lay.bias, out=lin.Y)
            torch.cuda.synchronize()
            if first is not None:
                launches += per
            now = time.perf_counter() - t0
            if now > 1.0 and now - last > 0.05:
                last = now
                met = amdsmi.amdsmi_get_gpu_metrics_info(h)
                if first is None:
                    first = met
                    t_first = time.perf_counter()
                clks = met.get("current_gfxclks")
                u = met.get("current_uclk")
                if isinstance(u, (int, float)) and 0 < u < 100000:
                    uclk.append(float(u))
                if isinstance(clks, (list, tuple)):
                    clks = [int(c) for c in clks if isinstance(c, (int, float)) and 0 < c < 10000]
                    if clks:
                        samples.append(clks)
        end = amdsmi.amdsmi_get_gpu_metrics_info(h) if first is not None else None
        per_launch = (time.perf_counter() - t_first) / launches if launches else None
        del Xq, xsc
        if not samples or len({len(c) for c in samples}) != 1:
            return None
        a = np.array(samples, dtype=np.float64)
        per_xcd = a.mean(axis=0)
        out = {"source": "amdsmi GPU metrics (current_gfxclks), sampled in-process during "
                         f"{seconds:.0f} s of back-to-back launches of this kernel",
               "mhz_per_xcd": [round(float(v)) for v in per_xcd],
               "mhz_mean": round(float(per_xcd.mean()), 1),
               "mhz_min": round(float(per_xcd.min()), 1), "samples": len(samples),
               "memory_clock_mhz": round(float(np.mean(uclk)), 1) if uclk else None}
        out["power"] = power_over_window(amdsmi, h, first, end, per_launch, lin.ops)
        out["power"]["launches"] = launches
        return out
    except Exception:
        return None
    finally:
        try:
            amdsmi.amdsmi_shut_down()
        except Exception:
            pass


def power_over_window(amdsmi, h, first, end, seconds_per_launch, ops_per_launch):
    """Power figures between two snapshots of the GPU metrics table taken
    around back-to-back launches of one kernel (see clock_under_load): the
    share of the power manager's 1 ms intervals with the power limiter on,
    and the average socket power over the table's own interval (its energy
    counter over its timestamp). Joules per launch are that power times the
    measured time per launch, so a table refreshed on its own schedule does
    not skew them. None where a field is missing."""
    def num(m, k):
        v = m.get(k) if m is not None else None
        return float(v) if isinstance(v, (int, float)) else None

    try:
        cap = amdsmi.amdsmi_get_power_cap_info(h).get("power_cap")
        cap_w = float(cap) / 1e6 if isinstance(cap, (int, float)) and cap > 0 else None
    except Exception:
        cap_w = None
    d = {}
    for k in ("accumulation_counter", "ppt_residency_acc", "energy_accumulator",
              "firmware_timestamp"):
        a, b = num(first, k), num(end, k)
        d[k] = b - a if a is not None and b is not None else None
    out = {"power_limit_w": cap_w}
    if not d["accumulation_counter"] or not d["firmware_timestamp"]:
        return out
    seconds = d["firmware_timestamp"] * 1e-8
    out["window_s"] = round(seconds, 3)
    if d["ppt_residency_acc"] is not None:
        out["ppt_throttle_share"] = round(d["ppt_residency_acc"] / d["accumulation_counter"], 4)
    if d["energy_accumulator"] is not None and d["energy_accumulator"] > 0:
        watts = d["energy_accumulator"] * 2.0 ** -16 / seconds
        out["avg_power_w"] = round(watts, 1)
        if seconds_per_launch:
            joules = watts * seconds_per_launch
            out["joules_per_launch"] = round(joules, 5)
            if ops_per_launch:
                out["tops_per_watt"] = round(ops_per_launch / joules / 1e12, 3)
    return out


def power_table(layers, dev, seconds: float = 2.0, settle: float = 0.8):
    """Each kernel of the workload's layers run back to back: `settle`
    seconds to let the clock settle, then `seconds` measured. Per kernel:
    time per launch (HIP events), the XCD clock mean, and the socket power
    figures of power_over_window. The activation steps read inputs rotating
    over more than the 256 MB Infinity Cache. None without amdsmi."""
    try:
        import amdsmi
        amdsmi.amdsmi_init()
    except Exception:
        return None
    try:
        h = _amdsmi_handle(amdsmi, dev)
        if h is None:
            return None
        table = []

        def run(label, fn, ops_per_launch=0, nbytes=0):
            t0 = time.perf_counter()
            while time.perf_counter() - t0 < settle:
                for _ in range(10):
                    fn()
                torch.cuda.synchronize()
            first = amdsmi.amdsmi_get_gpu_metrics_info(h)
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            n, clocks, last = 0, [], 0.0
            a.record()
            t0 = time.perf_counter()
            while time.perf_counter() - t0 < seconds:
                for _ in range(10):
                    fn()
                n += 10
                torch.cuda.synchronize()
                if time.perf_counter() - last > 0.1:
                    last = time.perf_counter()
                    c = amdsmi.amdsmi_get_gpu_metrics_info(h).get("current_gfxclks")
                    if isinstance(c, (list, tuple)):
                        c = [v for v in c if isinstance(v, (int, float)) and 0 < v < 10000]
                        if c:
                            clocks.append(float(np.mean(c)))
            b.record()
            torch.cuda.synchronize()
            end = amdsmi.amdsmi_get_gpu_metrics_info(h)
            us = a.elapsed_time(b) * 1e3 / n
            e = {"kernel": label, "us_per_launch": round(us, 2), "launches": n,
                 "mhz_mean": round(float(np.mean(clocks)), 1) if clocks else None}
            if ops_per_launch:
                e["TOPS"] = round(ops_per_launch / us / 1e6, 1)
            if nbytes:
                e["GB_s"] = round(nbytes / us / 1e3, 1)
            e.update(power_over_window(amdsmi, h, first, end, us * 1e-6, ops_per_launch))
            table.append(e)
            log(f"power: {json.dumps(e)}")

        gen = torch.Generator(device=dev)
        gen.manual_seed(12)
        for lin in layers:
            M, K, N = lin.M, lin.lay.K, lin.lay.N
            shape = f"{M}x{K}->{N}"
            X = lin.xs[0]
            if lin.lay.protected:
                run(f"bf16_linear {shape}", lambda: ops.bf16_linear(X, lin.lay.W, lin.lay.bias,
                                                                    out=lin.Y), lin.ops)
                continue
            Xq = torch.empty(M, K, dtype=torch.int8, device=dev)
            xsc = torch.empty(M, dtype=torch.float32, device=dev)
            lin.quant(X, Xq, xsc)
            run(f"w8a8_linear {shape}", lambda: ops.w8a8_linear(
                Xq, xsc, lin.lay.Wq, lin.lay.w_scale, lin.lay.bias, out=lin.Y), lin.ops)
            nbuf = max(3, int(np.ceil(700e6 / (3 * M * K))))
            xs_in = [X.clone() for _ in range(nbuf)]
            qs = [torch.empty_like(Xq) for _ in range(nbuf)]
            rot = {"i": 0}

            def quant():
                i = rot["i"] = (rot["i"] + 1) % nbuf
                ops.w8a8_quant_act(xs_in[i], lin.lay.inv_lambda, Xq=qs[i], x_scale=xsc)
            run(f"w8a8_quant_act {M}x{K}", quant, 0, quant_bytes(M, K))
            if K <= 8192:
                sh, sc = ((torch.randn(K, device=dev, generator=gen) * sd).bfloat16()
                          for sd in (0.05, 0.1))

                def adaln():
                    i = rot["i"] = (rot["i"] + 1) % nbuf
                    ops.w8a8_adaln_quant_act(xs_in[i], sh, sc, lin.lay.inv_lambda, Xq=qs[i],
                                             x_scale=xsc)
                run(f"w8a8_adaln_quant_act {M}x{K}", adaln, 0, quant_bytes(M, K) + 4 * K)
            del xs_in, qs, Xq, xsc
        return table
    except Exception as exc:  # a missing metrics field: report it, keep going
        log(f"power table unavailable: {exc}")
        return None
    finally:
        try:
            amdsmi.amdsmi_shut_down()
        except Exception:
            pass


def quant_bytes(M, K) -> int:
    """Algorithmic bytes of one quant launch: read X (bf16) and inv_lambda,
    write Xq (int8) and x_scale."""
    return 2 * M * K + M * K + 4 * M + 4 * K


def quant_name_bytes(lin) -> tuple[str, int]:
    """Name and algorithmic bytes of a layer's activation step; the adaLN
    version also reads the two bf16 modulation vectors."""
    M, K = lin.M, lin.lay.K
    if lin.mod is None:
        return "w8a8_quant_act", quant_bytes(M, K)
    return "w8a8_adaln_quant_act", quant_bytes(M, K) + 4 * K


def dequant_bytes(fmt: str, N: int, K: int) -> int:
    """Algorithmic HBM bytes of decoding a GGUF weight [N, K] to bf16: the
    planes read once, the bf16 weights written once."""
    if fmt == "q8_0":
        return N * K + 2 * (N * K // 32) + 2 * N * K
    return N * K // 2 + 12 * (N * K // 256) + 4 * (N * K // 256) + 2 * N * K


# --------------------------------------------------------------------------
# CPU oracle baseline
# --------------------------------------------------------------------------

class _OracleLinear:
    """The oracle on the first `rows` token rows of one seeded linear: for a
    W8A8 layer smoothing + per-token quant + int32 GEMM + bf16 epilogue
    (weights prepared outside the timing), for a protected layer the bf16
    linear with binary64 sums."""

    def __init__(self, c, protected: bool):
        import oracle

        self.o = oracle
        self.c, self.protected = c, protected
        self.M, self.N, self.K = c["M"], c["N"], c["K"]
        self.X = c["X"].reshape(self.M, self.K)
        if not protected:
            lam = oracle.smooth_factors(oracle.act_absmax(c["X"], self.M, self.K), c["W"],
                                        self.N, self.K, 0.5)
            self.Wq, self.ws, self.il = oracle.prepare_weight(c["W"], lam, self.N, self.K)
        self.tq = 0.0   # quant-step seconds of the last run

    def run(self, rows: int) -> float:
        o, N, K = self.o, self.N, self.K
        t = time.perf_counter()
        if self.protected:
            o.bf16_linear(self.X[:rows], self.c["W"], self.c["bias"], rows, N, K)
            self.tq = 0.0
            return time.perf_counter() - t
        Xq, xs = o.quant_act(self.X[:rows], self.il, rows, K)
        t1 = time.perf_counter()
        Y = o.w8a8_linear(Xq, xs, self.Wq, self.ws, self.c["bias"], rows, N, K)
        dt = time.perf_counter() - t
        self.tq = t1 - t
        # the timed routine against the oracle's unfused int32 GEMM +
        # epilogue on its first and last row (guards the timed work itself)
        for r in (0, rows - 1):
            acc = o.gemm_i32(Xq[r:r + 1], self.Wq, 1, N, K)
            if not np.array_equal(o.epilogue(acc, xs[r:r + 1], self.ws, self.c["bias"], 1, N),
                                  Y[r:r + 1]):
                raise SystemExit(f"oracle w8a8_linear disagrees with gemm_i32 + epilogue, row {r}")
        return dt

    def rows_for(self, seconds: float) -> tuple[int, float]:
        """Rows whose run takes about `seconds` (a 16-row probe, then once
        more from a mid-sized run, which a small probe overstates on many
        cores), and the measured time of that run."""
        rows, dt = 16, self.run(16)
        for _ in range(2):
            if rows >= self.M or dt >= 0.8 * seconds:
                break
            rows = int(min(self.M, max(16, rows * seconds / max(dt, 1e-6))))
            rows = max(16, rows // 16 * 16)
            dt = self.run(rows)
        return rows, dt


def _host_info() -> dict:
    """The host the oracle ran on: CPU model, logical CPUs, and the CPUs
    this process may run on."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        allowed = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        allowed = None
    return {"cpu_model": model, "logical_cpus": os.cpu_count(), "cpus_allowed": allowed}


def cpu_baseline(workload: str, target_s: float = 10.0):
    """The CPU oracle timed on a bounded sample of the workload on this
    host's cores (OpenMP over token rows).

    ffn_up / ffn_down: the W8A8 linear on as many token rows as take about
    target_s (the whole linear up to three times when it is faster).
    dit_block / backbone: each distinct linear shape (W8A8 or protected) on
    a row sample of about target_s / shapes, extrapolated to the workload as
    the sum over shapes of (time per row x M x number of such linears)."""
    import oracle

    oracle.build()
    if workload in ("ffn_up", "ffn_down"):
        c = synth.ffn_down_case() if workload == "ffn_down" else synth.ffn_up_case()
        lin = _OracleLinear(c, False)
        M, N, K = lin.M, lin.N, lin.K
        rows, dt = lin.rows_for(target_s)
        reps, q = 1, lin.tq
        while rows >= M and dt < target_s and reps < 3:
            dt += lin.run(rows)
            q += lin.tq
            reps += 1
        tops = 2.0 * rows * N * K * reps / dt / 1e12
        what = f"{rows} of {M} token rows" if reps == 1 else f"{reps} runs of all {M} token rows"
        return {"value": round(tops, 6), "unit": "TOPS", "cores": oracle.num_threads(),
                "kind": "oracle", "host": _host_info(),
                "quant_GB_s": round((3 * rows * K + 4 * rows) * reps / q / 1e9, 3),
                "gemm_epilogue_TOPS": round(2.0 * rows * N * K * reps / (dt - q) / 1e12, 6),
                "sample": f"{what} of the {M}x{K}->{N} linear: smoothing + per-token quant + "
                          f"int32 GEMM + bf16 epilogue (weights prepared outside the timing), "
                          f"{dt:.1f} s"}
    if workload == "dit_block":
        # the four linears of a block, counted once per CFG branch (the two
        # branches' linears differ only in their seeded weights)
        shapes = [(synth.block_case(0, li), synth.BLOCK_SHAPES[li][0] == "ffn_down", 2)
                  for li in range(4)]
        label = "one DiT block, both CFG branches"
    elif workload == "backbone":
        flags = L.protected_layers(211, 17)
        counts = {}
        for i in range(211):
            key = (i % 4, flags[i])
            counts[key] = counts.get(key, 0) + 2          # both branches
        shapes = [(synth.block_case(0, li), prot, n) for (li, prot), n in sorted(counts.items())]
        label = "211 linears x 2 branches"
    else:
        return None
    per = []
    total_s = 0.0
    total_ops = 0
    for c, prot, count in shapes:
        lin = _OracleLinear(c, prot)
        rows, dt = lin.rows_for(target_s / len(shapes))
        row_s = dt / rows
        total_s += row_s * lin.M * count
        total_ops += 2 * lin.M * lin.N * lin.K * count
        per.append(f"{'bf16' if prot else 'W8A8'} {lin.M}x{lin.K}->{lin.N} x{count}: "
                   f"{rows} rows in {dt:.2f} s")
    return {"value": round(total_ops / total_s / 1e12, 6), "unit": "TOPS",
            "cores": oracle.num_threads(), "kind": "oracle (extrapolated)", "host": _host_info(),
            "step_s_extrapolated": round(total_s, 2),
            "sample": f"{label}: each distinct linear timed on a row sample, the step's time "
                      f"extrapolated as the sum over shapes of time per row x {synth.TOKENS} "
                      f"rows x count (" + "; ".join(per) + ")"}


# --------------------------------------------------------------------------
# roofline traffic from committed counters
# --------------------------------------------------------------------------

def counter_traffic(workload: str):
    """HBM bytes per GEMM launch from the rocprofv3 counter summary in
    profiles/, if it was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", f"gemm_{workload}_counters.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("kernel_source_sha256") != sources_sha(GEMM_SOURCES):
        return None
    return d.get("hbm_bytes_per_launch")


# The counter passes. HBM traffic of the GEMM comes from two rocprofv3
# counter runs over the same short launch sequence (--counter-run): one with
# FETCH_SIZE, one with WRITE_SIZE (KiB per dispatch). Both counters are
# calibrated against a plain streaming kernel (y = -x over COPY_BYTES, larger
# than the 256 MB last-level cache, so it reads and writes COPY_BYTES of HBM
# each); --counters-from turns the two CSVs into the summary that
# counter_traffic() reads.
COPY_BYTES = 512 << 20


def counter_run(layers, dev, reps: int = 3, codes: str = "workload", path: str = "w8a8"):
    """codes="uniform" replaces the workload's int8 codes (X and W) by
    uniform random ones in [-127, 127], to compare the clock the GPU holds
    under the two (same launches, same scales). path="bf16" runs the
    workload's protected layer (bf16_linear) instead of the W8A8 one;
    path="act" its activation step (w8a8_quant_act, or w8a8_adaln_quant_act
    where the layer's input is modulated)."""
    if path == "act":
        lin = max((x for x in layers if not x.lay.protected), key=lambda x: x.ops)
        ws = L.Workspace(dev)
        Xq, xs = ws.get(lin.M, lin.lay.K)
        src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(reps):
            lin.quant(lin.xs[0], Xq, xs)
            torch.cuda.synchronize()
            torch.neg(src, out=dst)
            torch.cuda.synchronize()
        step = "w8a8_quant_act" if lin.mod is None else "w8a8_adaln_quant_act"
        log(f"counter run: {reps} x {step} {lin.M}x{lin.lay.K}, {reps} x neg over "
            f"{COPY_BYTES} bytes")
        return lin
    if path == "bf16":
        lin = max((x for x in layers if x.lay.protected), key=lambda x: x.ops)
        src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(reps):
            ops.bf16_linear(lin.xs[0], lin.lay.W, lin.lay.bias, out=lin.Y)
            torch.cuda.synchronize()
            torch.neg(src, out=dst)
            torch.cuda.synchronize()
        log(f"counter run: {reps} x bf16_linear {lin.M}x{lin.lay.K}->{lin.lay.N}, "
            f"{reps} x neg over {COPY_BYTES} bytes")
        return lin
    lin = max((x for x in layers if not x.lay.protected), key=lambda x: x.ops)
    ws = L.Workspace(dev)
    Xq, xs = ws.get(lin.M, lin.lay.K)
    ops.w8a8_quant_act(lin.xs[0], lin.lay.inv_lambda, Xq=Xq, x_scale=xs)
    Wq = lin.lay.Wq
    if codes == "uniform":
        g = torch.Generator(device=dev)
        g.manual_seed(7)
        Xq.copy_(torch.randint(-127, 128, Xq.shape, generator=g, device=dev, dtype=torch.int8))
        Wq = torch.randint(-127, 128, Wq.shape, generator=g, device=dev, dtype=torch.int8)
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        ops.w8a8_linear(Xq, xs, Wq, lin.lay.w_scale, lin.lay.bias, out=lin.Y)
        torch.cuda.synchronize()
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
    log(f"counter run: {reps} x w8a8_linear {lin.M}x{lin.lay.K}->{lin.lay.N} ({codes} codes), "
        f"{reps} x neg over {COPY_BYTES} bytes")
    return lin


def _counter_means(run_dir: str, counter: str):
    """Mean counter value per dispatch for the GEMM and the calibration
    kernel, from a rocprofv3 counter_collection.csv under run_dir."""
    import csv
    import glob

    files = glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {run_dir}")
    per = {}
    with open(files[0]) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter:
                continue
            name = r["Kernel_Name"]
            kind = "gemm" if "gemm" in name else ("copy" if "neg" in name else None)
            if kind is None:
                continue
            key = (kind, r.get("Dispatch_Id", r.get("Correlation_Id")))
            per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
    out = {}
    for kind in ("gemm", "copy"):
        vals = [v for (k, _), v in per.items() if k == kind]
        if not vals:
            raise SystemExit(f"no {kind} dispatch with {counter} in {files[0]}")
        out[kind] = float(np.mean(vals))
    return out


def counters_from(fetch_dir: str, write_dir: str, workload: str, lin_shape):
    M, N, K = lin_shape
    fe = _counter_means(fetch_dir, "FETCH_SIZE")
    wr = _counter_means(write_dir, "WRITE_SIZE")
    f_fetch = COPY_BYTES / (fe["copy"] * 1024.0)
    f_write = COPY_BYTES / (wr["copy"] * 1024.0)
    traffic = fe["gemm"] * 1024.0 * f_fetch + wr["gemm"] * 1024.0 * f_write
    d = {
        "kernel_source_sha256": sources_sha(GEMM_SOURCES),
        "workload": f"w8a8_linear {M}x{K}->{N}",
        "fetch_kib_per_launch": round(fe["gemm"], 1),
        "write_kib_per_launch": round(wr["gemm"], 1),
        "calibration": {"kernel": "y = -x (float32)", "bytes_read": COPY_BYTES,
                        "bytes_written": COPY_BYTES,
                        "fetch_kib": round(fe["copy"], 1), "write_kib": round(wr["copy"], 1),
                        "fetch_factor": round(f_fetch, 4), "write_factor": round(f_write, 4)},
        "hbm_bytes_per_launch": int(round(traffic)),
        "algorithmic_bytes_per_launch": M * K + N * K + 2 * M * N + 4 * M + 4 * N + 2 * N,
        "commands": [
            f"rocprofv3 --pmc FETCH_SIZE --output-format csv -d {fetch_dir} -o run -- "
            f"python -u bench.py --workload {workload} --counter-run",
            f"rocprofv3 --pmc WRITE_SIZE --output-format csv -d {write_dir} -o run -- "
            f"python -u bench.py --workload {workload} --counter-run",
            f"python bench.py --workload {workload} --counters-from {fetch_dir} {write_dir}",
        ],
    }
    path = os.path.join(ROOT, "profiles", f"gemm_{workload}_counters.json")
    with open(path, "w") as f:
        json.dump(d, f, indent=1)
        f.write("\n")
    print(json.dumps(d))


# --------------------------------------------------------------------------

def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="ffn_up",
                    choices=["ffn_up", "ffn_down", "dit_block", "backbone", "q8_0_ffn_up",
                             "q4_k_ffn_up", "adaln_ffn_up"])
    ap.add_argument("--pool", type=int, default=4, help="distinct inputs rotated over steps")
    ap.add_argument("--graph", action="store_true",
                    help="the step time with each step replayed from a captured HIP graph "
                         "(per-kernel figures stay eager)")
    ap.add_argument("--branch-streams", action="store_true",
                    help="dit_block / backbone: the step time with the two CFG branches issued "
                         "on two streams (per-kernel figures stay single-stream)")
    ap.add_argument("--adaln", action="store_true",
                    help="dit_block / backbone: the QKV and FFN-up inputs go through the fused "
                         "adaLN step (w8a8_adaln_quant_act) instead of w8a8_quant_act")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-accuracy", action="store_true",
                    help="skip the error report against a binary64 product")
    ap.add_argument("--no-clock", action="store_true",
                    help="skip reading the XCD clocks under load (amdsmi)")
    ap.add_argument("--no-eager", action="store_true",
                    help="skip timing the eager Torch pipeline beside the fused path")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--counter-run", action="store_true",
                    help="only the short launch sequence the counter passes profile")
    ap.add_argument("--counter-codes", choices=["workload", "uniform"], default="workload",
                    help="int8 codes of the counter run: the workload's, or uniform random")
    ap.add_argument("--counter-path", choices=["w8a8", "bf16", "act"], default="w8a8",
                    help="what the counter run launches: the W8A8 linear, the protected bf16 "
                         "one, or the activation step (the fused adaLN step where the input "
                         "is modulated)")
    ap.add_argument("--power-table", action="store_true",
                    help="only each kernel of the workload back to back, with its socket "
                         "power, power-limiter share, clock and joules per launch")
    ap.add_argument("--counters-from", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarise two rocprofv3 counter runs into profiles/ (no GPU)")
    args = ap.parse_args()

    if args.counters_from:
        shapes = {"ffn_up": (synth.TOKENS, 16384, 4096), "ffn_down": (synth.TOKENS, 4096, 16384)}
        counters_from(*args.counters_from, args.workload, shapes[args.workload])
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only and has no multi-GPU path "
              "(the W8A8 linear shards by CFG branch or token rows with no exchange "
              "between GPUs); run it with --gpus 1", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    props = torch.cuda.get_device_properties(dev)
    log(f"device {props.name} {getattr(props, 'gcnArchName', '')} CUs {props.multi_processor_count}")

    t_build = time.perf_counter()
    layers = build_workload(args.workload, dev, args.pool)
    if args.adaln:
        if args.workload not in ("dit_block", "backbone"):
            raise SystemExit("--adaln applies to --workload dit_block and backbone")
        modulate(layers, dev, 11)
    torch.cuda.synchronize()
    log(f"workload {args.workload}: {len(layers)} linears prepared in "
        f"{time.perf_counter() - t_build:.1f} s")
    if args.counter_run:
        counter_run(layers, dev, codes=args.counter_codes, path=args.counter_path)
        return
    if args.power_table:
        print(json.dumps({"workload": args.workload, "power_table": power_table(layers, dev)}))
        return

    # per-kernel durations inside the timed steps (events between kernels)
    step_ms_ev, _, quant_us, gemm_us = measure(layers, args.steps, args.warmup, dev, True)
    gemm_each = measure.gemm_each
    # the step time proper, without per-kernel events
    if args.branch_streams and args.workload not in ("dit_block", "backbone"):
        raise SystemExit("--branch-streams applies to --workload dit_block and backbone")
    step_ms, wall_ms, _, _ = measure(layers, args.steps, args.warmup, dev, False,
                                     branch_streams=args.branch_streams, graph=args.graph)
    total_ops = sum(lin.ops for lin in layers)
    value = total_ops / (step_ms * 1e-3) / 1e12

    w8 = [i for i, lin in enumerate(layers) if not lin.lay.protected and not lin.lay.weight_only]
    prot = [i for i, lin in enumerate(layers) if lin.lay.protected]
    gg = [i for i, lin in enumerate(layers) if lin.lay.weight_only]
    dom = max(w8, key=lambda i: gemm_us[i]) if w8 else None
    kernels = {}
    for i in gg:
        lin = layers[i]
        M, N, K = lin.M, lin.lay.N, lin.lay.K
        g, q = float(gemm_us[i]), float(quant_us[i])
        fmt = "q8_0" if lin.lay.q8_0 else "q4_k"
        dq_bytes = dequant_bytes(fmt, N, K)
        kernels[f"{fmt}_dequantize_{N}x{K}_in_step"] = {
            "us": round(q, 2), "GB_s": round(dq_bytes / q / 1e3, 1),
            "frac_hbm": round(dq_bytes / q / 1e3 / PEAK_HBM_GBS, 4)}
        kernels[f"{fmt}_bf16_gemm_{M}x{K}x{N}"] = {
            "us": round(g, 2), "TFLOPS": round(2 * M * N * K / g / 1e6, 1),
            "frac_bf16_peak": round(2 * M * N * K / g / 1e6 / PEAK_BF16_TFLOPS, 4)}
    for shape_key in sorted({(layers[i].M, layers[i].lay.N, layers[i].lay.K) for i in w8}):
        idx = [i for i in w8 if (layers[i].M, layers[i].lay.N, layers[i].lay.K) == shape_key]
        M, N, K = shape_key
        g = float(np.mean(gemm_us[idx]))
        q = float(np.mean(quant_us[idx]))
        kernels[f"w8a8_linear_{M}x{K}x{N}"] = {
            "us": round(g, 2), "TOPS": round(2 * M * N * K / g / 1e6, 1),
            "frac_int8_peak": round(2 * M * N * K / g / 1e6 / PEAK_INT8_TOPS, 4), "count": len(idx)}
        qname, qb = quant_name_bytes(layers[idx[0]])
        kernels[f"{qname}_{M}x{K}_in_step"] = {
            "us": round(q, 2), "GB_s": round(qb / q / 1e3, 1),
            "frac_hbm": round(qb / q / 1e3 / PEAK_HBM_GBS, 4)}
    for shape_key in sorted({(layers[i].M, layers[i].lay.N, layers[i].lay.K) for i in prot}):
        idx = [i for i in prot if (layers[i].M, layers[i].lay.N, layers[i].lay.K) == shape_key]
        M, N, K = shape_key
        g = float(np.mean(gemm_us[idx]))
        kernels[f"bf16_linear_{M}x{K}x{N}"] = {
            "us": round(g, 2), "TFLOPS": round(2 * M * N * K / g / 1e6, 1),
            "frac_bf16_peak": round(2 * M * N * K / g / 1e6 / PEAK_BF16_TFLOPS, 4),
            "count": len(idx)}
    # the quant kernel alone with HBM-resident (not cache-resident) inputs
    seen = set()
    for i in w8:
        lin = layers[i]
        if lin.lay.K in seen:
            continue
        seen.add(lin.lay.K)
        med, lo, hi = quant_isolated(lin, dev)
        qname, by = quant_name_bytes(lin)
        kernels[f"{qname}_{lin.M}x{lin.lay.K}_hbm"] = {
            "us": round(med, 2), "us_min": round(lo, 2), "us_max": round(hi, 2),
            "GB_s": round(by / med / 1e3, 1), "frac_hbm": round(by / med / 1e3 / PEAK_HBM_GBS, 4),
            "bytes": by}
        # per-channel absmax over tokens (calibration of lambda)
        med, lo, hi = absmax_isolated(lin, dev)
        kernels[f"act_absmax_{lin.M}x{lin.lay.K}_hbm"] = {
            "us": round(med, 2), "us_min": round(lo, 2), "us_max": round(hi, 2),
            "GB_s": round(2 * lin.M * lin.lay.K / med / 1e3, 1),
            "frac_hbm": round(2 * lin.M * lin.lay.K / med / 1e3 / PEAK_HBM_GBS, 4)}
        # fragility statistics (calibration-time, not part of the step):
        # one read of X
        med, lo, hi = moments_isolated(lin, dev)
        one = 2 * lin.M * lin.lay.K
        kernels[f"act_moments_{lin.M}x{lin.lay.K}_hbm"] = {
            "us": round(med, 2), "us_min": round(lo, 2), "us_max": round(hi, 2),
            "bytes_read": one, "GB_s": round(one / med / 1e3, 1),
            "frac_hbm": round(one / med / 1e3 / PEAK_HBM_GBS, 4)}

    roofline = None
    if dom is None and gg:
        i = gg[0]
        ach = layers[i].ops / (gemm_us[i] * 1e-6) / 1e12
        fmt = "Q8_0" if layers[i].lay.q8_0 else "Q4_K"
        roofline = {"bound": "mfma", "kernel": f"bf16 GEMM of the {fmt} weight-only linear",
                    "achieved": round(ach, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(ach / PEAK_BF16_TFLOPS, 4), "traffic": None,
                    "ops_per_launch": layers[i].ops, "avg_launch_us": round(float(gemm_us[i]), 2)}
    if dom is not None:
        lin = layers[dom]
        ach = lin.ops / (gemm_us[dom] * 1e-6) / 1e12
        roofline = {"bound": "mfma", "kernel": "w8a8_linear (INT8 MFMA GEMM + fused epilogue)",
                    "achieved": round(ach, 1), "peak": PEAK_INT8_TOPS, "unit": "TOP/s",
                    "frac": round(ach / PEAK_INT8_TOPS, 4),
                    "traffic": counter_traffic(args.workload),
                    "ops_per_launch": lin.ops, "avg_launch_us": round(float(gemm_us[dom]), 2),
                    "launch_us_p10_p50_p90": [round(float(v), 2) for v in
                                              np.percentile(gemm_each[:, dom], [10, 50, 90])]}
        clk = None if args.no_clock else clock_under_load(lin, dev)
        if clk is not None:
            clk["peak_clock_mhz"] = PEAK_CLOCK_MHZ
            clk["frac_at_measured_clock"] = round(
                ach / (PEAK_INT8_TOPS * clk["mhz_mean"] / PEAK_CLOCK_MHZ), 4)
        roofline["clock"] = clk

    eager = None
    if dom is not None and not args.no_eager and layers[dom].mod is None:
        lin = layers[dom]
        fused = float(quant_us[dom] + gemm_us[dom])
        us, us_mm, diff = eager_torch(lin, dev)
        eager = {"kind": "the layer as eager Torch ops (smoothing, absmax, round, clamp, "
                         "torch._int_mm, dequantization, bias), one pass each",
                 "shape": [lin.M, lin.lay.K, lin.lay.N], "us": round(us, 2),
                 "int_mm_us": round(us_mm, 2), "fused_us": round(fused, 2),
                 "speedup": round(us / fused, 3), "mean_abs_diff_rel": round(diff, 6)}

    accuracy = None
    if not args.no_accuracy and args.workload in ("ffn_up", "ffn_down"):
        log("error against a binary64 product on the host ...")
        accuracy = accuracy_report(layers, dev)

    cpu = None
    if not args.no_cpu_baseline and not args.adaln and args.workload in (
            "ffn_up", "ffn_down", "dit_block", "backbone"):
        log("timing the CPU oracle on a bounded sample ...")
        cpu = cpu_baseline(args.workload, args.cpu_seconds)

    M0 = layers[0].M
    cfg = {"workload": {"ffn_up": "DiT FFN up-projection 4608x4096->16384, one branch",
                        "ffn_down": "DiT FFN down-projection 4608x16384->4096, W8A8 and protected bf16",
                        "dit_block": "one DiT block (qkv, attn_out, ffn_up, ffn_down protected), both CFG branches",
                        "backbone": "211 linears x 2 branches, 17 protected per branch",
                        "adaln_ffn_up": "DiT FFN up-projection 4608x4096->16384 behind its adaLN modulation (fused into the activation quantization)",
                        "q8_0_ffn_up": "DiT FFN up-projection 4608x4096->16384 with GGUF Q8_0 weights",
                        "q4_k_ffn_up": "DiT FFN up-projection 4608x4096->16384 with GGUF Q4_K weights"}[args.workload],
           "tokens": M0, "linears": len(layers), "protected": len(prot),
           "adaln_inputs": sum(lin.mod is not None for lin in layers),
           "input_pool": args.pool if args.workload in ("ffn_up", "ffn_down", "adaln_ffn_up") else None,
           "smoothquant_alpha": 0.5}
    if args.adaln:
        cfg["workload"] += ", QKV and FFN-up inputs through the fused adaLN step"
    if args.branch_streams:
        cfg["workload"] += ", the two branches on two streams"
    if args.graph:
        cfg["workload"] += ", each step replayed from a HIP graph"
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "TOPS", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(step_ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if gg and not w8 else "int8",
        "data": "synthetic", "config": cfg, "roofline": roofline, "cpu_baseline": cpu,
        "eager_torch": eager, "accuracy": accuracy, "kernels": kernels, "ms_per_step_with_kernel_events": round(step_ms_ev, 4),
        "host_wall_ms_per_step": round(wall_ms, 4),
        "device": {"name": props.name, "arch": getattr(props, "gcnArchName", ""),
                   "cus": props.multi_processor_count},
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
