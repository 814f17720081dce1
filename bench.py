#!/usr/bin/env python3
"""Throughput of the fibattn hot path on one MI355X.

One step = one layer of the 60M-model shape (B=8, H=8, T=1024, d_head=64, bf16,
W=8, Fibonacci base K=15, alpha=1): RoPE of k at true positions, the forward that
rotates q where it loads it (o, lse, R q) and the backward (dq, dk, dv, dalpha, with
R^T carrying dq, dk back to the unrotated inputs), all in libfibattn.so's HIP kernels
on one stream.  Inputs are seeded N(0,1) tensors resident in HBM; several buffer sets
rotate so that the 256 MB last-level cache cannot hold a step's working set.  Steps
are replayed from a HIP graph holding one step per buffer set back to back.

Printed: one JSON line with queries*heads per second, the roofline of the dominant
kernel (algorithmic bytes per launch over its mean launch duration, timed with HIP
events on the launch stream), and the fp64 CPU oracle timed on the host's cores as
a reported baseline.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0  # MI355X HBM3E, published
ROPE_BASE = 10000.0    # theta_rope of the 60M model (Section 3)
METRIC = "fwd+bwd queries·heads/s at T=1024 and T=4096; achieved HBM GB/s vs peak"


def parse_args():
    p = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=40)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", default="layer_60m_fixed_T1024")
    p.add_argument("--sets", type=int, default=0, help="buffer sets to rotate (0: more than twice the 256 MB last-level cache between reuses)")
    p.add_argument("--eager", action="store_true", help="launch eagerly instead of replaying graphs")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=10.0, help="target length of the oracle sample")
    p.add_argument("--no-t4096", action="store_true", help="skip the T=4096 figure")
    p.add_argument("--no-gqa", action="store_true", help="skip the grouped-heads figure")
    p.add_argument("--no-learned-alpha", action="store_true", help="skip the device-alpha figure")
    p.add_argument("--no-rope-on-load", action="store_true",
                   help="skip the figure of RoPE applied to q inside the forward")
    p.add_argument("--no-integer-offsets", action="store_true",
                   help="skip the continuous vs rounded-offset stagger figure")
    p.add_argument("--no-configs", action="store_true",
                   help="skip the per-workload 16-layer sequence figures")
    p.add_argument("--copy-probe-mb", type=int, default=0,
                   help="also run one plain device copy of this many MiB (counter calibration)")
    return p.parse_args()


# HBM traffic per launch of the layer_60m_fixed_T1024 kernels, from two rocprofv3 --pmc
# passes (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch) over
#   bench.py --eager --steps 10 --warmup 2 --no-cpu-baseline --no-t4096 --no-gqa
#            --no-learned-alpha --no-integer-offsets --no-rope-on-load --no-configs --copy-probe-mb 256
# each scaled by what the same counter reads for the plain 256 MiB device copy of that run.
# They hold only for the kernel sources they were taken on (COUNTER_SOURCES_SHA).
COUNTER_SOURCES_SHA = "344e437b3afa06225bb4aeb4eea21d3a8b2183039bad721361a2dcbfe099f86c"
COUNTER_WORKLOAD = "layer_60m_fixed_T1024"
COUNTER_KIB = {  # kernel: (FETCH_SIZE, WRITE_SIZE) mean KiB per dispatch
    "forward": (12407.4, 16750.9),
    "bwd_dq": (20800.6, 10426.2),
    "bwd_dkdv": (18547.8, 16613.7),
    "rope": (4124.9, 8192.0),
}
COPY_PROBE_KIB = (262144.0, 131093.7, 262144.0)  # bytes moved each way; FETCH_SIZE; WRITE_SIZE


def kernel_sources_sha() -> str:
    d = os.path.join(ROOT, "paper_2606_28560_amd", "csrc")
    h = hashlib.sha256()
    for n in sorted(os.listdir(d)):
        if n.endswith((".hip", ".h")):
            h.update(n.encode())
            with open(os.path.join(d, n), "rb") as f:
                h.update(f.read())
    return h.hexdigest()


def hbm_traffic(kernel: str, workload: str):
    """Calibrated HBM bytes per launch, or None when the counters do not apply."""
    if workload != COUNTER_WORKLOAD or kernel not in COUNTER_KIB or kernel_sources_sha() != COUNTER_SOURCES_SHA:
        return None
    fetch, write = COUNTER_KIB[kernel]
    moved, copy_fetch, copy_write = COPY_PROBE_KIB
    return (fetch * moved / copy_fetch + write * moved / copy_write) * 1024.0


# algorithmic bytes per query-head (s = bytes per element, D = d_head)
def alg_bytes(kernel: str, D: int, s: int) -> int:
    return {
        "forward": 4 * D * s + 4,        # read q, k, v; write o, lse
        "forward_rope_q": 5 * D * s + 4, # read raw q, k, v; write o, lse, R q
        "bwd_dq": 6 * D * s + 8,         # read q, k, v, o, dO, lse; write dq, Delta
        "bwd_dkdv": 6 * D * s + 8,       # read q, k, v, dO, lse, Delta; write dk, dv
        "rope": 4 * D * s,               # read q, k; write R q, R k (one launch)
        "rope_k": 2 * D * s,             # read k; write R k
        "fwd+bwd": 12 * D * s + 8,       # forward + backward compulsory traffic
    }[kernel]


# the library kernel timed under each timing id in a Step -> its algorithmic-bytes key
STEP_ALG = {"forward": "forward_rope_q", "bwd_dq": "bwd_dq", "bwd_dkdv": "bwd_dkdv", "rope": "rope_k"}


class Step:
    """Buffers of one rotation set and the launches of one step: RoPE of k, the forward
    that rotates q where it loads it (writing R q for the backward), the backward."""

    def __init__(self, wl, call, set_index, kv_heads=None):
        import torch

        from paper_2606_28560_amd import inputs
        from paper_2606_28560_amd import fibattn as F

        self.F = F
        self.call = call
        hkv = kv_heads or wl.H
        x = inputs.attention_inputs(wl.B, wl.H, wl.T, wl.D, wl.dtype, wl.case, 1000 + set_index,
                                    names=("q", "dO"))
        x.update(inputs.attention_inputs(wl.B, hkv, wl.T, wl.D, wl.dtype, wl.case, 1000 + set_index,
                                         names=("k", "v")))
        dev = "cuda"
        self.q, self.k, self.v, self.dO = (x[n].to(dev) for n in ("q", "k", "v", "dO"))
        self.grouped = hkv != wl.H
        self.qr, self.o = torch.empty_like(self.q), torch.empty_like(self.q)
        self.kr = torch.empty_like(self.k)
        self.dq, self.dk, self.dv = torch.empty_like(self.q), torch.empty_like(self.k), torch.empty_like(self.v)
        self.lse = torch.empty((wl.B, wl.H, wl.T), device=dev, dtype=torch.float32)
        self.da = torch.empty(1, device=dev, dtype=torch.float32)
        need = F.fibattn_backward_workspace_bytes(wl.B, wl.H, wl.T, wl.D, call.W, len(call.base))
        self.ws = torch.empty(need, device=dev, dtype=torch.uint8)

    def forward(self):
        self.forward_q_on_load(True)

    def forward_two_launch(self):
        # one RoPE launch for q and k, then the forward on the rotated rows
        F, c = self.F, self.call
        if self.grouped:  # q and k have different head counts (one launch for both)
            F.fibattn_rope_qk_table(self.q, self.k, ROPE_BASE, q_out=self.qr, k_out=self.kr)
        else:
            F.fibattn_rope_qk(self.q, self.k, ROPE_BASE, q_out=self.qr, k_out=self.kr)
        F.fibattn_forward(self.qr, self.kr, self.v, c.W, c.base, c.alpha, o=self.o, lse=self.lse)

    def forward_q_on_load(self, keep_q: bool):
        # RoPE of k alone, then the forward that rotates each query row where it loads it
        # (keep_q: it also writes R q for a backward)
        F, c = self.F, self.call
        F.fibattn_rope(self.k, ROPE_BASE, out=self.kr)
        F.fibattn_forward_rope_q(self.q, self.kr, self.v, c.W, c.base, c.alpha, ROPE_BASE, o=self.o,
                                 lse=self.lse, q_out=self.qr if keep_q else None, keep_q=keep_q)

    def backward(self):
        # gradients w.r.t. the raw (unrotated) q, k: R^T is applied inside the backward
        F, c = self.F, self.call
        F.fibattn_backward(self.qr, self.kr, self.v, self.o, self.lse, self.dO, c.W, c.base, c.alpha,
                           dq=self.dq, dk=self.dk, dv=self.dv, dalpha=self.da, workspace=self.ws,
                           rope_base=ROPE_BASE)

    def __call__(self):
        self.forward()
        self.backward()


MALL_BYTES = 256 * 2**20  # MI355X last-level (Infinity) cache


def buffer_sets(per_set_bytes: int) -> int:
    """Buffer sets to rotate so that more than twice the last-level cache lies between
    two uses of one set (and at least 6 sets of the small ones)."""
    n = -(-2 * MALL_BYTES // per_set_bytes) + 1
    return max(n, 6 if per_set_bytes < 128 * 2**20 else 2)


def step_bytes(wl, call, kv_heads=None) -> int:
    """Device bytes of one Step's buffers (inputs, RoPE outputs, outputs, workspace)."""
    s = 2 if wl.dtype == "bf16" else 4
    hkv = kv_heads or wl.H
    qrow, kvrow = wl.B * wl.H * wl.T * wl.D * s, wl.B * hkv * wl.T * wl.D * s
    from paper_2606_28560_amd import fibattn as F
    ws = F.fibattn_backward_workspace_bytes(wl.B, wl.H, wl.T, wl.D, call.W, len(call.base))
    return 5 * qrow + 5 * kvrow + 4 * wl.B * wl.H * wl.T + ws


def capture(fn):
    import torch

    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()  # warm the allocator-free path once outside the graph
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def timed(run, steps: int, warmup: int):
    """Mean ms per step over `steps` calls of run(i), after `warmup` calls."""
    import torch

    for i in range(warmup):
        run(i)
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    t0.record()
    for i in range(steps):
        run(i)
    t1.record()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - w0) * 1e3 / steps
    return t0.elapsed_time(t1) / steps, wall


def timed_steps(fns, steps: int, warmup: int, eager: bool, whole: bool = True):
    """(mean ms per step, host wall ms per step) over `steps` steps after `warmup`, step i
    running fns[i % n], one function per buffer set.  With graphs, the n steps of one
    rotation over the buffer sets are captured back to back in one graph, as the layers
    of a model's training step are captured together; the timed region replays it
    steps // n times and then single-step graphs for the remaining steps, so it runs
    exactly `steps` steps, continuing the rotation where the warm-up left it.  (Replaying
    one single-step graph per step leaves the GPU idle for several microseconds between
    replays on this runtime: `one_graph_per_step_ms` in the output.)  whole: round `steps`
    up to whole rotations (the figures); the headline passes False and runs exactly the
    steps asked for."""
    import torch

    n = len(fns)
    if whole:
        steps = -(-steps // n) * n
    if eager:
        return timed(lambda i: fns[i % n](), steps, warmup)
    start = warmup % n
    singles = [capture(f) for f in fns]
    rot = capture(lambda: [fns[(start + j) % n]() for j in range(n)])
    for i in range(warmup):
        singles[i % n].replay()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    t0.record()
    for _ in range(steps // n):
        rot.replay()
    for j in range(steps % n):
        singles[(start + j) % n].replay()
    t1.record()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - w0) * 1e3 / steps
    return t0.elapsed_time(t1) / steps, wall


def kernel_time(F, sets, kernel: str, steps: int, per_step: int):
    """Mean launch duration (ms) of one library kernel over `steps` eager steps.  The
    library launches that kernel with a HIP event pair that takes the dispatch's own
    start and end timestamps (hipExtLaunchKernel on the launch stream), the interval a
    kernel-trace profile reports.  A spin kernel (no memory traffic) ahead of each step
    keeps the queue busy, as in the graph-replayed steps."""
    import torch

    torch.cuda.synchronize()
    F.fibattn_timing_begin(kernel, steps * per_step)
    for i in range(steps):
        torch.cuda._sleep(400_000)
        sets[i % len(sets)]()
    ms, n = F.fibattn_timing_end()
    return ms, n


def cpu_baseline(wl, call, target_s: float):
    """The fp64 oracle (as it stands) on a bounded sample of the same step."""
    import oracle
    from paper_2606_28560_amd import inputs

    b = wl.B  # the whole layer: B x H x T query-heads (OpenMP over the B*H pairs)
    x = inputs.attention_inputs(b, wl.H, wl.T, wl.D, wl.dtype, wl.case, 1000)
    q, k, v, dO = (x[n].double().numpy() for n in ("q", "k", "v", "dO"))
    reps = 0
    t0 = time.perf_counter()
    while True:
        qr, kr = oracle.rope(q), oracle.rope(k)
        oracle.forward(qr, kr, v, call.W, call.base, call.alpha)
        dq, dk, dv, da, _ = oracle.backward(qr, kr, v, dO, call.W, call.base, call.alpha)
        oracle.rope(dq, transpose=True)
        oracle.rope(dk, transpose=True)
        reps += 1
        el = time.perf_counter() - t0
        if el >= target_s or reps >= 1000:
            break
    qh = reps * b * wl.H * wl.T
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), "")
    except OSError:
        pass
    return {
        "value": qh / el,
        "unit": "queries·heads/s",
        "cores": min(oracle.num_threads(), b * wl.H),
        "kind": "oracle",
        "sample": f"{reps} x the full step (RoPE, forward, backward, R^T) of one layer "
                  f"({b}x{wl.H}x{wl.T} query-heads), {el:.1f} s",
        "openmp_threads": oracle.num_threads(),
        "nproc": len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count(),
        "cpu_model": model,
    }


def t4096_figure(steps: int, warmup: int, eager: bool):
    """fwd+bwd step at the 4x-length shape (B=4, H=8, T=4096, coprime layer 1)."""
    from paper_2606_28560_amd import workloads

    wl = workloads.workload("extrap_coprime16_T4096")
    call = wl.calls[1]
    sets = [Step(wl, call, i) for i in range(buffer_sets(step_bytes(wl, call)))]
    ms, _ = timed_steps(sets, steps, warmup, eager)
    msf, _ = timed_steps([s.forward for s in sets], steps, warmup, eager)
    qh = wl.queries_heads
    from paper_2606_28560_amd import fibattn as F
    kt = {k: round(kernel_time(F, sets, k, steps, 1)[0], 6) for k in ("forward", "bwd_dq", "bwd_dkdv", "rope")}
    # fwd+bwd compulsory bytes over the three attention kernels' summed launch durations
    s = 2 if wl.dtype == "bf16" else 4
    attn_ms = kt["forward"] + kt["bwd_dq"] + kt["bwd_dkdv"]
    frac = alg_bytes("fwd+bwd", wl.D, s) * qh / (attn_ms * 1e-3) / 1e9 / PEAK_HBM_GBS
    kfrac = {k: round(alg_bytes(STEP_ALG[k], wl.D, s) * qh / (kt[k] * 1e-3) / 1e9 / PEAK_HBM_GBS, 4) for k in kt}
    return {"workload": wl.name, "alpha": float(call.alpha), "ms_per_step": ms,
            "value": qh / (ms * 1e-3), "fwd_only_ms": msf, "fwd_only_value": qh / (msf * 1e-3),
            "kernels_mean_ms": kt, "kernels_frac": kfrac, "attention_kernels_ms": attn_ms,
            "attention_frac": round(frac, 4)}


def rope_on_load_figure(steps: int, warmup: int, eager: bool, rounds: int = 3):
    """RoPE applied to q where the forward loads it, against one RoPE launch for q and k
    ahead of the forward: forward only (no R q written) at the T=1024 layer and at the
    4x-length layer, and the T=1024 training step (R q written for the backward).  The
    variants alternate over `rounds` rounds; medians."""
    import statistics

    import torch

    from paper_2606_28560_amd import fibattn as F
    from paper_2606_28560_amd import workloads

    out = {}
    cases = [("layer_60m_fixed_T1024", 0, True), ("extrap_coprime16_T4096", 1, False)]
    for name, ci, train in cases:
        wl = workloads.workload(name)
        call = wl.calls[ci]
        sets = [Step(wl, call, i) for i in range(buffer_sets(step_bytes(wl, call)))]
        variants = {"two_launch_fwd": lambda st: st.forward_two_launch(),
                    "on_load_fwd": lambda st: st.forward_q_on_load(False)}
        if train:
            variants["two_launch_step"] = lambda st: (st.forward_two_launch(), st.backward())
            variants["on_load_step"] = lambda st: st()
        runs = {v: [lambda st=st, fn=fn: fn(st) for st in sets] for v, fn in variants.items()}
        res = {v: [] for v in variants}
        for _ in range(rounds):
            for vname in variants:
                res[vname].append(timed_steps(runs[vname], steps, warmup, eager)[0])
        fig = {v + "_ms": statistics.median(t) for v, t in res.items()}
        # launch durations of the rotating forward and of the RoPE launch on k alone
        fsets = [lambda st=st: st.forward_q_on_load(False) for st in sets]
        fig["on_load_kernels_ms"] = {k: round(kernel_time(F, fsets, k, steps, 1)[0], 6) for k in ("forward", "rope")}
        fig["alpha"] = float(call.alpha)
        out[name] = fig
        del sets, runs
        torch.cuda.synchronize()
    return out


def integer_offsets_figure(steps: int, warmup: int, eager: bool, layer: int = 3):
    """Attention forward + backward of a static-stagger layer (B=16, H=8, T=1024, W=8)
    on continuous offsets alpha * f (interpolated) and on the same offsets rounded to
    integers (one row per rung)."""
    import dataclasses

    import numpy as np

    from paper_2606_28560_amd import schedules, workloads

    wl = workloads.workload("stagger16_T1024")
    call = next(c for c in wl.calls if c.W == 8 and c.layer == layer)
    rounded = dataclasses.replace(call, base=schedules.integer_base(call.alpha, call.base),
                                  alpha=np.float32(1.0))
    out = {"workload": wl.name, "layer": layer, "alpha": float(call.alpha)}
    for tag, c in (("continuous", call), ("integer", rounded)):
        from paper_2606_28560_amd import fibattn as F
        sets = [Step(wl, c, i) for i in range(buffer_sets(step_bytes(wl, c)))]
        ms, _ = timed_steps([lambda st=st: attn_one(F, st) for st in sets], steps, warmup, eager)
        out[tag + "_ms"] = ms
        out[tag + "_value"] = wl.queries_heads / (ms * 1e-3)
        del sets
    out["integer_speedup"] = out["continuous_ms"] / out["integer_ms"]
    return out


def gqa_figure(steps: int, warmup: int, eager: bool, kv_heads: int = 2):
    """The 60M model's layer with its grouped key/value heads (8 query heads, 2 key/value
    heads; B=8, T=1024, W=8, Fibonacci, alpha=1): the full step (RoPE of k, the forward
    rotating q on load, backward) and per-kernel launch durations."""
    from paper_2606_28560_amd import fibattn as F
    from paper_2606_28560_amd import workloads

    wl = workloads.workload("layer_60m_fixed_T1024")
    call = wl.calls[0]
    sets = [Step(wl, call, i, kv_heads=kv_heads)
            for i in range(buffer_sets(step_bytes(wl, call, kv_heads)))]
    ms, _ = timed_steps(sets, steps, warmup, eager)
    kt = {}
    for k in ("forward", "bwd_dq", "bwd_dkdv", "rope"):
        kms, n = kernel_time(F, sets, k, steps, 1)
        kt[k] = round(kms * n / steps, 6)  # per step
    qh = wl.queries_heads
    # algorithmic bytes per query-head with G query heads per key/value head: the k, v
    # (and dk, dv) terms shrink by G
    G, D, s = wl.H // kv_heads, wl.D, 2 if wl.dtype == "bf16" else 4
    grouped = {"forward": 3 * D * s + 2 * D * s // G + 4, "bwd_dq": 4 * D * s + 2 * D * s // G + 8,
               "bwd_dkdv": 2 * D * s + 4 * D * s // G + 8, "rope": 2 * D * s // G}
    frac = {k: round(grouped[k] * qh / (kt[k] * 1e-3) / 1e9 / PEAK_HBM_GBS, 4) for k in grouped if kt.get(k)}
    return {"workload": wl.name, "H": wl.H, "H_kv": kv_heads, "ms_per_step": ms,
            "value": qh / (ms * 1e-3), "kernels_ms_per_step": kt, "buffer_sets": len(sets),
            "alg_bytes_per_qh": grouped, "kernels_frac": frac}


def learned_alpha_figure(steps: int, warmup: int, eager: bool, layer: int = 0):
    """Learned-alpha layer of the pow2/fib workload (B=32, H=8, T=1024, W=10, Fibonacci
    base, alpha = 0.5 + sigmoid(theta)) with theta resident on the device: theta ->
    alpha and rung table, in the RoPE launch of k -> forward rotating q -> backward with
    dtheta, against the same launches with alpha passed from the host."""
    import torch

    from paper_2606_28560_amd import fibattn as F
    from paper_2606_28560_amd import inputs, workloads

    wl = workloads.workload("pow2_fib_learned16_T1024")
    call = next(c for c in wl.calls if c.base_name == "fib15" and c.layer == layer)
    theta = torch.tensor(inputs.thetas(16, case=5)[layer:layer + 1], dtype=torch.float32, device="cuda")
    sets = [Step(wl, call, i) for i in range(buffer_sets(step_bytes(wl, call)))]
    dev = []
    for st in sets:
        st.theta, st.alpha = theta, torch.empty_like(theta)
        st.table = torch.empty(F.lib().fibattn_device_table_bytes(), device="cuda", dtype=torch.uint8)
        st.dtheta = torch.empty_like(theta)
        # a device table's rung count is not known on the host: the workspace for K = 0
        st.ws = torch.empty(F.fibattn_backward_workspace_bytes(wl.B, wl.H, wl.T, wl.D, call.W, 0),
                            device="cuda", dtype=torch.uint8)

        def run_dev(st=st):
            c = st.call
            F.fibattn_rope_qk_table(None, st.k, ROPE_BASE, theta=st.theta, base=c.base, W=c.W, table=st.table,
                                    alpha=st.alpha, k_out=st.kr)
            F.fibattn_forward_rope_q_dt(st.q, st.kr, st.v, c.W, st.table, ROPE_BASE, o=st.o, lse=st.lse,
                                        q_out=st.qr)
            F.fibattn_backward_dt(st.qr, st.kr, st.v, st.o, st.lse, st.dO, c.W, st.table, dq=st.dq,
                                  dk=st.dk, dv=st.dv, dalpha=st.da, dtheta=st.dtheta, workspace=st.ws,
                                  rope_base=ROPE_BASE)
        dev.append(run_dev)
    out = {"workload": wl.name, "layer": layer, "alpha": float(call.alpha)}
    runs = {"device_alpha": dev, "host_alpha": sets}
    # The two steps alternate over three rounds and the medians are reported: whichever
    # is measured first otherwise carries the GPU's ramp-up (7% on one run).
    ms_r = {tag: [] for tag in runs}
    kt_r = {tag: {} for tag in runs}
    for _ in range(3):
        for tag, fns in runs.items():
            ms_r[tag].append(timed_steps(fns, steps, warmup, eager)[0])
            for k in ("forward", "bwd_dq", "bwd_dkdv", "rope"):
                kms, n = kernel_time(F, fns, k, steps, 1)
                if n:
                    kt_r[tag].setdefault(k, []).append(kms)
    for tag in runs:
        ms = statistics.median(ms_r[tag])
        out[tag + "_ms"] = ms
        out[tag + "_value"] = wl.queries_heads / (ms * 1e-3)
        out[tag + "_kernels_ms"] = {k: round(statistics.median(v), 6) for k, v in kt_r[tag].items()}
    return out


class LayerSet:
    """Buffers of one rotation set for attention-only layer calls (q, k post-RoPE)."""

    def __init__(self, wl, call, set_index):
        import torch

        from paper_2606_28560_amd import inputs

        x = inputs.attention_inputs(wl.B, wl.H, wl.T, wl.D, wl.dtype, wl.case, 2000 + set_index)
        self.q, self.k, self.v, self.dO = (x[n].to("cuda") for n in ("q", "k", "v", "dO"))
        del x
        self.o, self.dq = torch.empty_like(self.q), torch.empty_like(self.q)
        self.dk, self.dv = torch.empty_like(self.k), torch.empty_like(self.v)
        self.lse = torch.empty((wl.B, wl.H, wl.T), device="cuda", dtype=torch.float32)
        self.da = torch.empty(1, device="cuda", dtype=torch.float32)
        from paper_2606_28560_amd import fibattn as F
        need = max(F.fibattn_backward_workspace_bytes(wl.B, wl.H, wl.T, wl.D, c.W, len(c.base))
                   for c in wl.calls)
        self.ws = torch.empty(need, device="cuda", dtype=torch.uint8)


def sequence_figure(F, wl, calls, sets, backward: bool, steps: int, warmup: int, eager: bool):
    """One pass over `calls` (a 16-layer sequence), layer l on buffer set l % len(sets),
    each layer an attention forward (and backward) on its own alpha and W."""
    def run_seq():
        for l, c in enumerate(calls):
            st = sets[l % len(sets)]
            F.fibattn_forward(st.q, st.k, st.v, c.W, c.base, c.alpha, o=st.o, lse=st.lse)
            if backward:
                F.fibattn_backward(st.q, st.k, st.v, st.o, st.lse, st.dO, c.W, c.base, c.alpha,
                                   dq=st.dq, dk=st.dk, dv=st.dv, dalpha=st.da, workspace=st.ws)
    if eager:
        run = lambda i: run_seq()  # noqa: E731
    else:
        g = capture(run_seq)
        run = lambda i: g.replay()  # noqa: E731
    ms, _ = timed(run, steps, warmup)
    s = 2 if wl.dtype == "bf16" else 4
    qh = wl.queries_heads * len(calls)
    byt = alg_bytes("fwd+bwd" if backward else "forward", wl.D, s) * qh
    return {"layers": len(calls), "ms": ms, "ms_per_layer": ms / len(calls), "value": qh / (ms * 1e-3),
            "alg_GBs": byt / (ms * 1e-3) / 1e9, "frac": byt / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS}


def config_figures(steps: int, warmup: int, eager: bool):
    """Attention forward + backward (no RoPE) of each workload's 16-layer sequence at its
    own shape: the stagger sweep once per W, the 4x-length coprime stagger forward-only
    and forward + backward, the pow2/fib learned-alpha layers once per base.  queries·heads/s
    and the fraction of 8 TB/s for the algorithmic bytes (fwd+bwd 12·d·s+8, fwd 4·d·s+4 per
    query-head)."""
    import torch

    from paper_2606_28560_amd import fibattn as F
    from paper_2606_28560_amd import workloads

    out = {}
    for name in ("stagger16_T1024", "extrap_coprime16_T4096", "pow2_fib_learned16_T1024"):
        wl = workloads.workload(name)
        per = step_bytes(wl, wl.calls[0])
        n = max(2, -(-2 * MALL_BYTES // per) + 1)
        sets = [LayerSet(wl, wl.calls[0], i) for i in range(n)]
        fig = {"B": wl.B, "H": wl.H, "T": wl.T, "d_head": wl.D, "buffer_sets": n}
        if name == "stagger16_T1024":
            for W in sorted(set(c.W for c in wl.calls)):
                calls = [c for c in wl.calls if c.W == W]
                fig[f"W{W}"] = sequence_figure(F, wl, calls, sets, True, steps, warmup, eager)
        elif name == "extrap_coprime16_T4096":
            fig["forward"] = sequence_figure(F, wl, wl.calls, sets, False, steps, warmup, eager)
            fig["fwd+bwd"] = sequence_figure(F, wl, wl.calls, sets, True, steps, warmup, eager)
        else:
            for b in ("pow2_11", "fib15"):
                calls = [c for c in wl.calls if c.base_name == b]
                fig[b] = sequence_figure(F, wl, calls, sets, True, steps, warmup, eager)
        out[name] = fig
        del sets
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    return out


def main():
    args = parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}): "
              "the library has no multi-GPU path; rerun with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2606_28560_amd import fibattn as F
    from paper_2606_28560_amd import workloads

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    F.lib()
    wl = workloads.workload(args.workload)
    call = wl.calls[0]
    s = 2 if wl.dtype == "bf16" else 4
    nsets = args.sets or buffer_sets(step_bytes(wl, call))
    print(f"# workload {wl.name}: B{wl.B} H{wl.H} T{wl.T} D{wl.D} {wl.dtype} W{call.W} "
          f"{call.base_name} alpha={float(call.alpha)}; {nsets} buffer sets", file=sys.stderr, flush=True)
    sets = [Step(wl, call, i) for i in range(nsets)]
    torch.cuda.synchronize()

    ms, wall_ms = timed_steps(sets, args.steps, args.warmup, args.eager, whole=False)
    qh = wl.queries_heads
    print(f"# step {ms:.4f} ms (host wall {wall_ms:.4f} ms/step)", file=sys.stderr, flush=True)

    # the same steps with one single-step graph replayed per step (launch-gap comparison)
    one_ms = None
    if not args.eager:
        graphs = [capture(st) for st in sets]
        one_ms, _ = timed(lambda i: graphs[i % nsets].replay(), args.steps, args.warmup)
        del graphs

    # attention only (forward + backward kernels, no RoPE)
    ms_attn, _ = timed_steps([lambda st=st: attn_one(F, st) for st in sets], args.steps, args.warmup, args.eager,
                             whole=False)

    # per-kernel mean durations (eager steps, library HIP events on the launch stream)
    kt = {}
    for kname in ("forward", "bwd_dq", "bwd_dkdv", "rope"):
        kms, n = kernel_time(F, sets, kname, args.steps, 1)
        kt[kname] = {"mean_ms": kms, "launches": n,
                     "frac": alg_bytes(STEP_ALG[kname], wl.D, s) * qh / (kms * 1e-3) / 1e9 / PEAK_HBM_GBS}
    per_step = {k: v["mean_ms"] for k, v in kt.items()}
    dom = max(per_step, key=per_step.get)
    units = qh  # query-heads per launch
    achieved = alg_bytes(STEP_ALG[dom], wl.D, s) * units / (kt[dom]["mean_ms"] * 1e-3) / 1e9
    roofline = {"bound": "hbm", "kernel": dom, "achieved": achieved, "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS, "traffic": hbm_traffic(dom, wl.name),
                "bytes_per_launch": alg_bytes(STEP_ALG[dom], wl.D, s) * units,
                "mean_launch_ms": kt[dom]["mean_ms"]}

    result = {
        "metric": METRIC,
        "value": qh / (ms * 1e-3),
        "unit": "queries·heads/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": wl.name, "B": wl.B, "H": wl.H, "T": wl.T, "d_head": wl.D,
                   "W": call.W, "base": call.base_name, "alpha": float(call.alpha),
                   "step": "rope(k) + forward rotating q on load + backward (dq, dk w.r.t. unrotated q, k)",
                   "launch": "eager" if args.eager else f"hip_graph of {nsets} steps (one per buffer set)",
                   "buffer_sets": nsets},
        "one_graph_per_step_ms": one_ms,
        "roofline": roofline,
        "attention_only": {"ms_per_step": ms_attn, "value": qh / (ms_attn * 1e-3),
                           "alg_GBs": alg_bytes("fwd+bwd", wl.D, s) * qh / (ms_attn * 1e-3) / 1e9,
                           "frac": alg_bytes("fwd+bwd", wl.D, s) * qh / (ms_attn * 1e-3) / 1e9
                           / PEAK_HBM_GBS},
        "kernels": kt,
    }
    if not args.no_t4096:
        result["t4096"] = t4096_figure(max(5, args.steps // 4), 2, args.eager)
    if not args.no_gqa:
        result["gqa"] = gqa_figure(max(5, args.steps // 4), 2, args.eager)
    if not args.no_learned_alpha:
        result["learned_alpha"] = learned_alpha_figure(max(5, args.steps // 4), 2, args.eager)
    if not args.no_rope_on_load:
        result["rope_on_load"] = rope_on_load_figure(max(5, args.steps // 4), 2, args.eager)
    if not args.no_integer_offsets:
        result["integer_offsets"] = integer_offsets_figure(max(5, args.steps // 4), 2, args.eager)
    if not args.no_configs:
        result["configs"] = config_figures(max(3, args.steps // 8), 1, args.eager)
    if args.copy_probe_mb:
        a = torch.empty(args.copy_probe_mb * 2**20, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        result["copy_probe_bytes"] = a.numel()
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, call, args.cpu_seconds)
    print(json.dumps(result), flush=True)


def attn_one(F, st):
    c = st.call
    F.fibattn_forward(st.qr, st.kr, st.v, c.W, c.base, c.alpha, o=st.o, lse=st.lse)
    F.fibattn_backward(st.qr, st.kr, st.v, st.o, st.lse, st.dO, c.W, c.base, c.alpha,
                       dq=st.dq, dk=st.dk, dv=st.dv, dalpha=st.da, workspace=st.ws)


if __name__ == "__main__":
    main()
