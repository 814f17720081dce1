"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Small cases span several workgroups and a ragged tail (T not a multiple of the 16-
to 64-query tile) in both storage dtypes and both head sizes, including the edge
cases of the method: T = 1, T < W, no rungs, all rungs inside the window, all rungs
masked, a rung landing exactly on row 0 (zero row beyond it), integer and
non-integer alpha, the maximum window and rung count.  Full-size cases run the five
workloads' shapes (a subset of their layers) in the launch configuration the
benchmark uses.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_28560_amd import inputs, schedules, workloads
from paper_2606_28560_amd import fibattn as F
from tests.parity import compare, gpu_run, oracle_run, rope_flip_size, rope_rounding_slack

pytestmark = pytest.mark.gpu

FIB = schedules.FIB15
POW2 = schedules.POW2_11


def _case_inputs(B, H, T, D, dtype, seed):
    return inputs.attention_inputs(B, H, T, D, dtype, 100 + seed, 0)


SMALL = [
    # (B, H, T, D, dtype, W, base, alpha)
    (1, 2, 128, 32, "fp32", 8, FIB, 1.0),
    (2, 3, 333, 32, "fp32", 8, FIB, 0.7310586),
    (1, 2, 300, 64, "fp32", 6, FIB, 1.5),
    (2, 2, 257, 64, "fp32", 3, POW2, 0.5),
    (1, 3, 333, 64, "bf16", 8, FIB, 1.0),
    (2, 2, 300, 64, "bf16", 12, FIB, 1.3),
    (1, 2, 290, 32, "bf16", 10, POW2, 0.8),
    (1, 1, 1, 64, "bf16", 8, FIB, 1.0),            # single position
    (1, 2, 5, 32, "fp32", 8, FIB, 1.0),            # T < W
    (1, 2, 77, 64, "fp32", 0, [], 1.0),            # no rungs, window of one
    (1, 2, 77, 32, "fp32", 12, FIB[:5], 1.0),      # every rung inside the window
    (1, 2, 40, 64, "bf16", 4, [50, 60, 70], 1.0),  # every rung masked (d > T-1)
    (1, 2, 64, 32, "fp32", 2, [1, 13, 40], 1.0),   # d = 13 and 40 land on row 0
    (1, 1, 300, 64, "fp32", 128, FIB, 1.1),        # maximum window
    (1, 1, 700, 32, "fp32", 0, list(range(3, 99, 3)), 0.9),  # K = 32
    (1, 2, 200, 64, "bf16", 8, FIB, 0.01),         # tiny alpha: all rungs in the window
    # 320 workgroups: 40 per XCD, so the reversed second run of the block order is
    # a partial one (8 positions)
    (1, 5, 4096, 64, "bf16", 8, FIB, 1.0),
    (1, 5, 4096, 64, "bf16", 8, FIB, 0.9),
    # the matrix-core kernels' window limit: their band tile reaches exactly 16 keys
    # back (W = 16), one below the first W the generic kernels take (W = 17); W = 0 with
    # alpha = 0.9 has a rung at d = 0.9 whose row r0 is the query itself
    (1, 2, 300, 64, "bf16", 16, FIB, 1.0),
    (1, 2, 300, 64, "bf16", 16, FIB, 0.7310586),
    (2, 1, 333, 64, "bf16", 13, FIB, 1.0),
    (2, 1, 333, 64, "bf16", 13, POW2, 1.3),
    (1, 2, 257, 64, "bf16", 0, FIB, 1.0),
    (1, 2, 257, 64, "bf16", 0, FIB, 0.9),
    (1, 2, 290, 64, "bf16", 17, FIB, 1.0),
    (1, 2, 290, 64, "bf16", 17, FIB, 1.2),
]


@pytest.mark.parametrize("B,H,T,D,dtype,W,base,alpha", SMALL)
def test_small_parity(B, H, T, D, dtype, W, base, alpha):
    idx = SMALL.index((B, H, T, D, dtype, W, base, alpha))
    x = _case_inputs(B, H, T, D, dtype, idx)
    print(f"small case {idx}: B{B} H{H} T{T} D{D} {dtype} W{W} K{len(base)} alpha={alpha}", flush=True)
    got = gpu_run(x["q"], x["k"], x["v"], x["dO"], W, base, alpha)
    ref = oracle_run(x["q"], x["k"], x["v"], x["dO"], W, base, alpha)
    rep = compare(got, ref, dtype, f"case {idx}")
    if "dalpha" in ref:
        print(f"dalpha {got['dalpha']:.6g} ref {ref['dalpha']:.6g} L1 {ref['l1']:.4g}", flush=True)
    print(rep, flush=True)


def _full_calls(wl):
    """A subset of each workload's layer calls: the first, the last and two interior."""
    n = len(wl.calls)
    picks = sorted(set([0, n - 1, n // 3, (2 * n) // 3]))
    return [(wl, c) for c in picks]


FULL = [pc for w in workloads.all_workloads() for pc in _full_calls(w)]


@pytest.mark.parametrize("wl,ci", FULL, ids=[f"{w.name}-call{c}" for w, c in FULL])
def test_full_size_parity(wl, ci):
    call = wl.calls[ci]
    print(f"full case {wl.name} call {ci}: layer {call.layer} W{call.W} {call.base_name} "
          f"alpha={float(call.alpha):.7f}", flush=True)
    x = workloads.layer_inputs(wl, ci)
    got = gpu_run(x["q"], x["k"], x["v"], x["dO"], call.W, call.base, call.alpha, backward=wl.backward)
    ref = oracle_run(x["q"], x["k"], x["v"], x["dO"], call.W, call.base, call.alpha, backward=wl.backward)
    rep = compare(got, ref, wl.dtype, f"{wl.name} call {ci}")
    if "dalpha" in ref:
        print(f"dalpha {got['dalpha']:.6g} ref {ref['dalpha']:.6g} L1 {ref['l1']:.4g}", flush=True)
    print(rep, flush=True)


@pytest.mark.parametrize("layer", [3, 11])
def test_integer_offsets_from_rounded_base(layer):
    # static stagger on integer offsets: the rounded base with alpha = 1 runs the
    # kernels that read one row per rung; the oracle gets the same table
    wl = workloads.workload("stagger16_T1024")
    a = schedules.alpha_linear_stagger(16)[layer]
    base = schedules.integer_base(a, FIB)
    print(f"integer offsets: layer {layer} alpha {float(a):.7f} base {base}", flush=True)
    x = inputs.attention_inputs(4, wl.H, wl.T, wl.D, wl.dtype, wl.case, 200 + layer)
    got = gpu_run(x["q"], x["k"], x["v"], x["dO"], 8, base, 1.0)
    ref = oracle_run(x["q"], x["k"], x["v"], x["dO"], 8, base, 1.0)
    compare(got, ref, wl.dtype, f"integer offsets layer {layer}")


def test_backward_at_extrapolation_length():
    # the T = 4096 workload is forward-only; the backward at that shape is checked too
    wl = workloads.workload("extrap_coprime16_T4096")
    call = wl.calls[1]
    x = inputs.attention_inputs(1, 4, wl.T, wl.D, wl.dtype, wl.case, 99)
    got = gpu_run(x["q"], x["k"], x["v"], x["dO"], call.W, call.base, call.alpha)
    ref = oracle_run(x["q"], x["k"], x["v"], x["dO"], call.W, call.base, call.alpha)
    compare(got, ref, wl.dtype, "T4096 backward")


@pytest.mark.parametrize("dtype,D,transpose,B,H,T", [
    ("fp32", 32, False, 2, 3, 1029), ("fp32", 64, True, 2, 3, 1029),
    ("bf16", 64, False, 2, 3, 1029), ("bf16", 32, True, 2, 3, 1029),
    # at least 2^17 rows: the bf16 d_head 64 launch of one tensor takes two positions per
    # lane group; T = 3999 leaves a ragged last workgroup of positions
    ("bf16", 64, False, 1, 33, 3999), ("bf16", 64, True, 1, 33, 3999)])
def test_rope_parity(dtype, D, transpose, B, H, T):
    x = _case_inputs(B, H, T, D, dtype, 50)["q"]
    got = F.fibattn_rope(x.cuda(), 10000.0, transpose).double().cpu().numpy()
    ref = oracle.rope(x, 10000.0, transpose)
    err = np.abs(got - ref).max()
    if dtype == "fp32":
        assert err <= 1e-5
    else:
        assert err <= 2e-2 * np.abs(ref).max()


def test_rope_in_place():
    x = _case_inputs(1, 2, 100, 64, "fp32", 51)["k"].cuda()
    y = F.fibattn_rope(x, 10000.0)
    F.fibattn_rope(x, 10000.0, out=x)
    assert torch.equal(x, y)


PIPE = [
    # (dtype, D, W, alpha): bf16/64/W<=16 applies R^T in the backward kernels' epilogue;
    # the others run the generic kernels followed by an R^T launch
    ("bf16", 64, 8, 0.85),
    ("bf16", 64, 8, 1.0),
    ("fp32", 64, 8, 0.85),
    ("fp32", 32, 6, 1.2),
    ("bf16", 64, 20, 0.9),
]


@pytest.mark.parametrize("dtype,D,W,alpha", PIPE)
def test_pipeline_with_rope(dtype, D, W, alpha):
    # raw q, k -> RoPE -> attention forward -> backward returning gradients w.r.t. the
    # raw q, k; the oracle runs the same chain (its rotated q, k rounded to the
    # storage dtype, as the pipeline stores them)
    B, H, T = 1, 2, 200
    x = _case_inputs(B, H, T, D, dtype, 60 + PIPE.index((dtype, D, W, alpha)))
    Q, K = F.fibattn_rope_qk(x["q"].cuda(), x["k"].cuda(), 10000.0)
    V, G = x["v"].cuda(), x["dO"].cuda()
    o, lse = F.fibattn_forward(Q, K, V, W, FIB, alpha)
    dq, dk, dv, da = F.fibattn_backward(Q, K, V, o, lse, G, W, FIB, alpha, rope_base=10000.0)
    torch.cuda.synchronize()
    eq, ek = oracle.rope(x["q"]), oracle.rope(x["k"])  # exact rotations
    rq, rk = (inputs.round_to(r.astype(np.float32), dtype).double().numpy() for r in (eq, ek))
    slack = rope_rounding_slack(x["q"].double().numpy(), x["k"].double().numpy(), eq, ek, dtype, W, FIB, alpha)
    if dtype == "fp32":
        np.testing.assert_allclose(Q.double().cpu().numpy(), rq, atol=1e-5, rtol=0)
    else:  # the oracle's rounding, or the other neighbour where a float32 rotation may flip it
        assert np.all(np.abs(Q.double().cpu().numpy() - rq) <= rope_flip_size(x["q"].double().numpy(), eq))
    ro, rl = oracle.forward(rq, rk, x["v"], W, FIB, alpha)
    rdq, rdk, rdv, rda, l1 = oracle.backward(rq, rk, x["v"], x["dO"], W, FIB, alpha)
    rdq, rdk = oracle.rope(rdq, transpose=True), oracle.rope(rdk, transpose=True)
    got = {"o": o, "lse": lse, "dq": dq, "dk": dk, "dv": dv}
    got = {kk: vv.double().cpu().numpy() for kk, vv in got.items()}
    got["dalpha"] = float(da.item())
    compare(got, {"o": ro, "lse": rl, "dq": rdq, "dk": rdk, "dv": rdv, "dalpha": rda, "l1": l1},
            dtype, f"pipeline {dtype} D{D} W{W}", lse_slack=slack)


ROPE_Q = [
    # (B, H, H_kv, T, D, dtype, W, alpha): bf16 with d_head 64 and W <= 16 rotates q inside
    # the forward (1, 2 or 4 query heads per workgroup, integer and interpolated offsets,
    # ragged tails, a single position, the window limit); the other shapes run the RoPE
    # launch on q, then the forward
    (2, 2, 2, 300, 64, "bf16", 8, 1.0),
    (1, 3, 3, 333, 64, "bf16", 8, 0.85),
    (1, 8, 2, 300, 64, "bf16", 12, 1.0),
    (1, 4, 2, 257, 64, "bf16", 16, 0.9),
    (1, 2, 2, 1, 64, "bf16", 0, 1.0),
    (1, 2, 2, 200, 64, "fp32", 8, 0.85),
    (1, 2, 1, 150, 128, "bf16", 8, 1.0),
    (1, 2, 2, 150, 64, "bf16", 20, 0.9),  # past the matrix-core window limit
]


@pytest.mark.parametrize("B,H,Hkv,T,D,dtype,W,alpha", ROPE_Q)
def test_forward_rotating_q_on_load(B, H, Hkv, T, D, dtype, W, alpha):
    # raw q and rotated k -> the forward that rotates q itself -> the backward with R^T
    # fused; the oracle runs the same chain on its own rotations, rounded to the storage
    # dtype (the lse bound allows for the rounding flips of a float32 rotation)
    idx = ROPE_Q.index((B, H, Hkv, T, D, dtype, W, alpha))
    print(f"rope-q case {idx}: B{B} H{H}/{Hkv} T{T} D{D} {dtype} W{W} alpha={alpha}", flush=True)
    x = _gqa_inputs(B, H, Hkv, T, D, dtype, 110 + idx)
    q = x["q"].cuda()
    K = F.fibattn_rope(x["k"].cuda(), 10000.0)
    V, G = x["v"].cuda(), x["dO"].cuda()
    o, lse, Q = F.fibattn_forward_rope_q(q, K, V, W, FIB, alpha, 10000.0)
    dq, dk, dv, da = F.fibattn_backward(Q, K, V, o, lse, G, W, FIB, alpha, rope_base=10000.0)
    torch.cuda.synchronize()
    eq, ek = oracle.rope(x["q"]), oracle.rope(x["k"])  # exact rotations
    rq, rk = (inputs.round_to(r.astype(np.float32), dtype).double().numpy() for r in (eq, ek))
    slack = rope_rounding_slack(x["q"].double().numpy(), x["k"].double().numpy(), eq, ek, dtype, W, FIB, alpha)
    if dtype == "fp32":
        np.testing.assert_allclose(Q.double().cpu().numpy(), rq, atol=1e-5, rtol=0)
    else:  # the oracle's rounding, or the other neighbour where a float32 rotation may flip it
        assert np.all(np.abs(Q.double().cpu().numpy() - rq) <= rope_flip_size(x["q"].double().numpy(), eq))
    ro, rl = oracle.forward(rq, rk, x["v"], W, FIB, alpha)
    rdq, rdk, rdv, rda, l1 = oracle.backward(rq, rk, x["v"], x["dO"], W, FIB, alpha)
    rdq, rdk = oracle.rope(rdq, transpose=True), oracle.rope(rdk, transpose=True)
    got = {"o": o, "lse": lse, "dq": dq, "dk": dk, "dv": dv}
    got = {kk: vv.double().cpu().numpy() for kk, vv in got.items()}
    got["dalpha"] = float(da.item())
    compare(got, {"o": ro, "lse": rl, "dq": rdq, "dk": rdk, "dv": rdv, "dalpha": rda, "l1": l1},
            dtype, f"rope-q case {idx}", lse_slack=slack)
    if dtype == "bf16" and D == 64 and W <= 16:
        # forward only (no q_out): the same kernel without the store, so the same bits;
        # and q_out may be q itself (each query row is read by its own wave only)
        o2, l2, none = F.fibattn_forward_rope_q(q, K, V, W, FIB, alpha, 10000.0, keep_q=False)
        q3 = q.clone()
        o3, l3, Q3 = F.fibattn_forward_rope_q(q3, K, V, W, FIB, alpha, 10000.0, q_out=q3)
        torch.cuda.synchronize()
        assert none is None and torch.equal(o2, o) and torch.equal(l2, lse)
        assert Q3.data_ptr() == q3.data_ptr() and torch.equal(q3, Q) and torch.equal(o3, o) and torch.equal(l3, lse)
    else:
        # outside the matrix-core kernels the rotated rows need a buffer: refused before
        # any launch
        with pytest.raises(F.FibattnError):
            F.fibattn_forward_rope_q(q, K, V, W, FIB, alpha, 10000.0, keep_q=False)


@pytest.mark.parametrize("name,ci", [("layer_60m_fixed_T1024", 0), ("extrap_coprime16_T4096", 1)])
def test_forward_rotating_q_on_load_full_size(name, ci):
    # forward only at the workload's shape: raw q, the keys rotated by the RoPE launch,
    # nothing written but o and lse
    wl = workloads.workload(name)
    call = wl.calls[ci]
    print(f"rope-q full size {name} call {ci}: alpha={float(call.alpha):.7f}", flush=True)
    x = workloads.layer_inputs(wl, ci, names=("q", "k", "v"))
    K = F.fibattn_rope(x["k"].cuda(), 10000.0)
    o, lse, _ = F.fibattn_forward_rope_q(x["q"].cuda(), K, x["v"].cuda(), call.W, call.base, call.alpha,
                                         10000.0, keep_q=False)
    torch.cuda.synchronize()
    eq, ek = oracle.rope(x["q"]), oracle.rope(x["k"])
    rq, rk = (inputs.round_to(r.astype(np.float32), wl.dtype).double().numpy() for r in (eq, ek))
    slack = rope_rounding_slack(x["q"].double().numpy(), x["k"].double().numpy(), eq, ek, wl.dtype, call.W,
                                call.base, call.alpha)
    ro, rl = oracle.forward(rq, rk, x["v"], call.W, call.base, call.alpha)
    print(compare({"o": o.double().cpu().numpy(), "lse": lse.double().cpu().numpy()}, {"o": ro, "lse": rl},
                  wl.dtype, f"rope-q full size {name}", lse_slack=slack), flush=True)


HEAD128 = [
    # (B, H, H_kv, T, D, dtype, W, base, alpha): d_head = 128 runs the generic kernels
    (1, 2, 2, 260, 128, "fp32", 8, FIB, 0.7310586),
    (2, 2, 1, 200, 128, "bf16", 8, FIB, 1.0),
    (1, 4, 4, 150, 128, "bf16", 12, POW2, 1.3),
]


@pytest.mark.parametrize("B,H,Hkv,T,D,dtype,W,base,alpha", HEAD128)
def test_head_dim_128_parity(B, H, Hkv, T, D, dtype, W, base, alpha):
    idx = HEAD128.index((B, H, Hkv, T, D, dtype, W, base, alpha))
    print(f"d_head 128 case {idx}: B{B} H{H}/{Hkv} T{T} {dtype} W{W} alpha={alpha}", flush=True)
    x = _gqa_inputs(B, H, Hkv, T, D, dtype, 70 + idx)
    got = gpu_run(x["q"], x["k"], x["v"], x["dO"], W, base, alpha)
    ref = oracle_run(x["q"], x["k"], x["v"], x["dO"], W, base, alpha)
    compare(got, ref, dtype, f"d_head 128 case {idx}")


def test_head_dim_128_rope_pipeline():
    x = inputs.attention_inputs(1, 2, 130, 128, "bf16", 77, 0)
    Q, K = F.fibattn_rope_qk(x["q"].cuda(), x["k"].cuda(), 10000.0)
    V, G = x["v"].cuda(), x["dO"].cuda()
    o, lse = F.fibattn_forward(Q, K, V, 8, FIB, 0.9)
    dq, dk, dv, da = F.fibattn_backward(Q, K, V, o, lse, G, 8, FIB, 0.9, rope_base=10000.0)
    torch.cuda.synchronize()
    eq, ek = oracle.rope(x["q"]), oracle.rope(x["k"])  # exact rotations
    rq, rk = (inputs.round_to(r.astype(np.float32), "bf16").double().numpy() for r in (eq, ek))
    slack = rope_rounding_slack(x["q"].double().numpy(), x["k"].double().numpy(), eq, ek, "bf16", 8, FIB, 0.9)
    ro, rl = oracle.forward(rq, rk, x["v"], 8, FIB, 0.9)
    rdq, rdk, rdv, rda, l1 = oracle.backward(rq, rk, x["v"], x["dO"], 8, FIB, 0.9)
    rdq, rdk = oracle.rope(rdq, transpose=True), oracle.rope(rdk, transpose=True)
    got = {kk: vv.double().cpu().numpy() for kk, vv in
           {"o": o, "lse": lse, "dq": dq, "dk": dk, "dv": dv}.items()}
    got["dalpha"] = float(da.item())
    compare(got, {"o": ro, "lse": rl, "dq": rdq, "dk": rdk, "dv": rdv, "dalpha": rda, "l1": l1},
            "bf16", "d_head 128 pipeline", lse_slack=slack)


GQA = [
    # (B, H, H_kv, T, D, dtype, W, base, alpha): grouped key/value heads.  bf16 d64
    # W<=16 runs the matrix-core kernels, whose dk/dv workgroup takes 4, 2 or 1 query
    # heads of a group side by side (G = 4, 8: four; G = 2: two; G = 3: one at a time)
    (2, 4, 2, 333, 32, "fp32", 8, FIB, 0.7310586),
    (1, 4, 1, 300, 64, "fp32", 6, FIB, 1.0),
    (2, 4, 2, 300, 64, "bf16", 8, FIB, 1.0),
    (1, 8, 2, 333, 64, "bf16", 8, FIB, 0.9),
    (1, 8, 1, 290, 64, "bf16", 10, POW2, 1.3),
    (1, 6, 2, 257, 64, "bf16", 8, FIB, 1.0),
    (1, 6, 2, 257, 64, "bf16", 12, FIB, 0.75),
    (1, 4, 2, 150, 64, "bf16", 20, FIB, 1.1),
    # several passes per group over 16 tiles: G = 8 (two passes of four), both offset
    # kinds, and G = 3 (three passes of one)
    (1, 8, 1, 1024, 64, "bf16", 8, FIB, 1.0),
    (1, 8, 1, 1024, 64, "bf16", 8, FIB, 0.9),
    (1, 9, 3, 1024, 64, "bf16", 8, FIB, 1.0),
]


def _gqa_inputs(B, H, Hkv, T, D, dtype, seed):
    x = inputs.attention_inputs(B, H, T, D, dtype, 300 + seed, 0, names=("q", "dO"))
    x.update(inputs.attention_inputs(B, Hkv, T, D, dtype, 300 + seed, 0, names=("k", "v")))
    return x


@pytest.mark.parametrize("B,H,Hkv,T,D,dtype,W,base,alpha", GQA)
def test_grouped_heads_parity(B, H, Hkv, T, D, dtype, W, base, alpha):
    idx = GQA.index((B, H, Hkv, T, D, dtype, W, base, alpha))
    print(f"gqa case {idx}: B{B} H{H} Hkv{Hkv} T{T} D{D} {dtype} W{W} alpha={alpha}", flush=True)
    x = _gqa_inputs(B, H, Hkv, T, D, dtype, idx)
    got = gpu_run(x["q"], x["k"], x["v"], x["dO"], W, base, alpha)
    ref = oracle_run(x["q"], x["k"], x["v"], x["dO"], W, base, alpha)
    assert got["dk"].shape == (B, Hkv, T, D)
    compare(got, ref, dtype, f"gqa case {idx}")


WS_CASES = [
    # (B, H, H_kv, T, W, base, alpha), bf16 d_head 64: the matrix-core backward, whose
    # dq kernel hands every rung entry's (tau dS, p) to dk/dv through the workspace
    (2, 4, 4, 300, 8, FIB, 1.0),     # integer offsets, ragged tail
    (1, 4, 4, 333, 8, FIB, 0.85),    # interpolated offsets
    (1, 8, 2, 257, 10, POW2, 1.2),   # four query heads per key/value head in a workgroup
    (1, 8, 1, 200, 8, FIB, 0.9),     # eight per key/value head: two passes
    (1, 6, 2, 190, 6, FIB, 1.0),     # three per key/value head: one at a time
]


@pytest.mark.parametrize("B,H,Hkv,T,W,base,alpha", WS_CASES)
def test_backward_ignores_workspace_contents(B, H, Hkv, T, W, base, alpha):
    # The workspace is filled with all-ones bytes (NaN as float32, float64 and as
    # bfloat16 pairs) before the call: a term the dk/dv kernel read without the dq
    # kernel having written it would make dk or dv NaN.
    idx = WS_CASES.index((B, H, Hkv, T, W, base, alpha))
    print(f"workspace case {idx}: B{B} H{H} Hkv{Hkv} T{T} W{W} alpha={alpha}", flush=True)
    x = _gqa_inputs(B, H, Hkv, T, 64, "bf16", 120 + idx)
    need = F.fibattn_backward_workspace_bytes(B, H, T, 64, W, len(base))
    ws = torch.full((need,), 0xFF, device="cuda", dtype=torch.uint8)
    got = gpu_run(x["q"], x["k"], x["v"], x["dO"], W, base, alpha, workspace=ws)
    ref = oracle_run(x["q"], x["k"], x["v"], x["dO"], W, base, alpha)
    compare(got, ref, "bf16", f"workspace case {idx}")


def test_workspace_reused_across_rung_tables():
    # one workspace, sized for the longer base, serves three backward calls whose rung
    # tables differ in length and distances (stale terms of an earlier call unused)
    B, H, T = 1, 4, 400
    ws = torch.empty(F.fibattn_backward_workspace_bytes(B, H, T, 64, 12, len(FIB)), device="cuda",
                     dtype=torch.uint8)
    for c, (W, base, alpha) in enumerate([(8, FIB, 1.3), (12, POW2, 0.9), (6, FIB[:9], 1.0)]):
        print(f"reuse call {c}: W{W} K{len(base)} alpha={alpha}", flush=True)
        x = _case_inputs(B, H, T, 64, "bf16", 60 + c)
        got = gpu_run(x["q"], x["k"], x["v"], x["dO"], W, base, alpha, workspace=ws)
        ref = oracle_run(x["q"], x["k"], x["v"], x["dO"], W, base, alpha)
        compare(got, ref, "bf16", f"reuse call {c}")


@pytest.mark.parametrize("alpha", [1.0, 0.7])
def test_grouped_heads_full_size(alpha):
    # the 60M model's layer with its 2 key/value heads: B = 8, H = 8, T = 1024
    print(f"gqa full size alpha={alpha}", flush=True)
    x = _gqa_inputs(8, 8, 2, 1024, 64, "bf16", 50 + int(alpha * 10))
    got = gpu_run(x["q"], x["k"], x["v"], x["dO"], 8, FIB, alpha)
    ref = oracle_run(x["q"], x["k"], x["v"], x["dO"], 8, FIB, alpha)
    compare(got, ref, "bf16", f"gqa full alpha {alpha}")


@pytest.mark.parametrize("dtype,D,W,alpha", [("bf16", 64, 8, 0.85), ("fp32", 32, 6, 1.0)])
def test_grouped_heads_pipeline_with_rope(dtype, D, W, alpha):
    # RoPE of q (4 heads) and k (2 heads), attention, backward with R^T fused: dk is
    # the group sum, rotated back
    B, H, Hkv, T = 1, 4, 2, 200
    x = _gqa_inputs(B, H, Hkv, T, D, dtype, 90 + D)
    Q = F.fibattn_rope(x["q"].cuda(), 10000.0)
    K = F.fibattn_rope(x["k"].cuda(), 10000.0)
    V, G = x["v"].cuda(), x["dO"].cuda()
    o, lse = F.fibattn_forward(Q, K, V, W, FIB, alpha)
    dq, dk, dv, da = F.fibattn_backward(Q, K, V, o, lse, G, W, FIB, alpha, rope_base=10000.0)
    torch.cuda.synchronize()
    eq, ek = oracle.rope(x["q"]), oracle.rope(x["k"])  # exact rotations
    rq, rk = (inputs.round_to(r.astype(np.float32), dtype).double().numpy() for r in (eq, ek))
    slack = rope_rounding_slack(x["q"].double().numpy(), x["k"].double().numpy(), eq, ek, dtype, W, FIB, alpha)
    ro, rl = oracle.forward(rq, rk, x["v"], W, FIB, alpha)
    rdq, rdk, rdv, rda, l1 = oracle.backward(rq, rk, x["v"], x["dO"], W, FIB, alpha)
    rdq, rdk = oracle.rope(rdq, transpose=True), oracle.rope(rdk, transpose=True)
    got = {"o": o, "lse": lse, "dq": dq, "dk": dk, "dv": dv}
    got = {kk: vv.double().cpu().numpy() for kk, vv in got.items()}
    got["dalpha"] = float(da.item())
    compare(got, {"o": ro, "lse": rl, "dq": rdq, "dk": rdk, "dv": rdv, "dalpha": rda, "l1": l1},
            dtype, f"gqa pipeline {dtype} D{D}", lse_slack=slack)


def test_rope_qk_matches_two_single_launches():
    x = _case_inputs(2, 3, 333, 64, "bf16", 52)
    q, k = x["q"].cuda(), x["k"].cuda()
    qa, ka = F.fibattn_rope_qk(q, k, 10000.0)
    assert torch.equal(qa, F.fibattn_rope(q, 10000.0)) and torch.equal(ka, F.fibattn_rope(k, 10000.0))


def test_deterministic_and_stream_independent():
    x = _case_inputs(2, 2, 500, 64, "bf16", 70)
    args = (x["q"], x["k"], x["v"], x["dO"], 10, FIB, 0.77)
    a = gpu_run(*args)
    b = gpu_run(*args)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        c = gpu_run(*args)
    for name in a:
        assert np.array_equal(a[name], b[name]), name
        assert np.array_equal(a[name], c[name]), name


# ---- general strides: q, k, v, o, dO, dq, dk, dv as views with contiguous rows ----

def _placed(x, how, slot=0):
    """A device view of x ([B,H,T,D], CPU) with the same values in placement `how`:
    "bthd" = a transposed [B,T,H,D] buffer; "qkv" = one slot of a [B,T,3,H,D] buffer
    (a fused projection output); "tslice" = the first T rows of each head of a NaN-filled
    [B,H,T+37,D] buffer (packed rows, larger head and batch strides); "packed" =
    contiguous."""
    B, H, T, D = x.shape
    if how == "packed":
        return x.cuda().contiguous()
    if how == "tslice":
        buf = torch.full((B, H, T + 37, D), float("nan"), dtype=x.dtype, device="cuda")
        buf[:, :, :T].copy_(x)
        return buf[:, :, :T]
    if how == "bthd":
        buf = torch.empty((B, T, H, D), dtype=x.dtype, device="cuda")
        buf.copy_(x.transpose(1, 2))
        return buf.transpose(1, 2)
    buf = torch.full((B, T, 3, H, D), float("nan"), dtype=x.dtype, device="cuda")
    buf[:, :, slot].copy_(x.transpose(1, 2))
    return buf[:, :, slot].transpose(1, 2)


STRIDED = [
    # (B, H, Hkv, T, D, dtype, W, alpha, placement of inputs, placement of outputs)
    (2, 4, 4, 300, 64, "bf16", 8, 1.0, "bthd", "packed"),     # matrix-core kernels, integer
    (2, 4, 4, 300, 64, "bf16", 8, 0.85, "qkv", "bthd"),       # interpolating, fused-qkv inputs
    (1, 8, 2, 257, 64, "bf16", 8, 1.0, "bthd", "bthd"),       # grouped heads
    (2, 3, 3, 200, 32, "fp32", 6, 0.7310586, "qkv", "bthd"),  # generic kernels
    (1, 4, 2, 130, 128, "bf16", 10, 1.2, "bthd", "qkv"),      # d_head 128, outputs in a qkv buffer
    # packed rows with non-packed head strides: the matrix-core kernels' strided instances
    (2, 4, 4, 300, 64, "bf16", 8, 1.0, "tslice", "tslice"),
    (1, 8, 2, 257, 64, "bf16", 8, 0.85, "tslice", "packed"),
    (2, 2, 2, 200, 64, "bf16", 12, 1.0, "packed", "tslice"),
]


@pytest.mark.parametrize("B,H,Hkv,T,D,dtype,W,alpha,pin,pout", STRIDED)
@pytest.mark.parametrize("rope_base", [0.0, 10000.0])
def test_strided_layouts(B, H, Hkv, T, D, dtype, W, alpha, pin, pout, rope_base):
    x = _gqa_inputs(B, H, Hkv, T, D, dtype, 61 + D)
    q, k, v, dO = (_placed(x[n], pin, s) for n, s in (("q", 0), ("k", 1), ("v", 2), ("dO", 0)))
    o = _placed(torch.zeros((B, H, T, D), dtype=x["q"].dtype), pout, 0)
    dq = _placed(torch.zeros((B, H, T, D), dtype=x["q"].dtype), pout, 0)
    dk = _placed(torch.zeros((B, Hkv, T, D), dtype=x["q"].dtype), pout, 1)
    dv = _placed(torch.zeros((B, Hkv, T, D), dtype=x["q"].dtype), pout, 2)
    assert not (q.is_contiguous() and o.is_contiguous())
    _, lse = F.fibattn_forward(q, k, v, W, FIB, alpha, o=o)
    _, _, _, da = F.fibattn_backward(q, k, v, o, lse, dO, W, FIB, alpha, dq=dq, dk=dk, dv=dv,
                                     rope_base=rope_base)
    torch.cuda.synchronize()
    ref = oracle_run(x["q"], x["k"], x["v"], x["dO"], W, FIB, alpha)
    if rope_base:
        ref["dq"] = oracle.rope(ref["dq"], rope_base, transpose=True)
        ref["dk"] = oracle.rope(ref["dk"], rope_base, transpose=True)
    got = {n_: t.double().cpu().numpy() for n_, t in (("o", o), ("lse", lse), ("dq", dq), ("dk", dk),
                                                       ("dv", dv))}
    got["dalpha"] = float(da.item())
    compare(got, ref, dtype, f"strided {pin}->{pout} B{B} H{H}/{Hkv} T{T} D{D} {dtype}")
    if pout == "qkv":
        # the outputs wrote only their own slot: the NaN fill of the other two survives
        for t, slot in ((o, 0), (dq, 0), (dk, 1), (dv, 2)):
            others = [s_ for s_ in range(3) if s_ != slot]
            assert torch.isnan(t._base[:, :, others].float()).all().item()
    if pout == "tslice":
        # nothing written past each head's T rows
        for t in (o, dq, dk, dv):
            assert torch.isnan(t._base[:, :, T:].float()).all().item()


ROPE_Q_STRIDED = [
    # (B, H, Hkv, T, D, dtype, W, alpha, placement of q, k, v, placement of o and q_out)
    (2, 4, 4, 300, 64, "bf16", 8, 1.0, "qkv", "bthd"),
    (1, 8, 2, 257, 64, "bf16", 12, 0.85, "tslice", "tslice"),
    (1, 4, 4, 200, 64, "bf16", 16, 1.0, "bthd", "packed"),
    (1, 2, 2, 200, 64, "fp32", 8, 0.85, "qkv", "bthd"),  # the RoPE launch, then the forward
    # the same past the matrix-core window, on 2^17+ rows of q: the RoPE launch of one
    # strided tensor with two positions per lane group, a ragged last position block
    (1, 33, 33, 3999, 64, "bf16", 20, 0.9, "bthd", "bthd"),
]


@pytest.mark.parametrize("B,H,Hkv,T,D,dtype,W,alpha,pin,pout", ROPE_Q_STRIDED)
def test_forward_rotating_q_on_load_strided(B, H, Hkv, T, D, dtype, W, alpha, pin, pout):
    # the same o, lse and R q bits as the packed call: placement changes addressing only
    x = _gqa_inputs(B, H, Hkv, T, D, dtype, 171 + D)
    K = F.fibattn_rope(x["k"].cuda(), 10000.0)
    q, k, v = _placed(x["q"], pin, 0), _placed(K.cpu(), pin, 1), _placed(x["v"], pin, 2)
    o = _placed(torch.zeros((B, H, T, D), dtype=x["q"].dtype), pout, 0)
    qo = _placed(torch.zeros((B, H, T, D), dtype=x["q"].dtype), pout, 1)
    assert not (q.is_contiguous() and o.is_contiguous())
    o1, l1, q1 = F.fibattn_forward_rope_q(q, k, v, W, FIB, alpha, 10000.0, o=o, q_out=qo)
    o2, l2, q2 = F.fibattn_forward_rope_q(x["q"].cuda(), K, x["v"].cuda(), W, FIB, alpha, 10000.0)
    torch.cuda.synchronize()
    assert o1.data_ptr() == o.data_ptr() and q1.data_ptr() == qo.data_ptr()
    assert torch.equal(o1, o2) and torch.equal(l1, l2) and torch.equal(q1, q2)
    if pout == "tslice":
        for t in (o1, q1):
            assert torch.isnan(t._base[:, :, T:].float()).all().item()
