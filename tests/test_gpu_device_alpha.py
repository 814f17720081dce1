"""GPU: the device-resident alpha path (rung table built on the device from a device
alpha, alpha = 0.5 + sigmoid(theta), dtheta), against the host table and the oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_28560_amd import fibattn as F
from paper_2606_28560_amd import inputs, schedules, workloads
from tests.parity import compare, oracle_run, rope_flip_size, rope_rounding_slack

pytestmark = pytest.mark.gpu

FIB = schedules.FIB15
POW2 = schedules.POW2_11


def _table_fields(buf):
    """(n, d0, w, f, W) of a device table read back (the library's layout: int n, int W,
    then int d0[32], float w[32], int f[32])."""
    raw = buf.cpu().numpy()
    n, W = (int(x) for x in raw[:8].view(np.int32))
    d0 = raw[8:136].view(np.int32)
    w = raw[136:264].view(np.float32)
    f = raw[264:392].view(np.int32)
    return n, d0, w, f, W


def _device_alphas():
    out = [np.float32(a) for a in (0.5, 0.7310586, 1.0, 1.2333333, 1.5, 0.01, 3.0)]
    out += list(schedules.alpha_linear_stagger(16)) + list(schedules.alpha_coprime_stagger(16))
    out += list(schedules.alpha_from_theta(inputs.thetas(16, case=5)))
    return out


@pytest.mark.parametrize("base,W", [(FIB, 8), (FIB, 6), (FIB, 12), (POW2, 10), ([3, 7, 11, 40], 2)])
def test_device_table_equals_host_table(base, W):
    alphas = _device_alphas()
    a_dev = torch.tensor(alphas, dtype=torch.float32, device="cuda")
    for idx, a in enumerate(alphas):
        buf = F.fibattn_device_table(a_dev[idx:idx + 1], base, W)
        torch.cuda.synchronize()
        n, d0, w, f, tw = _table_fields(buf)
        host = F.fibattn_rung_table(float(a), base, W)
        assert n == len(host), (float(a), n, len(host))
        assert tw == W
        for r, (hd0, hw, hf) in enumerate(host):
            assert (int(d0[r]), float(w[r]), int(f[r])) == (hd0, hw, hf), (float(a), r)


def _dev_run(x, W, base, alpha, rope=0.0, poison=True, table_W=None):
    Q, K, V, G = (x[n].cuda().contiguous() for n in ("q", "k", "v", "dO"))
    a_dev = torch.tensor([alpha], dtype=torch.float32, device="cuda")
    table = F.fibattn_device_table(a_dev, base, W if table_W is None else table_W)
    o = torch.empty_like(Q)
    lse = torch.empty(Q.shape[:3], device="cuda", dtype=torch.float32)
    dq, dk, dv = torch.empty_like(Q), torch.empty_like(K), torch.empty_like(V)
    da = torch.empty(1, device="cuda", dtype=torch.float32)
    if poison:
        for t in (o, lse, dq, dk, dv, da):
            t.fill_(float("nan"))
    F.fibattn_forward_dt(Q, K, V, W, table, o=o, lse=lse)
    F.fibattn_backward_dt(Q, K, V, o, lse, G, W, table, dq=dq, dk=dk, dv=dv, dalpha=da, rope_base=rope)
    torch.cuda.synchronize()
    res = {kk: vv.double().cpu().numpy() for kk, vv in
           {"o": o, "lse": lse, "dq": dq, "dk": dk, "dv": dv}.items()}
    res["dalpha"] = float(da.item())
    return res


DEV = [
    # (B, H, H_kv, T, D, dtype, W, base, alpha)
    (1, 2, 2, 300, 32, "fp32", 8, FIB, 0.7310586),
    (2, 2, 2, 257, 64, "fp32", 6, POW2, 1.0),
    (1, 3, 3, 333, 64, "bf16", 8, FIB, 1.0),
    (2, 2, 2, 300, 64, "bf16", 10, FIB, 1.2333333),
    (1, 8, 2, 290, 64, "bf16", 8, FIB, 0.9),
    (1, 2, 1, 200, 64, "bf16", 20, POW2, 0.8),
]


@pytest.mark.parametrize("B,H,Hkv,T,D,dtype,W,base,alpha", DEV)
def test_device_alpha_parity(B, H, Hkv, T, D, dtype, W, base, alpha):
    idx = DEV.index((B, H, Hkv, T, D, dtype, W, base, alpha))
    print(f"device alpha case {idx}: B{B} H{H}/{Hkv} T{T} D{D} {dtype} W{W} alpha={alpha}", flush=True)
    x = inputs.attention_inputs(B, H, T, D, dtype, 400 + idx, 0, names=("q", "dO"))
    x.update(inputs.attention_inputs(B, Hkv, T, D, dtype, 400 + idx, 0, names=("k", "v")))
    got = _dev_run(x, W, base, alpha)
    ref = oracle_run(x["q"], x["k"], x["v"], x["dO"], W, base, alpha)
    compare(got, ref, dtype, f"device alpha case {idx}")


@pytest.mark.parametrize("alpha", [float("nan"), 0.0, -1.0, float("inf")])
def test_invalid_device_alpha_gives_nan(alpha):
    x = inputs.attention_inputs(1, 2, 100, 64, "bf16", 450, 0)
    got = _dev_run(x, 8, FIB, alpha, poison=False)
    for name in ("o", "lse", "dq", "dk", "dv"):
        assert np.all(np.isnan(got[name])), name
    assert np.isnan(got["dalpha"])


@pytest.mark.parametrize("dtype,D,table_W,W", [("bf16", 64, 8, 12), ("bf16", 64, 20, 17),
                                               ("fp32", 32, 8, 6)])
def test_table_used_with_another_window_gives_nan(dtype, D, table_W, W):
    # a table records its W: with another W its in-window rule would have dropped or
    # kept the wrong rungs, so every output is NaN (matrix-core and generic kernels)
    x = inputs.attention_inputs(1, 2, 150, D, dtype, 451, 0)
    got = _dev_run(x, W, FIB, 0.9, poison=False, table_W=table_W)
    for name in ("o", "lse", "dq", "dk", "dv"):
        assert np.all(np.isnan(got[name])), name
    assert np.isnan(got["dalpha"])


def test_alpha_from_theta_and_dtheta():
    theta = inputs.thetas(64, case=7).astype(np.float32)
    t_dev = torch.tensor(theta, device="cuda")
    a = F.fibattn_alpha_from_theta(t_dev).cpu().numpy()
    ref = (0.5 + 1.0 / (1.0 + np.exp(-theta.astype(np.float64))))
    assert np.array_equal(a, ref.astype(np.float32))  # float64 sigmoid, one rounding
    da = torch.linspace(-3.0, 5.0, 64, device="cuda", dtype=torch.float32)
    dt = F.fibattn_dtheta(t_dev, da).cpu().numpy()
    sg = 1.0 / (1.0 + np.exp(-theta.astype(np.float64)))
    np.testing.assert_allclose(dt, da.cpu().numpy() * sg * (1 - sg), rtol=1e-6, atol=1e-7)


@pytest.mark.parametrize("base,W", [(FIB, 8), (POW2, 10), (FIB, 20)])
def test_table_from_theta_equals_table_from_alpha(base, W):
    theta = torch.tensor(inputs.thetas(16, case=5).astype(np.float32), device="cuda")
    for l in range(16):
        a_ref = F.fibattn_alpha_from_theta(theta[l:l + 1])
        t_ref = F.fibattn_device_table(a_ref, base, W)
        a = torch.full((1,), float("nan"), device="cuda")
        t = F.fibattn_device_table_theta(theta[l:l + 1], base, W, alpha=a)
        torch.cuda.synchronize()
        assert torch.equal(a, a_ref)
        # the same table (n, W, d0, w, f); only the theta table records d alpha / d theta
        assert torch.equal(t[:392], t_ref[:392])
        sg = 1.0 / (1.0 + np.exp(-float(theta[l].item())))
        assert t[392:400].cpu().numpy().view(np.float64)[0] == sg * (1.0 - sg)
        assert np.isnan(t_ref[392:400].cpu().numpy().view(np.float64)[0])


@pytest.mark.parametrize("dtype,D,W", [("bf16", 64, 8), ("fp32", 32, 8), ("bf16", 64, 20)])
def test_backward_dtheta_equals_separate_dtheta(dtype, D, W):
    # dtheta written by the backward (matrix-core and generic kernels) is bitwise the
    # value fibattn_dtheta computes from the stored dalpha; a table built from alpha
    # gives NaN
    x = inputs.attention_inputs(1, 4, 200, D, dtype, 452, 0)
    Q, K, V, G = (x[n].cuda() for n in ("q", "k", "v", "dO"))
    theta = torch.tensor([0.37], device="cuda")
    table = F.fibattn_device_table_theta(theta, FIB, W)
    o, lse = F.fibattn_forward_dt(Q, K, V, W, table)
    da, dth = torch.empty(1, device="cuda"), torch.full((1,), float("nan"), device="cuda")
    F.fibattn_backward_dt(Q, K, V, o, lse, G, W, table, dalpha=da, dtheta=dth)
    ref = F.fibattn_dtheta(theta, da)
    torch.cuda.synchronize()
    assert np.isfinite(float(dth.item())) and torch.equal(dth, ref)
    table_a = F.fibattn_device_table(F.fibattn_alpha_from_theta(theta), FIB, W)
    F.fibattn_backward_dt(Q, K, V, o, lse, G, W, table_a, dalpha=da, dtheta=dth)
    torch.cuda.synchronize()
    assert np.isnan(float(dth.item()))


@pytest.mark.parametrize("dtype,D,H,Hkv", [("bf16", 64, 8, 2), ("bf16", 64, 4, 4), ("fp32", 32, 6, 3)])
def test_rope_qk_table_equals_separate_launches(dtype, D, H, Hkv):
    # RoPE of q and of k with fewer heads, and the table from theta, in one launch: the
    # same bits as fibattn_rope on each tensor and fibattn_device_table_theta
    x = inputs.attention_inputs(2, H, 300, D, dtype, 453, 0, names=("q",))
    x.update(inputs.attention_inputs(2, Hkv, 300, D, dtype, 453, 0, names=("k",)))
    q, k = x["q"].cuda(), x["k"].cuda()
    theta = torch.tensor([-0.42], device="cuda")
    alpha = torch.full((1,), float("nan"), device="cuda")
    qo, ko, table = F.fibattn_rope_qk_table(q, k, 10000.0, theta=theta, base=FIB, W=8, alpha=alpha)
    rq, rk = F.fibattn_rope(q, 10000.0), F.fibattn_rope(k, 10000.0)
    ta = torch.full((1,), float("nan"), device="cuda")
    tref = F.fibattn_device_table_theta(theta, FIB, 8, alpha=ta)
    torch.cuda.synchronize()
    assert torch.equal(qo, rq) and torch.equal(ko, rk)
    assert torch.equal(table[:400], tref[:400]) and torch.equal(alpha, ta)
    # without theta: RoPE only, the table untouched
    t2 = torch.full_like(table, 7)
    qo2, ko2, _ = F.fibattn_rope_qk_table(q, k, 10000.0, table=t2)
    torch.cuda.synchronize()
    assert torch.equal(qo2, rq) and torch.equal(ko2, rk) and bool((t2 == 7).all())
    # k alone, the table job on that launch
    a3 = torch.full((1,), float("nan"), device="cuda")
    qo3, ko3, t3 = F.fibattn_rope_qk_table(None, k, 10000.0, theta=theta, base=FIB, W=8, alpha=a3)
    torch.cuda.synchronize()
    assert qo3 is None and torch.equal(ko3, rk)
    assert torch.equal(t3[:400], tref[:400]) and torch.equal(a3, ta)


DEV_ROPE_Q = [
    # (B, H, H_kv, T, W, alpha): the forward rotating q on load with a device table
    (1, 8, 2, 300, 8, 0.9),
    (2, 2, 2, 257, 16, 1.0),
    (1, 3, 3, 1, 0, 1.2333333),
]


@pytest.mark.parametrize("B,H,Hkv,T,W,alpha", DEV_ROPE_Q)
def test_device_alpha_rotating_q_on_load(B, H, Hkv, T, W, alpha):
    # device alpha -> table; RoPE of k; forward rotating q with the device table;
    # backward with R^T: the oracle runs the same chain on its own rounded rotations
    idx = DEV_ROPE_Q.index((B, H, Hkv, T, W, alpha))
    print(f"device alpha rope-q case {idx}: B{B} H{H}/{Hkv} T{T} W{W} alpha={alpha}", flush=True)
    x = inputs.attention_inputs(B, H, T, 64, "bf16", 470 + idx, 0, names=("q", "dO"))
    x.update(inputs.attention_inputs(B, Hkv, T, 64, "bf16", 470 + idx, 0, names=("k", "v")))
    q, V, G = x["q"].cuda(), x["v"].cuda(), x["dO"].cuda()
    table = F.fibattn_device_table(torch.tensor([alpha], dtype=torch.float32, device="cuda"), FIB, W)
    K = F.fibattn_rope(x["k"].cuda(), 10000.0)
    o, lse, Q = F.fibattn_forward_rope_q_dt(q, K, V, W, table, 10000.0)
    o2, l2, none = F.fibattn_forward_rope_q_dt(q, K, V, W, table, 10000.0, keep_q=False)
    ws = torch.empty(F.fibattn_backward_workspace_bytes(B, H, T, 64, W, 0), device="cuda", dtype=torch.uint8)
    dq, dk, dv, da = F.fibattn_backward_dt(Q, K, V, o, lse, G, W, table, workspace=ws, rope_base=10000.0)
    torch.cuda.synchronize()
    assert none is None and torch.equal(o2, o) and torch.equal(l2, lse)
    eq, ek = oracle.rope(x["q"]), oracle.rope(x["k"])
    rq, rk = (inputs.round_to(r.astype(np.float32), "bf16").double().numpy() for r in (eq, ek))
    assert np.all(np.abs(Q.double().cpu().numpy() - rq) <= rope_flip_size(x["q"].double().numpy(), eq))
    slack = rope_rounding_slack(x["q"].double().numpy(), x["k"].double().numpy(), eq, ek, "bf16", W, FIB, alpha)
    ro, rl = oracle.forward(rq, rk, x["v"], W, FIB, alpha)
    rdq, rdk, rdv, rda, l1 = oracle.backward(rq, rk, x["v"], x["dO"], W, FIB, alpha)
    rdq, rdk = oracle.rope(rdq, transpose=True), oracle.rope(rdk, transpose=True)
    got = {kk: vv.double().cpu().numpy() for kk, vv in {"o": o, "lse": lse, "dq": dq, "dk": dk, "dv": dv}.items()}
    got["dalpha"] = float(da.item())
    compare(got, {"o": ro, "lse": rl, "dq": rdq, "dk": rdk, "dv": rdv, "dalpha": rda, "l1": l1}, "bf16",
            f"device alpha rope-q case {idx}", lse_slack=slack)


@pytest.mark.parametrize("on_load", [False, True])
def test_learned_alpha_step_in_a_graph(on_load):
    # theta (device) -> alpha -> rung table -> RoPE -> forward -> backward -> dtheta,
    # captured once and replayed with theta changed in place between replays: every
    # replay follows the new theta with no host involvement.  on_load: the prologue
    # rotates k alone and the forward rotates q where it loads it
    wl = workloads.workload("pow2_fib_learned16_T1024")
    B, H, T, D, W = 2, 4, 256, 64, 10
    x = inputs.attention_inputs(B, H, T, D, "bf16", 460, 0)
    q, k, v, dO = (x[n].cuda() for n in ("q", "k", "v", "dO"))
    theta = torch.tensor([0.3], device="cuda", dtype=torch.float32)
    alpha = torch.empty_like(theta)
    table = torch.empty(F.lib().fibattn_device_table_bytes(), device="cuda", dtype=torch.uint8)
    qr, kr, o = torch.empty_like(q), torch.empty_like(k), torch.empty_like(q)
    lse = torch.empty((B, H, T), device="cuda", dtype=torch.float32)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    da, dth = torch.empty(1, device="cuda"), torch.empty(1, device="cuda")
    ws = torch.empty(F.fibattn_backward_workspace_bytes(B, H, T, D, W, 0), device="cuda", dtype=torch.uint8)
    base = wl.calls[0].base

    def step():  # RoPE, theta -> alpha and table in one launch; dtheta from the backward
        if on_load:
            F.fibattn_rope_qk_table(None, k, 10000.0, theta=theta, base=base, W=W, table=table, alpha=alpha,
                                    k_out=kr)
            F.fibattn_forward_rope_q_dt(q, kr, v, W, table, 10000.0, o=o, lse=lse, q_out=qr)
        else:
            F.fibattn_rope_qk_table(q, k, 10000.0, theta=theta, base=base, W=W, table=table, alpha=alpha,
                                    q_out=qr, k_out=kr)
            F.fibattn_forward_dt(qr, kr, v, W, table, o=o, lse=lse)
        F.fibattn_backward_dt(qr, kr, v, o, lse, dO, W, table, dq=dq, dk=dk, dv=dv, dalpha=da,
                              dtheta=dth, workspace=ws, rope_base=10000.0)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()  # warm-up outside capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    eq, ek = oracle.rope(x["q"]), oracle.rope(x["k"])  # exact rotations
    rq, rk = (inputs.round_to(r.astype(np.float32), "bf16").double().numpy() for r in (eq, ek))
    for rep, th in enumerate((0.3, -0.8, 1.7)):
        theta.fill_(th)
        g.replay()
        torch.cuda.synchronize()
        a = float(alpha.item())
        assert a == float(schedules.alpha_from_theta(np.float32(th)))
        slack = rope_rounding_slack(x["q"].double().numpy(), x["k"].double().numpy(), eq, ek, "bf16", W, base, a)
        ro, rl = oracle.forward(rq, rk, x["v"], W, base, a)
        rdq, rdk, rdv, rda, l1 = oracle.backward(rq, rk, x["v"], x["dO"], W, base, a)
        rdq, rdk = oracle.rope(rdq, transpose=True), oracle.rope(rdk, transpose=True)
        got = {kk: vv.double().cpu().numpy() for kk, vv in
               {"o": o, "lse": lse, "dq": dq, "dk": dk, "dv": dv}.items()}
        got["dalpha"] = float(da.item())
        compare(got, {"o": ro, "lse": rl, "dq": rdq, "dk": rdk, "dv": rdv, "dalpha": rda, "l1": l1},
                "bf16", f"graph replay {rep}", lse_slack=slack)
        sg = 1.0 / (1.0 + np.exp(-float(np.float32(th))))
        assert abs(float(dth.item()) - got["dalpha"] * sg * (1 - sg)) <= 1e-5 * max(1.0, abs(got["dalpha"]))
        # against the oracle: the chain rule through alpha = 0.5 + sigmoid(theta)
        assert abs(float(dth.item()) - rda * sg * (1 - sg)) <= 2e-2 * max(1.0, abs(rda * sg * (1 - sg)))
