"""Helpers for GPU-vs-oracle parity tests.

Tolerances (written out here, used by every parity test):
  * float32 storage: max |x - x_ref| <= 1e-5 for o, lse, dq, dk, dv;
    |dalpha - ref| <= 1e-5 * max(1, A), A = sum |f_k dL/dw| (the L1 mass of the terms
    of dalpha: with |dalpha| ~ 1e3 the float32 ulp alone is ~1e-4, so an absolute
    1e-5 bound is unattainable for any float32 implementation);
  * bfloat16 storage with float32 arithmetic: max |x - x_ref| <= 2e-2 * max |x_ref|
    per tensor for o, dq, dk, dv; lse (a float32 output) within 1e-3 absolute;
    |dalpha - ref| <= 2e-2 * max(1, |ref|) (relative to dalpha itself: a zero or
    sign-flipped dalpha fails it).
The oracle reads the very same rounded inputs, upcast to float64.  Pipelines that rotate
q and k on the GPU (RoPE before the attention) add rope_rounding_slack to the bfloat16
lse bound: the rounding of a rotated element to bfloat16 is decided in float32 there and
in float64 here, so an element whose exact value lies within the float32 error of a
rounding midpoint may land on either neighbour.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2606_28560_amd import fibattn as F

TOL_FP32 = 1e-5
TOL_BF16_REL = 2e-2
TOL_BF16_LSE = 1e-3


def to_gpu(t):
    return t.to("cuda").contiguous()


def gpu_run(q, k, v, dO, W, base, alpha, backward=True, poison=True, workspace=None):
    """Runs the HIP path on CPU tensors; returns float64 numpy results.  `workspace`:
    the backward's workspace (a uint8 device tensor), else the binding allocates one."""
    Q, K, V = to_gpu(q), to_gpu(k), to_gpu(v)
    o = torch.empty_like(Q)
    lse = torch.empty(Q.shape[:3], device="cuda", dtype=torch.float32)
    if poison:
        o.fill_(float("nan")); lse.fill_(float("nan"))
    F.fibattn_forward(Q, K, V, W, base, alpha, o=o, lse=lse)
    out = {"o": o, "lse": lse}
    if backward:
        G = to_gpu(dO)
        dq, dk, dv = torch.empty_like(Q), torch.empty_like(K), torch.empty_like(V)
        da = torch.empty(1, device="cuda", dtype=torch.float32)
        if poison:
            for t in (dq, dk, dv, da):
                t.fill_(float("nan"))
        F.fibattn_backward(Q, K, V, o, lse, G, W, base, alpha, dq=dq, dk=dk, dv=dv, dalpha=da,
                           workspace=workspace)
        out.update(dq=dq, dk=dk, dv=dv, dalpha=da)
    torch.cuda.synchronize()
    res = {kk: vv.double().cpu().numpy() for kk, vv in out.items()}
    if "dalpha" in res:
        res["dalpha"] = float(res["dalpha"][0])
    return res


def oracle_run(q, k, v, dO, W, base, alpha, backward=True):
    o, lse = oracle.forward(q, k, v, W, base, alpha)
    res = {"o": o, "lse": lse}
    if backward:
        dq, dk, dv, da, l1 = oracle.backward(q, k, v, dO, W, base, alpha)
        res.update(dq=dq, dk=dk, dv=dv, dalpha=da, l1=l1)
    return res


def rope_flip_size(raw, exact):
    """Per element of a rotated tensor: the size of the bfloat16 rounding flip a float32
    rotation may cause (0 where both neighbours of the exact value's float32 error
    interval round alike); see rope_rounding_slack."""
    raw = np.abs(np.asarray(raw, dtype=np.float64))
    half = raw.shape[-1] // 2
    pair = raw[..., :half] + raw[..., half:]
    delta = 2.0 ** -20.5 * np.concatenate([pair, pair], axis=-1)
    lo = torch.from_numpy((exact - delta).astype(np.float32)).bfloat16().double().numpy()
    hi = torch.from_numpy((exact + delta).astype(np.float32)).bfloat16().double().numpy()
    return np.abs(hi - lo)


def rope_rounding_slack(raw_q, raw_k, rq, rk, dtype, W, base, alpha):
    """Extra lse tolerance per (b, h, i), natural-log units, for a bfloat16 pipeline whose
    rotated q, k were rounded on the GPU.  Everything here is oracle-side: raw_q, raw_k
    are the stored inputs, rq, rk the oracle's exact (unrounded) rotations, and the
    attended keys follow the oracle's rung table for (W, base, alpha).

    The GPU rotates in float32: the angle is reduced in float64 and rounded to float32
    (|angle| <= pi: error <= 2^-23), then sincosf (within 2 float32 ulps, 2^-23), so cos
    and sin are each within 2.4e-7 of the exact values; the two products and the sum add
    <= 2^-24 relative each.  Its unrounded value is thus within 3.6e-7 (|u| + |v|) =
    2^-21.4 (|u| + |v|) of the exact one (u, v: the pair's inputs); the bound used is
    twice that, 2^-20.5 (|u| + |v|).  An element whose exact value lies that
    close to a bfloat16 rounding midpoint may round either way; f is the size of that
    possible flip (0 elsewhere).  A logit s_ij = tau <q_i, k_j> then moves by at most
    tau sum_d (f_q |k| + |q| f_k + f_q f_k), and lse_i by at most the largest such move
    over the keys j it attends (lse is 1-Lipschitz in the max norm of the logits)."""
    if dtype != "bf16":
        return 0.0
    fq, fk = rope_flip_size(raw_q, rq), rope_flip_size(raw_k, rk)
    B, H, T, D = rq.shape
    G = H // rk.shape[1]
    tau = 1.0 / np.sqrt(D)
    # key offsets i - j a query may read: the window and each rung's rows r0 (and r1)
    offs = set(range(W + 1))
    for d0, w, _, _ in oracle.rungs(alpha, base, W):
        offs.add(d0)
        if w != 0.0:
            offs.add(d0 + 1)
    slack = np.zeros((B, H, T))
    aq, ak = np.abs(rq), np.abs(rk)
    for b in range(B):
        for h in range(H):
            kh = h // G
            # queries with a flip of their own, against the largest key element
            s = fq[b, h] @ (ak[b, kh] + fk[b, kh]).max(axis=0)
            # keys with a flip, against the queries that attend them
            for j in np.nonzero(fk[b, kh].any(axis=1))[0]:
                i = np.array(sorted(j + o for o in offs if j + o < T))
                s[i] += aq[b, h, i] @ fk[b, kh, j]
            slack[b, h] = tau * s
    return slack


def compare(got, ref, dtype, label="", lse_slack=0.0):
    """Asserts parity of every result present in `got`; returns the error report.
    lse_slack: extra bfloat16 lse tolerance per element (rope_rounding_slack)."""
    report = {}
    for name in ("o", "lse", "dq", "dk", "dv"):
        if name not in got:
            continue
        g, r = got[name], ref[name]
        assert np.all(np.isfinite(g)), f"{label} {name}: non-finite values (unwritten rows?)"
        err = float(np.max(np.abs(g - r))) if g.size else 0.0
        scale = float(np.max(np.abs(r))) if r.size else 0.0
        if dtype == "fp32":
            bound = TOL_FP32
        elif name == "lse":
            excess = np.abs(g - r) - (TOL_BF16_LSE + lse_slack)
            worst = np.unravel_index(np.argmax(excess), excess.shape) if g.size else ()
            bound = TOL_BF16_LSE + (float(np.broadcast_to(lse_slack, g.shape)[worst]) if g.size else 0.0)
            err = float(np.abs(g - r)[worst]) if g.size else 0.0
        else:
            bound = TOL_BF16_REL * scale
        report[name] = (err, bound)
        assert err <= bound, f"{label} {name}: max abs err {err:.3e} > bound {bound:.3e}"
    if "dalpha" in got:
        err = abs(got["dalpha"] - ref["dalpha"])
        if dtype == "fp32":
            bound = TOL_FP32 * max(1.0, ref["l1"])
        else:
            bound = TOL_BF16_REL * max(1.0, abs(ref["dalpha"]))
        report["dalpha"] = (err, bound)
        assert np.isfinite(got["dalpha"]), f"{label} dalpha not finite"
        assert err <= bound, f"{label} dalpha: {got['dalpha']} vs {ref['dalpha']} (err {err:.3e} > {bound:.3e})"
    return report
