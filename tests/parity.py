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
The oracle reads the very same rounded inputs, upcast to float64.
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


def compare(got, ref, dtype, label=""):
    """Asserts parity of every result present in `got`; returns the error report."""
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
            bound = TOL_BF16_LSE
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
