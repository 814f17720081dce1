"""The allocation-free backward (fibattn_backward_noalloc) against the workspace one.

Same kernels, so the outputs must be bitwise those of fibattn_backward_gqa on the same
inputs; three calls in a row on the library's one static scratch array, each smaller
than the one before (the later calls find the earlier calls' contents in it), over
the matrix-core and the generic kernels.  The smallest call is also checked against
the fp64 oracle.
"""
import pytest
import torch

from paper_2606_28560_amd import fibattn as F
from paper_2606_28560_amd import inputs, schedules
from tests.parity import compare, oracle_run

pytestmark = pytest.mark.gpu

CALLS = [
    # (B, H, H_kv, T, D, dtype, W, base, alpha, rope_base)
    (4, 8, 8, 1024, 64, "bf16", 8, schedules.FIB15, 0.9, 10000.0),
    (1, 4, 2, 333, 64, "bf16", 12, schedules.FIB15, 1.0, 0.0),
    (1, 2, 1, 200, 32, "fp32", 8, schedules.POW2_11, 0.7310586, 0.0),
]


def _inputs(B, H, Hkv, T, D, dtype, seed):
    x = inputs.attention_inputs(B, H, T, D, dtype, 300 + seed, 0, names=("q", "dO"))
    x.update(inputs.attention_inputs(B, Hkv, T, D, dtype, 300 + seed, 0, names=("k", "v")))
    return {n: t.cuda() for n, t in x.items()}


def _outputs(q, k):
    nan = float("nan")
    return (torch.full_like(q, nan), torch.full_like(k, nan), torch.full_like(k, nan),
            torch.full((1,), nan, device="cuda", dtype=torch.float32))


def test_noalloc_backward_matches_workspace_backward():
    for n, (B, H, Hkv, T, D, dtype, W, base, alpha, rope) in enumerate(CALLS):
        print(f"no-alloc call {n}: B{B} H{H}/{Hkv} T{T} D{D} {dtype} W{W} K{len(base)} "
              f"alpha={alpha} rope={rope}", flush=True)
        x = _inputs(B, H, Hkv, T, D, dtype, n)
        o, lse = F.fibattn_forward(x["q"], x["k"], x["v"], W, base, alpha)
        ws = torch.full((F.fibattn_backward_workspace_bytes(B, H, T, D, W, len(base)),), 255,
                        device="cuda", dtype=torch.uint8)
        ref = _outputs(x["q"], x["k"])
        F.fibattn_backward(x["q"], x["k"], x["v"], o, lse, x["dO"], W, base, alpha, dq=ref[0], dk=ref[1],
                           dv=ref[2], dalpha=ref[3], workspace=ws, rope_base=rope)
        got = _outputs(x["q"], x["k"])
        F.fibattn_backward_noalloc(x["q"], x["k"], x["v"], o, lse, x["dO"], W, base, alpha, dq=got[0],
                                   dk=got[1], dv=got[2], dalpha=got[3], rope_base=rope)
        torch.cuda.synchronize()
        for name, a, b in zip(("dq", "dk", "dv", "dalpha"), got, ref):
            assert torch.equal(a.view(torch.int16 if a.dtype == torch.bfloat16 else torch.int32),
                               b.view(torch.int16 if b.dtype == torch.bfloat16 else torch.int32)), \
                f"call {n}: {name} differs from the workspace backward"
        if n == len(CALLS) - 1:
            cpu = {k_: t.cpu() for k_, t in x.items()}
            r = oracle_run(cpu["q"], cpu["k"], cpu["v"], cpu["dO"], W, base, alpha)
            res = {"dq": got[0], "dk": got[1], "dv": got[2]}
            res = {k_: t.double().cpu().numpy() for k_, t in res.items()}
            res["dalpha"] = float(got[3].item())
            print(compare(res, r, dtype, f"no-alloc call {n}"), flush=True)


def test_noalloc_rejects_problems_beyond_the_scratch():
    # 32 x 8 heads at T = 16384, K = 15: ~270 MB of scratch > 64 MiB; refused before launch
    q = torch.empty((32, 8, 16384, 64), device="cuda", dtype=torch.bfloat16)
    lse = torch.empty((32, 8, 16384), device="cuda", dtype=torch.float32)
    da = torch.empty(1, device="cuda", dtype=torch.float32)
    assert F.fibattn_backward_workspace_bytes(32, 8, 16384, 64, 8, 15) > F.SCRATCH_BYTES
    with pytest.raises(F.FibattnError) as ei:
        F.fibattn_backward_noalloc(q, q, q, q, lse, q, 8, schedules.FIB15, 1.0, dq=q, dk=q, dv=q, dalpha=da)
    assert ei.value.status == 5
