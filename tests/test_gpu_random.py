"""GPU parity over seeded random configurations: the HIP path (through the C ABI)
against the fp64 oracle, forward and backward, at shapes drawn from the space the
library accepts rather than from the workloads: storage type, head size, grouped
heads, ragged lengths (T not a multiple of any tile), windows on both sides of the
matrix-core limit (W <= 16), the Fibonacci, power-of-2 and arbitrary increasing base
tables, integer and non-integer alpha.  Each case is fixed by its seed, so a failure
names a reproducible configuration."""
import numpy as np
import pytest

from paper_2606_28560_amd import inputs, schedules
from tests.parity import compare, gpu_run, oracle_run

pytestmark = pytest.mark.gpu

N_CASES = 64


def _config(seed):
    rng = np.random.default_rng(9000 + seed)
    dtype = "bf16" if rng.random() < 0.7 else "fp32"
    # bfloat16 with d_head 64 (the matrix-core kernels) is the common case
    D = 64 if (dtype == "bf16" and rng.random() < 0.75) else int(rng.choice([32, 64, 128]))
    H_kv = int(rng.choice([1, 2, 3, 4]))
    G = int(rng.choice([1, 1, 2, 3, 4]))
    H = H_kv * G
    B = int(rng.choice([1, 2]))
    T = int(rng.integers(1, 700))
    W = int(rng.choice([0, 1, 4, 8, 12, 15, 16, 17, 24])) if D != 128 else int(rng.integers(0, 17))
    kind = rng.random()
    if kind < 0.45:
        base = schedules.FIB15
    elif kind < 0.7:
        base = schedules.POW2_11
    else:
        K = int(rng.integers(1, 33))
        base = sorted(int(x) for x in rng.choice(np.arange(1, 1200), size=K, replace=False))
    alpha = 1.0 if rng.random() < 0.3 else float(np.float32(rng.uniform(0.3, 2.5)))
    return B, H, H_kv, T, D, dtype, W, base, alpha


@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_configuration(seed):
    B, H, H_kv, T, D, dtype, W, base, alpha = _config(seed)
    print(f"random case {seed}: B{B} H{H}/{H_kv} T{T} D{D} {dtype} W{W} K{len(base)} alpha={alpha}",
          flush=True)
    x = inputs.attention_inputs(B, H, T, D, dtype, 600 + seed, 0, names=("q", "dO"))
    x.update(inputs.attention_inputs(B, H_kv, T, D, dtype, 600 + seed, 0, names=("k", "v")))
    got = gpu_run(x["q"], x["k"], x["v"], x["dO"], W, base, alpha)
    ref = oracle_run(x["q"], x["k"], x["v"], x["dO"], W, base, alpha)
    compare(got, ref, dtype, f"random case {seed}")


@pytest.mark.parametrize("seed", range(16))
def test_random_step_with_q_rotated_on_load(seed):
    # the layer step's chain (RoPE of k, the forward rotating q, the backward with R^T)
    # at random matrix-core shapes; the oracle on its own rotations rounded to bfloat16
    import torch

    import oracle
    from paper_2606_28560_amd import fibattn as F
    from tests.parity import rope_flip_size, rope_rounding_slack

    rng = np.random.default_rng(9500 + seed)
    H_kv = int(rng.choice([1, 2, 4]))
    H = H_kv * int(rng.choice([1, 2, 3, 4]))
    B, T, W = int(rng.choice([1, 2])), int(rng.integers(1, 600)), int(rng.integers(0, 17))
    base = schedules.FIB15 if rng.random() < 0.6 else schedules.POW2_11
    alpha = 1.0 if rng.random() < 0.4 else float(np.float32(rng.uniform(0.4, 2.0)))
    print(f"random rope-q case {seed}: B{B} H{H}/{H_kv} T{T} W{W} K{len(base)} alpha={alpha}", flush=True)
    x = inputs.attention_inputs(B, H, T, 64, "bf16", 700 + seed, 0, names=("q", "dO"))
    x.update(inputs.attention_inputs(B, H_kv, T, 64, "bf16", 700 + seed, 0, names=("k", "v")))
    K = F.fibattn_rope(x["k"].cuda(), 10000.0)
    V, G = x["v"].cuda(), x["dO"].cuda()
    o, lse, Q = F.fibattn_forward_rope_q(x["q"].cuda(), K, V, W, base, alpha, 10000.0)
    dq, dk, dv, da = F.fibattn_backward(Q, K, V, o, lse, G, W, base, alpha, rope_base=10000.0)
    torch.cuda.synchronize()
    eq, ek = oracle.rope(x["q"]), oracle.rope(x["k"])
    rq, rk = (inputs.round_to(r.astype(np.float32), "bf16").double().numpy() for r in (eq, ek))
    assert np.all(np.abs(Q.double().cpu().numpy() - rq) <= rope_flip_size(x["q"].double().numpy(), eq))
    slack = rope_rounding_slack(x["q"].double().numpy(), x["k"].double().numpy(), eq, ek, "bf16", W, base, alpha)
    ro, rl = oracle.forward(rq, rk, x["v"], W, base, alpha)
    rdq, rdk, rdv, rda, l1 = oracle.backward(rq, rk, x["v"], x["dO"], W, base, alpha)
    rdq, rdk = oracle.rope(rdq, transpose=True), oracle.rope(rdk, transpose=True)
    got = {kk: vv.double().cpu().numpy() for kk, vv in {"o": o, "lse": lse, "dq": dq, "dk": dk, "dv": dv}.items()}
    got["dalpha"] = float(da.item())
    compare(got, {"o": ro, "lse": rl, "dq": rdq, "dk": rdk, "dv": rdv, "dalpha": rda, "l1": l1}, "bf16",
            f"random rope-q case {seed}", lse_slack=slack)
