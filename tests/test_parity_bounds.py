"""The parity bounds themselves (CPU): compare() must reject wrong results.

Negative controls at full size: the oracle's own results for whole workload layers,
with dalpha replaced by 0, by -dalpha_ref, or scaled past the bound, must fail the
bfloat16 check; a dalpha within 2e-2 of the reference must pass.  A per-tensor
mistake (one output row zeroed) must fail as well.
"""
import numpy as np
import pytest

from paper_2606_28560_amd import inputs, schedules, workloads
from tests.parity import compare, oracle_run


def _full_case(name):
    if name == "layer_60m":  # the 60M model's layer, alpha = 1
        wl = workloads.workload("layer_60m_fixed_T1024")
        c = wl.calls[0]
        x = workloads.layer_inputs(wl, 0)
        return x, c.W, c.base, c.alpha
    if name == "learned_pow2":  # B = 32, W = 10, power-of-2 base, alpha = 0.5 + sigmoid(theta)
        wl = workloads.workload("pow2_fib_learned16_T1024")
        c = wl.calls[0]
        x = workloads.layer_inputs(wl, 0)
        return x, c.W, c.base, c.alpha
    # B1 H8 T1024 with a stagger alpha (interpolated rungs): |dalpha| is ~1/1800 of the
    # L1 mass of its terms
    x = inputs.attention_inputs(1, 8, 1024, 64, "bf16", 7, 0)
    return x, 8, schedules.FIB15, float(schedules.alpha_linear_stagger()[5])


@pytest.fixture(scope="module", params=["layer_60m", "learned_pow2", "stagger_interp"])
def full_ref(request):
    x, W, base, alpha = _full_case(request.param)
    ref = oracle_run(x["q"], x["k"], x["v"], x["dO"], W, base, alpha)
    return request.param, ref


def _got(ref, dalpha):
    g = {n: ref[n].copy() for n in ("o", "lse", "dq", "dk", "dv")}
    g["dalpha"] = dalpha
    return g


def test_dalpha_bound_rejects_zero_and_sign_flip(full_ref):
    name, ref = full_ref
    da = ref["dalpha"]
    assert abs(da) > 1.0, f"{name}: dalpha_ref {da} too small to test a relative bound"
    for bad in (0.0, -da, 1.03 * da, 0.97 * da):
        with pytest.raises(AssertionError):
            compare(_got(ref, bad), ref, "bf16", name)
    compare(_got(ref, 1.015 * da), ref, "bf16", name)
    compare(_got(ref, da), ref, "bf16", name)


def test_float32_dalpha_bound_rejects_zero_and_sign_flip(full_ref):
    name, ref = full_ref
    da = ref["dalpha"]
    for bad in (0.0, -da):
        with pytest.raises(AssertionError):
            compare(_got(ref, bad), ref, "fp32", name)


def test_tensor_bounds_reject_a_missing_row(full_ref):
    name, ref = full_ref
    for t in ("o", "dq", "dk", "dv"):
        g = _got(ref, ref["dalpha"])
        flat = g[t].reshape(-1, g[t].shape[-1])
        r = int(np.argmax(np.abs(flat).max(axis=1)))  # the row holding the largest value
        flat[r] = 0.0
        with pytest.raises(AssertionError):
            compare(g, ref, "bf16", f"{name} {t}")
