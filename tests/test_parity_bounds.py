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


def _float32_rope(raw, base=10000.0):
    """The rotation a float32 kernel computes (float64-reduced angle, cos/sin rounded to
    float32, one fused multiply-add per output), before bfloat16 rounding: an emulation
    independent of rope_flip_size, to check that it flags every flip such a kernel can
    make."""
    a = np.asarray(raw, dtype=np.float64)
    B, H, T, D = a.shape
    half = D // 2
    ang = np.arange(T)[:, None] * base ** (-2.0 * np.arange(half) / D)[None, :]
    r = (ang - 2 * np.pi * np.rint(ang / (2 * np.pi))).astype(np.float32).astype(np.float64)
    c = np.cos(r).astype(np.float32).astype(np.float64)
    s = np.sin(r).astype(np.float32).astype(np.float64)
    u, v = a[..., :half], a[..., half:]
    x0 = (u * c - (v * s).astype(np.float32)).astype(np.float32)
    x1 = (v * c + (u * s).astype(np.float32)).astype(np.float32)
    return np.concatenate([x0, x1], axis=-1).astype(np.float64)


def test_rope_rounding_slack_covers_float32_rotation():
    # every element where a float32 rotation rounds to a different bfloat16 value than the
    # exact one is flagged, the lse of the flipped inputs stays within 1e-3 + slack, and
    # most queries keep the plain 1e-3 bound (slack only where a flagged element is read)
    import oracle
    from tests.parity import TOL_BF16_LSE, rope_flip_size, rope_rounding_slack

    x = inputs.attention_inputs(1, 4, 400, 64, "bf16", 412, 0)
    raw_q, raw_k = x["q"].double().numpy(), x["k"].double().numpy()
    eq, ek = oracle.rope(x["q"]), oracle.rope(x["k"])
    rq, rk = (inputs.round_to(r.astype(np.float32), "bf16").double().numpy() for r in (eq, ek))
    gq, gk = (inputs.round_to(_float32_rope(r).astype(np.float32), "bf16").double().numpy()
              for r in (raw_q, raw_k))
    assert (gq != rq).sum() + (gk != rk).sum() > 0  # the case exercises flips
    for g, r, raw, e in ((gq, rq, raw_q, eq), (gk, rk, raw_k, ek)):
        f = rope_flip_size(raw, e)
        assert np.all(f[g != r] > 0)
        assert np.all(np.abs(g - r) <= f + 1e-30)
    slack = rope_rounding_slack(raw_q, raw_k, eq, ek, "bf16", 8, schedules.FIB15, 1.0)
    _, l_ref = oracle.forward(rq, rk, x["v"], 8, schedules.FIB15, 1.0)
    _, l_flip = oracle.forward(gq, gk, x["v"], 8, schedules.FIB15, 1.0)
    assert np.all(np.abs(l_flip - l_ref) <= TOL_BF16_LSE + slack)
    assert np.median(slack) < 1e-4 and (slack > TOL_BF16_LSE).mean() < 0.1
