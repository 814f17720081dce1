"""Pins of the fp64 CPU oracle against facts that do not come from the oracle itself.

Each test checks the oracle (oracle/) against one of:
  * a brute-force construction on tiny inputs (explicit per-query lists of row-weight
    vectors at continuous positions i - d, then textbook softmax attention);
  * a dense formulation with interpolation matrices, differentiated by torch autograd
    (an independent derivation of dq, dk, dv and dalpha);
  * a library routine where the method reduces to one (torch SDPA with a boolean mask
    at integer alpha, Section 2 "Implementation note"; sliding-window and full causal
    attention when there are no rungs);
  * closed forms (q = 0 gives a uniform softmax), hand-worked examples and the paper's
    printed distance count (tests/golden/), finite differences, and invariants.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2606_28560_amd import schedules

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
FIB = list(schedules.FIB15)
POW2 = list(schedules.POW2_11)


def rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


# ---------------------------------------------------------------------------
# independent constructions used as pins
# ---------------------------------------------------------------------------

def fl32_distances(alpha, base):
    """Rung distances as float32 products, as Python floats."""
    a = np.float32(alpha)
    return [float(a * np.float32(f)) for f in base]


def brute_force(q, k, v, W, base, alpha):
    """Attention over explicit per-query lists of virtual keys.

    Each attended item is a weight vector over the T rows: a window distance is a
    one-hot at i - delta; a rung distance d is the linear interpolation at the
    continuous position p = i - d between rows floor(p) and floor(p) + 1.  Rungs whose
    distance lies within [0, W] are already in the window (the set is a union), and
    rungs with d > i reach before position 0."""
    B, H, T, D = q.shape
    tau = 1.0 / math.sqrt(D)
    ds = sorted(set(d for d in fl32_distances(alpha, base) if d > W))
    o = np.zeros_like(q)
    lse = np.zeros((B, H, T))
    for b in range(B):
        for h in range(H):
            for i in range(T):
                items = []
                for delta in range(W + 1):
                    if i - delta >= 0:
                        e = np.zeros(T); e[i - delta] = 1.0; items.append(e)
                for d in ds:
                    if d <= i:
                        p = i - d
                        lo = math.floor(p); fr = p - lo
                        e = np.zeros(T)
                        e[lo] += 1.0 - fr
                        if fr > 0:
                            e[lo + 1] += fr
                        items.append(e)
                E = np.array(items)
                s = tau * (E @ k[b, h]) @ q[b, h, i]
                m = s.max()
                lse[b, h, i] = m + math.log(np.exp(s - m).sum())
                pr = np.exp(s - lse[b, h, i])
                o[b, h, i] = pr @ (E @ v[b, h])
    return o, lse


def dense_autograd(q, k, v, dO, W, base, alpha):
    """Forward as one softmax over T window columns plus one column per rung, where the
    rung's key and value are (1 - w) S0 K + w S1 K with constant shift matrices S0, S1
    (S1 has no entry for row -1: zero padding).  w = w32 + (a - alpha) * f so that
    autograd sees dw/da = f while the value is the float32 fraction.  Each rung's weight
    also carries a zero per-query offset leaf, whose gradient is the per-entry
    dL/dw; the L1 mass sum |f dL/dw| is summed from those.  Returns
    (o, lse, dq, dk, dv, dalpha, l1)."""
    B, H, T, D = q.shape
    tau = 1.0 / math.sqrt(D)
    Q = torch.tensor(q, dtype=torch.float64, requires_grad=True)
    Kleaf = torch.tensor(k, dtype=torch.float64, requires_grad=True)
    Vleaf = torch.tensor(v, dtype=torch.float64, requires_grad=True)
    # grouped heads: each key/value head serves H / Hkv consecutive query heads
    Kt = Kleaf.repeat_interleave(H // k.shape[1], dim=1)
    V = Vleaf.repeat_interleave(H // k.shape[1], dim=1)
    a = torch.tensor(float(np.float32(alpha)), dtype=torch.float64, requires_grad=True)
    rungs = []
    seen = set()
    for f, d in zip(base, fl32_distances(alpha, base)):
        if d > W and d not in seen:
            seen.add(d)
            rungs.append((f, d))
    idx = torch.arange(T)
    rel = idx[:, None] - idx[None, :]
    band = (rel >= 0) & (rel <= W)
    S = tau * Q @ Kt.transpose(-1, -2)
    S = S.masked_fill(~band, float("-inf"))
    cols = [S]
    vals = []
    offs = []  # per-(b, h, query) weight offsets, one leaf per rung
    for f, d in rungs:
        d0 = math.floor(d)
        w32 = d - d0
        wq = torch.zeros((B, H, T, 1), dtype=torch.float64, requires_grad=True)
        offs.append((f, wq))
        w = w32 + (a - float(np.float32(alpha))) * f + wq
        S0 = (rel == d0).to(torch.float64)
        S1 = (rel == d0 + 1).to(torch.float64)
        K0, K1 = S0 @ Kt, S1 @ Kt
        V0, V1 = S0 @ V, S1 @ V
        Kk = (1 - w) * K0 + w * K1
        Vk = (1 - w) * V0 + w * V1
        logit = tau * (Q * Kk).sum(-1, keepdim=True)
        incl = torch.tensor([d <= i for i in range(T)])[:, None]
        logit = logit.masked_fill(~incl, float("-inf"))
        cols.append(logit)
        vals.append(Vk)
    Z = torch.cat(cols, dim=-1)
    lse = torch.logsumexp(Z, dim=-1)
    P = torch.exp(Z - lse[..., None])
    o = P[..., :T] @ V
    for j, Vk in enumerate(vals):
        o = o + P[..., T + j:T + j + 1] * Vk
    L = (o * torch.tensor(dO)).sum()
    L.backward()
    l1 = sum(float((f * wq.grad).abs().sum()) for f, wq in offs)
    return (o.detach().numpy(), lse.detach().numpy(), Q.grad.numpy(), Kleaf.grad.numpy(),
            Vleaf.grad.numpy(), float(a.grad), l1)


# ---------------------------------------------------------------------------
# P1 brute force, P2 autograd
# ---------------------------------------------------------------------------

CASES = [
    # (T, D, W, base, alpha)
    (24, 4, 2, FIB[:8], 1.0),
    (24, 4, 3, FIB[:8], 0.7310586),
    (32, 8, 0, FIB[:9], 1.5),
    (32, 8, 5, POW2[:6], 0.5),
    (30, 4, 1, POW2[:5], 1.2),
    (20, 2, 4, [3, 7, 11], 1.37),
    (17, 4, 16, FIB[:7], 0.9),     # window covers everything but the far rungs
    (16, 4, 2, FIB[:7], 0.0625 * 16),
]


@pytest.mark.parametrize("T,D,W,base,alpha", CASES)
def test_forward_matches_brute_force(T, D, W, base, alpha):
    q, k, v = rand((1, 2, T, D), 1), rand((1, 2, T, D), 2), rand((1, 2, T, D), 3)
    o, lse = oracle.forward(q, k, v, W, base, alpha)
    ob, lb = brute_force(q, k, v, W, base, alpha)
    np.testing.assert_allclose(o, ob, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, lb, rtol=0, atol=1e-12)


@pytest.mark.parametrize("T,D,W,base,alpha", CASES)
def test_forward_backward_match_autograd(T, D, W, base, alpha):
    q, k, v, dO = (rand((2, 1, T, D), s) for s in (11, 12, 13, 14))
    o, lse = oracle.forward(q, k, v, W, base, alpha)
    dq, dk, dv, da, l1 = oracle.backward(q, k, v, dO, W, base, alpha)
    oa, la, dqa, dka, dva, daa, l1a = dense_autograd(q, k, v, dO, W, base, alpha)
    np.testing.assert_allclose(o, oa, atol=1e-12)
    np.testing.assert_allclose(lse, la, atol=1e-12)
    np.testing.assert_allclose(dq, dqa, atol=1e-11)
    np.testing.assert_allclose(dk, dka, atol=1e-11)
    np.testing.assert_allclose(dv, dva, atol=1e-11)
    assert abs(da - daa) <= 1e-10 * max(1.0, l1)
    # the L1 mass that scales the float32 dalpha tolerance, from autograd's per-entry
    # gradients (zero when no rung is included anywhere)
    assert abs(l1 - l1a) <= 1e-10 * max(1.0, l1a)


@pytest.mark.parametrize("Hkv,case", [(1, 1), (2, 3), (2, 5)])
def test_grouped_heads_match_autograd(Hkv, case):
    # k, v with fewer heads, read by groups of query heads; autograd sums the group's
    # gradients into the shared dk, dv through repeat_interleave
    T, D, W, base, alpha = CASES[case]
    q, dO = rand((2, 4, T, D), 21), rand((2, 4, T, D), 24)
    k, v = rand((2, Hkv, T, D), 22), rand((2, Hkv, T, D), 23)
    o, lse = oracle.forward(q, k, v, W, base, alpha)
    dq, dk, dv, da, l1 = oracle.backward(q, k, v, dO, W, base, alpha)
    oa, la, dqa, dka, dva, daa, l1a = dense_autograd(q, k, v, dO, W, base, alpha)
    assert dk.shape == k.shape and dv.shape == v.shape
    np.testing.assert_allclose(o, oa, atol=1e-12)
    np.testing.assert_allclose(lse, la, atol=1e-12)
    np.testing.assert_allclose(dq, dqa, atol=1e-11)
    np.testing.assert_allclose(dk, dka, atol=1e-11)
    np.testing.assert_allclose(dv, dva, atol=1e-11)
    assert abs(da - daa) <= 1e-10 * max(1.0, l1)
    assert abs(l1 - l1a) <= 1e-10 * max(1.0, l1a)


def test_grouped_heads_equal_repeated_heads():
    # sharing a key/value head is the same as giving each query head its own copy,
    # with dk, dv summed over the copies
    T, D, W, base, alpha, G = 40, 8, 4, FIB[:9], 0.83, 3
    q, dO = rand((2, 6, T, D), 31), rand((2, 6, T, D), 34)
    k, v = rand((2, 2, T, D), 32), rand((2, 2, T, D), 33)
    kr, vr = np.repeat(k, G, axis=1), np.repeat(v, G, axis=1)
    o, lse = oracle.forward(q, k, v, W, base, alpha)
    orr, lr = oracle.forward(q, kr, vr, W, base, alpha)
    np.testing.assert_allclose(o, orr, rtol=0, atol=1e-14)
    np.testing.assert_allclose(lse, lr, rtol=0, atol=1e-14)
    dq, dk, dv, da, l1 = oracle.backward(q, k, v, dO, W, base, alpha)
    dqr, dkr, dvr, dar, l1r = oracle.backward(q, kr, vr, dO, W, base, alpha)
    np.testing.assert_allclose(dq, dqr, rtol=0, atol=1e-14)
    np.testing.assert_allclose(dk, dkr.reshape(2, 2, G, T, D).sum(2), rtol=0, atol=1e-12)
    np.testing.assert_allclose(dv, dvr.reshape(2, 2, G, T, D).sum(2), rtol=0, atol=1e-12)
    assert abs(da - dar) <= 1e-12 * max(1.0, l1) and abs(l1 - l1r) <= 1e-12 * l1


# ---------------------------------------------------------------------------
# P3 integer alpha == boolean-mask attention (library SDPA)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("W,base", [(8, FIB), (6, FIB), (8, POW2), (0, FIB)])
def test_integer_alpha_equals_boolean_mask_sdpa(W, base):
    T, D = 96, 8
    q, k, v = (rand((2, 2, T, D), s) for s in (21, 22, 23))
    o, lse = oracle.forward(q, k, v, W, base, 1.0)
    i = np.arange(T)[:, None]; j = np.arange(T)[None, :]
    rel = i - j
    M = ((rel >= 0) & (rel <= W)) | np.isin(rel, np.array(base))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(q), torch.tensor(k), torch.tensor(v), attn_mask=torch.tensor(M))
    np.testing.assert_allclose(o, ref.numpy(), atol=1e-12)


# ---------------------------------------------------------------------------
# P5 special cases reducing to textbook attention
# ---------------------------------------------------------------------------

def test_no_rungs_is_sliding_window():
    T, D, W = 40, 8, 5
    q, k, v = (rand((1, 3, T, D), s) for s in (31, 32, 33))
    o, _ = oracle.forward(q, k, v, W, [], 1.0)
    rel = np.arange(T)[:, None] - np.arange(T)[None, :]
    M = (rel >= 0) & (rel <= W)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(q), torch.tensor(k), torch.tensor(v), attn_mask=torch.tensor(M))
    np.testing.assert_allclose(o, ref.numpy(), atol=1e-12)


def test_full_window_is_causal_attention():
    T, D = 33, 8
    q, k, v, dO = (rand((1, 2, T, D), s) for s in (41, 42, 43, 44))
    o, _ = oracle.forward(q, k, v, T - 1, [], 1.0)
    Q, K, V = (torch.tensor(x, requires_grad=True) for x in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(Q, K, V, is_causal=True)
    np.testing.assert_allclose(o, ref.detach().numpy(), atol=1e-12)
    (ref * torch.tensor(dO)).sum().backward()
    dq, dk, dv, da, _ = oracle.backward(q, k, v, dO, T - 1, [], 1.0)
    np.testing.assert_allclose(dq, Q.grad.numpy(), atol=1e-11)
    np.testing.assert_allclose(dk, K.grad.numpy(), atol=1e-11)
    np.testing.assert_allclose(dv, V.grad.numpy(), atol=1e-11)
    assert da == 0.0


def test_single_position():
    q, k, v = (rand((2, 2, 1, 8), s) for s in (51, 52, 53))
    o, lse = oracle.forward(q, k, v, 8, FIB, 1.0)
    np.testing.assert_allclose(o, v, atol=0)
    np.testing.assert_allclose(lse, (q * k).sum(-1) / math.sqrt(8), atol=1e-15)


# ---------------------------------------------------------------------------
# P4 closed forms at q = 0 and the paper's distance count
# ---------------------------------------------------------------------------

def test_paper_distance_count_at_full_context():
    g = json.load(open(os.path.join(GOLDEN, "paper_counts.json")))
    T, W, alpha, base = g["T"], g["W"], g["alpha"], g["base"]
    q = np.zeros((1, 1, T, 1)); k = np.zeros_like(q)
    v = np.arange(T, dtype=np.float64).reshape(1, 1, T, 1)
    o, lse = oracle.forward(q, k, v, W, base, alpha)
    counts = np.rint(np.exp(lse[0, 0])).astype(int)
    np.testing.assert_allclose(np.exp(lse[0, 0]), counts, rtol=1e-12)
    assert counts[-1] == g["distinct_distances_full_context"]
    assert all(c == g["distinct_distances_full_context"] for c in counts[max(base):])
    # with v_j = j the output is i minus the mean attended distance
    for i in (0, 5, 8, 13, 100, 600, 987, 1023):
        dists = [dl for dl in range(W + 1) if dl <= i] + [f for f in base if f > W and f <= i]
        assert counts[i] == len(dists)
        assert abs(o[0, 0, i, 0] - (i - np.mean(dists))) < 1e-9


def test_uniform_softmax_weights_non_integer_alpha():
    # q = 0: every entry has probability 1/|E(i)|; with v_j = j the rung entry is worth
    # exactly i - d (linear interpolation of a linear function).
    T, W, alpha = 200, 6, 0.7
    q = np.zeros((1, 1, T, 1)); k = rand((1, 1, T, 1), 5)
    v = np.arange(T, dtype=np.float64).reshape(1, 1, T, 1)
    o, lse = oracle.forward(q, k, v, W, FIB, alpha)
    ds = sorted(set(d for d in fl32_distances(alpha, FIB) if d > W))
    for i in (0, 3, 6, 7, 9, 15, 50, 199):
        dists = [float(x) for x in range(min(W, i) + 1)] + [d for d in ds if d <= i]
        assert abs(lse[0, 0, i] - math.log(len(dists))) < 1e-12
        assert abs(o[0, 0, i, 0] - (i - np.mean(dists))) < 1e-9


# ---------------------------------------------------------------------------
# P6 hand-worked examples
# ---------------------------------------------------------------------------

def test_hand_examples():
    g = json.load(open(os.path.join(GOLDEN, "hand_examples.json")))
    for c in g["cases"]:
        T = c["T"]
        q = np.zeros((1, 1, T, 1)); k = np.zeros_like(q)
        v = np.array(c["v"]).reshape(1, 1, T, 1)
        dO = np.ones_like(q)
        o, lse = oracle.forward(q, k, v, c["W"], c["base"], c["alpha"])
        np.testing.assert_allclose(o[0, 0, :, 0], c["o"], atol=1e-15, err_msg=c["name"])
        np.testing.assert_allclose(lse[0, 0], c["lse"], atol=1e-15, err_msg=c["name"])
        _, _, _, da, _ = oracle.backward(q, k, v, dO, c["W"], c["base"], c["alpha"])
        assert abs(da - c["dalpha"]) < 1e-14, c["name"]


# ---------------------------------------------------------------------------
# P7 / P9 finite differences, P8 nonzero dalpha at integer alpha
# ---------------------------------------------------------------------------

def _loss(o, dO):
    return float((o * dO).sum())


def test_dalpha_finite_difference_off_kinks():
    T, D, W = 96, 8, 4
    alpha = np.float32(0.7310586)
    tab = oracle.rungs(alpha, FIB, W)
    # away from kinks: every d_k is far from an integer and from i
    gaps = [min(float(w), 1 - float(w)) / f for (_, w, f, _) in tab]
    h = min(gaps) / 8
    assert h > 1e-6
    q, k, v, dO = (rand((1, 2, T, D), s) for s in (61, 62, 63, 64))
    d0 = [t[0] for t in tab]; f = [t[2] for t in tab]
    w = np.array([float(t[1]) for t in tab])
    _, _, _, da, _ = oracle.backward_table(q, k, v, dO, W, d0, w, f)
    lp = _loss(oracle.forward_table(q, k, v, W, d0, w + h * np.array(f), f)[0], dO)
    lm = _loss(oracle.forward_table(q, k, v, W, d0, w - h * np.array(f), f)[0], dO)
    fd = (lp - lm) / (2 * h)
    assert abs(fd - da) <= 1e-6 * max(1.0, abs(da)), (fd, da)


@pytest.mark.parametrize("alpha", [1.0, 0.9])
def test_input_gradients_finite_difference(alpha):
    T, D, W = 48, 4, 3
    q, k, v, dO = (rand((1, 1, T, D), s) for s in (71, 72, 73, 74))
    dq, dk, dv, _, _ = oracle.backward(q, k, v, dO, W, FIB, alpha)
    rng = np.random.default_rng(7)
    h = 1e-5
    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        for _ in range(6):
            idx = (0, 0, int(rng.integers(T)), int(rng.integers(D)))
            xp = x.copy(); xp[idx] += h
            xm = x.copy(); xm[idx] -= h
            args_p = {"q": q, "k": k, "v": v}; args_p[name] = xp
            args_m = {"q": q, "k": k, "v": v}; args_m[name] = xm
            lp = _loss(oracle.forward(args_p["q"], args_p["k"], args_p["v"], W, FIB, alpha)[0], dO)
            lm = _loss(oracle.forward(args_m["q"], args_m["k"], args_m["v"], W, FIB, alpha)[0], dO)
            fd = (lp - lm) / (2 * h)
            assert abs(fd - g[idx]) <= 1e-7 * max(1.0, abs(g[idx])), (name, idx, fd, g[idx])


def test_dalpha_nonzero_at_integer_alpha():
    # Section 2: interpolation keeps a nonzero gradient to alpha even when every rung
    # sits on an integer position.
    T, D, W = 128, 8, 8
    q, k, v, dO = (rand((1, 2, T, D), s) for s in (81, 82, 83, 84))
    _, _, _, da, l1 = oracle.backward(q, k, v, dO, W, FIB, 1.0)
    assert abs(da) > 1e-3 * l1 > 0


# ---------------------------------------------------------------------------
# P10 invariants
# ---------------------------------------------------------------------------

def test_causality():
    T, D, W = 80, 8, 4
    q, k, v = (rand((1, 1, T, D), s) for s in (91, 92, 93))
    o, lse = oracle.forward(q, k, v, W, FIB, 0.8)
    i0 = 37
    q2, k2, v2 = q.copy(), k.copy(), v.copy()
    q2[:, :, i0 + 1:] += 3.0; k2[:, :, i0 + 1:] -= 2.0; v2[:, :, i0 + 1:] *= 5.0
    o2, lse2 = oracle.forward(q2, k2, v2, W, FIB, 0.8)
    np.testing.assert_array_equal(o[:, :, :i0 + 1], o2[:, :, :i0 + 1])
    np.testing.assert_array_equal(lse[:, :, :i0 + 1], lse2[:, :, :i0 + 1])


def test_batch_head_permutation_equivariance():
    T, D, W = 40, 4, 3
    q, k, v, dO = (rand((3, 2, T, D), s) for s in (95, 96, 97, 98))
    dq, dk, dv, da, _ = oracle.backward(q, k, v, dO, W, FIB, 1.2)
    perm = [2, 0, 1]
    dq2, dk2, dv2, da2, _ = oracle.backward(q[perm][:, ::-1], k[perm][:, ::-1], v[perm][:, ::-1],
                                            dO[perm][:, ::-1], W, FIB, 1.2)
    np.testing.assert_array_equal(dq[perm][:, ::-1], dq2)
    np.testing.assert_array_equal(dv[perm][:, ::-1], dv2)
    assert abs(da - da2) <= 1e-12 * max(1, abs(da))


# ---------------------------------------------------------------------------
# rung table readings and schedules
# ---------------------------------------------------------------------------

def test_rung_table_inclusion_and_float32_offsets():
    # alpha = 1, W = 8: rungs 1, 2, 3, 5, 8 lie in the window; 10 rungs remain.
    tab = oracle.rungs(1.0, FIB, 8)
    assert [t[0] for t in tab] == FIB[5:]
    assert all(t[1] == 0 for t in tab)
    # float32 offsets: alpha_3 = fl32(0.7) times 610 rounds to exactly 427 in float32,
    # while the float64 product 426.99999... would floor to 426.
    a3 = schedules.alpha_linear_stagger(16)[3]
    assert float(a3) * 610 < 427
    tab = {t[2]: t for t in oracle.rungs(a3, FIB, 8)}
    assert tab[610][0] == 427 and tab[610][1] == 0
    # alpha = 0.5: rung 13 at 6.5 is inside W = 8 and dropped
    assert [t[2] for t in oracle.rungs(0.5, FIB, 8)][0] == 21


def test_rung_table_rejects_bad_input():
    with pytest.raises(ValueError):
        oracle.rungs(0.0, FIB, 8)
    with pytest.raises(ValueError):
        oracle.rungs(1.0, [2, 1], 8)
    with pytest.raises(ValueError):
        oracle.rungs(1.0, [0, 1], 8)


def test_schedules_match_paper_and_library():
    lin = oracle.alpha_schedule("linear")
    assert lin[0] == np.float32(0.5) and lin[-1] == np.float32(1.5)
    cop = oracle.alpha_schedule("coprime")
    # the coprime map l -> 7l mod 16 is an involution, so it permutes the ramp values
    assert sorted(cop.tolist()) == sorted(lin.tolist())
    assert all((7 * ((7 * l) % 16)) % 16 == l for l in range(16))
    assert cop[1] == lin[7] and cop[2] == lin[14]
    assert oracle.alpha_from_theta(0.0) == np.float32(1.0)
    th = np.random.default_rng(3).standard_normal(16)
    np.testing.assert_array_equal(oracle.alpha_schedule("learned", theta=th), schedules.alpha_from_theta(th))
    np.testing.assert_array_equal(lin, schedules.alpha_linear_stagger())
    np.testing.assert_array_equal(cop, schedules.alpha_coprime_stagger())
    np.testing.assert_array_equal(oracle.alpha_schedule("fixed"), schedules.alpha_fixed())


def test_rope_is_a_rotation_and_transpose_inverts_it():
    x = rand((1, 2, 50, 8), 99)
    y = oracle.rope(x, 10000.0)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)
    np.testing.assert_allclose(oracle.rope(y, 10000.0, transpose=True), x, atol=1e-13)
    # position 0 is the identity; position t pairs (j, j + D/2) rotate by t * 1e4^(-2j/D)
    np.testing.assert_array_equal(y[:, :, 0], x[:, :, 0])
    t, j, D = 7, 1, 8
    ang = t * 10000.0 ** (-2 * j / D)
    a, b = x[0, 0, t, j], x[0, 0, t, j + D // 2]
    assert abs(y[0, 0, t, j] - (a * math.cos(ang) - b * math.sin(ang))) < 1e-14
    # relative-position property: <R_t q, R_s k> depends on t - s only
    q = rand((1, 1, 1, 8), 5)[0, 0, 0]; kk = rand((1, 1, 1, 8), 6)[0, 0, 0]
    X = np.zeros((1, 1, 40, 8)); X[0, 0, :] = q
    Y = np.zeros((1, 1, 40, 8)); Y[0, 0, :] = kk
    RQ, RK = oracle.rope(X), oracle.rope(Y)
    assert abs(RQ[0, 0, 20] @ RK[0, 0, 13] - RQ[0, 0, 30] @ RK[0, 0, 23]) < 1e-12
