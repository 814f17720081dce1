"""Host-only checks of the C ABI (no GPU): the library loads, exports every entry
point include/fibattn.h declares, builds the same rung table as the oracle's
independent code, and rejects invalid arguments before touching the device."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2606_28560_amd import fibattn as F
from paper_2606_28560_amd import schedules, workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    src = open(os.path.join(ROOT, "include", "fibattn.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(fibattn_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    names = header_functions()
    assert len(names) >= 8
    L = F.lib()
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(F.EXPORTED)


def _all_alphas():
    al = [1.0, 0.5, 1.5, 0.7310586, 0.01, 3.7]
    for w in workloads.all_workloads():
        al += [float(c.alpha) for c in w.calls]
    return sorted(set(al))


@pytest.mark.parametrize("W", [0, 6, 8, 10, 12])
def test_rung_table_matches_oracle(W):
    for base in (schedules.FIB15, schedules.POW2_11, (3, 7, 11, 1000)):
        for a in _all_alphas():
            lib_tab = F.fibattn_rung_table(a, base, W)
            orc_tab = [(d0, w, f) for (d0, w, f, _) in oracle.rungs(a, base, W)]
            assert lib_tab == orc_tab, (a, base, W)


def test_stagger_float32_floor_cases():
    # float32 products that round up to an integer where the float64 product does not
    lin = schedules.alpha_linear_stagger(16)
    hits = []
    for l, a in enumerate(lin):
        for f in schedules.FIB15:
            if np.floor(np.float32(a) * np.float32(f)) != np.floor(float(a) * f):
                hits.append((l, f))
    assert hits == [(3, 610), (5, 144), (6, 610), (10, 144), (12, 610)]
    tab = {f: (d0, w) for d0, w, f in F.fibattn_rung_table(lin[3], schedules.FIB15, 8)}
    assert tab[610] == (427, 0.0)


def test_integer_base_rounds_half_to_even():
    # alpha = 0.5 by hand: 0.5 f = 0.5, 1, 1.5, 2.5, 4, 6.5, 10.5, 17, 27.5, 44.5, 72,
    # 116.5, 188.5, 305, 493.5 -> half to even 0, 1, 2, 2, 4, 6, 10, 17, 28, 44, 72,
    # 116, 188, 305, 494; 0 and the repeated 2 dropped
    assert schedules.integer_base(0.5, schedules.FIB15) == (
        1, 2, 4, 6, 10, 17, 28, 44, 72, 116, 188, 305, 494)
    assert schedules.integer_base(1.0, schedules.FIB15) == schedules.FIB15
    assert schedules.integer_base(2.0, schedules.POW2_11) == tuple(1 << j for j in range(1, 12))


@pytest.mark.parametrize("layer", [0, 3, 7, 11, 15])
def test_integer_base_gives_integer_rungs(layer):
    # a pre-rounded base with alpha = 1 is the integer path: every weight 0, every
    # distance one of the rounded offsets beyond the window, equal to the oracle's
    a = schedules.alpha_linear_stagger(16)[layer]
    base = schedules.integer_base(a, schedules.FIB15)
    assert all(b2 > b1 for b1, b2 in zip(base, base[1:])) and base[0] >= 1
    lib_tab = F.fibattn_rung_table(1.0, base, 8)
    assert all(w == 0.0 for _, w, _ in lib_tab)
    assert [d0 for d0, _, _ in lib_tab] == [b for b in base if b > 8]
    ref = oracle.rungs(1.0, base, 8)
    assert [(int(r[0]), float(r[1]), int(r[2])) for r in ref] == [(d, w, f) for d, w, f in lib_tab]


def test_rung_table_rejects_bad_input():
    for alpha, base in ((0.0, [1, 2]), (-1.0, [1]), (float("nan"), [1]), (1.0, [2, 2]),
                        (1.0, [0, 3]), (1.0, list(range(1, 40)))):
        with pytest.raises(F.FibattnError):
            F.fibattn_rung_table(alpha, base, 8)


def test_invalid_arguments_return_codes_without_gpu():
    L = F.lib()
    b = (ctypes.c_int32 * 15)(*schedules.FIB15)
    one = ctypes.c_float(1.0)
    # null pointers
    assert L.fibattn_forward(None, None, None, None, None, 1, 1, 8, 64, 8, b, 15, one, 1, None) == 1
    # bad sizes
    assert L.fibattn_forward(16, 16, 16, 16, 16, 0, 1, 8, 64, 8, b, 15, one, 1, None) == 1
    assert L.fibattn_forward(16, 16, 16, 16, 16, 1, 1, 8, 96, 8, b, 15, one, 1, None) == 2
    assert L.fibattn_forward(16, 16, 16, 16, 16, 1, 1, 8, 64, 129, b, 15, one, 1, None) == 2
    assert L.fibattn_forward(16, 16, 16, 16, 16, 1, 1, 8, 64, 8, b, 15, one, 9, None) == 1
    # one head's rows must stay below 2^31 bytes (32-bit row offsets in the kernels)
    assert L.fibattn_forward(16, 16, 16, 16, 16, 1, 1, 1 << 24, 64, 8, b, 15, one, 1, None) == 2
    assert L.fibattn_forward(16, 16, 16, 16, 16, 1, 1, 1 << 22, 128, 8, b, 15, one, 0, None) == 2
    assert L.fibattn_backward_workspace_bytes(1, 1, 1 << 24, 64, 8, 15) == 0
    assert L.fibattn_backward_workspace_bytes(1, 1, (1 << 24) - 1, 64, 8, 15) > 0
    # the workspace size does not depend on the storage type: a bfloat16 shape beyond
    # the float32 limit still gets its size, and the bfloat16 call checks against it
    assert L.fibattn_backward_workspace_bytes(1, 1, 1 << 23, 64, 8, 15) > 4 * 15 * (1 << 23)
    assert L.fibattn_backward(16, 16, 16, 16, 16, 16, 16, 16, 16, 16, 16, 256,
                              1, 1, 1 << 23, 64, 8, b, 15, one, ctypes.c_float(0.0), 1, None) == 3
    # workspace
    zero = ctypes.c_float(0.0)
    assert L.fibattn_backward(16, 16, 16, 16, 16, 16, 16, 16, 16, 16, None, 0,
                              1, 1, 8, 64, 8, b, 15, one, zero, 1, None) == 3
    # rope_base must be 0 (no rotation) or > 1
    assert L.fibattn_backward(16, 16, 16, 16, 16, 16, 16, 16, 16, 16, 16, 1 << 30,
                              1, 1, 8, 64, 8, b, 15, one, ctypes.c_float(0.5), 1, None) == 1
    assert L.fibattn_backward_workspace_bytes(1, 1, 8, 48, 8, 15) == 0
    assert L.fibattn_backward_workspace_bytes(8, 8, 1024, 64, 8, 15) > 8 * 8 * 1024 * 4
    # the matrix-core shapes (d_head 64, W <= 16) add a 4-byte term per query and rung:
    # K of them, or 32 (the most a table holds) for a device table (K = 0)
    n = 8 * 8 * 1024
    ws = L.fibattn_backward_workspace_bytes
    assert ws(8, 8, 1024, 64, 8, 15) >= 4 * n + 8 * (n // 64) + 4 * 15 * n
    assert ws(8, 8, 1024, 64, 8, 0) >= 4 * n + 8 * (n // 64) + 4 * 32 * n
    assert ws(8, 8, 1024, 64, 8, 15) - ws(8, 8, 1024, 64, 8, 11) == 4 * 4 * n
    assert ws(8, 8, 1024, 32, 8, 15) < 4 * n + 4 * 15 * n   # generic kernels: no terms
    assert ws(8, 8, 1024, 64, 17, 15) < 4 * n + 4 * 15 * n
    # rope
    assert L.fibattn_rope(None, None, 1, 1, 8, 64, ctypes.c_float(1e4), 0, 1, None) == 1
    assert L.fibattn_rope(16, 16, 1, 1, 8, 64, ctypes.c_float(1.0), 0, 1, None) == 1
    assert L.fibattn_rope(16, 16, 1, 1, 8, 96, ctypes.c_float(1e4), 0, 1, None) == 2
    assert L.fibattn_rope(18, 16, 1, 1, 8, 64, ctypes.c_float(1e4), 0, 1, None) == 1  # misaligned
    assert L.fibattn_rope_qk(16, 16, 16, None, 1, 1, 8, 64, ctypes.c_float(1e4), 1, None) == 1
    assert L.fibattn_rope_qk(16, 16, 16, 16, 1, 1, 8, 64, ctypes.c_float(1.0), 1, None) == 1
    assert L.fibattn_rope_qk(16, 16, 16, 16, 1, 1, 8, 48, ctypes.c_float(1e4), 1, None) == 2
    # grouped heads: H_kv must divide H
    for hkv in (0, 3, 16):
        assert L.fibattn_forward_gqa(16, 16, 16, 16, 16, 1, 8, hkv, 8, 64, 8, b, 15, one, 1, None) == 1
        assert L.fibattn_backward_gqa(16, 16, 16, 16, 16, 16, 16, 16, 16, 16, 16, 1 << 30,
                                      1, 8, hkv, 8, 64, 8, b, 15, one, zero, 1, None) == 1
    # queries rotated on load: q_out aligned or null, rope_base > 1, H_kv dividing H; a null
    # q_out only where the rotation runs inside the forward (bf16, d_head 64, W <= 16)
    rq, r4 = L.fibattn_forward_rope_q, ctypes.c_float(1e4)
    assert rq(16, 16, 16, 16, 16, 18, 1, 8, 8, 8, 64, 8, b, 15, one, r4, 1, None) == 1
    assert rq(16, 16, 16, 16, 16, 16, 1, 8, 8, 8, 64, 8, b, 15, one, ctypes.c_float(1.0), 1, None) == 1
    assert rq(16, 16, 16, 16, 16, 16, 1, 8, 3, 8, 64, 8, b, 15, one, r4, 1, None) == 1
    assert rq(None, 16, 16, 16, 16, 16, 1, 8, 8, 8, 64, 8, b, 15, one, r4, 1, None) == 1
    assert rq(16, 16, 16, 16, 16, 16, 1, 8, 8, 8, 48, 8, b, 15, one, r4, 1, None) == 2
    assert rq(16, 16, 16, 16, 16, None, 1, 8, 8, 8, 64, 8, b, 15, one, r4, 0, None) == 2   # float32
    assert rq(16, 16, 16, 16, 16, None, 1, 8, 8, 8, 64, 20, b, 15, one, r4, 1, None) == 2  # W > 16
    # with placements: the layouts are checked before any launch
    rqs = L.fibattn_forward_rope_q_strided
    assert rqs(16, 16, 16, 16, 16, 16, None, 1, 8, 8, 8, 64, 8, b, 15, one, r4, 1, None) == 1
    bad_lay = (ctypes.c_int64 * 15)(*([8 * 64 * 8, 64 * 8, 64] * 4 + [8 * 64 * 8, 64 * 8, 3]))
    assert rqs(16, 16, 16, 16, 16, 16, bad_lay, 1, 8, 8, 8, 64, 8, b, 15, one, r4, 1, None) == 1
    # the same from a device table: the table pointer is required
    rqd = L.fibattn_forward_rope_q_dt
    assert rqd(16, 16, 16, 16, 16, 16, 1, 8, 8, 8, 64, 8, None, r4, 1, None) == 1
    assert rqd(16, 16, 16, 16, 16, 16, 1, 8, 8, 8, 64, 8, 16, ctypes.c_float(0.5), 1, None) == 1
    assert rqd(16, 16, 16, 16, 16, None, 1, 8, 8, 8, 64, 8, 16, r4, 0, None) == 2
    # k alone through the prologue launch: q and q_out null together, or neither
    rt = L.fibattn_rope_qk_table
    assert rt(None, 16, 16, 16, 1, 8, 8, 8, 64, r4, None, None, b, 15, 8, None, 1, None) == 1
    assert rt(16, 16, None, 16, 1, 8, 8, 8, 64, r4, None, None, b, 15, 8, None, 1, None) == 1
    # device alpha: the base table is checked on the host, pointers before any launch
    bad = (ctypes.c_int32 * 3)(5, 3, 8)
    assert L.fibattn_device_table(16, bad, 3, 8, 16, None) == 1
    assert L.fibattn_device_table(None, b, 15, 8, 16, None) == 1
    assert L.fibattn_device_table(16, b, 15, 8, 18, None) == 1  # misaligned table
    assert L.fibattn_device_table_bytes() >= 8 + 3 * 4 * 32 + 8
    assert L.fibattn_forward_dt(16, 16, 16, 16, 16, 1, 2, 2, 8, 64, 8, None, 1, None) == 1
    assert L.fibattn_forward_dt(16, 16, 16, 16, 16, 1, 8, 3, 8, 64, 8, 16, 1, None) == 1
    assert L.fibattn_backward_dt(16, 16, 16, 16, 16, 16, 16, 16, 16, 16, None, None, 0,
                                 1, 1, 1, 8, 64, 8, 16, zero, 1, None) == 3
    assert L.fibattn_device_table_theta(None, None, b, 15, 8, 16, None) == 1
    # RoPE + table: H_kv must divide H; a theta needs an aligned table and a valid base
    assert L.fibattn_rope_qk_table(16, 16, 16, 16, 1, 8, 3, 8, 64, ctypes.c_float(1e4), None, None, b, 15, 8,
                                   None, 1, None) == 1
    assert L.fibattn_rope_qk_table(16, 16, 16, 16, 1, 8, 2, 8, 64, ctypes.c_float(1e4), 16, None, b, 15, 8,
                                   None, 1, None) == 1
    assert L.fibattn_rope_qk_table(16, 16, 16, 16, 1, 8, 2, 8, 64, ctypes.c_float(0.5), None, None, b, 15, 8,
                                   None, 1, None) == 1
    assert L.fibattn_device_table_theta(16, None, b, 15, -1, 16, None) == 1
    assert L.fibattn_alpha_from_theta(16, 16, 0, None) == 1
    assert L.fibattn_dtheta(16, None, 16, 4, None) == 1
    for s in range(5):
        assert F.status_string(s)


def test_strided_layouts_are_checked_before_any_launch():
    """Bad layouts return a status on the host.  Every call here fails validation
    before any launch (the pointers are dummies)."""
    L = F.lib()
    b = (ctypes.c_int32 * 15)(*schedules.FIB15)
    one, zero = ctypes.c_float(1.0), ctypes.c_float(0.0)

    def lay(*rows):
        arr = (ctypes.c_int64 * (3 * len(rows)))()
        for a, r in enumerate(rows):
            arr[3 * a:3 * a + 3] = r
        return arr

    good = (8 * 8 * 64, 8 * 64, 64)  # packed [B, 8, 8, 64]

    def fwd(ls, T=8):
        return L.fibattn_forward_strided(16, 16, 16, 16, 16, ls, 1, 8, 8, T, 64, 8, b, 15, one, 1, None)

    assert fwd(None) == 1
    assert fwd(lay(good, good, good, (-64, 64, 64))) == 1                # negative stride
    assert fwd(lay(good, (8 * 8 * 64, 8 * 64, 60), good, good)) == 1     # rows not 16-byte aligned
    assert fwd(lay(good, good, (8 * 8 * 64 + 4, 8 * 64, 64), good)) == 1  # batch stride misaligned
    assert fwd(lay(good, good, (0, 0, 1 << 26), good), T=64) == 2        # row offsets >= 2^31 bytes

    def bwd(ls):
        return L.fibattn_backward_strided(16, 16, 16, 16, 16, 16, 16, 16, 16, 16, 16, 1 << 30, ls,
                                          1, 8, 8, 8, 64, 8, b, 15, one, zero, 1, None)

    assert bwd(None) == 1
    assert bwd(lay(*([good] * 7 + [(0, 0, 12)]))) == 1                   # dv rows misaligned
    assert bwd(lay(*([good] * 5 + [(0, -8, 64)] + [good] * 2))) == 1     # dq head stride negative


def test_noalloc_backward_refuses_problems_beyond_its_scratch_without_gpu():
    # the size check comes before any pointer is read or any HIP call is made
    L = F.lib()
    b = (ctypes.c_int32 * 15)(*schedules.FIB15)
    one, zero = ctypes.c_float(1.0), ctypes.c_float(0.0)
    need = F.fibattn_backward_workspace_bytes(32, 8, 16384, 64, 8, 15)
    assert need > F.SCRATCH_BYTES
    st = L.fibattn_backward_noalloc(*([16] * 10), 32, 8, 8, 16384, 64, 8, b, 15, one, zero, 1, None)
    assert st == 5 and "scratch" in F.status_string(st)
    # bad sizes are refused as by the other entry points
    assert L.fibattn_backward_noalloc(*([16] * 10), 0, 8, 8, 1024, 64, 8, b, 15, one, zero, 1, None) == 1
    assert L.fibattn_backward_noalloc(*([16] * 10), 1, 8, 3, 1024, 64, 8, b, 15, one, zero, 1, None) == 1
