"""Host-side logic of bench.py (CPU): the byte accounting against the hot path's
compulsory traffic, the buffer rotation that keeps the last-level cache from serving a
step, the guard on the stored HBM counter figures, the one-GPU contract and the CPU
baseline record."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from paper_2606_28560_amd import workloads  # noqa: E402


def test_algorithmic_bytes_per_query_head():
    # d_head 64, bfloat16: forward 516 B, fwd+bwd 1544 B (q, k, v in, o, lse out; then q,
    # k, v, o, dO, lse in, dq, dk, dv out); the two backward kernels 776 B each
    assert bench.alg_bytes("forward", 64, 2) == 516
    assert bench.alg_bytes("fwd+bwd", 64, 2) == 1544
    assert bench.alg_bytes("bwd_dq", 64, 2) == bench.alg_bytes("bwd_dkdv", 64, 2) == 776
    assert bench.alg_bytes("rope", 64, 2) == 512
    # the step's forward rotates q on load: it also writes R q; its RoPE launch takes k only
    assert bench.alg_bytes("forward_rope_q", 64, 2) == 516 + 128
    assert bench.alg_bytes("rope_k", 64, 2) == 256
    assert set(bench.STEP_ALG) == {"forward", "bwd_dq", "bwd_dkdv", "rope"}
    # float32 with d_head 32 moves the same bytes per query-head
    assert bench.alg_bytes("fwd+bwd", 32, 4) == 1544


@pytest.mark.parametrize("per_set_mib", [20, 57, 88, 130, 300, 2000])
def test_buffer_sets_exceed_twice_the_last_level_cache(per_set_mib):
    per = per_set_mib * 2**20
    n = bench.buffer_sets(per)
    # between two uses of one set, the other n - 1 sets move more than 2x the cache
    assert (n - 1) * per > 2 * bench.MALL_BYTES
    if per < 128 * 2**20:
        assert n >= 6


def test_step_bytes_of_the_60m_layer():
    wl = workloads.workload("layer_60m_fixed_T1024")
    c = wl.calls[0]
    row = 8 * 8 * 1024 * 64 * 2
    from paper_2606_28560_amd import fibattn as F
    ws = F.fibattn_backward_workspace_bytes(8, 8, 1024, 64, c.W, len(c.base))
    assert bench.step_bytes(wl, c) == 10 * row + 4 * 8 * 8 * 1024 + ws
    assert bench.buffer_sets(bench.step_bytes(wl, c)) == 8


def test_stored_traffic_applies_only_to_its_sources_and_workload(monkeypatch):
    if bench.kernel_sources_sha() == bench.COUNTER_SOURCES_SHA:
        t = bench.hbm_traffic("bwd_dq", bench.COUNTER_WORKLOAD)
        fetch, write = bench.COUNTER_KIB["bwd_dq"]
        moved, cf, cw = bench.COPY_PROBE_KIB
        assert t == pytest.approx((fetch * moved / cf + write * moved / cw) * 1024)
    assert bench.hbm_traffic("bwd_dq", "stagger16_T1024") is None
    assert bench.hbm_traffic("not_a_kernel", bench.COUNTER_WORKLOAD) is None
    monkeypatch.setattr(bench, "COUNTER_SOURCES_SHA", "0" * 64)
    assert bench.hbm_traffic("bwd_dq", bench.COUNTER_WORKLOAD) is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_cpu_baseline_record():
    wl = workloads.workload("layer_60m_fixed_T1024")
    rec = bench.cpu_baseline(wl, wl.calls[0], 0.01)  # one repetition of the layer
    assert rec["kind"] == "oracle" and rec["unit"] == "queries·heads/s"
    assert rec["value"] > 0 and 1 <= rec["cores"] <= rec["openmp_threads"]
    assert rec["nproc"] >= 1 and "query-heads" in rec["sample"]
