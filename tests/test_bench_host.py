"""Host logic of the benchmark (no GPU): the one-GPU refusal, the algorithmic
work behind the roofline entry (closed forms on a small workload), the
committed HBM counter profile and the guard that withholds it once the kernel
sources change, and the host thread count of the oracle baseline."""
import json
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import gen  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and "--gpus 2" in r.stderr


def test_stage_work_closed_forms():
    # C = 30 clusters: C_eff = 30 for the sequence of 40 and 25 for that of 25
    w = gen.config_speech(B=2, H=3, N=40, d=32, C=30, lengths=np.array([40, 25], np.int32))
    nsum = (40 + 25) * 3
    cn = (30 * 40 + 25 * 25) * 3           # sum over units of C_eff n
    flops, unit, bound, peak = bench.stage_work(w, "centroid_attn", 32)
    assert (unit, bound) == ("TFLOP/s", "mfma") and peak == bench.PEAKS["fp32_mfma_TFLOPs"]
    assert flops == 2 * (2 * cn * 32)      # Q^c K^T and A^c V
    assert bench.stage_work(w, "attn_tile", 32)[0] == flops
    ops, unit, bound, _ = bench.stage_work(w, "kmeans", 0)
    assert unit == "TOP/s" and ops == 2 * 64 * w.L * cn
    byts, unit, bound, peak = bench.stage_work(w, "hash", 0)
    assert (unit, bound) == ("GB/s", "hbm") and byts == nsum * 32 * 4 + nsum * 8
    assert bench.stage_work(w, "output", 0)[0] == nsum * 32 * 4 + nsum * 4
    # the T rows: C_eff k_eff = 30 * 32 and 25 * 25 per head
    assert bench.stage_work(w, "output", 32)[0] == 2 * nsum * 32 * 4 + 2 * 3 * (30 * 32 + 25 * 25) * 32 * 4
    assert bench.stage_work(w, "centroids", 0)[0] == nsum * 32 * 4 + nsum * 4 + 3 * (30 + 25) * 32 * 4
    wb = gen.config_sweep(64, dtype="bf16", H=2, C=10)
    assert bench.stage_work(wb, "attn_tile", 0)[3] == bench.PEAKS["bf16_mfma_TFLOPs"]
    with pytest.raises(ValueError):
        bench.stage_work(w, "nonsense", 0)


@pytest.mark.parametrize("profile", ["speech_b32h6n800_d32_f32", "sweep_b1h8n32768_d64_f32",
                                     "long_b1h8n65536_d64_bf16"])
def test_counter_profile_is_withheld_when_sources_change(monkeypatch, profile):
    """Each committed counter profile holds the key of the bench line's
    roofline kernel (the i-clustered tile kernel), and the bench reports it
    only while the kernel sources hash to the recorded value."""
    path = os.path.join(ROOT, "profiles", profile + "_hbm_counters.json")
    with open(path) as f:
        prof = json.load(f)
    key = "attn_tile (iclustered)"
    assert prof["kernels"][key]["hbm_bytes_per_launch"] > 0
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: prof["source_sha256"])
    assert bench.measured_traffic(key, profile) == prof["kernels"][key]["hbm_bytes_per_launch"]
    assert bench.measured_traffic("no such kernel", profile) is None
    assert bench.measured_traffic(key, "no_such_workload") is None
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "0" * 64)
    assert bench.measured_traffic(key, profile) is None


def test_kernel_source_hash_is_stable():
    h0 = bench.kernel_source_hash()
    assert len(h0) == 64 and h0 == bench.kernel_source_hash()


def test_cpu_threads(monkeypatch):
    monkeypatch.setenv("OMP_NUM_THREADS", "1")
    assert bench.cpu_threads() == 1
    monkeypatch.setenv("OMP_NUM_THREADS", "")
    assert bench.cpu_threads() >= 1


def test_centroid_stage_priced_by_its_own_reads_when_fused():
    """With the centroid sums formed inside the one-launch K-means (grids that
    cover every compute unit), the centroid stage reads only the workgroups'
    fp64 parts, and its algorithmic bytes say so."""
    import gen
    wl = gen.config_long()
    ws = gen.make_config(3, N=32768, dtype="f32")
    assert bench.fused_centroid_sums(wl, 256) and not bench.fused_centroid_sums(ws, 256)
    B, H, N, D = wl.q.shape
    nwg = (N + 2047) // 2048
    want = B * H * wl.C * nwg * D * 8 + B * H * wl.C * D * 4 + B * H * wl.C * 4
    assert bench.stage_work(wl, "centroids", wl.topk, 256)[0] == want
    B, H, N, D = ws.q.shape
    assert bench.stage_work(ws, "centroids", ws.topk, 256)[0] == B * H * N * (D * 4 + 4) + B * H * ws.C * D * 4
