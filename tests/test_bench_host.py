"""Host-side logic of bench.py (CPU only, no GPU)."""
import json
import os
import subprocess
import sys

import pytest

import bench
from paper_2609_36070_amd.workloads import WORKLOADS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("n", [2, 8])
def test_more_than_one_gpu_is_refused_before_any_gpu_work(n):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", str(n)],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""          # no JSON line


@pytest.mark.parametrize("name", ["large_shared_train", "tiny"])
def test_stage_flops_add_up_to_the_step_convention(name):
    """The per-stage FLOPs (used for the per-stage rates and the roofline)
    partition the step's 6 T (k f + f_s) d forward and twice that backward."""
    w = WORKLOADS[name]
    fwd, bwd = bench.stage_flops(w)
    assert sum(v[0] for v in fwd.values()) == pytest.approx(w.fwd_flops(), rel=1e-12)
    assert sum(v[0] for v in bwd.values()) == pytest.approx(2.0 * w.fwd_flops(), rel=1e-12)


def test_traffic_record_is_reported_only_for_the_current_sources(monkeypatch):
    recs = [p for p in os.listdir(os.path.join(ROOT, "profiles")) if p.startswith("traffic_")]
    assert recs, "a traffic record is committed under profiles/"
    with open(os.path.join(ROOT, "profiles", recs[0])) as fh:
        rec = json.load(fh)
    for key in ("kernel", "workload", "read_bytes_per_launch", "write_bytes_per_launch",
                "fetch_scale", "write_scale", "source_sha256", "commands"):
        assert key in rec, key
    monkeypatch.setattr(bench, "source_sha256", lambda: rec["source_sha256"])
    got = bench.measured_traffic(rec["kernel"], rec["workload"])
    assert got == rec["read_bytes_per_launch"] + rec["write_bytes_per_launch"]
    monkeypatch.setattr(bench, "source_sha256", lambda: "0" * 64)
    assert bench.measured_traffic(rec["kernel"], rec["workload"]) is None
    assert bench.measured_traffic("no such kernel", rec["workload"]) is None


def test_hbm_bytes_follow_the_per_kernel_formulas():
    """Route 2Td + 2dE + 4TE + 8Tk and combine 2Rd + 2Td (shared) + 2Td + 8R
    (236.6 MB and 2.35 GB at the large-shared layer)."""
    w = WORKLOADS["large_shared_train"]
    b = bench.hbm_bytes(w)
    assert b["route"] == 236_568_576
    assert b["combine"] == 2_349_858_816
    assert b["dw_router"] == 2 * w.T * w.d + 4 * w.T * w.E + 4 * w.d * w.E
    assert "reverse_combine" in b
    assert "reverse_combine" not in bench.hbm_bytes(WORKLOADS["large_shared"])


def test_expert_roofline_closed_forms():
    """Large experts are bound by their FLOPs, tiny ones by their weights,
    empty ones cost nothing."""
    w = WORKLOADS["many_experts"]
    big = 10 ** 6
    t = bench.expert_roofline_ms(w, [big])
    assert t == pytest.approx(1e3 * 6.0 * big * w.d * w.f / (bench.PEAK_BF16_TFLOPS * 1e12))
    t1 = bench.expert_roofline_ms(w, [1])
    assert t1 == pytest.approx(1e3 * (6.0 * w.d * w.f + 4.0 * w.d + 4.0 * w.f) / (bench.PEAK_HBM_GBS * 1e9))
    assert bench.expert_roofline_ms(w, [0, 0]) == 0.0
