"""Host-side logic of bench.py (no GPU): the algorithmic work per kernel class that the roofline
divides by, the counter records it attaches only while the kernel source is unchanged, and the
refusal of more than one GPU."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
import workloads  # noqa: E402


def test_algorithmic_flops_of_the_gpt2s_workload():
    cfg, w = workloads.model_cfg(2), workloads.WORKLOADS[2]
    B, L = w["B"], w["L"]
    M = B * L
    assert bench.algorithmic_units("gemm_mlp_down", cfg, B, L) == (2.0 * M * 3072 * 768, "TFLOP/s", "mfma")
    assert bench.algorithmic_units("gemm_qkv", cfg, B, L)[0] == 2.0 * M * 768 * 2304
    assert bench.algorithmic_units("attention", cfg, B, L)[0] == 4.0 * B * L * L * 768
    # the vocabulary projection counts the rows it actually projects
    assert bench.algorithmic_units("gemm_vocab", cfg, B, L)[0] == 2.0 * M * 768 * 50257
    assert bench.algorithmic_units("gemm_vocab", cfg, B, L, rows=8192.5)[0] == 2.0 * 8192.5 * 768 * 50257
    assert bench.algorithmic_units("attention", cfg, B, L, rows=100)[0] == 4.0 * 100 * L * 768
    assert bench.algorithmic_units("layernorm", cfg, B, L) == (None, None, None)


def test_launch_rows_follow_the_compacted_loop():
    """Rows of the timed launches: every launch takes all B L rows, except the vocabulary
    projection (the still-masked rows of its step) and, in a trimmed loop, the last layer's
    attention, attention output and MLPs (the same rows)."""
    cfg = workloads.model_cfg(2, n_layers=3)
    B, L, T = 2, 8, 4
    M = B * L
    masked = [16, 12, 7, 3]                       # before steps 4, 3, 2, 1
    assert bench.launch_rows("gemm_mlp_up", cfg, B, L, T, 5, None, True) == M
    # vocabulary: one launch per step, wrapping into the next loop after T launches
    assert bench.launch_rows("gemm_vocab", cfg, B, L, T, 6, masked, False) == (16 + 12 + 7 + 3 + 16 + 12) / 6
    # three layers per step: launches 0, 1 take all rows; the last layer's GEMMs are a gated pair
    # (usual tiles, then 64-row tiles), of which the small-tile launch does the listed rows here
    assert bench.launch_rows("gemm_mlp_down", cfg, B, L, T, 8, masked, True) == (4 * M + 0 + 16 + 0 + 12) / 8
    assert bench.launch_rows("gemm_mlp_down", cfg, B, L, T, 6, masked, False) == M
    assert bench.launch_rows("gemm_qkv", cfg, B, L, T, 6, masked, True) == M
    # the attention has one listed-query launch per step
    assert bench.launch_rows("attention", cfg, B, L, T, 3, masked, True) == (2 * M + 16) / 3
    # above the gate the usual tiles do the rows
    big = [5000, 4000, 3000, 2000]
    assert bench.launch_rows("gemm_mlp_up", cfg, B, L, T, 4, big, True) == (2 * M + 5000 + 0) / 4


def _record(tmp_path, sha, cls="gemm_mlp_down"):
    (tmp_path / "profiles").mkdir()
    (tmp_path / "src.hip").write_bytes(b"kernel source\n")
    rec = {"kernel_class": cls, "workload": "gpt2s-mask-bf16", "source": "src.hip", "source_sha256": sha,
           "traffic_bytes_per_launch": 123.0}
    (tmp_path / "profiles" / "traffic_x.md").write_text("# t\n\ntraffic-json: " + json.dumps(rec) + "\n")


def test_traffic_record_only_while_the_source_is_unchanged(tmp_path, monkeypatch):
    import hashlib
    good = hashlib.sha256(b"kernel source\n").hexdigest()
    _record(tmp_path, good)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.recorded_traffic("gemm_mlp_down", "gpt2s-mask-bf16") == 123.0
    assert bench.recorded_traffic("gemm_mlp_up", "gpt2s-mask-bf16") is None
    # a record taken on one workload says nothing about another workload's launches
    assert bench.recorded_traffic("gemm_mlp_down", "gpt2s-mask-b128-bf16") is None
    (tmp_path / "src.hip").write_bytes(b"kernel source, edited\n")
    assert bench.recorded_traffic("gemm_mlp_down", "gpt2s-mask-bf16") is None


def test_committed_traffic_records_parse():
    for cls in ("gemm_mlp_down", "gemm_mlp_up"):
        t = bench.recorded_traffic(cls, "gpt2s-mask-bf16")
        assert t is None or 1e8 < t < 1e9, (cls, t)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in (r.stdout + r.stderr)
