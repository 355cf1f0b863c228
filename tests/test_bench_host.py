"""Host-side logic of bench.py (no GPU): the algorithmic work it divides by
the measured launch times, the one-GPU guard, and the rule that a counter
record of HBM traffic is replayed only while its kernel's sources are
unchanged."""
import hashlib
import json
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from synth import make_inputs  # noqa: E402


def test_work_per_launch_matches_the_shapes():
    """Algorithmic FLOPs per launch, written out independently for a small
    shape: projections 2 x rows x out x in, the layer tail the O projection
    plus both FFN products, attention 4 x d per (query, visible key) pair
    with the candidate's own key counted."""
    inp = make_inputs([5, 0, 9], [4, 3, 0], 64, 2, 1, 256, dtype="bf16", seed=0)
    R, d, F = 7, 64, 256
    pairs = 4 * (5 + 1) + 3 * (0 + 1) + 0 * (9 + 1)
    w = bench.kernel_work(inp)
    assert w["rank.gemm_qkv"] == ("mfma", 2.0 * R * (3 * d) * d)
    assert w["rank.oproj_ffn"] == ("mfma", 2.0 * R * d * d + 2.0 * R * F * d + 2.0 * R * d * F)
    assert w["rank.attn"] == ("mfma", 4.0 * d * pairs)
    # tokens read and LN1 written, two bytes each, for a bf16 model
    assert w["rank.init_ln1"] == ("hbm", R * d * 4.0)
    # the whole step: L layers of q|k|v (3d^2), O (d^2), FFN (2dF) per row,
    # attention, and the score head's dot product
    flops = 1 * (R * 2.0 * (3 * d * d + d * d + 2 * d * F) + 4.0 * d * pairs) + 2.0 * d * R
    assert bench.path_flops(inp) == flops


def test_headline_work_figures():
    """The headline shape (64 users x 2000 candidates over 1024-row
    histories, d 512, d_ff 2048): 201 GFLOP for q|k|v, 604 for the tail and
    269 for attention per layer."""
    inp = make_inputs([1024] * 2, [2000] * 2, 512, 8, 1, 2048, dtype="bf16", seed=0)
    w = bench.kernel_work(inp)
    scale = 32   # 2 of 64 users drawn here
    assert abs(w["rank.gemm_qkv"][1] * scale - 201.326592e9) < 1e3
    assert abs(w["rank.oproj_ffn"][1] * scale - 603.979776e9) < 1e3
    assert abs(w["rank.attn"][1] * scale - 268.6976e9) < 1e3


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert p.returncode == 2
    assert "one GPU" in p.stderr and p.stdout == ""


def test_traffic_record_needs_unchanged_sources(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_text("// kernel source\n")
    sha = hashlib.sha1(src.read_bytes()).hexdigest()[:12]
    (tmp_path / "profiles").mkdir()
    rec = {"sources": ["k.hip"], "source_sha1": sha, "hbm_read_bytes": 100.0, "hbm_write_bytes": 50.0,
           "fetch_factor": 0.5, "write_factor": 1.0}
    (tmp_path / "profiles" / "traffic.json").write_text(json.dumps({"w": {"attn": rec}}))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("rank.attn", "w") == 150
    assert "x2.000 and x1.000" in bench.traffic_provenance("rank.attn", "w")
    assert bench.measured_traffic("rank.attn", "other_workload") is None
    src.write_text("// kernel source, edited\n")
    assert bench.measured_traffic("rank.attn", "w") is None
