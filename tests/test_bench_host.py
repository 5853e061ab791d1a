"""Host logic of bench.py (CPU only): the one-GPU contract, the per-projection weight
layout and the reading of the rocprofv3 traffic summaries."""
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stdout + r.stderr


def test_weight_layout_rule():
    # auto: row-major only for one or two tokens of matrices under 16384 rows
    assert not bench.weight_tiled("auto", 1, 6144)
    assert not bench.weight_tiled("auto", 2, 16383)
    assert bench.weight_tiled("auto", 1, 19456)      # Qwen3-4B gate/up
    assert bench.weight_tiled("auto", 1, 128256)     # Llama-3.2-3B LM head
    assert bench.weight_tiled("auto", 3, 2560)
    assert bench.weight_tiled("tiled", 1, 8)
    assert not bench.weight_tiled("row-major", 512, 5120)


def _summary(tmp_path, sha, rows):
    d = tmp_path / "profiles"
    d.mkdir(exist_ok=True)
    lines = ["# HBM traffic", "source-sha256: %s" % sha, "",
             "| launch | kernel | grid | dispatches | FETCH_SIZE KiB | WRITE_SIZE KiB | traffic bytes | algorithmic bytes |",
             "|---|---|---|---|---|---|---|---|"]
    lines += ["| %s | k | 1 | 1 | 1.0 | 1.0 | %d | 1 |" % (n, v) for n, v in rows]
    (d / "traffic_w_bf16x3_tiled.md").write_text("\n".join(lines) + "\n")


def test_traffic_summary_read_only_while_sources_match(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "gemm_source_sha", lambda: "abc")
    names = ["qkv", "o"]
    assert bench.measured_traffic("w", "bf16x3", "tiled", names) is None       # no summary
    _summary(tmp_path, "abc", [("qkv", 100), ("o", 50)])
    assert bench.measured_traffic("w", "bf16x3", "tiled", names) == {"qkv": 100.0, "o": 50.0}
    assert bench.measured_traffic("w", "bf16x3", "tiled", names + ["down"]) is None  # a launch missing
    _summary(tmp_path, "stale", [("qkv", 100), ("o", 50)])
    assert bench.measured_traffic("w", "bf16x3", "tiled", names) is None       # kernels changed since
