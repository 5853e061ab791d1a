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
    # auto: row-major only for one token under 6144 rows and two tokens under about 12 M elements
    assert not bench.weight_tiled("auto", 1, 5120, 3072)   # Llama-3.2-3B QKV
    assert not bench.weight_tiled("auto", 1, 2560, 9728)   # Qwen3-4B Down: wide K, few rows
    assert bench.weight_tiled("auto", 1, 6144, 2560)       # Qwen3-4B QKV
    assert bench.weight_tiled("auto", 1, 8192, 3072)
    assert bench.weight_tiled("auto", 1, 19456, 2560)      # Qwen3-4B gate/up
    assert bench.weight_tiled("auto", 1, 128256, 3072)     # Llama-3.2-3B LM head
    assert not bench.weight_tiled("auto", 2, 2560, 4096)   # Qwen3-4B O: 10.5 M elements
    assert bench.weight_tiled("auto", 2, 5120, 2560)       # 13.1 M elements
    assert bench.weight_tiled("auto", 2, 2560, 9728)       # Qwen3-4B Down at two tokens
    assert bench.weight_tiled("auto", 3, 2560, 2560)
    assert bench.weight_tiled("tiled", 1, 8, 8)
    assert not bench.weight_tiled("row-major", 512, 5120, 3072)


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


class _FakeSp:
    SPLITEE_PREC_F32, SPLITEE_PREC_BF16, SPLITEE_PREC_BF16X3 = 0, 1, 2
    PRECS = {"f32": 0, "bf16": 1, "bf16x3": 2}


class _FakePath:
    def __init__(self, M, step_masks, projs, layers):
        self.projs, self.M, self.step_masks, self.layers_per_step = projs, M, step_masks, layers
        self.w_dtype, self.layout, self.tiled, self.nsets, self.row0 = "bf16", "tiled", [True] * len(projs), 1, 0

    def gemm_bytes(self):
        return [2.0 * p.N * p.K + (8.0 if self.step_masks else 4.0) * self.M * p.K + 8.0 * self.M * p.N
                for p in self.projs]


def test_leg_summary_picks_the_dominant_launch_and_the_whole_step():
    import workloads as WL
    projs = WL.QWEN3_4B.projections()
    path = _FakePath(1024, False, projs, 36)
    us = [100.0, 80.0, 300.0, 160.0]
    head, roof = bench.leg_summary(_FakeSp, path, 30.0, us, [20.0, 25.0, 20.0, 60.0], 2, "none")
    assert roof["kernel"].startswith("gate_up") and roof["bound"] == "mfma"
    fl = 2.0 * 1024 * 19456 * 2560
    assert roof["achieved"] == round(fl / 300e-6 / 1e12, 1)
    assert roof["mfma_issued_frac"] == round(3 * fl / 300e-6 / 1e12 / 2500.0, 4)
    step_fl = 36 * sum(2.0 * 1024 * p.N * p.K for p in projs)
    assert roof["step"]["achieved"] == round(step_fl / 30e-3 / 1e12, 1)
    assert roof["step"]["noise_mask_share"] == round(36 * 125.0 / 30e3, 4)
    assert head["value"] == round(step_fl / 30e-3 / 1e12, 3)
    # decode: bandwidth-bound, one mask launch per step
    dpath = _FakePath(1, True, projs, 36)
    _, droof = bench.leg_summary(_FakeSp, dpath, 1.8, [9.0, 7.0, 20.0, 13.0], [30.0], 2, "none")
    assert droof["bound"] == "hbm" and droof["step"]["bound"] == "hbm"
    assert droof["achieved"] == round(dpath.gemm_bytes()[2] / 20e-6 / 1e9, 1)
    assert droof["step"]["noise_mask_share"] == round(30.0 / 1800.0, 4)
