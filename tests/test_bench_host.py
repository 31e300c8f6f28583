"""Host-side logic of bench.py (no GPU): the one-GPU guard, the issue-bound peak of the score
passes, the compression roofline, the source hash that ties stored counters to the code, and the
traffic summary's calibration arithmetic."""
import json
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr + r.stdout


def test_score_issue_peak():
    # MFMA 2d flops at 2.5 PFLOP/s, then one exp2 (8 lanes per SIMD cycle) and fma + add (16 lanes
    # per SIMD cycle each) on 256 CUs x 4 SIMDs at 2.4 GHz: 2.04e-13 s per logit at d = 128, so
    # the vector work of a 16x16x32 MFMA's 64 logits (16 cycles) equals the MFMA's own 16 cycles
    t = bench.score_logit_seconds(128, "bf16")
    simd_hz = 256 * 4 * 2.4e9
    assert t == pytest.approx(256 / 2.5e15 + 1 / (8 * simd_hz) + 2 / (16 * simd_hz), rel=1e-12)
    assert 2 * 128 / t / 1e12 == pytest.approx(1254.1, abs=0.1)
    assert 2.5e15 / (2 * 128 / t) == pytest.approx(2.0, rel=0.01)


def test_compression_roof_of_the_128k_layer():
    # 128K prompt, batch 8, 28/4 heads, d 128, w 64, bf16, a 25 % layer (T = 4 * 32768 rows):
    # MFMA 2*28*64*128*131072*8 flops = 481 GFLOP at 2.5 PFLOP/s = 192 us; HBM per sequence
    # 2*(4*131072*128 + 4*131072*128) + 4*131072 + 2*28*64*128 bytes = 269.4 MB over 8 TB/s
    roof, roof2 = bench.compress_roof_seconds(8, 131072, 28, 4, 128, 64, 2, 131072.0, "bf16")
    hbm = 8 * (2 * (4 * 131072 * 128 + 4 * 131072 * 128) + 4 * 131072 + 2 * 28 * 64 * 128)
    assert roof == pytest.approx(hbm / 8e12, rel=1e-12)
    assert roof * 1e6 == pytest.approx(269.4, abs=0.1)
    # computing the window LSE too: the GEMM twice (384.8 us) against K read twice (403.6 us)
    k = 8 * 2 * 4 * 131072 * 128
    assert roof2 == pytest.approx(max(2 * 8 * 2 * 28 * 64 * 128 * 131072 / 2.5e15, (hbm + k) / 8e12), rel=1e-12)
    assert roof / roof2 == pytest.approx(0.6675, abs=1e-4)
    assert bench.percentile([5, 1, 4, 2, 3], 0.5) == 3 and bench.percentile([1, 2], 0.1) == pytest.approx(1.1)


def test_source_hash_ignores_comments_but_not_code(tmp_path, monkeypatch):
    csrc = tmp_path / "paper_2609_03235_amd" / "csrc"
    shutil.copytree(os.path.join(ROOT, "paper_2609_03235_amd", "csrc"), csrc,
                    ignore=shutil.ignore_patterns("*.o", "_build"))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    base = bench.source_sha("gather")
    src = csrc / "select_kernels.hip"
    text = src.read_text()
    src.write_text("// a new comment\n/* and a block\n   comment */\n" + text.replace("\n", "\n\n", 3))
    assert bench.source_sha("gather") == base
    assert bench.source_sha("score_colsum") == bench.source_sha("score_lse")
    assert "constexpr int U = 8;" in text
    src.write_text(text.replace("constexpr int U = 8;", "constexpr int U = 4;", 1))
    assert bench.source_sha("gather") != base


def _csv(path, counter, rows):
    with open(path, "w") as fh:
        fh.write("Dispatch_Id,Kernel_Name,Counter_Name,Counter_Value\n")
        for i, (name, v) in enumerate(rows):
            fh.write(f'{i + 1},"{name}",{counter},{v}\n')


def test_traffic_summary_scales_by_the_copy(tmp_path, monkeypatch):
    mib = 8
    kib = mib * 1024.0
    fill = "void at::native::vectorized_elementwise_kernel<4, at::native::FillFunctor<float>>(int)"
    copy = "void at::native::vectorized_elementwise_kernel<4, at::native::AUnaryFunctor<MulFunctor<float>>>(int)"
    gather = "void sgdkv::copy_rows_kernel<256>(sgdkv::CompressArgs)"
    # the three copies move kib each: FETCH_SIZE counts half of it, WRITE_SIZE all of it; a later
    # multiplication (input generation) and a large fill must not count
    _csv(tmp_path / "f.csv", "FETCH_SIZE", [(fill, 0.0), (copy, kib / 2), (copy, kib / 2 + 2), (copy, kib / 2 + 3),
                                            (copy, 3 * kib), (fill, 4 * kib), (gather, 100.0), (gather, 102.0)])
    _csv(tmp_path / "w.csv", "WRITE_SIZE", [(fill, kib), (copy, kib), (copy, kib), (copy, kib),
                                            (copy, 9 * kib), (fill, 4 * kib), (gather, 50.0), (gather, 50.0)])
    out = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "traffic_path", lambda wl, r, w: str(out))
    args = type("A", (), dict(calibrate_copy_mib=mib, workload="tiny", ratio=0.25, obs_window=0))()
    bench.summarize_traffic(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), args)
    d = json.loads(out.read_text())
    ff = kib / (kib / 2 + 2)  # median of the three copies' fetch
    assert d["calibration"]["fetch_factor"] == pytest.approx(ff)
    assert d["calibration"]["write_factor"] == pytest.approx(1.0)
    g = d["kernels"]["gather"]
    assert g["dispatches"] == 2
    assert g["hbm_bytes_per_launch"] == round(1024 * (101.0 * ff + 50.0))
    assert set(d["kernels"]) == {"gather"}
