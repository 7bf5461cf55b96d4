"""Host-side logic of bench.py: the one-GPU guard, rocprofv3 counter ingestion, and the
source hash that retires counters when a kernel's source or compile flags change."""

import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def _write_csv(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp",
                                          "End_Timestamp"])
        w.writeheader()
        for r in rows:
            w.writerow(r)


def _load(path):
    with open(path) as f:
        return json.load(f)


def _row(kernel, counter, value, t0=0, t1=1000):
    return {"Kernel_Name": kernel, "Counter_Name": counter, "Counter_Value": value, "Start_Timestamp": t0,
            "End_Timestamp": t1}


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_hbm_counters_scale_by_the_copy(tmp_path, monkeypatch):
    """Bytes per launch = mean counter value per dispatch x (copy bytes / the copy's counter)."""
    monkeypatch.setattr(bench, "COUNTERS", str(tmp_path / "hbm.json"))
    k_stats = "void tgvkv::(anonymous namespace)::score_stats_text_kernel<128, 1, 1>(tgvkv::Shape, ...)"
    k_dec = "void tgvkv::(anonymous namespace)::decode_kernel<128, 1, tgvkv::ContigRows<128> >(tgvkv::Shape)"
    fetch, write = tmp_path / "f.csv", tmp_path / "w.csv"
    _write_csv(fetch, [_row(k_stats, "FETCH_SIZE", 1000), _row(k_dec, "FETCH_SIZE", 100),
                       _row(k_dec, "FETCH_SIZE", 300)])
    _write_csv(write, [_row(k_stats, "WRITE_SIZE", 10), _row(k_dec, "WRITE_SIZE", 4), _row(k_dec, "WRITE_SIZE", 4)])
    cf, cw = tmp_path / "cf.csv", tmp_path / "cw.csv"
    _write_csv(cf, [_row("copy", "FETCH_SIZE", bench.COPY_BYTES // 2048), _row("fill", "FETCH_SIZE", 3)])
    _write_csv(cw, [_row("copy", "WRITE_SIZE", bench.COPY_BYTES // 1024)])
    bench.ingest_counters(str(fetch), str(write), str(cf), str(cw), workload="w", decode_steps=7)
    rec = _load(bench.COUNTERS)["w"]
    assert rec["score_text"]["fetch_bytes"] == pytest.approx(1000 * 2048)
    assert rec["score_text"]["write_bytes"] == pytest.approx(10 * 1024)
    assert rec["decode"]["bytes_per_launch"] == pytest.approx(200 * 2048 + 4 * 1024)  # mean over dispatches
    assert rec["decode"]["decode_steps"] == 7
    # the record is used only while the source hash matches, and for decode the step count too
    assert bench.traffic_for("score_text", "w") == pytest.approx(1000 * 2048 + 10 * 1024)
    assert bench.traffic_for("decode", "w", decode_steps=7) is not None
    assert bench.traffic_for("decode", "w", decode_steps=8) is None


def test_mfma_counters_and_their_reading(tmp_path, monkeypatch):
    """Per-launch means of the matrix-core counters, and the busy fraction with busy cycles
    summed over 1024 SIMDs and GPU-active cycles over 8 XCDs."""
    monkeypatch.setattr(bench, "MFMA_COUNTERS", str(tmp_path / "mfma.json"))
    k = "void tgvkv::(anonymous namespace)::score_vision_kernel<128, 4, 4, false>(tgvkv::Shape, int)"
    rows = []
    for counter, value in (("SQ_INSTS_MFMA", 1000), ("SQ_VALU_MFMA_BUSY_CYCLES", 16000),
                           ("GRBM_GUI_ACTIVE", 8 * 500), ("SQ_INSTS_VALU", 7000),
                           ("SQ_INSTS_VALU_TRANS_F32", 900)):
        rows.append(_row(k, counter, value, 0, 2000))
    path = tmp_path / "p.csv"
    _write_csv(path, rows)
    bench.ingest_mfma_counters(str(path), "w")
    rec = _load(bench.MFMA_COUNTERS)["w"]["score_vision"]
    assert rec["mfma_instrs"] == 1000 and rec["pmc_run_launch_ns"] == 2000
    assert bench.mfma_for("score_vision", "w") == rec
    summ = bench.mfma_summary(rec, launch_ms=0.002)
    # 16000 busy cycles over 1024 SIMDs x 500 cycles per XCD
    assert summ["mfma_busy_frac"] == pytest.approx(16000 / (1024 * 500), abs=1e-4)
    assert summ["issued_tflops"] == pytest.approx(1000 * 16384 / 2e-6 / 1e12, rel=1e-3)
    assert summ["valu_instrs_per_mfma"] == pytest.approx(7.0)


def test_source_hash_follows_sources_and_flags(monkeypatch):
    from paper_2606_03075_amd import build
    h_score = bench.source_hash(bench.KERNEL_SOURCES["score_text"])
    h_decode = bench.source_hash(bench.KERNEL_SOURCES["decode"])
    assert h_score != h_decode
    # the scoring sources compile with their own flags, and the hash sees them
    assert build.device_flags("score.hip") != build.device_flags("decode.hip")
    monkeypatch.setattr(build, "NO_IEEE_SOURCES", ())
    assert bench.source_hash(bench.KERNEL_SOURCES["score_text"]) != h_score
    assert bench.source_hash(bench.KERNEL_SOURCES["decode"]) == h_decode
