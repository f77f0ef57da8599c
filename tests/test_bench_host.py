"""Host logic of bench.py that runs without a GPU: the one-GPU contract, the
phase-stamp summary and the traffic records keyed to kernel sources."""
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 2
    assert "one MI355X" in r.stderr
    assert r.stdout.strip() == ""


def _tile_rows(launches, wgs, loop_ticks, epi_ticks, apart, mode=3, rows=100):
    out = []
    for k in range(launches):
        for w in range(wgs):
            t0 = k * apart + 10 * w
            t1 = t0 + loop_ticks + 7 * w
            t2 = t1 + epi_ticks + 5 * w
            out.append((t0, t1, t2, w | (mode << 32) | (rows << 40)))
    return np.array(out, dtype=np.int64)


def test_phase_stamp_summary_of_known_phases():
    # Three fused launches of four workgroups, 200 us apart: main loops of
    # 80 us plus 0.07 us per workgroup index, epilogues of 16 us plus 0.05 us.
    tile = _tile_rows(3, 4, 8000, 1600, 20000)
    rng = np.random.default_rng(3)
    tile = tile[rng.permutation(len(tile))]  # the summary sorts by start
    coop = np.zeros((4, 256, 6), np.int64)
    phases = np.array([0, 275, 301, 341, 578])  # product, reduction, update, barrier
    n_iter = 4
    for s in range(4):
        for i in range(n_iter - 1):
            coop[s, i, :5] = 587 * i + 3 * s + phases
    coop[0, 0, 5] = n_iter
    out = bench.summarize_phase_stamps(tile, coop)

    f = out["tile_fused"]
    assert f["launches"] == 3
    assert f["main_loop_us"] == pytest.approx(80.0 + 0.07 * 1.5)
    assert f["main_loop_max_us"] == pytest.approx(80.0 + 0.07 * 3)
    assert f["epilogue_us"] == pytest.approx(16.0 + 0.05 * 1.5)
    assert f["epilogue_max_us"] == pytest.approx(16.0 + 0.05 * 3)
    end = 30 + 8000 + 21 + 1600 + 15  # last workgroup's end within a launch
    assert f["span_us"] == pytest.approx(end * 0.01)
    assert f["gap_before_us_median"] == pytest.approx((20000 - end) * 0.01)

    c = out["cooperative"]
    assert c["iterations"] == n_iter
    assert c["product_us"] == pytest.approx(2.75)
    assert c["reduction_us"] == pytest.approx(0.26)
    assert c["update_us"] == pytest.approx(0.40)
    assert c["barrier_us"] == pytest.approx(2.37)
    assert c["iteration_us"] == pytest.approx(5.87)


def test_phase_stamp_summary_skips_store_and_few_column_launches():
    store = _tile_rows(2, 4, 8000, 900, 20000, mode=2)
    few = _tile_rows(2, 4, 800, 100, 20000, rows=5) + np.array([40000, 40000, 40000, 0])
    coop = np.zeros((4, 256, 6), np.int64)
    out = bench.summarize_phase_stamps(np.concatenate([store, few]), coop)
    assert "tile_fused" not in out and "cooperative" not in out


def test_traffic_records_follow_their_sources(monkeypatch):
    r = bench.hessian_roofline(262144, 4096, 4.0)
    assert r["achieved"] == pytest.approx(262144 * 4096 * 4096 / 4e-3 / 1e12)
    assert r["frac"] == pytest.approx(r["achieved"] / bench.BF16_MFMA_PEAK_TFLOPS)
    monkeypatch.setattr(bench, "kernel_sources_sha1",
                        lambda files=None: bench.HESSIAN_TRAFFIC["sources_sha1"])
    assert bench.hessian_roofline(262144, 4096, 4.0)["traffic"] == \
        bench.HESSIAN_TRAFFIC["bytes_per_launch"]
    monkeypatch.setattr(bench, "kernel_sources_sha1", lambda files=None: "0" * 40)
    assert bench.hessian_roofline(262144, 4096, 4.0)["traffic"] is None


def test_source_hashes_cover_the_kernel_files():
    a = bench.kernel_sources_sha1()
    b = bench.kernel_sources_sha1(bench.HESSIAN_SOURCES)
    assert len(a) == 40 and len(b) == 40 and a != b
