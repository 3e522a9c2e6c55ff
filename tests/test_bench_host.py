"""Host logic of bench.py that needs no GPU: the critical-path model behind
the stage-pipelined passes' latency roofline."""
import numpy as np

import bench


def test_pipeline_depth():
    # register pass: two stages per wave above 16 stages, one below
    assert bench.pipeline_depth(1, 32) == 16
    assert bench.pipeline_depth(1, 12) == 12
    # grid pass: one position per stage
    assert bench.pipeline_depth(3, 64) == 64


def test_latency_roofline_counts_critical_hops():
    # two instances of the register pass (S = 32, depth 16): searches are one
    # per augmentation (column 0), iterations summed over searches (column 1)
    stats = np.zeros((2, 10), dtype=np.int64)
    stats[0, 0], stats[0, 1] = 10, 50  # 10 searches of 5 iterations
    stats[1, 0], stats[1, 1] = 12, 48  # 12 searches of 4 iterations
    hand = {"lds_wave_ns": 100.0, "device_neighbour_ns": 500.0, "device_same_xcd_ns": 300.0}
    r = bench.latency_roofline(1, stats, 32, 1e-3, hand, None, "k")
    hops0 = 10 * 15 + 2 * (50 - 10)  # (H - 1) per search + 2 per later iteration
    hops1 = 12 * 15 + 2 * (48 - 12)
    assert r["bound"] == "latency"
    assert r["model"]["critical_hops"] == max(hops0, hops1)
    assert abs(r["achieved"] - max(hops0, hops1) / 1e-3) < 1e-6
    assert abs(r["peak"] - 1e9 / 100.0) < 1e-6
    assert abs(r["frac"] - max(hops0, hops1) * 100e-9 / 1e-3) < 1e-12


def test_latency_roofline_grid_uses_search_count_and_device_handoff():
    stats = np.zeros((1, 10), dtype=np.int64)
    stats[0, 0], stats[0, 1], stats[0, 8] = 40, 120, 25  # 40 paths from 25 searches
    hand = {"lds_wave_ns": 100.0, "device_neighbour_ns": 500.0, "device_same_xcd_ns": 300.0}
    r = bench.latency_roofline(3, stats, 64, 2e-3, hand, None, "k")
    assert r["model"]["critical_hops"] == 25 * 63 + 2 * (120 - 25)
    assert r["model"]["hop_floor_ns"] == 500.0


def test_latency_roofline_without_calibration():
    stats = np.ones((1, 10), dtype=np.int64)
    hand = {"lds_wave_ns": -1.0, "device_neighbour_ns": -1.0, "device_same_xcd_ns": -1.0}
    r = bench.latency_roofline(1, stats, 32, 1e-3, hand, None, "k")
    assert r["frac"] is None and r["bound"] == "latency"
