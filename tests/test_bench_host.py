"""bench.py's host-side parts (no GPU): the algorithmic byte counts against
the sizes of the five workloads, the roofline peak from the unit counts, the
traffic records and their source hashes, and the one-GPU guard."""
import os
import subprocess
import sys

import numpy as np

import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_algorithmic_bytes_of_the_fused_workloads():
    # x, delta (B,D,L) + B, C (B,L,N) in the input dtype, A (D,N) and Dskip (D)
    # fp32, y (B,D,L) and h_last (B,D,N) fp32: the sizes of the workloads
    expect = {
        "selective_f32_b2_d256_n16_l512": 3_326_976,
        "selective_bf16_b8_d1536_n16_l2048": 203_266_048,
        "selective_f32_b1_d5120_n16_l65536": 4_035_596_288,
        "selective_f32_b4_d2048_n16_l8192_stress": 810_164_224,
    }
    for name, nbytes in expect.items():
        assert bench.algorithmic_bytes(wl.workload(name)) == nbytes, name


def test_roofline_peaks_are_the_published_ones():
    # the line's roofline is HBM-bound against 8 TB/s; the fp32 arithmetic is
    # reported beside it against the fp32 vector peak, 157.3 TFLOP/s
    # (256 CUs x 4 SIMDs x 32 lanes x 2 flops per FMA x 2.4 GHz)
    assert bench.HBM_PEAK_GBS == 8000.0
    assert abs(bench.FP32_PEAK_TFLOPS - 256 * 4 * 32 * 2 * 2.4e9 / 1e12) < 0.1
    # mul, mul, FMA, FMA per element; the exp2 is not a flop
    assert bench.FLOP_PER_ELEM == 6.0


def test_default_workload_is_the_largest_single_gpu_one():
    w = wl.workload(bench.DEFAULT_WORKLOAD)
    fused = [wl.workload(n) for n in wl.WORKLOADS if wl.workload(n).path != "affine"]
    assert w.elems == max(v.elems for v in fused)
    assert (w.B, w.D, w.N, w.L, w.dtype) == (1, 5120, 16, 65536, "f32")


def test_traffic_records_match_their_sources_and_workloads():
    for name, rec in bench.TRAFFIC_RECORDS.items():
        w = wl.workload(name)
        path = os.path.join(ROOT, "profiles", rec)
        assert os.path.exists(path), rec
        text = open(path).read()
        t = bench.measured_traffic(w)
        if f"kernel_source_sha256: {bench.kernel_source_sha256(w.path)}" not in text:
            assert t is None, rec  # a record taken on other sources is not reported
            continue
        alg = 12 * w.elems if w.path == "affine" else bench.algorithmic_bytes(w)
        # every algorithmic byte moves at least once, and not many twice
        assert t is not None and alg <= t <= 1.2 * alg, (rec, t, alg)
    for name, rec in bench.BWD_TRAFFIC_RECORDS.items():
        w = wl.workload(name)
        path = os.path.join(ROOT, "profiles", rec)
        assert os.path.exists(path), rec
        text = open(path).read()
        t = bench.measured_traffic(w, bwd=True)
        if f"kernel_source_sha256: {bench.kernel_source_sha256('bwd')}" not in text:
            assert t is None, rec
            continue
        # every gradient and input moves at least once; on top, the tile
        # checkpoints (B*D*L/8*16 fp32) are read and the per-workgroup shares of
        # dB and dC (B * D/16 * L * 16 fp32 each) written and read back
        es = 2 if w.dtype == "bf16" else 4
        alg = (3 * es + 8) * w.B * w.D * w.L + (2 * es + 8) * w.B * w.L * w.N
        extra = 4 * w.B * w.D * w.L * 2 + 2 * 2 * 4 * w.B * (w.D // 16) * w.L * 16
        assert t is not None and alg <= t <= 1.2 * (alg + extra), (rec, t, alg, extra)
    # no record for a workload without one, and the hashes differ by path
    assert bench.measured_traffic(wl.workload("selective_f32_b2_d256_n16_l512")) is None
    assert bench.measured_traffic(wl.workload("selective_f32_b2_d256_n16_l512"), bwd=True) is None
    assert bench.kernel_source_sha256("affine") != bench.kernel_source_sha256("selective")
    assert bench.kernel_source_sha256("bwd") != bench.kernel_source_sha256("selective")


def test_launch_stats_fields():
    st = bench.launch_stats(100e-6, np.array([101e-6, 99e-6, 100e-6]))
    assert abs(st["mean"] - 100.0) < 1e-9
    assert abs(st["median"] - 100.0) < 1e-9
    assert st["spread_launches"] == 3


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr


def test_launch_stats_of_graph_replays():
    st = bench.launch_stats(5e-6, np.array([5.1e-6, 4.9e-6]), graph=True)
    assert st["spread_replays"] == 2 and "spread_launches" not in st
    assert "graph" in st["method"]


def test_graph_backward_is_refused():
    # the backward allocates a workspace per call: no graph capture
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--graph", "--pass",
                          "bwd", "--no-cpu"], capture_output=True, text=True, timeout=300)
    assert res.returncode == 2
    assert "cannot be captured" in res.stderr
