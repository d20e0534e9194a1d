"""Host-side logic of bench.py: the size sweep's crossovers, the spread statistics of the timed
passes, and the single-GPU contract of the command line."""
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _pt(n, res, same, mapped):
    return {"N": n, "bytes": n * 8192, "resident_GBps": res, "resident_same_buffer_GBps": same, "mapped_GBps": mapped}


def test_size_crossovers_synthetic_curve():
    # rates rise with size to a plateau; a repeated buffer beats rotated ones until the 4th point
    pts = [_pt(256, 500, 480, 40), _pt(512, 1000, 1100, 45), _pt(1024, 3000, 3600, 50),
           _pt(2048, 6000, 6100, 55), _pt(4096, 7000, 7050, 56), _pt(8192, 7200, 7200, 56)]
    c = bench.size_crossovers(pts)
    assert c["resident_plateau_GBps"] == 7200
    assert c["dispatch"]["N"] == 2048                  # first rate >= half the plateau (3600); 3000 is below
    assert c["mall"]["N"] == 2048                      # from here on same-buffer <= 1.02 x rotated
    assert c["largest_repeat_gain"]["bytes"] == 1024 * 8192   # 3600 / 3000
    assert abs(c["largest_repeat_gain"]["same_buffer_over_rotated"] - 1.2) < 1e-12
    assert c["mapped_equals_resident"] is None


def test_size_crossovers_dispatch_threshold_and_mapped():
    pts = [_pt(256, 100, 100, 120), _pt(512, 3600, 3600, 50), _pt(1024, 7200, 7200, 50)]
    c = bench.size_crossovers(pts)
    assert c["dispatch"]["N"] == 512                   # exactly half the plateau counts
    assert c["mapped_equals_resident"]["N"] == 256     # host-mapped at least as fast as resident
    assert c["mall"]["N"] == 256                       # no point where the repeat beats rotation by > 2 %


def test_size_crossovers_no_mall_when_last_point_repeats_faster():
    pts = [_pt(256, 1000, 1000, 40), _pt(512, 2000, 2100, 40)]
    assert bench.size_crossovers(pts)["mall"] is None


def test_spread_statistics():
    ms = [3.0, 1.0, 2.0, 5.0, 4.0]
    s = bench.spread(ms)
    assert s["n"] == 5 and s["median"] == 3.0
    assert s["iqr"] == [2.0, 4.0]
    lo, hi = s["ci95_median"]
    assert 1.0 <= lo <= 3.0 <= hi <= 5.0
    assert bench.spread(ms) == s                       # the bootstrap is seeded
    assert s["ms_per_token"] == ms                     # the passes in the order they ran


def test_spread_single_pass():
    s = bench.spread([7.25])
    assert s["median"] == 7.25 and s["iqr"] == [7.25, 7.25] and s["ci95_median"] == [7.25, 7.25]


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr) or "1 GPU" in (r.stdout + r.stderr) or "single" in (r.stdout + r.stderr)


def test_oracle_threads_records_the_cap(monkeypatch):
    avail = len(os.sched_getaffinity(0))
    monkeypatch.delenv("OMP_NUM_THREADS", raising=False)
    assert bench.oracle_threads() == (avail, avail, None)
    if avail > 1:
        monkeypatch.setenv("OMP_NUM_THREADS", "1")
        assert bench.oracle_threads() == (1, avail, "OMP_NUM_THREADS=1")
    monkeypatch.setenv("OMP_NUM_THREADS", str(avail + 7))      # a cap above the cores is no cap
    assert bench.oracle_threads() == (avail, avail, None)


def test_size_crossovers_without_mapped_arm():
    pts = [{"N": n, "bytes": n * 8192, "resident_GBps": r, "resident_same_buffer_GBps": r}
           for n, r in ((256, 500), (512, 4000), (1024, 7000))]
    c = bench.size_crossovers(pts)
    assert c["dispatch"]["N"] == 512 and c["mapped_equals_resident"] == "not measured"


def test_probe_and_gemv_oracle_baselines_on_small_inputs():
    import synth
    buf = synth.grid_f32((1 << 16) + 3, seed=0, stream=1)
    r = bench.probe_cpu_baseline(buf)
    assert r["kind"] == "oracle" and r["sums_equal"] and r["value"] > 0 and r["single_thread"]["cores"] == 1
    assert r["cores"] >= 1 and r["cores_available"] >= r["cores"]
    W = [synth.normal16((64, 256), 0.02, "f16", seed=0, stream=5 + i) for i in range(3)]
    x = synth.normal16(256, 1.0, "f16", seed=0, stream=9)
    g = bench.gemv_cpu_baseline(W, x, "f16", 0.05, "three small matrices")
    assert g["value"] > 0 and g["single_thread"]["calls"] >= 1 and g["sample"].startswith("three small")


def test_measured_ceiling_second_denominator():
    rows = {"probe": {"resident_GBps": 7000.0, "roofline": {"achieved": 7000.0}},
            "gemv_f16": {"roofline": {"achieved": 3500.0}},
            "endpoints": {"GBps": {"resident": 1.0}}}
    pc = bench.measured_ceiling(7140.0, rows)
    assert pc["GBps"] == 7000.0 and pc["frac"] == 1.02
    assert rows["gemv_f16"]["frac_of_probe"] == 0.5
    assert "frac_of_probe" not in rows["probe"] and "frac_of_probe" not in rows["endpoints"]
    assert bench.measured_ceiling(7140.0, {"gemv_f16": {"roofline": {"achieved": 1.0}}}) is None
