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
