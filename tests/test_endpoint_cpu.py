"""Endpoint selection (Alg. 2, Sec. 8.1) on the CPU: the oracle against the paper's Table 12 and
its theta-sensitivity statement, planted mistakes in the oracle caught by those pins, the library's
C selection against the oracle, and the page-residency query on real mappings."""
import importlib.util
import json
import mmap
import os

import numpy as np
import pytest

from oracle import endpoint as ep

from paper_2608_12114_amd import wsr

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLD = json.load(open(os.path.join(ROOT, "tests", "golden", "endpoint_policy.json")))
W = 1e9     # any working set: Table 12 gives path times, so rates are W / t


def rate(t_ms):
    return None if t_ms is None else W / (t_ms * 1e-3)


def table_case(row, theta, mod=ep):
    # a resident time of null is the GH200 set that exceeds device memory: a capacity limit
    excluded = ("resident",) if row["resident_ms"] is None else ()
    return mod.select_endpoint(W, rate(row["map_ms"]), rate(row["resident_ms"]), rate(row["copy_ms"]),
                               theta=theta, excluded=excluded)


# ---- pins of the oracle ----------------------------------------------------------------------

def pin_table12(mod):
    for row in GOLD["rows"]:
        assert table_case(row, GOLD["theta"], mod) == (row["rule"], row["by_tie"]), row["platform"]


def pin_theta_sweep(mod):
    lo, hi = GOLD["theta_sweep"]["lo"], GOLD["theta_sweep"]["hi"]
    for theta in np.linspace(lo, hi, 19):
        for row in GOLD["rows"]:
            assert table_case(row, float(theta), mod)[0] == row["rule"], (theta, row["platform"])


def pin_gh200_below_its_gap(mod):
    gh = [r for r in GOLD["rows"] if r["platform"].startswith("GH200")][0]
    gap = GOLD["gh200_gap_pct"] / 100
    assert table_case(gh, gap * 0.5, mod)[0] == GOLD["gh200_below_gap"]
    assert table_case(gh, 0.0, mod)[0] == "copy"


def pin_band_never_overrides_a_clear_resident_lead(mod):
    """Map is never chosen over a resident endpoint that is faster by more than theta."""
    rng = np.random.default_rng(0)
    for _ in range(2000):
        t = rng.uniform(1, 100, size=3)
        theta = float(rng.choice([0.0, 0.02, 0.05, 0.1, 0.2]))
        choice, _ = mod.select_endpoint(W, rate(t[0]), rate(t[1]), rate(t[2]), theta=theta)
        if t[0] > t[1] * (1 + theta) + 1e-9:
            assert choice != "map"
        assert choice in ep.ENDPOINTS
        # the choice is map or the fastest endpoint
        assert choice == "map" or t[ep.ENDPOINTS.index(choice)] == t.min()


def pin_stops_and_drops(mod):
    assert mod.select_endpoint(W, 1e9, 1e12, 1e9, mapped_resident=False)[0] == "storage-bound"
    # resident fastest by far, but its arm failed or evicted the mapping: copy beats map here
    assert mod.select_endpoint(W, 1e9, 1e12, 2e9, resident_ok=False)[0] == "copy"
    assert mod.select_endpoint(W, 1e9, 1e12, 2e9, excluded=("resident", "copy"))[0] == "map"
    assert mod.select_endpoint(W, None, None, None)[0] == "none"
    assert mod.select_endpoint(W, 5e10, 7e12, 5.5e10)[0] == "resident"


PINS = [pin_table12, pin_theta_sweep, pin_gh200_below_its_gap, pin_band_never_overrides_a_clear_resident_lead,
        pin_stops_and_drops]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_oracle_pin(pin):
    pin(ep)


MUTANTS = {
    "no_tie_band": ("survivors[\"map\"] - t_min <= theta * t_min", "survivors[\"map\"] - t_min <= 0 * t_min"),
    "band_on_wrong_side": ("survivors[\"map\"] - t_min <= theta * t_min", "t_min - survivors[\"map\"] <= theta * t_min"),
    "slowest_wins": ("fastest = min(survivors", "fastest = max(survivors"),
    "rate_not_time": ("return w_bytes / rate_bytes_per_s * 1e3", "return rate_bytes_per_s / w_bytes * 1e3"),
    "no_storage_stop": ("    if not mapped_resident:\n        return \"storage-bound\", False\n", ""),
    "resident_kept": ("        times[\"resident\"] = None\n", "        pass\n"),
    "exclusions_ignored": ("        times[e] = None\n", "        pass\n"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, tmp_path):
    find, repl = MUTANTS[name]
    src = open(ep.__file__).read()
    assert src.count(find) == 1, name
    path = tmp_path / f"endpoint_{name}.py"
    path.write_text(src.replace(find, repl))
    spec = importlib.util.spec_from_file_location(f"endpoint_{name}", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    caught = []
    for pin in PINS:
        try:
            pin(mod)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"no pin caught mutant {name}"


# ---- the library's selection against the oracle ------------------------------------------------

CODE = {"map": wsr.WSR_EP_MAP, "resident": wsr.WSR_EP_RESIDENT, "copy": wsr.WSR_EP_COPY,
        "storage-bound": wsr.WSR_EP_STORAGE_BOUND, "none": wsr.WSR_EP_NONE}
BIT = {"map": 1 << wsr.WSR_EP_MAP, "resident": 1 << wsr.WSR_EP_RESIDENT, "copy": 1 << wsr.WSR_EP_COPY}


def lib_select(w, b_map, b_res, b_copy, theta=0.05, mapped_resident=True, resident_ok=True, excluded=()):
    mask = sum(BIT[e] for e in excluded)
    return wsr.wsr_select_endpoint(w, b_map or 0.0, b_res or 0.0, b_copy or 0.0, theta, mapped_resident,
                                   resident_ok, mask)


def test_library_matches_table12():
    for row in GOLD["rows"]:
        excluded = ("resident",) if row["resident_ms"] is None else ()
        code, times = lib_select(W, rate(row["map_ms"]), rate(row["resident_ms"]), rate(row["copy_ms"]),
                                 excluded=excluded)
        assert code == CODE[row["rule"]], row["platform"]
        assert times[0] == pytest.approx(row["map_ms"]) and times[2] == pytest.approx(row["copy_ms"])


def test_library_matches_oracle_random():
    rng = np.random.default_rng(1)
    for _ in range(5000):
        w = float(rng.uniform(1e6, 3e11))
        rates = [None if rng.random() < 0.15 else float(w / rng.uniform(1e-3, 5.0)) for _ in range(3)]
        if rng.random() < 0.3:          # near-ties around the band
            rates[0] = rates[1] * float(rng.uniform(0.9, 1.1)) if rates[1] else rates[0]
        theta = float(rng.choice([0.0, 0.01, 0.02, 0.05, 0.1, 0.2]))
        mr, rok = bool(rng.random() > 0.05), bool(rng.random() > 0.1)
        exc = tuple(e for e in ep.ENDPOINTS if rng.random() < 0.1)
        want = ep.select_endpoint(w, *rates, theta=theta, mapped_resident=mr, resident_ok=rok, excluded=exc)[0]
        got, _ = lib_select(w, *rates, theta=theta, mapped_resident=mr, resident_ok=rok, excluded=exc)
        assert got == CODE[want], (w, rates, theta, mr, rok, exc)


def test_library_argument_checks():
    with pytest.raises(wsr.WsrError):
        wsr.wsr_select_endpoint(0.0, 1.0, 1.0, 1.0)
    with pytest.raises(wsr.WsrError):
        wsr.wsr_select_endpoint(1.0, 1.0, 1.0, 1.0, theta=-0.1)
    with pytest.raises(wsr.WsrError):
        wsr.wsr_select_endpoint(1.0, 1.0, 1.0, 1.0, excluded=1)       # bit 0 names no endpoint


# ---- page residency ----------------------------------------------------------------------------

def test_resident_pages_of_a_file_mapping(tmp_path):
    page = mmap.PAGESIZE
    path = tmp_path / "w.bin"
    path.write_bytes(os.urandom(64 * page))
    with open(path, "rb") as f:
        m = mmap.mmap(f.fileno(), 64 * page, prot=mmap.PROT_READ)
        a = np.frombuffer(m, dtype=np.uint8)
        assert int(a[::page].sum()) >= 0                 # fault every page in
        r, t = wsr.wsr_host_resident_pages(a.ctypes.data, a.nbytes)
        assert (r, t) == (64, 64)
        # an unaligned sub-range spans the pages it touches
        r, t = wsr.wsr_host_resident_pages(a.ctypes.data + 10, 2 * page)
        assert (r, t) == (3, 3)
        del a
        m.close()


def test_resident_pages_of_untouched_anonymous_memory():
    page = mmap.PAGESIZE
    m = mmap.mmap(-1, 32 * page)
    a = np.frombuffer(m, dtype=np.uint8)
    r, t = wsr.wsr_host_resident_pages(a.ctypes.data, a.nbytes)
    assert t == 32 and r == 0
    a[: 8 * page : page] = 1                              # write-fault the first 8 pages
    r, _ = wsr.wsr_host_resident_pages(a.ctypes.data, a.nbytes)
    assert r == 8
    del a
    m.close()


def test_resident_pages_rejects_unmapped_range():
    page = mmap.PAGESIZE
    m = mmap.mmap(-1, 4 * page)
    a = np.frombuffer(m, dtype=np.uint8)
    base = a.ctypes.data
    del a
    m.close()
    with pytest.raises(wsr.WsrError):
        wsr.wsr_host_resident_pages(base, 4 * page)
