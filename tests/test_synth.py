"""The seeded input generators: determinism, random access, encoders, distributions."""
from fractions import Fraction

import numpy as np
import pytest
from scipy import stats

import synth


def test_counter_random_access_and_threads():
    a = synth.normal16((64, 100), 0.02, "bf16", seed=0, stream=3, threads=1)
    b = synth.normal16((64, 100), 0.02, "bf16", seed=0, stream=3, threads=8)
    assert np.array_equal(a, b)
    # any row (odd start element included) regenerates on its own
    for r in (0, 1, 17, 63):
        row = synth.normal16(100, 0.02, "bf16", seed=0, stream=3, e0=r * 100)
        assert np.array_equal(row, a[r])
    odd = synth.normal16(7, 0.02, "bf16", seed=0, stream=3, e0=101)
    assert np.array_equal(odd, a.ravel()[101:108])
    # streams and seeds are distinct
    assert not np.array_equal(a, synth.normal16((64, 100), 0.02, "bf16", seed=0, stream=4))
    assert not np.array_equal(a, synth.normal16((64, 100), 0.02, "bf16", seed=1, stream=3))


def test_q4_and_scales_rows():
    full = synth.q4_codes(10, 64, seed=0, stream=5)
    part = synth.q4_codes(3, 64, seed=0, stream=5, row0=4)
    assert np.array_equal(full[4:7], part)
    s = synth.q4_scales(10, 64, seed=0, stream=6)
    assert np.array_equal(s[4:7], synth.q4_scales(3, 64, seed=0, stream=6, row0=4))
    sv = s.view(np.float16).astype(np.float64)
    assert sv.min() >= 0.005 - 1e-5 and sv.max() <= 0.02


def _rne_exact(v: float, mbits: int, bias: int) -> float:
    """Round-to-nearest-even by exact rational arithmetic (finite results only)."""
    if v == 0:
        return 0.0
    a = Fraction(abs(v))
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    ulp_e = max(e - mbits, 1 - bias - mbits)
    q = a / Fraction(2) ** ulp_e
    fl = q.numerator // q.denominator
    rem = q - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    r = float(fl * Fraction(2) ** ulp_e)
    return -r if v < 0 else r


def _edge_values():
    rng = np.random.default_rng(0)
    v = list(rng.standard_normal(20000) * np.exp2(rng.integers(-30, 20, 20000)))
    v += [0.0, -0.0, 1.0, -1.0, 65504.0, 65519.99, 65520.0, 1e6, 2.0 ** -24, 2.0 ** -25,
          2.0 ** -25 * 1.0000001, 2.0 ** -14, 2.0 ** -14 * (1 - 2 ** -11), 3 * 2.0 ** -26,
          1 + 2.0 ** -11, 1 + 3 * 2.0 ** -11, 1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, 0.1, 1e-40, 3e38, 3.4e38]
    return np.array(v, dtype=np.float64)


def test_f16_encoder_matches_numpy():
    v = _edge_values()
    got = synth.encode16(v, "f16")
    with np.errstate(over="ignore"):        # the overflow-to-infinity cases are intended
        want = v.astype(np.float16).view(np.uint16)
    assert np.array_equal(got, want)


def test_bf16_encoder_matches_exact_rounding():
    v = _edge_values()
    got = synth.encode16(v, "bf16").astype(np.uint32) << 16
    gotf = got.view(np.float32).astype(np.float64)
    for a, g in zip(v, gotf):
        if abs(a) < 3.3e38:
            assert g == _rne_exact(float(a), 7, 127), a
    # ties: 1 + 2^-8 is halfway between 1 and 1 + 2^-7 -> even (1); 1 + 3*2^-8 -> 1 + 2^-6
    assert synth.encode16([1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8], "bf16").tolist() == [0x3F80, 0x3F82]


def test_grid_values():
    x = synth.grid_f32(1 << 16, seed=0, stream=1)
    assert x.min() >= -1.0 and x.max() < 1.0
    assert np.all(x.astype(np.float64) * 2 ** 23 == np.round(x.astype(np.float64) * 2 ** 23))
    assert abs(x.mean()) < 0.01


def _implied_probabilities(fmt, sigma):
    q, alias = synth.table_arrays(fmt, sigma)
    cap = float(1 << 48)
    spill = np.bincount(alias, weights=cap - q.astype(np.float64), minlength=65536)
    return (q.astype(np.float64) + spill) / 2.0 ** 64


def _rounded_normal_mass(fmt, sigma):
    """Independent: scipy's normal CDF over the interval of reals that rounds to each code."""
    codes = np.arange(0x7C00 if fmt == "f16" else 0x7F80, dtype=np.uint32).astype(np.uint16)
    if fmt == "f16":
        v = codes.view(np.float16).astype(np.float64)
    else:
        v = (codes.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    mid = 0.5 * (v[1:] + v[:-1])
    lo = np.concatenate([[0.0], mid]) / sigma
    hi = np.concatenate([mid, [np.inf]]) / sigma
    p = stats.norm.sf(lo) - stats.norm.sf(hi)
    p[0] *= 2.0                       # +0 owns (-h, h)
    full = np.zeros(65536)
    full[: codes.size] = p
    full[0x8001: 0x8000 + codes.size] = p[1:]
    return full


@pytest.mark.parametrize("fmt,sigma", [("f16", 1.0), ("f16", 0.02), ("bf16", 1.0), ("bf16", 0.02)])
def test_sampling_table_matches_rounded_normal(fmt, sigma):
    got = _implied_probabilities(fmt, sigma)
    want = _rounded_normal_mass(fmt, sigma)
    assert abs(got.sum() - 1.0) < 1e-12
    assert np.all(np.abs(got - want) <= 1e-14 + 1e-6 * want)
    assert got[0x7C00:0x8000].sum() == 0 and got[0xFC00:].sum() == 0 if fmt == "f16" else True


def test_normal_draws_follow_the_table():
    n = 4_000_000
    a = synth.normal16(n, 0.02, "f16", seed=0, stream=11)
    p = _implied_probabilities("f16", 0.02)
    counts = np.bincount(a, minlength=65536)
    big = p * n > 50                                   # chi-square over well-populated codes
    chi2 = float((((counts[big] - n * p[big]) ** 2) / (n * p[big])).sum())
    dof = int(big.sum()) - 1
    assert stats.chi2.sf(chi2, dof) > 1e-4, (chi2, dof)
    w = a.view(np.float16).astype(np.float64)
    assert abs(w.mean()) < 1e-4 and abs(w.std() - 0.02) < 1e-4
    one = synth.lib().synth_normal16_one(synth.table("f16", 0.02).ctypes.data, 0, 11, 12345)
    assert one == a[12345]


def test_int4_uniform():
    c = synth.q4_codes(1000, 64, seed=0, stream=2)
    codes = np.concatenate([c & 0xF, c >> 4]).ravel()
    counts = np.bincount(codes, minlength=16)
    assert counts.min() > 0.9 * codes.size / 16 and counts.max() < 1.1 * codes.size / 16


def test_int8_uniform_and_rows():
    c = synth.i8_codes(2000, 128, seed=0, stream=3)
    counts = np.bincount(c.view(np.uint8).ravel(), minlength=256)
    assert counts.min() > 0.85 * c.size / 256 and counts.max() < 1.15 * c.size / 256
    assert c.min() == -128 and c.max() == 127
    part = synth.i8_codes(3, 128, seed=0, stream=3, row0=7)
    assert np.array_equal(c[7:10], part)
    assert synth.int8(0, 3, 7 * 128 + 5) == c[7, 5]
    s = synth.i8_scales(500, seed=0, stream=4).view(np.float16).astype(np.float64)
    assert s.min() >= synth.I8_SCALE_LO * (1 - 2 ** -10) and s.max() <= synth.I8_SCALE_HI
