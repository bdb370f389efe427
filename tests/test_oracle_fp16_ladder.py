"""Pins for the oracle's fp16 rounding and ladder (CPU only)."""
import bisect
from fractions import Fraction

import numpy as np
import pytest

from oracle import fp16, ladder

# ---------------------------------------------------------------- fp16 rounding


def _all_finite_f16():
    bits = np.arange(0x10000, dtype=np.uint32).astype(np.uint16)
    vals = bits.view(np.float16).astype(np.float64)
    ok = np.isfinite(vals) & (bits != 0x8000)
    pairs = sorted((Fraction(float(v)), int(b)) for v, b in zip(vals[ok], bits[ok]))
    return [p[0] for p in pairs], [p[1] for p in pairs]


_F16_VALS, _F16_BITS = _all_finite_f16()


def _rne_bruteforce(x):
    """Nearest fp16 by exact rational comparison, ties to the even pattern
    (IEEE 754 roundTiesToEven), overflow to +-inf beyond the max + half ulp."""
    fx = Fraction(float(x))
    top = Fraction(65504) + Fraction(16)  # 65504 + half an ulp (32/2)
    if fx >= top:
        return 0x7C00
    if fx <= -top:
        return 0xFC00
    if fx > _F16_VALS[-1]:
        return _F16_BITS[-1]
    if fx < _F16_VALS[0]:
        return _F16_BITS[0]
    i = bisect.bisect_left(_F16_VALS, fx)
    if i < len(_F16_VALS) and _F16_VALS[i] == fx:
        return _F16_BITS[i]
    lo, hi = i - 1, i
    dl, dh = fx - _F16_VALS[lo], _F16_VALS[hi] - fx
    if dl < dh:
        b = _F16_BITS[lo]
    elif dh < dl:
        b = _F16_BITS[hi]
    else:
        b = _F16_BITS[lo] if _F16_BITS[lo] % 2 == 0 else _F16_BITS[hi]
    return 0 if b == 0x8000 else b


def test_fp16_direct_rounding_vectors():
    # 1 + 2^-11 + 2^-40 lies just above the midpoint: a single rounding gives 0x3C01,
    # a detour through fp32 (which drops the 2^-40) would give the even 0x3C00.
    assert fp16.from_f64(np.array([1 + 2.0 ** -11 + 2.0 ** -40]))[0] == 0x3C01
    assert fp16.from_f64(np.array([1 + 2.0 ** -11]))[0] == 0x3C00       # tie -> even
    assert fp16.from_f64(np.array([1 + 3 * 2.0 ** -11]))[0] == 0x3C02   # tie -> even
    assert fp16.from_f64(np.array([-0.0]))[0] == 0x0000                 # canonical zero
    assert fp16.from_f64(np.array([2.0 ** -25 + 2.0 ** -60]))[0] == 0x0001  # subnormal, above half
    assert fp16.from_f64(np.array([2.0 ** -25]))[0] == 0x0000           # tie -> even (zero)
    assert fp16.from_f64(np.array([65520.0]))[0] == 0x7C00              # rounds to inf


def test_fp16_matches_bruteforce_rne():
    r = np.random.default_rng(7)
    xs = np.concatenate([
        r.standard_normal(400) * 10.0 ** r.integers(-9, 5, 400),
        (r.integers(-2048, 2048, 200) + 0.5) * 2.0 ** r.integers(-24, 6, 200),  # exact ties
        np.array([5e-8, 6e-8, 6.1e-5, 6.104e-5, 65503.9, 65519.99, -65519.0]),
    ])
    got = fp16.from_f64(xs)
    for x, g in zip(xs, got):
        assert int(g) == _rne_bruteforce(x), (x, hex(int(g)), hex(_rne_bruteforce(x)))


# ---------------------------------------------------------------- ladder


def test_tiny_ladder_token_bands():
    lv = ladder.ladder("tiny", 2048)
    toks = {L: 64 * int((lv == L).sum()) for L in ladder.LEVELS}
    # newest 256 exact, next 512 int8, next 768 int4, oldest 512 int2
    assert toks == {16: 256, 8: 512, 4: 768, 2: 512, 1: 0, 0: 0}
    assert lv[-1] == 16 and lv[0] == 2


@pytest.mark.parametrize("T,expect", [
    (16384, (16, 60, 84, 71, 25)),
    (32768, (16, 124, 173, 148, 51)),
    (131072, (16, 508, 711, 609, 204)),
    (1048576, (16, 4092, 5728, 4910, 1638)),
])
def test_graded_ladder_bands(T, expect):
    lv = ladder.ladder("graded", T)
    got = tuple(int((lv == L).sum()) for L in (16, 8, 4, 2, 1))
    assert got == expect
    nb = len(lv)
    R = nb - 16
    # 25 / 35 / 40 % age bands of the non-exact blocks, oldest 10 % as centroids
    assert abs(got[1] - 0.25 * R) < 1 and abs(got[2] - 0.35 * R) < 2
    assert abs(got[4] - 0.10 * nb) < 1


def _rank(lv):
    return np.array([ladder.ORDER[int(x)] for x in lv])


@pytest.mark.parametrize("profile", ["tiny", "graded", "rdv2"])
def test_ladder_monotone_in_age_and_time(profile):
    prev = None
    for nb in range(1, 2600):
        lv = ladder.ladder(profile, nb * 64)
        rk = _rank(lv)
        # older blocks never hold a more precise level than newer ones
        assert np.all(np.diff(rk) >= 0), nb
        if prev is not None:
            # appending a block never promotes an existing block
            assert np.all(rk[:-1] <= prev), nb
        prev = rk


def test_ladder_separate_floors_would_promote():
    # the reason for cumulative floors: flooring 25 % and 35 % separately moves the
    # int4/int2 boundary by two blocks at R = 20 and would promote a block.
    def sep(nb):
        R = nb - 16
        n8, n4 = 25 * R // 100, 35 * R // 100
        return [16 + n8, 16 + n8 + n4]
    assert sep(36)[1] - sep(35)[1] == 2
    lv35, lv36 = ladder.ladder("graded", 35 * 64), ladder.ladder("graded", 36 * 64)
    assert np.all(_rank(lv36)[:-1] <= _rank(lv35))
