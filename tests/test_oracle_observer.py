"""Pins for the oracle's causal mass observer, EMA and analytic allocation
(CPU only)."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import fp16, observer
from paper_2608_23599_amd import synth


def _qk(seed, n_obs, G, T):
    k, _ = synth.kv_unit(300 + seed, 0, 0, T)
    q = synth.queries(300 + seed, n_obs, G).reshape(n_obs, G, 128)
    return q, k


def test_masses_sum_to_one():
    q, k = _qk(1, 5, 3, 700)
    m = observer.observe_mass(q, k)
    assert m.shape == (11,)
    assert abs(m.sum() - 1.0) < 1e-12 and np.all(m >= 0)


def test_equal_keys_give_visible_token_shares():
    """All keys equal: each query spreads its mass evenly over the keys it sees,
    so a block's mass is the mean over queries of (its visible tokens) /
    (visible tokens) -- exact rationals."""
    T, n_obs, G = 200, 7, 2
    k = np.tile(fp16.from_f64(np.linspace(-1, 1, 128)), (T, 1))
    q = synth.queries(302, n_obs, G).reshape(n_obs, G, 128)
    m = observer.observe_mass(q, k)
    for b in range(4):
        want = Fraction(0)
        for i in range(n_obs):
            vis = T - n_obs + i + 1
            lo, hi = 64 * b, min(64 * b + 64, vis)
            want += Fraction(max(hi - lo, 0), vis)
        want /= n_obs
        assert abs(m[b] - float(want)) < 1e-13


def test_causal_rows_are_single_queries_on_their_prefix():
    """The mask and positions: the n_obs-query mass equals the mean of one-query
    masses, each on the prefix its query sees (no mask needed there)."""
    T, n_obs, G = 333, 4, 3
    q, k = _qk(3, n_obs, G, T)
    m = observer.observe_mass(q, k)
    acc = np.zeros_like(m)
    for i in range(n_obs):
        vis = T - n_obs + i + 1
        mi = observer.observe_mass(q[i:i + 1], k[:vis])
        acc[:len(mi)] += mi
    np.testing.assert_allclose(m, acc / n_obs, rtol=1e-12, atol=1e-15)


def test_gqa_identical_heads_equal_one_head():
    T, n_obs = 256, 3
    q, k = _qk(4, n_obs, 1, T)
    m1 = observer.observe_mass(q, k)
    m4 = observer.observe_mass(np.repeat(q, 4, axis=1), k)
    np.testing.assert_allclose(m4, m1, rtol=1e-13, atol=1e-16)


def test_dominant_key_takes_the_mass():
    T = 300
    k = np.zeros((T, 128), dtype=np.uint16)
    k[70] = fp16.from_f64(np.full(128, 2.0))
    q = fp16.from_f64(np.full((2, 1, 128), 2.0))
    m = observer.observe_mass(q, k)
    # logit gap 128 * 4 / sqrt(128) ~ 45.25: every other block holds < 64 e^-45
    assert m[1] >= 1 - 1e-15
    assert np.all(np.delete(m, 1) < 64 * np.exp(-45))


def test_ema_blend():
    a, b = np.array([0.5, 0.25, 0.25]), np.array([0.0, 1.0, 0.0])
    np.testing.assert_allclose(observer.ema(a, b), [0.45, 0.325, 0.225], rtol=1e-15)
    np.testing.assert_array_equal(observer.ema(np.full(3, np.nan), b, 1.0), b)


def test_key_range_and_query_norm():
    k = np.zeros((100, 128))
    k[3, 5], k[40, 5] = -3.0, 4.0   # channel 5 spans 7 in block 0
    k[64, 9], k[99, 9] = 1.5, -0.5  # partial block 1 spans 2 in channel 9
    e = observer.key_range(fp16.from_f64(k))
    assert list(e) == [7.0, 2.0]
    q = np.zeros((2, 2, 128))
    q[0, 1, 0], q[0, 1, 1] = 3.0, 4.0
    q[1, 0, 7] = 4.5
    assert observer.query_norm(fp16.from_f64(q)) == 5.0


@pytest.mark.parametrize("x,level", [(0.0, 1), (1.0, 1), (1.0000001, 2), (3.0, 2), (3.5, 4), (15.0, 4),
                                     (15.25, 8), (255.0, 8), (255.5, 16), (1e30, 16)])
def test_bit_depth_thresholds(x, level):
    """b* = ceil(log2(x + 1)) -> smallest ladder level >= b* (1 clamps b* = 0)."""
    import math
    b = math.ceil(math.log2(x + 1)) if x < 1e29 else 99
    assert observer.bit_level(x) == level
    assert level == min([L for L in (1, 2, 4, 8, 16) if L >= b] or [16])


def _nearest_level(b):
    """The level of {1, 2, 4, 8, 16} nearest to an integer bit depth b (b >= 0),
    ties to the larger level; b <= 1 clamps to 1."""
    best = None
    for L in (1, 2, 4, 8, 16):
        if best is None or abs(L - b) < abs(best - b) or (abs(L - b) == abs(best - b) and L > best):
            best = L
    return best


def test_bit_depth_nearest_level():
    """The "nearest available discrete level" reading of section 3.3: for every
    integer b* the level nearest to it (ties up), found by brute force over the
    ladder, equals bit_level(x, "nearest") both at the smallest x with that b*
    and at the largest (x = 2^b* - 1)."""
    import math
    assert [_nearest_level(b) for b in range(14)] == [1, 1, 2, 4, 4, 4, 8, 8, 8, 8, 8, 8, 16, 16]
    for b in range(0, 20):
        hi = 2.0 ** b - 1.0                     # largest x with ceil(log2(x + 1)) == b
        lo = 2.0 ** (b - 1) - 1.0 if b else 0.0  # x a little above it has b* == b
        xs = [hi] + ([lo + 2.0 ** (b - 1) * 1e-9] if b else [])
        for x in xs:
            assert math.ceil(math.log2(x + 1)) == b
            assert observer.bit_level(x, "nearest") == _nearest_level(b), (b, x)
    # the two readings differ exactly at b* = 5 and b* = 9..11
    for b in range(0, 20):
        up = observer.bit_level(2.0 ** b - 1.0, "up")
        near = observer.bit_level(2.0 ** b - 1.0, "nearest")
        assert (up != near) == (b in (5, 9, 10, 11)), b


def test_allocate_nearest_reading():
    """The formula test's setting under both readings: x = m / 2, so masses 6 (x = 3,
    b* = 2), 30 (x = 15, b* = 4), 60 (x = 30, b* = 5), 510 (x = 255, b* = 8), 4000
    (x = 2000, b* = 11) and 5000 (x = 2500, b* = 12) give 2, 4, 4, 8, 8, 16 when
    rounded to the nearest level and 2, 4, 8, 8, 16, 16 when rounded up."""
    T = 64 * 10 + 5
    e = np.full(11, 2.0)
    qn, c, tau = 4.0, 1.0, 11.0 * 8.0
    m = np.array([0, 2, 6, 30, 60, 510, 4000, 5000, 1, 1, 1], dtype=np.float32)
    assert list(observer.allocate(m, e, qn, T, c, tau, window=2, rounding="nearest")) == \
        [1, 1, 2, 4, 4, 8, 8, 16, 1, 16, 16]
    assert list(observer.allocate(m, e, qn, T, c, tau, window=2, rounding="up")) == \
        [1, 1, 2, 4, 8, 8, 16, 16, 1, 16, 16]


def test_allocate_formula_window_and_monotone():
    T = 64 * 10 + 5          # 11 blocks, the last partial
    e = np.full(11, 2.0)
    qn, c, tau = 4.0, 1.0, 11.0 * 8.0
    # x = c qn e N m / (2 tau) = 4 * 2 * 11 * m / (2 * 88) = m / 2
    m = np.array([0, 2, 2.5, 6, 30, 510, 600, 1, 1, 1, 1], dtype=np.float32)
    lv = observer.allocate(m, e, qn, T, c, tau, window=2)
    assert list(lv) == [1, 1, 2, 2, 4, 8, 16, 1, 1, 16, 16]
    # more mass never lowers a level
    for scale in (0.5, 2.0, 4.0):
        lv2 = observer.allocate(m * np.float32(scale), e, qn, T, c, tau, window=2)
        assert np.all(lv2 >= lv) if scale >= 1.0 else np.all(lv2 <= lv)
    # the partial last block is exact even with no window
    assert observer.allocate(np.zeros(11, np.float32), e, qn, T, c, tau, window=0)[-1] == 16
