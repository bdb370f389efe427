"""Pins for the oracle's block quantizers, centroid state and demotion (CPU only)."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import fp16, quant
from paper_2608_23599_amd import synth


def _block(seed=0, scale=1.0):
    k, _ = synth.kv_unit(100 + seed, 0, 0, 64)
    x = fp16.to_f64(k) * scale
    return fp16.to_f64(fp16.from_f64(x))


@pytest.mark.parametrize("bits", [8, 4, 2])
def test_scalar_codes_are_nearest_levels(bits):
    """Brute force: each code is the reconstruction level c*s16+z16 nearest to x,
    computed with exact rationals (the rint/division/clamp must implement this)."""
    x = _block(1)[:, :16]
    codes, s16, z16 = quant.quantize_scalar(x, bits)
    s = fp16.to_f64(s16)
    z = fp16.to_f64(z16)
    qmax = (1 << bits) - 1
    for d in range(x.shape[1]):
        lv = [Fraction(c) * Fraction(s[d]) + Fraction(z[d]) for c in range(qmax + 1)]
        for j in range(x.shape[0]):
            fx = Fraction(x[j, d])
            errs = [abs(fx - v) for v in lv]
            best = min(errs)
            cands = [c for c in range(qmax + 1) if errs[c] == best]
            assert codes[j, d] in cands


@pytest.mark.parametrize("bits", [8, 4, 2])
def test_scalar_error_bound_and_range(bits):
    x = _block(2)
    codes, s16, z16 = quant.quantize_scalar(x, bits)
    qmax = (1 << bits) - 1
    assert codes.min() >= 0 and codes.max() <= qmax
    s = fp16.to_f64(s16)
    s64 = (x.max(0) - x.min(0)) / qmax
    xh = quant.dequant_scalar(codes, s16, z16)
    bound = s / 2 + qmax * np.abs(s64 - s) + 1e-12
    assert np.all(np.abs(x - xh) <= bound[None, :])
    # the minimum of every channel is stored exactly as the zero and gets code 0
    assert np.array_equal(fp16.to_f64(z16), x.min(0))
    assert np.all(codes[x.argmin(0), np.arange(x.shape[1])] == 0)


def test_dequant_is_exact_in_fp64():
    x = _block(3, scale=37.0)
    for bits in (8, 4, 2):
        codes, s16, z16 = quant.quantize_scalar(x, bits)
        xh = quant.dequant_scalar(codes, s16, z16)
        s, z = fp16.to_f64(s16), fp16.to_f64(z16)
        for j in range(0, 64, 7):
            for d in range(0, 128, 5):
                assert Fraction(xh[j, d]) == Fraction(int(codes[j, d])) * Fraction(s[d]) + Fraction(z[d])


def test_constant_channel_and_scale_rounding():
    x = _block(4)
    x[:, 5] = 1.5
    codes, s16, z16 = quant.quantize_scalar(x, 4)
    assert s16[5] == 0 and np.all(codes[:, 5] == 0)
    assert fp16.to_f64(z16)[5] == 1.5
    # the scale is one RNE rounding of the fp64 quotient
    rng_ = x.max(0) - x.min(0)
    assert np.array_equal(s16, fp16.from_f64(rng_ / 15.0))


@pytest.mark.parametrize("bits", [8, 4, 2])
def test_requantize_same_level_is_identity(bits):
    qmax = (1 << bits) - 1
    r = np.random.default_rng(bits)
    codes = r.integers(0, qmax + 1, size=(64, 128))
    codes[0] = 0
    codes[1] = qmax      # both extreme codes present in every channel
    s16 = fp16.from_f64(r.uniform(0.01, 2.0, 128))
    z16 = fp16.from_f64(r.standard_normal(128))
    xh = quant.dequant_scalar(codes, s16, z16)
    c2, s2, z2 = quant.quantize_scalar(xh, bits)
    assert np.array_equal(c2, codes) and np.array_equal(s2, s16) and np.array_equal(z2, z16)


def test_centroids_recover_separated_clusters():
    r = np.random.default_rng(11)
    protos = r.standard_normal((4, 128)) * 20
    member = np.array([j % 4 for j in range(64)])
    r.shuffle(member[4:])
    member[[0, 16, 32, 48]] = [0, 1, 2, 3]
    x = protos[member] + r.standard_normal((64, 128)) * 0.01
    x = fp16.to_f64(fp16.from_f64(x))
    cent16, ids = quant.kmeans_centroids(x)
    assert np.array_equal(ids, member)
    for k in range(4):
        m = x[member == k].mean(0)
        # the stored centroid is the cluster mean rounded once to fp16 (half an ulp)
        assert np.all(np.abs(fp16.to_f64(cent16[k]) - m) <= np.abs(m) * 2.0 ** -11 + 2.0 ** -24)


def test_centroid_ids_are_argmin_of_stored_centroids():
    x = _block(5)
    cent16, ids = quant.kmeans_centroids(x)
    c = fp16.to_f64(cent16)
    for j in range(64):
        dist = [sum((Fraction(x[j, d]) - Fraction(c[k, d])) ** 2 for d in range(128)) for k in range(4)]
        best = min(dist)
        # channel-sequential fp64 distances can only tie-break differently when the
        # exact distances are within rounding of each other
        assert dist[ids[j]] <= best * (1 + 1e-12)


def test_k1_centroid_is_block_mean():
    x = _block(6)
    cent16, ids = quant.kmeans_centroids(x, k=1)
    exact_mean = [sum(Fraction(v) for v in x[:, d]) / 64 for d in range(128)]
    assert np.array_equal(cent16[0], fp16.from_f64(np.array([float(m) for m in exact_mean])))
    assert np.all(ids == 0)


def test_lloyd_objective_does_not_increase():
    x = _block(7)
    c = x[[0, 16, 32, 48]].copy()
    prev = np.inf
    for _ in range(10):
        d = quant._sq_dist(x, c)
        a = d.argmin(1)
        obj = d[np.arange(64), a].sum()
        assert obj <= prev * (1 + 1e-12)
        prev = obj
        for k in range(4):
            if np.any(a == k):
                c[k] = x[a == k].mean(0)


def test_demote_chain_and_no_promotion():
    x = _block(8)
    rec = quant.encode_fp16(16, fp16.from_f64(x))
    chain = [8, 4, 2, 1]
    for lv in chain:
        rec = quant.demote(rec, lv)
        assert rec.level == lv
    with pytest.raises(quant.NotMonotone):
        quant.demote(rec, 2)
    r8 = quant.encode(8, x)
    with pytest.raises(quant.NotMonotone):
        quant.demote(r8, 8)
    with pytest.raises(quant.NotMonotone):
        quant.demote(r8, 16)
    # demotion re-encodes the current (already quantized) values
    d4 = quant.demote(r8, 4)
    c, s, z = quant.quantize_scalar(quant.decode(r8), 4)
    assert np.array_equal(d4.codes, c) and np.array_equal(d4.s16, s) and np.array_equal(d4.z16, z)


def test_mean_level_is_correctly_rounded_block_mean():
    """Level 0 stores the fp16 of the exact block mean (rational arithmetic here,
    numpy's own fp16 rounding for the reference), and decodes every row to it."""
    x = _block(9, scale=3.0)
    rec = quant.encode(0, x)
    exact_mean = [sum(Fraction(v) for v in x[:, d]) / 64 for d in range(128)]
    ref = np.array([float(m) for m in exact_mean]).astype(np.float16).view(np.uint16)
    ref = np.where(ref == 0x8000, 0, ref)  # negative zero is stored as +0
    assert rec.cent16.shape == (1, 128)
    assert np.array_equal(rec.cent16[0], ref)
    assert np.all(rec.ids == 0)
    dec = quant.decode(rec)
    assert np.array_equal(dec, np.repeat(fp16.to_f64(ref[None, :]), 64, axis=0))


def test_mean_level_demotion_from_centroid_weights_by_count():
    """Demoting a 4-centroid block to level 0 averages its reconstruction, i.e.
    the centroids weighted by their token counts."""
    x = _block(10)
    c1 = quant.encode(1, x)
    m = quant.demote(c1, 0)
    c = fp16.to_f64(c1.cent16)
    cnt = np.bincount(c1.ids, minlength=4)
    exact = [sum(Fraction(int(cnt[k])) * Fraction(c[k, d]) for k in range(4)) / 64 for d in range(128)]
    ref = np.array([float(e) for e in exact]).astype(np.float16).view(np.uint16)
    ref = np.where(ref == 0x8000, 0, ref)
    assert np.array_equal(m.cent16[0], ref)
    # level 0 is the bottom of the ladder: nothing is below it, and no promotion
    for to in (1, 2, 16):
        with pytest.raises(quant.NotMonotone):
            quant.demote(m, to)
    with pytest.raises(quant.NotMonotone):
        quant.demote(m, 0)
    chain = quant.encode_fp16(16, fp16.from_f64(x))
    for lv in (8, 4, 2, 1, 0):
        chain = quant.demote(chain, lv)
    assert chain.level == 0


@pytest.mark.parametrize("bits", [8, 4, 2])
def test_per_token_codes_are_nearest_levels(bits):
    """Per-token grouping (values read the paper's way): each token's codes are the
    nearest of its own 2^b levels c*s_t + z_t, with exact rationals, and every
    decoded value is within half a step of the input."""
    x = _block(12, scale=2.0)[:8]  # 8 tokens x 128 channels
    codes, s16, z16 = quant.quantize_scalar_per_token(x, bits)
    assert codes.shape == x.shape and s16.shape == (8,) and z16.shape == (8,)
    s, z = fp16.to_f64(s16), fp16.to_f64(z16)
    qmax = (1 << bits) - 1
    for t in range(8):
        assert z[t] == float(np.float16(x[t].min())) or z[t] == 0.0
        lv = [Fraction(c) * Fraction(s[t]) + Fraction(z[t]) for c in range(qmax + 1)]
        for d in range(0, 128, 7):
            fx = Fraction(x[t, d])
            errs = [abs(fx - v) for v in lv]
            assert errs[codes[t, d]] == min(errs)
    rec = quant.encode(bits, np.vstack([x] * 8), per_token=True)
    dec = quant.decode(rec)
    step = np.repeat(fp16.to_f64(rec.s16)[:, None], 128, axis=1)
    rng_lo = np.repeat(fp16.to_f64(rec.z16)[:, None], 128, axis=1)
    inside = np.vstack([x] * 8) >= rng_lo
    assert np.all(np.abs(dec - np.vstack([x] * 8))[inside] <= step[inside] / 2 + 1e-12)


def test_per_token_grouping_is_kept_down_the_ladder():
    x = _block(13)
    r8 = quant.encode(8, x, per_token=True)
    r4 = quant.demote(r8, 4)
    assert r4.per_token and r4.s16.shape == (64,)
    c, s, z = quant.quantize_scalar_per_token(quant.decode(r8), 4)
    assert np.array_equal(r4.codes, c) and np.array_equal(r4.s16, s) and np.array_equal(r4.z16, z)
    r1 = quant.demote(r4, 1)  # centroid state: no grouping, the flag only rides along
    assert r1.level == 1 and r1.per_token
    # per-token and per-channel differ on a block whose channels have different spreads
    xc = x * np.linspace(0.1, 3.0, 128)[None, :]
    xc = fp16.to_f64(fp16.from_f64(xc))
    assert not np.array_equal(quant.decode(quant.encode(4, xc)), quant.decode(quant.encode(4, xc, per_token=True)))
