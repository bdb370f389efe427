"""Pins for the oracle's Quest ranking, attention, residual, certificate and
rate accounting (CPU only)."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import fp16, quant, quest, attention, residual, accounting, certificate, cache
from oracle.ladder import ladder, EXACT, INT8, INT4, INT2, CENTROID
from paper_2608_23599_amd import synth

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_rates.json")))


def _seq_dot(q, k):
    acc = 0.0
    for a, b in zip(q, k):
        acc = acc + a * b
    return acc


def _seq_dot_f32(q, k):
    acc = np.float32(0.0)
    for a, b in zip(q.astype(np.float32), k.astype(np.float32)):
        acc = np.float32(acc + a * b)
    return acc


def test_box_bound_never_below_true_score():
    """Every term of the bound is >= the key's term (exact fp32 products) and
    round-to-nearest addition is monotone, so the fp32 bound is never below the same
    channel-ascending fp32 sum for any key of the page."""
    k, _ = synth.kv_unit(201, 0, 0, 512)
    q = synth.queries(201, 1, 4)[0]
    kmin, kmax = quest.page_boxes(k)
    ub = quest.box_upper_bounds(q, kmin, kmax)
    assert ub.dtype == np.float32
    kf, qf = fp16.to_f64(k), fp16.to_f64(q)
    for g in range(4):
        for p in range(kmin.shape[0]):
            best = max(_seq_dot_f32(qf[g], kf[j]) for j in range(16 * p, 16 * p + 16))
            assert ub[g, p] >= best
    assert np.all(fp16.to_f64(kmin)[:, None, :] <= fp16.to_f64(k).reshape(32, 16, 128))


def test_box_bound_within_fp32_error_of_exact_sum():
    """The bound against its exact rational value: recursive summation of n terms
    rounds to within (n - 1) * 2^-24 * sum |term| (each product is exact)."""
    k, _ = synth.kv_unit(203, 0, 0, 256)
    q = synth.queries(203, 1, 4)[0]
    kmin, kmax = quest.page_boxes(k)
    ub = quest.box_upper_bounds(q, kmin, kmax)
    qf, lo, hi = fp16.to_f64(q), fp16.to_f64(kmin), fp16.to_f64(kmax)
    for g in range(4):
        for p in range(kmin.shape[0]):
            terms = [Fraction(qf[g, d]) * Fraction(hi[p, d] if qf[g, d] >= 0 else lo[p, d]) for d in range(128)]
            exact = sum(terms)
            bound = 127 * Fraction(1, 2 ** 24) * sum(abs(t) for t in terms)
            assert abs(Fraction(float(ub[g, p])) - exact) <= bound


def test_box_bound_picks_corner_by_sign():
    """q_d >= 0 takes kmax_d, q_d < 0 takes kmin_d (small integers: exact in any order)."""
    q = np.zeros((1, 128))
    lo, hi = np.zeros((1, 128)), np.zeros((1, 128))
    q[0, :3], lo[0, :3], hi[0, :3] = [1, -1, 2], [-3, -5, 1], [2, 7, 4]
    ub = quest.box_upper_bounds(fp16.from_f64(q), fp16.from_f64(lo), fp16.from_f64(hi))
    assert ub[0, 0] == 1 * 2 + (-1) * (-5) + 2 * 4


def test_box_bound_fp32_channel_order():
    """The bound rounds to fp32 after every channel, in ascending channel order:
    terms (2^24, 1, -2^24) sum to 0 (2^24 + 1 rounds to 2^24), terms (2^24, -2^24, 1)
    to 1; fp64, or the descending order, would give 1 for the first."""
    def bound(qs, ks):
        q = np.zeros((1, 128))
        k = np.zeros((1, 128))
        q[0, :3], k[0, :3] = qs, ks
        kb = fp16.from_f64(k)
        return quest.box_upper_bounds(fp16.from_f64(q), kb, kb)[0, 0]
    assert bound([2048, 1, -2048], [8192, 1, 8192]) == 0.0
    assert bound([2048, -2048, 1], [8192, 8192, 1]) == 1.0


def test_page_size_one_is_exact_topk():
    r = np.random.default_rng(3)
    k = fp16.from_f64(r.integers(-8, 9, size=(300, 128)).astype(np.float64))
    q = fp16.from_f64(r.integers(-4, 5, size=(1, 128)).astype(np.float64))
    kmin, kmax = quest.page_boxes(k, page=1)
    sel = quest.quest_select(q, kmin, kmax, T=300, k=20, page=1)
    exact = [sum(Fraction(int(a)) * Fraction(int(b)) for a, b in zip(fp16.to_f64(q)[0], fp16.to_f64(k)[j]))
             for j in range(299)]
    order = sorted(range(299), key=lambda j: (-exact[j], j))
    assert list(sel) == sorted(order[:20])


def test_ties_go_to_lower_page_and_padding():
    k, _ = synth.kv_unit(202, 0, 0, 256)
    k = k.copy()
    k[64:80] = k[16:32]   # page 4 duplicates page 1
    kmin, kmax = quest.page_boxes(k)
    q = synth.queries(202, 1, 2)[0]
    s = quest.page_scores(q, kmin, kmax)
    assert s[1] == s[4]
    top = np.lexsort((np.arange(len(s)), -s))
    pos1, pos4 = list(top).index(1), list(top).index(4)
    assert pos1 < pos4
    sel = quest.select_top(s, 40)
    assert list(sel[:len(s)]) == list(range(len(s))) and np.all(sel[len(s):] == -1)


def test_quest_all_pages_equals_dense():
    k, v = synth.kv_unit(203, 0, 0, 1024)
    lv = ladder("tiny", 1024)
    uc = cache.UnitCache(k, v, lv)
    q = synth.queries(203, 1, 4)[0]
    kmin, kmax = quest.page_boxes(k)
    pages = quest.quest_select(q, kmin, kmax, T=1024, k=64)
    assert np.array_equal(pages[:63], np.arange(63))
    np.testing.assert_allclose(uc.decode_quest(q, pages), uc.decode_dense(q), rtol=0, atol=1e-14)


def test_attention_matches_bruteforce():
    k, v = synth.kv_unit(204, 0, 0, 96)
    q = synth.queries(204, 1, 3)[0]
    kh, vh = fp16.to_f64(k), fp16.to_f64(v)
    a = attention.attend(fp16.to_f64(q), kh, vh)
    b = attention.attend_bruteforce(fp16.to_f64(q).tolist(), kh.tolist(), vh.tolist())
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-13)


def test_all_exact_ladder_is_plain_attention():
    k, v = synth.kv_unit(205, 0, 0, 200)
    q = synth.queries(205, 1, 2)[0]
    uc = cache.UnitCache(k, v, ladder("exact", 200))
    ref = attention.attend_bruteforce(fp16.to_f64(q).tolist(), fp16.to_f64(k).tolist(), fp16.to_f64(v).tolist())
    np.testing.assert_allclose(uc.decode_dense(q), ref, rtol=1e-12, atol=1e-13)


def test_certificate_holds_for_graded_reconstruction():
    k, v = synth.kv_unit(206, 0, 0, 2048)
    uc = cache.UnitCache(k, v, ladder("tiny", 2048))
    kh, vh = uc.khat_vhat()
    kf, vf = fp16.to_f64(k), fp16.to_f64(v)
    qs = fp16.to_f64(synth.queries(206, 1, 8)[0])
    for g in range(8):
        bnd, err = certificate.bound(qs[g], kf, vf, kh, vh)
        assert err <= bnd
        assert err > 0


def test_residual_selection_pins():
    T = 512
    k, v = synth.kv_unit(207, 0, 0, T)
    uc = cache.UnitCache(k, v, ladder("tiny", T))
    m = synth.mass_unit(207, 0, 0, T)
    n = residual.n_keep(T, 2)
    assert n == 10
    idx, s = uc.select_residual(k, v, m, n)
    lv = np.repeat(uc.levels, 64)[:T]
    assert np.all(s[lv == 16] == 0)            # exact tokens have no distortion
    assert len(idx) == n and np.all(np.diff(idx) > 0)
    brute = sorted(range(T), key=lambda j: (-s[j], j))[:n]
    assert list(idx) == sorted(brute)
    # fraction 0 leaves the graded cache unchanged
    uc0 = cache.UnitCache(k, v, ladder("tiny", T))
    uc0.select_residual(k, v, m, 0)
    q = synth.queries(207, 1, 2)[0]
    np.testing.assert_array_equal(uc0.decode_dense(q), cache.UnitCache(k, v, ladder("tiny", T)).decode_dense(q))
    # with the residual, selected tokens read their exact values
    kh, vh = uc.khat_vhat()
    assert np.array_equal(vh[idx], fp16.to_f64(v[idx]))


def test_rd_score_on_centroid_block_is_equation():
    # for a centroid block the graded value IS the block value centroid of Eq. rdscore
    k, v = synth.kv_unit(208, 0, 0, 64)
    rec = quant.encode_fp16(1, v)
    c = fp16.to_f64(rec.cent16)
    a = synth.mass_unit(208, 0, 0, 64)
    s = residual.scores(fp16.to_f64(v), quant.decode(rec), a)
    for j in (0, 17, 63):
        e = sum((Fraction(x) - Fraction(y)) ** 2 for x, y in zip(fp16.to_f64(v)[j], c[rec.ids[j]]))
        assert abs(s[j] - float(a[j]) * float(e)) <= 1e-12 * s[j]


# ---------------------------------------------------------------- accounting


def test_level_bits_per_value():
    got = [accounting.block_bits(L) / (64 * 128) for L in (16, 8, 4, 2, 1, 0)]
    assert got == [16.0, 8.5, 4.5, 2.5, 1.015625, 0.25]
    # the one-centroid state costs one exact row per block and nothing per token
    assert accounting.block_bits(0) == accounting.row_bits(16)
    assert accounting.row_bits(0) == 0


def test_mean_blocks_attend_as_counted_single_keys():
    """Closed form: every token of a level-0 block has the same key and value, so
    the block acts as ONE key whose weight is multiplied by its token count
    (log-count added to the logit); residual tokens leave their block's count."""
    T = 64 * 6
    k, v = synth.kv_unit(211, 0, 0, T)
    lv = np.array([0, 0, 0, 0, 16, 16], dtype=np.int8)
    uc = cache.UnitCache(k, v, lv)
    m = synth.mass_unit(211, 0, 0, T)
    idx, _ = uc.select_residual(k, v, m, 40)
    q = synth.queries(211, 1, 3)[0]
    got = uc.decode_dense(q)
    kf, vf, qf = fp16.to_f64(k), fp16.to_f64(v), fp16.to_f64(q)
    res = set(int(j) for j in idx)
    for g in range(3):
        logits, vals = [], []
        for b in range(4):
            means_k = quant.decode(quant.encode(0, kf[64 * b:64 * b + 64]))[0]
            means_v = quant.decode(quant.encode(0, vf[64 * b:64 * b + 64]))[0]
            n = sum(1 for j in range(64 * b, 64 * b + 64) if j not in res)
            if n:
                logits.append(float(qf[g] @ means_k) / np.sqrt(128) + np.log(n))
                vals.append(means_v)
        # residual rows of the level-0 blocks, then the exact blocks, read exactly
        for j in sorted(r for r in res if r < 256) + list(range(256, T)):
            logits.append(float(qf[g] @ kf[j]) / np.sqrt(128))
            vals.append(vf[j])
        logits = np.array(logits)
        w = np.exp(logits - logits.max())
        ref = (w[:, None] * np.array(vals)).sum(0) / w.sum()
        np.testing.assert_allclose(got[g], ref, rtol=1e-10, atol=1e-12)


def test_rdv2_ladder_and_rates():
    """RD-V2: newest 16 blocks exact, older blocks one-centroid; growth only
    demotes exact blocks straight to level 0, once each; with 10.2% exact residual
    rows the resident rate at 128k tokens is 0.25 bpv of base plus the exact
    window plus 16 bits, a 32-bit index per row and one mask per block."""
    lv = ladder("rdv2", 131072)
    assert (lv == 16).sum() == 16 and (lv == 0).sum() == 2048 - 16 and np.all(lv[-16:] == 16)
    from oracle import ladder as lad
    for T0 in (64 * 16, 64 * 16 + 1, 5000):
        cr = lad.crossings("rdv2", T0, T0 + 64)
        assert all(o == 16 and n == 0 for _, o, n in cr)
        assert len(cr) == (1 if lad.n_blocks(T0) >= 16 else 0)
    n = residual.n_keep(131072, 102, 1000)
    assert n == 13369
    r = accounting.unit_rates(lv, 131072, nres=n)
    vals = 131072 * 2 * 128
    base = (16 * 64 * 128 * 16 + 2032 * 128 * 16) * 2
    res = n * (2 * 128 * 16 + 32) + 2048 * 64
    assert r["resident_bits"] == base + res
    assert abs(r["resident_bits"] / vals - 2.0217) < 1e-4


def test_tiny_and_llama_graded_rates():
    r = accounting.unit_rates(ladder("tiny", 2048), 2048)
    assert r["resident_bits"] / r["values"] == 6.4375
    r2 = accounting.unit_rates(ladder("graded", 16384), 16384)
    assert abs(r2["resident_bits"] / r2["values"] - 5.2613) < 5e-5


def test_paper_quest_rates():
    g = GOLD["quest_setting"]
    T, page, frac = g["T"], g["page_tokens"], g["page_fraction"]
    lv = ladder("exact", T)
    npages = T // page
    k = int(round(frac * npages))
    pages = np.arange(k)
    r = accounting.unit_rates(lv, T, page=page, pages=pages)
    res = r["resident_bits"] / r["values"]
    rd = r["read_bits"] / r["values"]
    assert res == pytest.approx(GOLD["quest_resident_bpv"]["value"], abs=1e-9)
    assert abs(rd - GOLD["quest_read_bpv_3b"]["value"]) < 0.005
    assert abs(rd - GOLD["quest_read_bpv_8b"]["value"]) < 0.005
    assert (accounting.BOX_BITS / (page * 2 * 128)) == GOLD["box_rate_bpv_64token_pages"]["value"]


def test_paper_per_token_bytes():
    for key in ("per_token_kib_qwen3_8b", "per_token_kib_qwen25_3b"):
        g = GOLD[key]
        bits = g["layers"] * g["kv_heads"] * 2 * accounting.row_bits(16, g["head_dim"])
        assert bits / 8 / 1024 == g["value"]
    g = GOLD["kv_gib_1m_qwen25_7b"]
    bits = g["tokens"] * g["layers"] * g["kv_heads"] * 2 * accounting.row_bits(16, g["head_dim"])
    assert round(bits / 8 / 2 ** 30, 2) == g["value"]


# Graded Compressed-Quest read rate (section 3.5, R_read equation), written out term by
# term by hand.  Per tensor block of 64 tokens x 128 channels: int b codes 128*b bits
# per row plus 2 * 128 * 16 bits of scale/zero per block; centroid state 2 bits of id
# per row plus 4 * 128 * 16 bits of centroids per block; exact 128 * 16 bits per row.
# Every term is doubled for K and V.  A plausible slip fails one of the two cases:
# scale/zero charged per page instead of per touched block (case 1 has two pages of
# one int2 block, case 2 two pages of one int4 block), the current page's block
# overhead dropped (case 2's current page lies in an int8 block), the current page
# left out or counted as a full page (case 1's is 8 rows), boxes counted for the
# ranked pages only instead of every closed page.
GRADED_QUEST_CASES = [
    dict(T=248, levels=[CENTROID, INT2, INT8, EXACT], pages=[1, 5, 6, 9, 12],
         terms=[15 * 2 * 128 * 16,       # boxes of the 15 closed pages (248 // 16)
                16 * 2 * 2,              # page 1: 16 rows of 2-bit centroid ids, block 0
                2 * 4 * 128 * 16,        # block 0 centroids, once
                32 * 2 * 128 * 2,        # pages 5, 6: 32 rows of int2 codes, block 1
                2 * 2 * 128 * 16,        # block 1 scale/zero, once for both pages
                16 * 2 * 128 * 8,        # page 9: 16 rows of int8 codes, block 2
                2 * 2 * 128 * 16,        # block 2 scale/zero
                16 * 2 * 128 * 16,       # page 12: 16 exact rows, block 3
                8 * 2 * 128 * 16],       # current page 15: tokens 240..247, 8 exact rows
         read_bits=241728, resident_bits=520448),
    dict(T=256, levels=[INT4, INT8, INT2, INT8], pages=[0, 3, 9],
         terms=[16 * 2 * 128 * 16,       # boxes of the 16 closed pages (256 // 16)
                32 * 2 * 128 * 4,        # pages 0, 3: 32 rows of int4 codes, block 0
                2 * 2 * 128 * 16,        # block 0 scale/zero, once for both pages
                16 * 2 * 128 * 2,        # page 9: 16 rows of int2 codes, block 2
                2 * 2 * 128 * 16,        # block 2 scale/zero
                16 * 2 * 128 * 8,        # current page 15 (always read): int8, block 3
                2 * 2 * 128 * 16],       # block 3 scale/zero, touched by the current page only
         read_bits=163840, resident_bits=None),
]


@pytest.mark.parametrize("case", GRADED_QUEST_CASES)
def test_graded_quest_read_rate_by_hand(case):
    assert sum(case["terms"]) == case["read_bits"]
    T = case["T"]
    r = accounting.unit_rates(case["levels"], T, page=16, pages=np.array(case["pages"]))
    assert r["read_bits"] == case["read_bits"]
    assert r["values"] == T * 2 * 128
    if case["resident_bits"] is not None:
        # 2 x (centroid 8320 + int2 20480 + int8 69632 + exact 131072) + 15 boxes
        assert r["resident_bits"] == 2 * (8320 + 20480 + 69632 + 131072) + 15 * 4096 == case["resident_bits"]
    # the same pages listed twice, unsorted, with -1 padding read the same bits
    padded = np.array(list(reversed(case["pages"])) + case["pages"][:1] + [-1, -1])
    assert accounting.unit_rates(case["levels"], T, page=16, pages=padded)["read_bits"] == case["read_bits"]


def test_quest_read_rate_with_residual_by_hand():
    """A Compressed-Quest read of a cache with exact residual rows: on top of the
    graded read of case 2 (163840 bits), the rows of the residual tokens inside the
    read set (2 * 128 * 16 + 32 bits each) and one 64-bit override mask per touched
    block; residual tokens outside the read set cost nothing."""
    case = GRADED_QUEST_CASES[1]  # pages 0, 3, 9 and current page 15 of T = 256
    res_idx = np.array([5, 40, 52, 100, 150, 200, 250, 255])
    # in the read set: 5 (page 0), 52 (page 3), 150 (page 9), 250, 255 (page 15);
    # outside: 40 (page 2), 100 (page 6), 200 (page 12)
    touched_blocks = 3  # blocks 0, 2, 3
    want = case["read_bits"] + 5 * (2 * 128 * 16 + 32) + touched_blocks * 64
    r = accounting.unit_rates(case["levels"], 256, page=16, nres=len(res_idx), pages=np.array(case["pages"]),
                              res_idx=res_idx)
    assert r["read_bits"] == want == 163840 + 20640 + 192
    with pytest.raises(ValueError):
        accounting.unit_rates(case["levels"], 256, page=16, nres=len(res_idx), pages=np.array(case["pages"]))
