"""GPU parity of every call of the C ABI against the CPU oracle, on seeded
synthetic workloads at sizes the oracle finishes in seconds (several tiles and a
ragged tail).  Codes, scales, zeros, centroids, ids, boxes, page sets and residual
sets must be bit-exact; attention outputs within 2e-3 max-abs."""
import numpy as np
import pytest

from oracle import fp16 as ofp16, ladder as olad, quest as oquest, residual as ores, cache as ocache, quant as oquant
from oracle import accounting as oacc
from paper_2608_23599_amd import synth
from tests._util import TOL, kv_all, oracle_units, compare_record, q_group, max_err

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    return torch


def _build(gpu, ks, vs, Hq, levels, **kw):
    return gpu.GradedCache.build(ks, vs, Hq=Hq, levels=levels, device="cuda", **kw)


def _order_keys(s):
    """Order-preserving 64-bit keys of fp64 scores (a +0 for -0), as the selection ranks them."""
    b = (np.asarray(s, dtype=np.float64) + 0.0).view(np.uint64)
    neg = (b >> np.uint64(63)) != 0
    return np.where(neg, ~b, b | np.uint64(1 << 63))


def check_rd_keys(cache, b, h, T, want_scores):
    """The residual selection ranks the tokens of (b, h) by keys it leaves at the head of
    its workspace, [B][Hkv][nblk_cap * 64] (tokens below T); they must be the oracle's
    fp64 scores bit for bit, not only select the same rows."""
    ws = cache.workspace(2)
    stride = cache.nblk_cap * 64
    keys = ws[: cache.B * cache.Hkv * stride * 8].view(_torch().int64).view(cache.B, cache.Hkv, stride)
    got = keys[b, h, :T].cpu().numpy().view(np.uint64)
    np.testing.assert_array_equal(got, _order_keys(want_scores))


@pytest.mark.parametrize("T", [2048, 1000])
def test_tiny_graded_codes_and_attention(gpu, T):
    """Workload 1 shapes (8 query / 2 KV heads, tiny ladder); T = 1000 leaves a
    partial exact block and a partial tile."""
    B_, Hq, Hkv = 1, 8, 2
    ks, vs = kv_all(1, B_, Hkv, T)
    lv = olad.ladder("tiny", T)
    cache = _build(gpu, ks, vs, Hq, lv)
    ucs = oracle_units(ks, vs, lv)
    for (b, h), uc in ucs.items():
        for blk in range(len(lv)):
            for tensor in (0, 1):
                compare_record(cache, uc, b, h, blk, tensor)
    q = synth.queries(1, B_, Hq)
    out = cache.decode(q).cpu().numpy()
    G = Hq // Hkv
    for (b, h), uc in ucs.items():
        ref = uc.decode_dense(q_group(q, b, h, G))
        assert max_err(out[b, h * G:(h + 1) * G], ref) <= TOL


def test_llama16k_centroids_and_attention(gpu):
    """Workload 2: 32 query / 8 KV heads, T = 16384, graded ladder with centroids."""
    B_, Hq, Hkv, T = 1, 32, 8, 16384
    ks, vs = kv_all(2, B_, Hkv, T)
    lv = olad.ladder("graded", T)
    cache = _build(gpu, ks, vs, Hq, lv)
    ucs = oracle_units(ks, vs, lv)
    r = np.random.default_rng(0)
    for (b, h), uc in ucs.items():
        blks = set(np.nonzero(lv == 1)[0][:6]) | set(r.choice(len(lv), 6, replace=False)) | {len(lv) - 1}
        for blk in sorted(blks):
            for tensor in (0, 1):
                compare_record(cache, uc, b, h, blk, tensor)
    q = synth.queries(2, B_, Hq)
    out = cache.decode(q).cpu().numpy()
    G = Hq // Hkv
    errs = []
    for (b, h), uc in ucs.items():
        ref = uc.decode_dense(q_group(q, b, h, G))
        errs.append(max_err(out[b, h * G:(h + 1) * G], ref))
    assert max(errs) <= TOL, errs


@pytest.mark.parametrize("T,topk", [(32768, 128), (4001, 64), (1024, 100)])
def test_quest_boxes_selection_and_sparse_attention(gpu, T, topk):
    """Workload 3 shapes: exact 16-token page boxes, box-bound top-k (ties to the
    lower page), attention over selected + current page.  T = 4001 has a partial
    current page; T = 1024 with top-100 selects every ranked page (= dense)."""
    B_, Hq, Hkv, page = 1, 32, 8, 16
    if T < 32768:
        Hq, Hkv = 8, 2
    ks, vs = kv_all(3, B_, Hkv, T)
    lv = olad.ladder("graded", T)
    cache = _build(gpu, ks, vs, Hq, lv, page=page)
    G = Hq // Hkv
    q = synth.queries(3, B_, Hq)
    pages = cache.quest_select(q, topk)
    out = cache.decode(q, pages=pages).cpu().numpy()
    pages = pages.cpu().numpy()
    for b in range(B_):
        for h in range(Hkv):
            kmin, kmax = oquest.page_boxes(ks[b, h])
            gmin, gmax = cache.boxes_host(b, h, T // page)
            np.testing.assert_array_equal(gmin, kmin)
            np.testing.assert_array_equal(gmax, kmax)
            want = oquest.quest_select(q_group(q, b, h, G), kmin, kmax, T, topk)
            np.testing.assert_array_equal(pages[b, h], want)
            uc = ocache.UnitCache(ks[b, h], vs[b, h], lv)
            ref = uc.decode_quest(q_group(q, b, h, G), want)
            assert max_err(out[b, h * G:(h + 1) * G], ref) <= TOL
            if topk >= (T - 1) // page:
                assert max_err(out[b, h * G:(h + 1) * G], uc.decode_dense(q_group(q, b, h, G))) <= TOL


def test_quest_read_skips_invalid_entries(gpu):
    """A Compressed-Quest read reads the ascending selected pages of the list and skips
    every entry below 0 or at or past the current page, wherever it stands: the output
    equals the oracle's read of the valid pages plus the current page."""
    T, Hq, Hkv, topk = 4099, 8, 2, 24
    ks, vs = kv_all(3, 1, Hkv, T)
    lv = olad.ladder("graded", T)
    cache = _build(gpu, ks, vs, Hq, lv, page=16)
    G = Hq // Hkv
    q = synth.queries(3, 1, Hq, step=5)
    cur = (T - 1) // 16
    lists = [[-1, 3, 4, -1, 17, 40, 41, 64, -1, 100, cur, 170, 200, cur + 3, 240, 255, -1, -1, 5000, -1, -1, -1, -1, -1],
             [0, 1, 2, -1, -1, 63, 64, 65, 66, 67, 68, -1, 127, 128, 129, 130, 131, 200, 201, 202, 203, 250, -1, cur]]
    assert all(len(x) == topk for x in lists)
    pages = _torch().from_numpy(np.array(lists, dtype=np.int32)[None]).cuda()
    out = cache.decode(q, pages=pages).cpu().numpy()
    for h in range(Hkv):
        uc = ocache.UnitCache(ks[0, h], vs[0, h], lv)
        valid = np.array([x for x in lists[h] if 0 <= x < cur], dtype=np.int32)
        ref = uc.decode_quest(q_group(q, 0, h, G), valid, 16)
        assert max_err(out[0, h * G:(h + 1) * G], ref) <= TOL


@pytest.mark.parametrize("page,T,topk", [(32, 6001, 40), (64, 8192, 30), (64, 3000, 50)])
def test_quest_larger_pages(gpu, page, T, topk):
    """Compressed-Quest with 32- and 64-token pages (the paper's own box granularity is
    a 64-token block): boxes, selection and attention over the selected pages plus the
    current page against the oracle; T = 3000 with top-50 selects every ranked page."""
    B_, Hq, Hkv = 1, 8, 2
    ks, vs = kv_all(3, B_, Hkv, T)
    lv = olad.ladder("graded", T)
    cache = _build(gpu, ks, vs, Hq, lv, page=page)
    G = Hq // Hkv
    q = synth.queries(3, B_, Hq, step=page)
    pages = cache.quest_select(q, topk)
    out = cache.decode(q, pages=pages).cpu().numpy()
    pages = pages.cpu().numpy()
    for h in range(Hkv):
        kmin, kmax = oquest.page_boxes(ks[0, h], page)
        gmin, gmax = cache.boxes_host(0, h, T // page)
        np.testing.assert_array_equal(gmin, kmin)
        np.testing.assert_array_equal(gmax, kmax)
        want = oquest.quest_select(q_group(q, 0, h, G), kmin, kmax, T, topk, page)
        np.testing.assert_array_equal(pages[0, h], want)
        uc = ocache.UnitCache(ks[0, h], vs[0, h], lv)
        ref = uc.decode_quest(q_group(q, 0, h, G), want, page)
        assert max_err(out[0, h * G:(h + 1) * G], ref) <= TOL
        if topk >= (T - 1) // page:
            assert max_err(out[0, h * G:(h + 1) * G], uc.decode_dense(q_group(q, 0, h, G))) <= TOL


def test_quest_read_with_more_splits_than_a_wavefront(gpu):
    """One (b, KV head) with top-600 pages: one wavefront per read page puts 151
    workgroups' partials into one merge, more than the 64 lanes that take the split
    weights (three splits per lane).  Pages bit-exact, output against the oracle."""
    T, Hq, Hkv, page, topk = 16384, 4, 1, 16, 600
    ks, vs = kv_all(33, 1, Hkv, T)
    lv = olad.ladder("graded", T)
    cache = _build(gpu, ks, vs, Hq, lv, page=page)
    q = synth.queries(33, 1, Hq)
    pages = cache.quest_select(q, topk)
    out = cache.decode(q, pages=pages).cpu().numpy()
    kmin, kmax = oquest.page_boxes(ks[0, 0])
    want = oquest.quest_select(q_group(q, 0, 0, Hq), kmin, kmax, T, topk)
    np.testing.assert_array_equal(pages.cpu().numpy()[0, 0], want)
    uc = ocache.UnitCache(ks[0, 0], vs[0, 0], lv)
    assert max_err(out[0], uc.decode_quest(q_group(q, 0, 0, Hq), want)) <= TOL


def test_quest_ties_go_to_lower_page(gpu):
    T, Hq, Hkv = 2048, 4, 1
    ks, vs = kv_all(31, 1, Hkv, T)
    ks[0, 0, 64 * 4:64 * 4 + 16] = ks[0, 0, 16:32]          # page 16 duplicates page 1
    ks[0, 0, 64 * 8:64 * 8 + 48] = ks[0, 0, 64 * 2:64 * 2 + 48]  # pages 32-34 duplicate 8-10
    lv = olad.ladder("exact", T)
    cache = _build(gpu, ks, vs, Hq, lv, page=16)
    q = synth.queries(31, 1, Hq)
    kmin, kmax = oquest.page_boxes(ks[0, 0])
    s = oquest.page_scores(q[0], kmin[:127], kmax[:127])
    for k in range(1, 127, 9):
        got = cache.quest_select(q, k).cpu().numpy()[0, 0]
        np.testing.assert_array_equal(got, oquest.select_top(s, k))


@pytest.mark.parametrize("T,Bn", [(8192, 2), (3000, 1), (9001, 1)])
def test_rd_residual_selection_and_attention(gpu, T, Bn):
    """Workload 4 shapes at reduced length: 28 query / 4 KV heads, 2% residual by
    attention mass x squared value error.  T = 9001 exceeds one 8192-key slice and
    is selected in two slices and a final pass."""
    Hq, Hkv = 28, 4
    ks, vs = kv_all(4, Bn, Hkv, T)
    lv = olad.ladder("graded", T)
    n = ores.n_keep(T, 2)
    cache = _build(gpu, ks, vs, Hq, lv, nres_cap=n)
    mass = np.stack([np.stack([synth.mass_unit(4, b, h, T) for h in range(Hkv)]) for b in range(Bn)])
    cache.rd_residual_select(ks, vs, mass, n)
    q = synth.queries(4, Bn, Hq)
    out = cache.decode(q).cpu().numpy()
    idx = cache.res_idx.cpu().numpy()
    msk = cache.res_mask.cpu().numpy().view(np.uint64)
    G = Hq // Hkv
    for b in range(Bn):
        for h in range(Hkv):
            uc = ocache.UnitCache(ks[b, h], vs[b, h], lv)
            want, sc = uc.select_residual(ks[b, h], vs[b, h], mass[b, h], n)
            np.testing.assert_array_equal(idx[b, h, :n], want)
            check_rd_keys(cache, b, h, T, sc)
            bits = np.zeros(len(lv), dtype=np.uint64)
            for t in want:
                bits[t // 64] |= np.uint64(1) << np.uint64(t % 64)
            np.testing.assert_array_equal(msk[b, h, :len(lv)], bits)
            ref = uc.decode_dense(q_group(q, b, h, G))
            assert max_err(out[b, h * G:(h + 1) * G], ref) <= TOL


def test_rd_zero_fraction_is_graded(gpu):
    T, Hq, Hkv = 2048, 4, 1
    ks, vs = kv_all(41, 1, Hkv, T)
    lv = olad.ladder("tiny", T)
    cache = _build(gpu, ks, vs, Hq, lv, nres_cap=64)
    q = synth.queries(41, 1, Hq)
    before = cache.decode(q).cpu().numpy()
    cache.rd_residual_select(ks, vs, np.ones((1, 1, T), np.float32), 0)
    after = cache.decode(q).cpu().numpy()
    np.testing.assert_array_equal(before, after)


def test_demote_chain_bit_exact(gpu):
    """gkv_demote: exact -> int8 -> int4 -> int2 -> centroid, each step re-encoding
    the current record; a promotion is rejected without touching the cache."""
    T, Hq, Hkv = 512, 4, 2
    ks, vs = kv_all(51, 1, Hkv, T)
    lv = olad.ladder("exact", T)
    cache = _build(gpu, ks, vs, Hq, lv, slack={8: 16, 4: 16, 2: 16, 1: 16})
    ucs = oracle_units(ks, vs, lv)
    for to in (8, 4, 2, 1):
        jobs = [(0, h, blk) for h in range(Hkv) for blk in (1, 3, 6)]
        cache.demote(jobs, [to] * len(jobs))
        for (b, h), uc in ucs.items():
            for blk in (1, 3, 6):
                uc.k_recs[blk] = oquant.demote(uc.k_recs[blk], to)
                uc.v_recs[blk] = oquant.demote(uc.v_recs[blk], to)
                uc.levels[blk] = to
                compare_record(cache, uc, b, h, blk, 0)
                compare_record(cache, uc, b, h, blk, 1)
    with pytest.raises(Exception):
        cache.demote([(0, 0, 1)], [2])
    # demote int8 straight to centroid
    cache.demote([(0, 0, 2)], [8])
    cache.demote([(0, 0, 2)], [1])
    uc = ucs[(0, 0)]
    uc.k_recs[2] = oquant.demote(oquant.demote(uc.k_recs[2], 8), 1)
    uc.v_recs[2] = oquant.demote(oquant.demote(uc.v_recs[2], 8), 1)
    uc.levels[2] = 1
    compare_record(cache, uc, 0, 0, 2, 0)
    compare_record(cache, uc, 0, 0, 2, 1)
    q = synth.queries(51, 1, Hq)
    out = cache.decode(q).cpu().numpy()
    for (b, h), uc in ucs.items():
        assert max_err(out[b, 2 * h:2 * h + 2], uc.decode_dense(q_group(q, b, h, 2))) <= TOL


def test_dense_plan_kept_through_appends_inside_a_block(gpu):
    """An append that opens no block (and demotes nothing) leaves the block tables and
    the version as they were, so a dense read keeps the plan in its workspace: the plan
    covers the last block whole and the attention masks its tokens past the length.
    Every step the kept-plan output equals, bit for bit, the output of a call with a
    fresh workspace (which plans anew) and matches the oracle within tolerance."""
    Hq, Hkv = 8, 2
    T0 = 64 * 40 - 3
    steps = 12  # step 3 opens block 40
    ks, vs = kv_all(6, 1, Hkv, T0 + steps)
    lv = olad.ladder("graded", T0)
    cache = _build(gpu, ks[:, :, :T0], vs[:, :, :T0], Hq, lv, extra_blocks=2,
                   slack={16: 8, 8: 8, 4: 8, 2: 8, 1: 8})
    ucs = {h: ocache.UnitCache(ks[0, h, :T0], vs[0, h, :T0], lv) for h in range(Hkv)}
    G = Hq // Hkv
    kept = 0
    for s in range(steps):
        t = T0 + s
        v0 = int(cache.c.version)
        moves = cache.append(ks[:, :, t], vs[:, :, t], profile="graded")
        for h in range(Hkv):
            ucs[h].append(ks[0, h, t], vs[0, h, t], "graded")
        if t % 64 or moves:
            assert (int(cache.c.version) != v0) == bool(moves)
        else:
            assert int(cache.c.version) != v0
        kept += int(cache.c.version) == v0
        q = synth.queries(6, 1, Hq, step=s)
        out = cache.decode(q)
        ws = cache._ws[(1, 0)]
        cache._ws[(1, 0)] = _torch().zeros_like(ws)
        fresh = cache.decode(q)
        cache._ws[(1, 0)] = ws
        assert _torch().equal(out, fresh)
        out = out.cpu().numpy()
        for h in range(Hkv):
            ref = ucs[h].decode_dense(q_group(q, 0, h, G))
            assert max_err(out[0, h * G:(h + 1) * G], ref) <= TOL
    assert kept >= steps - 3


def test_append_demote_boxes_and_quest_steps(gpu):
    """Workload 5 step at a small length: every step appends one token per KV head
    (boxes of completed pages, new exact block every 64 tokens), demotes the blocks
    whose level the ladder lowers, selects pages and decodes; all checked against
    the oracle at every step."""
    Hq, Hkv, page, topk = 8, 2, 16, 24
    T0 = 64 * 40 - 3
    steps = 70
    ks, vs = kv_all(5, 1, Hkv, T0 + steps)
    lv = olad.ladder("graded", T0)
    cache = _build(gpu, ks[:, :, :T0], vs[:, :, :T0], Hq, lv, page=page, extra_blocks=4,
                   slack={16: 8, 8: 8, 4: 8, 2: 8, 1: 8})
    ucs = {(0, h): ocache.UnitCache(ks[0, h, :T0], vs[0, h, :T0], lv) for h in range(Hkv)}
    G = Hq // Hkv
    for s in range(steps):
        t = T0 + s
        moves = cache.append(ks[:, :, t], vs[:, :, t], profile="graded")
        omoves = []
        for h in range(Hkv):
            omoves = ucs[(0, h)].append(ks[0, h, t], vs[0, h, t], "graded")
        assert sorted((blk, o, n) for b, h, blk, o, n in moves if h == 0) == sorted(omoves)
        q = synth.queries(5, 1, Hq, step=s)
        pages = cache.quest_select(q, topk)
        out = cache.decode(q, pages=pages).cpu().numpy()
        pages = pages.cpu().numpy()
        T = t + 1
        for h in range(Hkv):
            uc = ucs[(0, h)]
            kmin, kmax = oquest.page_boxes(ks[0, h, :T])
            want = oquest.quest_select(q_group(q, 0, h, G), kmin, kmax, T, topk)
            np.testing.assert_array_equal(pages[0, h], want)
            ref = uc.decode_quest(q_group(q, 0, h, G), want)
            assert max_err(out[0, h * G:(h + 1) * G], ref) <= TOL
            for b_, h_, blk, o, n in moves:
                if h_ == h:
                    compare_record(cache, uc, 0, h, blk, 0)
                    compare_record(cache, uc, 0, h, blk, 1)
        dense = cache.decode(q).cpu().numpy()
        for h in range(Hkv):
            assert max_err(dense[0, h * G:(h + 1) * G], ucs[(0, h)].decode_dense(q_group(q, 0, h, G))) <= TOL
    assert T > T0 + 64


def test_constant_channel_and_equal_rows(gpu):
    """Degenerate blocks: constant channels (scale 0, codes 0) and identical rows
    (every centroid equal, ties to centroid 0)."""
    T, Hq, Hkv = 256, 4, 1
    ks, vs = kv_all(61, 1, Hkv, T)
    ks[0, 0, :, 5] = ofp16.from_f64(np.array([1.5]))[0]
    vs[0, 0, 64:128] = vs[0, 0, 64]
    ks[0, 0, 128:192] = ks[0, 0, 130]
    lv = np.array([2, 1, 1, 16], dtype=np.int8)
    cache = _build(gpu, ks, vs, Hq, lv)
    uc = ocache.UnitCache(ks[0, 0], vs[0, 0], lv)
    for blk in range(4):
        compare_record(cache, uc, 0, 0, blk, 0)
        compare_record(cache, uc, 0, 0, blk, 1)
    q = synth.queries(61, 1, Hq)
    assert max_err(cache.decode(q).cpu().numpy()[0], uc.decode_dense(q[0])) <= TOL


def test_staged_attention_equals_one_call(gpu):
    """plan -> partials -> merge on one stream gives the one-call result bit for bit,
    for a dense read with residual rows and for a Compressed-Quest read."""
    torch = _torch()
    T, Hq, Hkv = 3000, 8, 2
    ks, vs = kv_all(4, 1, Hkv, T)
    lv = olad.ladder("graded", T)
    nres = ores.n_keep(T, 2)
    cache = _build(gpu, ks, vs, Hq, lv, nres_cap=nres, page=16)
    mass = np.stack([synth.mass_unit(4, 0, h, T) for h in range(Hkv)])[None]
    q = synth.queries(4, 1, Hq)
    qd = torch.from_numpy(q.view(np.int16)).cuda()
    # Compressed-Quest read (before the residual exists: it requires nres = 0)
    pages = cache.quest_select(q, 24)
    one = cache.decode(qd, pages=pages).clone()
    out = torch.full_like(one, float("nan"))
    cache.attn_plan(pages)
    cache.attn_partials(qd, pages)
    cache.attn_merge(out, pages)
    assert torch.equal(one, out)
    # dense read with residual rows
    cache.rd_residual_select(ks, vs, mass, nres)
    one = cache.decode(qd).clone()
    out = torch.full_like(one, float("nan"))
    cache.attn_plan()
    cache.attn_partials(qd)
    cache.attn_merge(out)
    assert torch.equal(one, out)


def test_quest_selection_beyond_register_keys(gpu):
    """More than 8192 ranked pages (T = 16 * 8300): the selection in two slices and a
    final pass must give the oracle's page set."""
    T, Hq, Hkv, page, topk = 16 * 8300 + 5, 4, 1, 16, 200
    ks, vs = kv_all(3, 1, Hkv, T)
    lv = olad.ladder("graded", T)
    cache = _build(gpu, ks, vs, Hq, lv, page=page)
    q = synth.queries(3, 1, Hq, step=7)
    pages = cache.quest_select(q, topk).cpu().numpy()
    kmin, kmax = oquest.page_boxes(ks[0, 0])
    want = oquest.quest_select(q_group(q, 0, 0, Hq), kmin, kmax, T, topk)
    np.testing.assert_array_equal(pages[0, 0], want)


@pytest.mark.parametrize("G", [1, 2, 3, 6, 8, 16])
def test_quest_selection_per_group_size(gpu, G):
    """Page sets for GQA group sizes 1..16: the scoring splits a group's heads over one,
    two or four wavefronts depending on the size, and each split must give the oracle's
    pages (ties to the lower page)."""
    T, Hkv, page, topk = 4001, 2, 16, 40
    Hq = G * Hkv
    ks, vs = kv_all(3, 1, Hkv, T)
    cache = _build(gpu, ks, vs, Hq, olad.ladder("graded", T), page=page)
    q = synth.queries(3, 1, Hq, step=G)
    pages = cache.quest_select(q, topk).cpu().numpy()
    for h in range(Hkv):
        kmin, kmax = oquest.page_boxes(ks[0, h])
        want = oquest.quest_select(q_group(q, 0, h, G), kmin, kmax, T, topk)
        np.testing.assert_array_equal(pages[0, h], want)


@pytest.mark.parametrize("k", [1, 100, 4096, 5000])
def test_quest_select_ties_across_slices(gpu, k):
    """16500 ranked pages built from three page contents, so every score is shared by
    thousands of pages and the k-th falls inside a tie: the winners must be the oracle's
    (ties to the lower page) whether the selection runs in 8192-page slices and a final
    pass (k <= 4096) or in one streamed pass (k = 5000)."""
    T, Hq, Hkv, page = 16 * 16500 + 3, 4, 1, 16
    r = np.random.default_rng(77)
    pat = r.standard_normal((3, page, 128)).astype(np.float16).view(np.uint16)
    which = r.integers(0, 3, size=(T + page - 1) // page)
    ks = np.ascontiguousarray(pat[which].reshape(-1, 128)[:T])[None, None]
    vs = np.zeros_like(ks)
    cache = _build(gpu, ks, vs, Hq, olad.ladder("exact", T), page=page)
    q = synth.queries(3, 1, Hq, step=3)
    kmin, kmax = oquest.page_boxes(ks[0, 0])
    n = (T - 1) // page
    s = oquest.page_scores(q[0], kmin[:n], kmax[:n])
    assert len(np.unique(s)) == 3
    got = cache.quest_select(q, k).cpu().numpy()[0, 0]
    np.testing.assert_array_equal(got, oquest.select_top(s, k))


def test_rd_residual_streamed_selection(gpu):
    """A residual of 5000 rows out of 9001 tokens (more than half of a 8192-key slice)
    takes the single streamed selection pass; residual set and mask bit-exact."""
    T, Hq, Hkv, n = 9001, 8, 1, 5000
    ks, vs = kv_all(4, 1, Hkv, T)
    lv = olad.ladder("graded", T)
    cache = _build(gpu, ks, vs, Hq, lv, nres_cap=n)
    mass = synth.mass_unit(4, 0, 0, T)[None, None]
    cache.rd_residual_select(ks, vs, mass, n)
    uc = ocache.UnitCache(ks[0, 0], vs[0, 0], lv)
    want, sc = uc.select_residual(ks[0, 0], vs[0, 0], mass[0, 0], n)
    np.testing.assert_array_equal(cache.res_idx.cpu().numpy()[0, 0, :n], want)
    check_rd_keys(cache, 0, 0, T, sc)
    q = synth.queries(4, 1, Hq)
    out = cache.decode(q).cpu().numpy()
    assert max_err(out[0], uc.decode_dense(q_group(q, 0, 0, Hq))) <= TOL


def test_quest_1m_sampled(gpu):
    """Workload 5 at its launch configuration (T = 2^20, 65,535 ranked pages, 32
    query / 8 KV heads, top-256): KV heads 0 and 7 hold their own seeded data and
    the other six repeat them, so that the selection and plan grids are the
    benchmarked ones.  For the two sampled heads: boxes, box-bound selection
    (bit-exact), attention over the selected pages (against the oracle, which
    encodes only the blocks the read set touches), then one append that opens a
    block and the demotions it triggers (bit-exact records)."""
    import types
    from oracle import attention as oattn
    T, Hq, Hkv, page, topk = 1 << 20, 32, 8, 16, 256
    G = Hq // Hkv
    samp = [0, Hkv - 1]
    data = {h: synth.kv_unit(5, 0, h, T + 1) for h in samp}
    ks = np.empty((1, Hkv, T + 1, 128), np.uint16)
    vs = np.empty((1, Hkv, T + 1, 128), np.uint16)
    for h in range(Hkv):
        ks[0, h], vs[0, h] = data[samp[h % 2]]
    lv = olad.ladder("graded", T)
    cache = _build(gpu, ks[:, :, :T], vs[:, :, :T], Hq, lv, page=page, extra_blocks=2,
                   slack={16: 2 * Hkv, 8: 8 * Hkv, 4: 8 * Hkv, 2: 8 * Hkv, 1: 8 * Hkv})
    q = synth.queries(5, 1, Hq, step=0)
    pages = cache.quest_select(q, topk)
    out = cache.decode(q, pages=pages).cpu().numpy()
    pages = pages.cpu().numpy()
    for h in samp:
        kmin, kmax = oquest.page_boxes(ks[0, h, :T])
        gmin, gmax = cache.boxes_host(0, h, T // page)
        np.testing.assert_array_equal(gmin, kmin)
        np.testing.assert_array_equal(gmax, kmax)
        want = oquest.quest_select(q_group(q, 0, h, G), kmin, kmax, T, topk)
        np.testing.assert_array_equal(pages[0, h], want)
        idx = oquest.read_tokens(want, T)
        kh = np.empty((len(idx), 128))
        vh = np.empty((len(idx), 128))
        for blk in np.unique(idx // 64):
            rows = slice(blk * 64, (blk + 1) * 64)
            sel = (idx // 64) == blk
            kh[sel] = oquant.decode(oquant.encode_fp16(int(lv[blk]), ks[0, h, rows]))[idx[sel] - blk * 64]
            vh[sel] = oquant.decode(oquant.encode_fp16(int(lv[blk]), vs[0, h, rows]))[idx[sel] - blk * 64]
        ref = oattn.unit_decode(q_group(q, 0, h, G), kh, vh)
        assert max_err(out[0, h * G:(h + 1) * G], ref) <= TOL
    # the next token opens block 2^14: every block whose level the ladder lowers is
    # re-encoded from its record
    moves = cache.append(ks[:, :, T], vs[:, :, T], profile="graded")
    lv1 = olad.ladder("graded", T + 1)
    want_moves = sorted((h, int(i), int(lv[i]), int(lv1[i])) for h in range(Hkv)
                        for i in range(len(lv)) if lv1[i] != lv[i])
    assert sorted((h, blk, o, n) for b, h, blk, o, n in moves) == want_moves
    assert moves
    for b, h, blk, old, new in moves:
        if h not in samp:
            continue
        rows = slice(blk * 64, (blk + 1) * 64)
        ko = oquant.demote(oquant.encode_fp16(old, ks[0, h, rows]), new)
        vo = oquant.demote(oquant.encode_fp16(old, vs[0, h, rows]), new)
        uc = types.SimpleNamespace(k_recs={blk: ko}, v_recs={blk: vo})
        compare_record(cache, uc, 0, h, blk, 0)
        compare_record(cache, uc, 0, h, blk, 1)


def _cert_compare(cache, uc, b, h):
    """The cache's per-block certificate numbers against the oracle's: fp32 rounded
    upwards from fp64, so never below and within a few ulps above."""
    nblk = len(uc.levels)
    got = cache.cert[b, h, :nblk, :3].cpu().numpy().astype(np.float64)
    want = np.stack([uc.kerr, uc.verr, uc.vmax], 1)
    assert np.all(got >= want * (1 - 1e-12))
    assert np.all(got <= want * (1 + 1e-6) + 1e-30)


def _bound_close(got, want):
    assert np.all(np.abs(got - want) <= 2e-3 * want + 1e-6), (got, want)


@pytest.mark.parametrize("prof,T,Bn", [("tiny", 2048, 1), ("graded", 5000, 2), ("int8", 2048, 1)])
def test_certificate_numbers_and_bound(gpu, prof, T, Bn):
    """Decode-time attention error certificate (section 3.6): per-block numbers written
    by the encoder and the per-head bound from the attention kernel and merge, against
    the oracle; the output equals the plain decode bit for bit."""
    torch = _torch()
    Hq, Hkv = 8, 2
    ks, vs = kv_all(6, Bn, Hkv, T)
    lv = np.full(T // 64, olad.INT8, np.int8) if prof == "int8" else olad.ladder(prof, T)
    cache = _build(gpu, ks, vs, Hq, lv)
    q = synth.queries(6, Bn, Hq)
    out, bnd = cache.decode_bound(q)
    assert torch.equal(out, cache.decode(q))
    bnd = bnd.cpu().numpy()
    G = Hq // Hkv
    for b in range(Bn):
        for h in range(Hkv):
            uc = ocache.UnitCache(ks[b, h], vs[b, h], lv)
            _cert_compare(cache, uc, b, h)
            _bound_close(bnd[b, h * G:(h + 1) * G], uc.certificate(q_group(q, b, h, G)))
    if prof == "int8":  # informative: well below the universal cap of 2 max ||v||
        assert np.all(bnd < 0.5 * 2 * cache.cert[..., 2].max().item())


def test_certificate_with_residual_rows(gpu):
    """Residual rows count as exact in the bound."""
    T, Hq, Hkv = 3000, 8, 2
    ks, vs = kv_all(7, 1, Hkv, T)
    lv = olad.ladder("graded", T)
    n = ores.n_keep(T, 2)
    cache = _build(gpu, ks, vs, Hq, lv, nres_cap=n)
    mass = np.stack([synth.mass_unit(7, 0, h, T) for h in range(Hkv)])[None]
    cache.rd_residual_select(ks, vs, mass, n)
    q = synth.queries(7, 1, Hq)
    _, bnd = cache.decode_bound(q)
    bnd = bnd.cpu().numpy()
    G = Hq // Hkv
    for h in range(Hkv):
        uc = ocache.UnitCache(ks[0, h], vs[0, h], lv)
        uc.select_residual(ks[0, h], vs[0, h], mass[0, h], n)
        _bound_close(bnd[0, h * G:(h + 1) * G], uc.certificate(q_group(q, 0, h, G)))


def test_certificate_through_appends_and_demotions(gpu):
    """Appends open exact blocks and raise the value norms; demotions raise the
    errors by the change of the reconstruction; the bound follows the oracle."""
    Hq, Hkv = 8, 2
    T0 = 64 * 40 - 3
    steps = 70
    ks, vs = kv_all(8, 1, Hkv, T0 + steps)
    lv = olad.ladder("graded", T0)
    cache = _build(gpu, ks[:, :, :T0], vs[:, :, :T0], Hq, lv, extra_blocks=4,
                   slack={16: 8, 8: 8, 4: 8, 2: 8, 1: 8})
    ucs = [ocache.UnitCache(ks[0, h, :T0], vs[0, h, :T0], lv) for h in range(Hkv)]
    nmoves = 0
    for s in range(steps):
        t = T0 + s
        nmoves += len(cache.append(ks[:, :, t], vs[:, :, t], profile="graded"))
        for h in range(Hkv):
            ucs[h].append(ks[0, h, t], vs[0, h, t], "graded")
    assert nmoves > 0
    q = synth.queries(8, 1, Hq)
    _, bnd = cache.decode_bound(q)
    bnd = bnd.cpu().numpy()
    G = Hq // Hkv
    for h in range(Hkv):
        _cert_compare(cache, ucs[h], 0, h)
        _bound_close(bnd[0, h * G:(h + 1) * G], ucs[h].certificate(q_group(q, 0, h, G)))


# ---------------------------------------------------------------- one-centroid state, RD-V2


@pytest.mark.parametrize("T,Bn", [(8192, 2), (3001, 1), (7464, 1)])
def test_rdv2_codes_residual_attention_and_bound(gpu, T, Bn):
    """RD-V2 (section 3.4): newest 16 blocks exact, older blocks one-centroid, and
    10.2% exact residual rows by Eq. rdscore against the block mean; 28 query / 4 KV
    heads.  Records, residual sets and masks bit-exact; attention and certificate
    against the oracle.  T = 7464 (117 blocks, 12 residual pseudo-blocks) puts the
    visit group that holds the last block and the first residual rows inside the
    plan's reordered range, onto a group of one-centroid blocks."""
    torch = _torch()
    Hq, Hkv = 28, 4
    ks, vs = kv_all(9, Bn, Hkv, T)
    lv = olad.ladder("rdv2", T)
    n = ores.n_keep(T, 102, 1000)
    cache = _build(gpu, ks, vs, Hq, lv, nres_cap=n)
    mass = np.stack([np.stack([synth.mass_unit(9, b, h, T) for h in range(Hkv)]) for b in range(Bn)])
    cache.rd_residual_select(ks, vs, mass, n)
    q = synth.queries(9, Bn, Hq)
    out, bnd = cache.decode_bound(q)
    assert torch.equal(out, cache.decode(q))
    out, bnd = out.cpu().numpy(), bnd.cpu().numpy()
    idx = cache.res_idx.cpu().numpy()
    G = Hq // Hkv
    for b in range(Bn):
        for h in range(Hkv):
            uc = ocache.UnitCache(ks[b, h], vs[b, h], lv)
            for blk in (0, 1, len(lv) // 2, len(lv) - 17, len(lv) - 16, len(lv) - 1):
                compare_record(cache, uc, b, h, blk, 0)
                compare_record(cache, uc, b, h, blk, 1)
            want, sc = uc.select_residual(ks[b, h], vs[b, h], mass[b, h], n)
            np.testing.assert_array_equal(idx[b, h, :n], want)
            check_rd_keys(cache, b, h, T, sc)
            ref = uc.decode_dense(q_group(q, b, h, G))
            assert max_err(out[b, h * G:(h + 1) * G], ref) <= TOL
            _cert_compare(cache, uc, b, h)
            _bound_close(bnd[b, h * G:(h + 1) * G], uc.certificate(q_group(q, b, h, G)))


def test_demote_every_level_to_mean(gpu):
    """gkv_demote to the one-centroid state from every other level, bit-exact, and
    attention over the result."""
    T, Hq, Hkv = 512, 4, 2
    ks, vs = kv_all(52, 1, Hkv, T)
    lv = np.array([16, 8, 4, 2, 1, 16, 16, 16], dtype=np.int8)
    cache = _build(gpu, ks, vs, Hq, lv, slack={0: 16})
    ucs = oracle_units(ks, vs, lv)
    jobs = [(0, h, blk) for h in range(Hkv) for blk in range(5)]
    cache.demote(jobs, [0] * len(jobs))
    for (b, h), uc in ucs.items():
        for blk in range(5):
            uc.k_recs[blk] = oquant.demote(uc.k_recs[blk], 0)
            uc.v_recs[blk] = oquant.demote(uc.v_recs[blk], 0)
            uc.levels[blk] = 0
            compare_record(cache, uc, b, h, blk, 0)
            compare_record(cache, uc, b, h, blk, 1)
    with pytest.raises(Exception):
        cache.demote([(0, 0, 1)], [1])
    q = synth.queries(52, 1, Hq)
    out = cache.decode(q).cpu().numpy()
    for (b, h), uc in ucs.items():
        assert max_err(out[b, 2 * h:2 * h + 2], uc.decode_dense(q_group(q, b, h, 2))) <= TOL


def test_rdv2_append_steps_with_quest_pages(gpu):
    """Decode steps on an RD-V2 ladder: appends open exact blocks and demote the
    block leaving the exact window straight to the one-centroid state; Compressed-
    Quest selects pages by their exact boxes and reads one-centroid pages as counted
    single keys; dense and sparse reads against the oracle at every step."""
    Hq, Hkv, page, topk = 8, 2, 16, 20
    T0 = 64 * 24 - 5
    steps = 70
    ks, vs = kv_all(53, 1, Hkv, T0 + steps)
    lv = olad.ladder("rdv2", T0)
    cache = _build(gpu, ks[:, :, :T0], vs[:, :, :T0], Hq, lv, page=page, extra_blocks=4, slack={16: 8, 0: 8})
    ucs = {(0, h): ocache.UnitCache(ks[0, h, :T0], vs[0, h, :T0], lv) for h in range(Hkv)}
    G = Hq // Hkv
    nmoves = 0
    for s in range(steps):
        t = T0 + s
        moves = cache.append(ks[:, :, t], vs[:, :, t], profile="rdv2")
        nmoves += len(moves)
        for h in range(Hkv):
            omoves = ucs[(0, h)].append(ks[0, h, t], vs[0, h, t], "rdv2")
        assert sorted((blk, o, n) for b, h, blk, o, n in moves if h == 0) == sorted(omoves)
        assert all(o == 16 and n == 0 for b, h, blk, o, n in moves)
        q = synth.queries(53, 1, Hq, step=s)
        pages = cache.quest_select(q, topk)
        out = cache.decode(q, pages=pages).cpu().numpy()
        dense = cache.decode(q).cpu().numpy()
        pages = pages.cpu().numpy()
        T = t + 1
        for h in range(Hkv):
            uc = ucs[(0, h)]
            kmin, kmax = oquest.page_boxes(ks[0, h, :T])
            want = oquest.quest_select(q_group(q, 0, h, G), kmin, kmax, T, topk)
            np.testing.assert_array_equal(pages[0, h], want)
            assert max_err(out[0, h * G:(h + 1) * G], uc.decode_quest(q_group(q, 0, h, G), want)) <= TOL
            assert max_err(dense[0, h * G:(h + 1) * G], uc.decode_dense(q_group(q, 0, h, G))) <= TOL
            for b_, h_, blk, o, n in moves:
                if h_ == h:
                    compare_record(cache, uc, 0, h, blk, 0)
                    compare_record(cache, uc, 0, h, blk, 1)
    assert nmoves == 2 * Hkv  # two blocks leave the exact window per KV head in 70 steps


@pytest.mark.parametrize("prof,frac,vtok", [("graded", (2, 100), False), ("rdv2", (102, 1000), False),
                                           ("graded", (2, 100), True)])
def test_rd128k_full_size_sampled(gpu, prof, frac, vtok):
    """The 128k decode step at its full size and launch configuration (B = 8, 28
    query / 4 KV heads, T = 131072): graded ladder with 2% residual rows, and RD-V2
    with 10.2%, and the graded ladder with values quantised per token.  Units (0, 0)
    and (7, 3) hold their own seeded data and are checked
    against the oracle (sampled records, residual set, attention); the other 30
    units repeat those two, so that the launch covers the whole grid."""
    from paper_2608_23599_amd import workloads
    wl = workloads.RD128K
    B, Hq, Hkv, T = wl.B, wl.Hq, wl.Hkv, wl.T
    samp = [(0, 0), (B - 1, Hkv - 1)]
    data = {u: synth.kv_unit(wl.id, *u, T) for u in samp}
    masses = {u: synth.mass_unit(wl.id, *u, T) for u in samp}
    ks = np.empty((B, Hkv, T, 128), np.uint16)
    vs = np.empty((B, Hkv, T, 128), np.uint16)
    mass = np.empty((B, Hkv, T), np.float32)
    for b in range(B):
        for h in range(Hkv):
            u = samp[(b * Hkv + h) % 2]
            ks[b, h], vs[b, h] = data[u]
            mass[b, h] = masses[u]
    lv = olad.ladder(prof, T)
    n = ores.n_keep(T, *frac)
    cache = _build(gpu, ks, vs, Hq, lv, nres_cap=n, v_per_token=vtok)
    cache.rd_residual_select(ks, vs, mass, n)
    q = synth.queries(wl.id, B, Hq)
    out_d = cache.decode(q)
    # the same call again gives the same bits (one-centroid runs zero their stale rows)
    assert _torch().equal(cache.decode(q), out_d)
    out = out_d.cpu().numpy()
    idx = cache.res_idx.cpu().numpy()
    G = Hq // Hkv
    for b, h in samp:
        uc = ocache.UnitCache(ks[b, h], vs[b, h], lv, v_per_token=vtok)
        for blk in (0, 1, 700, 1500, len(lv) - 17, len(lv) - 1):
            compare_record(cache, uc, b, h, blk, 0)
            compare_record(cache, uc, b, h, blk, 1)
        want, sc = uc.select_residual(ks[b, h], vs[b, h], mass[b, h], n)
        np.testing.assert_array_equal(idx[b, h, :n], want)
        check_rd_keys(cache, b, h, T, sc)
        assert max_err(out[b, h * G:(h + 1) * G], uc.decode_dense(q_group(q, b, h, G))) <= TOL


# ---------------------------------------------------------------- values grouped per token


def _units_per_token(ks, vs, lv):
    B, Hkv = ks.shape[:2]
    return {(b, h): ocache.UnitCache(ks[b, h], vs[b, h], lv, v_per_token=True) for b in range(B) for h in range(Hkv)}


@pytest.mark.parametrize("prof,T,Bn,Hq,Hkv", [("tiny", 2048, 1, 8, 2), ("graded", 5000, 2, 28, 4),
                                              ("tiny", 1000, 1, 32, 2)])
def test_per_token_values_codes_attention_and_bound(gpu, prof, T, Bn, Hq, Hkv):
    """Values quantised per token (one scale and zero per token over its channels):
    records bit-exact (keys stay per channel), attention and certificate against the
    oracle; G = 16 runs the kernel without packed query columns."""
    torch = _torch()
    ks, vs = kv_all(10, Bn, Hkv, T)
    lv = olad.ladder(prof, T)
    cache = _build(gpu, ks, vs, Hq, lv, v_per_token=True)
    ucs = _units_per_token(ks, vs, lv)
    for (b, h), uc in ucs.items():
        for blk in sorted(set(range(0, len(lv), 3)) | {len(lv) - 1}):
            compare_record(cache, uc, b, h, blk, 0)
            compare_record(cache, uc, b, h, blk, 1)
    q = synth.queries(10, Bn, Hq)
    out, bnd = cache.decode_bound(q)
    assert torch.equal(out, cache.decode(q))
    out, bnd = out.cpu().numpy(), bnd.cpu().numpy()
    G = Hq // Hkv
    for (b, h), uc in ucs.items():
        assert max_err(out[b, h * G:(h + 1) * G], uc.decode_dense(q_group(q, b, h, G))) <= TOL
        _cert_compare(cache, uc, b, h)
        _bound_close(bnd[b, h * G:(h + 1) * G], uc.certificate(q_group(q, b, h, G)))


def test_per_token_values_demotion_and_residual(gpu):
    """Demotion re-encodes per-token value records (8 -> 4 -> 2 -> centroid), and the
    residual scores values against their per-token reconstruction."""
    T, Hq, Hkv = 64 * 12, 8, 2
    ks, vs = kv_all(11, 1, Hkv, T)
    lv = olad.ladder("exact", T)
    n = ores.n_keep(T, 5)
    cache = _build(gpu, ks, vs, Hq, lv, nres_cap=n, slack={8: 16, 4: 16, 2: 16, 1: 16}, v_per_token=True)
    ucs = _units_per_token(ks, vs, lv)
    for to in (8, 4, 2, 1):
        jobs = [(0, h, blk) for h in range(Hkv) for blk in (0, 2, 5)]
        cache.demote(jobs, [to] * len(jobs))
        for (b, h), uc in ucs.items():
            for blk in (0, 2, 5):
                uc.k_recs[blk] = oquant.demote(uc.k_recs[blk], to)
                uc.v_recs[blk] = oquant.demote(uc.v_recs[blk], to)
                uc.levels[blk] = to
                compare_record(cache, uc, b, h, blk, 0)
                compare_record(cache, uc, b, h, blk, 1)
        if to == 4:  # residual selection over a mix of exact and per-token int4 blocks
            mass = np.stack([synth.mass_unit(11, 0, h, T) for h in range(Hkv)])[None]
            cache.rd_residual_select(ks, vs, mass, n)
            idx = cache.res_idx.cpu().numpy()
            for (b, h), uc in ucs.items():
                import copy
                want, sc = copy.deepcopy(uc).select_residual(ks[b, h], vs[b, h], mass[b, h], n)
                np.testing.assert_array_equal(idx[b, h, :n], want)
                check_rd_keys(cache, b, h, T, sc)
    q = synth.queries(11, 1, Hq)
    mass = np.stack([synth.mass_unit(11, 0, h, T) for h in range(Hkv)])[None]
    out = cache.decode(q).cpu().numpy()
    for (b, h), uc in ucs.items():
        # the residual chosen at int4 time, read over the demoted blocks
        sel = cache.res_idx.cpu().numpy()[b, h, :n]
        uc.res_idx = sel.astype(np.int32)
        uc.res_k = ks[b, h][sel]
        uc.res_v = vs[b, h][sel]
        assert max_err(out[b, 4 * h:4 * h + 4], uc.decode_dense(q_group(q, b, h, 4))) <= TOL


def test_per_token_values_quest_pages(gpu):
    T, Hq, Hkv, page, topk = 6000, 8, 2, 16, 40
    ks, vs = kv_all(12, 1, Hkv, T)
    lv = olad.ladder("graded", T)
    cache = _build(gpu, ks, vs, Hq, lv, page=page, v_per_token=True)
    q = synth.queries(12, 1, Hq)
    pages = cache.quest_select(q, topk)
    out = cache.decode(q, pages=pages).cpu().numpy()
    pages = pages.cpu().numpy()
    for (b, h), uc in _units_per_token(ks, vs, lv).items():
        assert max_err(out[b, 4 * h:4 * h + 4], uc.decode_quest(q_group(q, b, h, 4), pages[b, h])) <= TOL


def test_rdv2_long_context_runs(gpu):
    """RD-V2 beyond 4096 visits per (b, KV head) (T = 300,001: the plan's looped path),
    with a residual: one-centroid runs, their edges at residual-free and ragged
    places, against the oracle."""
    T, Hq, Hkv = 300001, 4, 1
    ks, vs = kv_all(13, 1, Hkv, T)
    lv = olad.ladder("rdv2", T)
    n = ores.n_keep(T, 1, 100)
    cache = _build(gpu, ks, vs, Hq, lv, nres_cap=n)
    mass = synth.mass_unit(13, 0, 0, T)[None, None]
    cache.rd_residual_select(ks, vs, mass, n)
    q = synth.queries(13, 1, Hq)
    out = cache.decode(q).cpu().numpy()
    uc = ocache.UnitCache(ks[0, 0], vs[0, 0], lv)
    uc.select_residual(ks[0, 0], vs[0, 0], mass[0, 0], n)
    assert max_err(out[0], uc.decode_dense(q_group(q, 0, 0, Hq))) <= TOL


# ---------------------------------------------------------------- multi-layer service


@pytest.mark.parametrize("skew", [False, True])
def test_layers_step_matches_per_layer_appends(gpu, skew):
    """gkv_layers_step on 3 layers (one call per decode step: appends, each layer's
    crossings, demotions, slot recycling) against the same layers stepped one by one
    with gkv_append / gkv_demote: identical levels, offsets, records, pool use and
    decode outputs at every step, and each layer against the oracle at the end.
    With skew, layer 1 starts from the ladder of a context 640 tokens shorter (its
    newer blocks exact), so its levels differ from the other layers' and its first
    step demotes blocks that theirs does not."""
    torch = _torch()
    L, Hq, Hkv, page = 3, 8, 2, 16
    T0 = 64 * 40 - 3
    steps = 70
    data = [kv_all(70 + l, 1, Hkv, T0 + steps) for l in range(L)]
    lv = olad.ladder("graded", T0)
    lvs = [lv] * L
    if skew:
        short = olad.ladder("graded", T0 - 640)
        lvs[1] = np.concatenate([short, np.full(len(lv) - len(short), 16, np.int8)])
        assert not np.array_equal(lvs[1], lv)
    slack = {16: 8, 8: 16, 4: 16, 2: 16, 1: 16}
    mk = lambda ks, vs, lvl: _build(gpu, ks[:, :, :T0], vs[:, :, :T0], Hq, lvl, page=page, extra_blocks=4,
                                    slack=slack)
    svc = gpu.LayerCaches([mk(*d, lvs[l]) for l, d in enumerate(data)], "graded")
    ref = [mk(*d, lvs[l]) for l, d in enumerate(data)]
    G = Hq // Hkv
    total = 0
    for s in range(steps):
        t = T0 + s
        kn = np.stack([d[0][:, :, t] for d in data])
        vn = np.stack([d[1][:, :, t] for d in data])
        n = svc.step(kn, vn)
        moves = [r.append(kn[l], vn[l], profile="graded") for l, r in enumerate(ref)]
        assert sum(len(m) for m in moves) == n
        if skew and s == 0:
            assert len(moves[1]) > len(moves[0])
        total += n
        q = synth.queries(71, 1, Hq, step=s)
        for l in range(L):
            a, b = svc.caches[l], ref[l]
            assert a.T == b.T == t + 1
            np.testing.assert_array_equal(a.level_host, b.level_host)
            np.testing.assert_array_equal(a.koff_host, b.koff_host)
            np.testing.assert_array_equal(a.voff_host, b.voff_host)
            assert all(a.pool.used(x) == b.pool.used(x) for x in gpu.LEVELS)
            assert torch.equal(a.decode(q), b.decode(q))
    assert total > 0
    for l, (ks, vs) in enumerate(data):
        T = T0 + steps
        uc = ocache.UnitCache(ks[0, 0, :T0], vs[0, 0, :T0], lvs[l])
        for t in range(T0, T):
            uc.append(ks[0, 0, t], vs[0, 0, t], "graded")
        for blk in range(T // 64):  # complete blocks (rows past T of the newest are not defined)
            compare_record(svc.caches[l], uc, 0, 0, blk, 0)
            compare_record(svc.caches[l], uc, 0, 0, blk, 1)
        q = synth.queries(71, 1, Hq, step=steps)
        out = svc.caches[l].decode(q).cpu().numpy()
        assert max_err(out[0, 0:G], uc.decode_dense(q_group(q, 0, 0, G))) <= TOL


def test_layers_step_more_layers_than_one_launch(gpu):
    """gkv_layers_step over 18 layers (more than the 16 one append launch serves),
    through steps that open no block and one that does, against the same layers
    appended one by one: identical levels, offsets, pool use and decode outputs."""
    torch = _torch()
    L, Hq, Hkv = 18, 4, 1
    T0 = 64 * 6 - 3
    steps = 5  # step 3 opens block 6
    data = [kv_all(90 + l, 1, Hkv, T0 + steps) for l in range(L)]
    lv = olad.ladder("graded", T0)
    slack = {16: 4, 8: 4, 4: 4, 2: 4, 1: 4}
    mk = lambda ks, vs: _build(gpu, ks[:, :, :T0], vs[:, :, :T0], Hq, lv, extra_blocks=2, slack=slack)
    svc = gpu.LayerCaches([mk(*d) for d in data], "graded")
    ref = [mk(*d) for d in data]
    for s_ in range(steps):
        t = T0 + s_
        kn = np.stack([d[0][:, :, t] for d in data])
        vn = np.stack([d[1][:, :, t] for d in data])
        n = svc.step(kn, vn)
        moves = [r.append(kn[l], vn[l], profile="graded") for l, r in enumerate(ref)]
        assert sum(len(m) for m in moves) == n
        q = synth.queries(91, 1, Hq, step=s_)
        for l in range(L):
            a, b = svc.caches[l], ref[l]
            assert a.T == b.T == t + 1
            np.testing.assert_array_equal(a.level_host, b.level_host)
            np.testing.assert_array_equal(a.koff_host, b.koff_host)
            np.testing.assert_array_equal(a.voff_host, b.voff_host)
            assert all(a.pool.used(x) == b.pool.used(x) for x in gpu.LEVELS)
            assert torch.equal(a.decode(q), b.decode(q))


def test_opened_block_rows_are_defined(gpu):
    """A block opened by an append gets zero rows past the token: free slots filled
    with NaN bit patterns (as recycled records can hold) must not reach the output
    (masked rows meet P = 0 in the P.V product, and 0 * NaN is NaN)."""
    T0, Hq, Hkv = 64 * 8, 4, 1
    ks, vs = kv_all(14, 1, Hkv, T0 + 3)
    lv = olad.ladder("tiny", T0)
    cache = _build(gpu, ks[:, :, :T0], vs[:, :, :T0], Hq, lv, extra_blocks=2, slack={16: 4, 8: 4, 4: 4, 2: 4})
    off = cache.pool.alloc(16)
    cache.pool.free(16, off)
    cache.arena[off:off + 4 * 16384] = 0xFF  # every free exact slot: fp16 NaN patterns
    uc = ocache.UnitCache(ks[0, 0, :T0], vs[0, 0, :T0], lv)
    for t in range(T0, T0 + 3):
        cache.append(ks[:, :, t], vs[:, :, t], profile="tiny")
        uc.append(ks[0, 0, t], vs[0, 0, t], "tiny")
        q = synth.queries(14, 1, Hq, step=t)
        out = cache.decode(q).cpu().numpy()
        assert np.all(np.isfinite(out))
        assert max_err(out[0], uc.decode_dense(q_group(q, 0, 0, Hq))) <= TOL


def test_graph_replays_match_eager(gpu):
    """A Compressed-Quest step and a dense step captured in one HIP graph: every
    replay, with eager work and synchronisations between replays, equals the eager
    result bit for bit (the calls allocate nothing and clear nothing on the device)."""
    torch = _torch()
    T, Hq, Hkv, page, topk = 5000, 8, 2, 16, 40
    ks, vs = kv_all(15, 1, Hkv, T)
    lv = olad.ladder("graded", T)
    cache = _build(gpu, ks, vs, Hq, lv, page=page)
    q = torch.from_numpy(synth.queries(15, 1, Hq).view(np.int16)).cuda()
    pages = torch.empty((1, Hkv, topk), dtype=torch.int32, device="cuda")
    out_q = torch.empty((1, Hq, 128), dtype=torch.float32, device="cuda")
    out_d = torch.empty_like(out_q)
    cache.quest_select(q, topk, out=pages)
    cache.decode(q, pages=pages, out=out_q)
    cache.decode(q, out=out_d)
    torch.cuda.synchronize()
    want = (pages.clone(), out_q.clone(), out_d.clone())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        cache.quest_select(q, topk, out=pages)
        cache.decode(q, pages=pages, out=out_q)
        cache.decode(q, out=out_d)
    for rep in range(3):
        pages.fill_(-7)
        out_q.zero_()
        out_d.zero_()
        cache.decode(q, out=torch.empty_like(out_d))  # eager work on the same workspace between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(pages, want[0]) and torch.equal(out_q, want[1]) and torch.equal(out_d, want[2]), rep


def test_quest128k_b8_full_size_sampled(gpu):
    """The Compressed-Quest 128k point at its full launch configuration (B = 8, 32
    query / 8 KV heads, T = 131072, 16-token pages, top-128): units (0, 0) and (7, 7)
    hold their own seeded data (the others repeat them) and their boxes, page sets
    (bit-exact) and sparse attention are checked against the oracle."""
    from oracle import attention as oattn
    B, Hq, Hkv, T, page, topk = 8, 32, 8, 131072, 16, 128
    G = Hq // Hkv
    samp = [(0, 0), (B - 1, Hkv - 1)]
    data = {u: synth.kv_unit(3, *u, T) for u in samp}
    ks = np.empty((B, Hkv, T, 128), np.uint16)
    vs = np.empty((B, Hkv, T, 128), np.uint16)
    for b in range(B):
        for h in range(Hkv):
            ks[b, h], vs[b, h] = data[samp[(b * Hkv + h) % 2]]
    lv = olad.ladder("graded", T)
    cache = _build(gpu, ks, vs, Hq, lv, page=page)
    q = synth.queries(3, B, Hq)
    pages = cache.quest_select(q, topk)
    out = cache.decode(q, pages=pages).cpu().numpy()
    pages = pages.cpu().numpy()
    for b, h in samp:
        kmin, kmax = oquest.page_boxes(ks[b, h])
        want = oquest.quest_select(q_group(q, b, h, G), kmin, kmax, T, topk)
        np.testing.assert_array_equal(pages[b, h], want)
        idx = oquest.read_tokens(want, T)
        kh = np.empty((len(idx), 128))
        vh = np.empty((len(idx), 128))
        for blk in np.unique(idx // 64):
            rows = slice(blk * 64, (blk + 1) * 64)
            sel = (idx // 64) == blk
            kh[sel] = oquant.decode(oquant.encode_fp16(int(lv[blk]), ks[b, h, rows]))[idx[sel] - blk * 64]
            vh[sel] = oquant.decode(oquant.encode_fp16(int(lv[blk]), vs[b, h, rows]))[idx[sel] - blk * 64]
        assert max_err(out[b, h * G:(h + 1) * G], oattn.unit_decode(q_group(q, b, h, G), kh, vh)) <= TOL


# ---------------------------------------------------------------- dense plan reuse


def test_dense_plan_reuse_follows_the_tables(gpu):
    """A dense read reuses the visit plan a workspace holds only for the same table
    state: two caches alternating on one workspace, an append (T grows), a demotion
    (levels and slots change), a residual selection (rows leave their blocks) and a
    Compressed-Quest read on the same workspace in between each give the output of a
    call with a fresh workspace, bit for bit.  The workspace's tag carries the
    cache's version after a dense call; a Compressed-Quest read (which lists its
    pages in the attention kernel) leaves it in place."""
    import ctypes
    torch = _torch()
    T, Hq, Hkv = 2048, 8, 2
    (ka, va), (kb, vb) = kv_all(40, 1, Hkv, T + 1), kv_all(41, 1, Hkv, T)
    lv = olad.ladder("tiny", T)
    A = _build(gpu, ka[:, :, :T], va[:, :, :T], Hq, lv, page=16, extra_blocks=2, nres_cap=64,
               slack={16: 4, 8: 4, 4: 4, 2: 4, 1: 4})
    Bc = _build(gpu, kb, vb, Hq, lv, page=16, extra_blocks=2, nres_cap=64, slack={16: 4, 8: 4, 4: 4, 2: 4, 1: 4})
    q = synth.queries(40, 1, Hq)
    nbytes = max(A.workspace(1, 0).numel(), A.workspace(1, 32).numel())
    shared = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")

    def dec(c, pages=None):
        out = torch.empty((1, Hq, 128), dtype=torch.float32, device="cuda")
        topk = 0 if pages is None else int(pages.shape[-1])
        st = gpu._attn(gpu._dptr(gpu._as_bits(q, "cuda")), ctypes.byref(c.c), gpu._dptr(pages), topk,
                       gpu._dptr(out), gpu._dptr(shared), shared.numel(), gpu._stream())
        assert st == 0
        return out

    def fresh(c, pages=None):
        c._ws = {}
        return c.decode(q, pages=pages)

    def tag():
        torch.cuda.synchronize()
        return int(shared[:8].cpu().numpy().view(np.uint64)[0])

    for c in (A, Bc, A, Bc, A):
        assert torch.equal(dec(c), fresh(c))
        assert tag() == c.c.version
    A.append(ka[:, :, T], va[:, :, T], profile="tiny")
    assert torch.equal(dec(A), fresh(A))
    Bc.demote([(0, 0, 5), (0, 1, 9)], [1, 2])  # int2 -> centroid, int4 -> int2
    assert torch.equal(dec(Bc), fresh(Bc))
    mass = np.stack([synth.mass_unit(41, 0, h, T) for h in range(Hkv)])[None]
    Bc.rd_residual_select(kb, vb, mass, 64)
    assert torch.equal(dec(Bc), fresh(Bc))
    before = tag()
    assert before == Bc.c.version
    pages = A.quest_select(q, 32)
    assert torch.equal(dec(A, pages), fresh(A, pages))
    assert tag() == before  # a Compressed-Quest read has no plan and leaves the dense one in place
    assert torch.equal(dec(Bc), fresh(Bc))
    assert torch.equal(dec(A), fresh(A))
    # the reused plan is the same one: the same call twice gives the same bits
    assert torch.equal(dec(A), dec(A))


# ---------------------------------------------------------------- Compressed-Quest with a residual


@pytest.mark.parametrize("page,T,topk,frac,Bn", [(16, 6001, 64, (2, 100), 2), (16, 4096, 60, (20, 100), 1),
                                                 (32, 5003, 40, (10, 100), 1), (64, 8192, 20, (10, 100), 1)])
def test_quest_read_with_residual_rows(gpu, page, T, topk, frac, Bn):
    """A Compressed-Quest read of a cache with exact residual rows (sections 3.4 and
    3.5): the rows of residual tokens in the selected pages or the current page
    override their graded entries (the oracle's decode_quest on the same residual),
    for 16-, 32- and 64-token pages, 2% to 20% residual rows, a partial current page;
    the read accounting matches the oracle's."""
    Hq, Hkv = 8, 2
    G = Hq // Hkv
    ks, vs = kv_all(44, Bn, Hkv, T)
    lv = olad.ladder("graded", T)
    n = ores.n_keep(T, *frac)
    cache = _build(gpu, ks, vs, Hq, lv, page=page, nres_cap=n)
    mass = np.stack([np.stack([synth.mass_unit(44, b, h, T) for h in range(Hkv)]) for b in range(Bn)])
    cache.rd_residual_select(ks, vs, mass, n)
    q = synth.queries(44, Bn, Hq)
    pages_d = cache.quest_select(q, topk)
    out = cache.decode(q, pages=pages_d).cpu().numpy()
    pages = pages_d.cpu().numpy()
    idx = cache.res_idx.cpu().numpy()
    res_bits = read_bits = 0
    for b in range(Bn):
        for h in range(Hkv):
            kmin, kmax = oquest.page_boxes(ks[b, h], page)
            want = oquest.quest_select(q_group(q, b, h, G), kmin, kmax, T, topk, page)
            np.testing.assert_array_equal(pages[b, h], want)
            uc = ocache.UnitCache(ks[b, h], vs[b, h], lv)
            ridx, _ = uc.select_residual(ks[b, h], vs[b, h], mass[b, h], n)
            np.testing.assert_array_equal(idx[b, h, :n], ridx)
            assert np.isin(ridx, oquest.read_tokens(want, T, page)).any()  # the read set holds residual rows
            ref = uc.decode_quest(q_group(q, b, h, G), want, page)
            assert max_err(out[b, h * G:(h + 1) * G], ref) <= TOL
            o = oacc.unit_rates(lv, T, page=page, nres=n, pages=want, res_idx=ridx)
            res_bits += o["resident_bits"]
            read_bits += o["read_bits"]
    r = cache.account(pages_d)
    assert r["resident_bits"] == res_bits and r["read_bits"] == read_bits


# ---------------------------------------------------------------- sequences of different lengths


def _ragged_levels(lens, Hkv, profile="graded"):
    nb = (max(lens) + 63) // 64
    lv = np.full((len(lens), Hkv, nb), 16, np.int8)
    for b, t in enumerate(lens):
        lv[b, :, :(t + 63) // 64] = olad.ladder(profile, t)
    return lv


def _check_ragged(cache, ucs, keys, q, lens, G, topk, page, live):
    """Dense and Compressed-Quest reads of every live sequence against its oracle unit
    (pages bit-exact; keys[b, h] is the unit's exact key stream), zeros for retired
    ones."""
    Hkv = cache.Hkv
    out = cache.decode(q).cpu().numpy()
    pages = cache.quest_select(q, topk)
    outq = cache.decode(q, pages=pages).cpu().numpy()
    pages = pages.cpu().numpy()
    for b in range(cache.B):
        if not live[b]:
            assert np.all(out[b] == 0) and np.all(outq[b] == 0) and np.all(pages[b] == -1)
            continue
        for h in range(Hkv):
            uc = ucs[b, h]
            assert uc.T == lens[b]
            qg = q_group(q, b, h, G)
            assert max_err(out[b, h * G:(h + 1) * G], uc.decode_dense(qg)) <= TOL
            kmin, kmax = oquest.page_boxes(keys[b, h][:lens[b]], page)
            want = oquest.quest_select(qg, kmin, kmax, lens[b], topk, page)
            np.testing.assert_array_equal(pages[b, h], want)
            assert max_err(outq[b, h * G:(h + 1) * G], uc.decode_quest(qg, want, page)) <= TOL


def test_ragged_batch_appends_retire_and_admit(gpu):
    """Four sequences of different lengths in one batch (section 3.7 serving: the block
    manager's incremental appends): each is its own oracle unit.  Dense and
    Compressed-Quest reads, then 70 decode steps of appends in which every sequence
    opens blocks and crosses ladder boundaries at its own length (records bit-exact);
    sequence 2 is retired at step 30 (its slots go back to the pool, its outputs are
    zero) and admitted again as a new, empty sequence at step 45."""
    torch = _torch()
    lens0 = [1000, 64 * 23 + 17, 700, 64 * 30 - 3]
    Bn, Hq, Hkv, page, topk, steps = 4, 8, 2, 16, 24, 70
    G = Hq // Hkv
    Tmax = max(lens0) + steps
    ks, vs = kv_all(46, Bn, Hkv, Tmax)
    kn2, vn2 = kv_all(47, 1, Hkv, steps)  # the admitted sequence's tokens
    lv = _ragged_levels(lens0, Hkv)
    cache = _build(gpu, ks[:, :, :max(lens0)], vs[:, :, :max(lens0)], Hq, lv, page=page, seq_lens=lens0,
                   extra_blocks=4, slack={16: 8, 8: 8, 4: 8, 2: 8, 1: 8})
    ucs, keys = {}, {}
    for b in range(Bn):
        for h in range(Hkv):
            t = lens0[b]
            ucs[b, h] = ocache.UnitCache(ks[b, h, :t], vs[b, h, :t], lv[b, h, :(t + 63) // 64])
            keys[b, h] = ks[b, h]
    lens = list(lens0)
    live = [True] * Bn
    q = synth.queries(46, Bn, Hq)
    _check_ragged(cache, ucs, keys, q, lens, G, topk, page, live)
    pos = list(lens0)  # next token of each sequence's own stream
    moves_seen = 0
    for s in range(steps):
        if s == 30:
            used = {L: cache.pool.used(L) for L in gpu.LEVELS}
            nb2 = (lens[2] + 63) // 64
            freed = {L: 2 * int((cache.level_host[2, :, :nb2] == L).sum()) for L in gpu.LEVELS}
            cache.retire(2)
            assert all(cache.pool.used(L) == used[L] - freed[L] for L in gpu.LEVELS)
            live[2] = False
            lens[2] = -1
            assert list(cache.lengths()) == lens
        if s == 45:
            cache.admit(2)
            live[2] = True
            lens[2] = 0
            pos[2] = 0
            ucs[2, 0] = ocache.UnitCache(kn2[0, 0, :0], vn2[0, 0, :0], [])
            ucs[2, 1] = ocache.UnitCache(kn2[0, 1, :0], vn2[0, 1, :0], [])
            keys[2, 0], keys[2, 1] = kn2[0, 0], kn2[0, 1]
        kn = np.zeros((Bn, Hkv, 128), np.uint16)
        vn = np.zeros((Bn, Hkv, 128), np.uint16)
        for b in range(Bn):
            if not live[b]:
                continue
            src_k, src_v = (kn2[0], vn2[0]) if (b == 2 and s >= 45) else (ks[b], vs[b])
            kn[b], vn[b] = src_k[:, pos[b]], src_v[:, pos[b]]
        moves = cache.append(kn, vn, profile="graded")
        want = []
        for b in range(Bn):
            if not live[b]:
                continue
            for h in range(Hkv):
                for blk, old, new in ucs[b, h].append(kn[b, h], vn[b, h], "graded"):
                    want.append((b, h, blk, old, new))
            pos[b] += 1
            lens[b] += 1
        assert sorted(moves) == sorted(want)
        moves_seen += len(moves)
        assert list(cache.lengths()) == lens
        if s % 23 == 22 or s == steps - 1:
            qs = synth.queries(46, Bn, Hq, step=s + 1)
            _check_ragged(cache, ucs, keys, qs, lens, G, topk, page, live)
    assert moves_seen > 0
    for b in range(Bn):
        for h in range(Hkv):
            for blk in range(lens[b] // 64):  # complete blocks
                compare_record(cache, ucs[b, h], b, h, blk, 0)
                compare_record(cache, ucs[b, h], b, h, blk, 1)
    r = cache.account()
    want_bits = sum(oacc.unit_rates(ucs[b, h].levels, lens[b], page=page)["resident_bits"]
                    for b in range(Bn) for h in range(Hkv))
    assert r["resident_bits"] == want_bits


def test_layers_step_with_sequences_of_different_lengths(gpu):
    """gkv_layers_step over two layers of a batch of three sequences of different
    lengths: every sequence opens blocks and crosses ladder boundaries at its own
    length; the service equals per-layer appends step by step (levels, offsets, pool
    use, decode outputs bit for bit)."""
    torch = _torch()
    L, Bn, Hq, Hkv, steps = 2, 3, 8, 2, 70
    lens = [64 * 10 - 1, 64 * 7 + 3, 64 * 12]
    data = [kv_all(80 + l, Bn, Hkv, max(lens) + steps) for l in range(L)]
    lv = _ragged_levels(lens, Hkv, "tiny")  # 4 exact, 8 int8, 12 int4 blocks: crossings at these lengths
    slack = {16: 16, 8: 16, 4: 16, 2: 16, 1: 8}
    mk = lambda ks, vs: _build(gpu, ks[:, :, :max(lens)], vs[:, :, :max(lens)], Hq, lv, page=16, extra_blocks=4,
                               slack=slack, seq_lens=lens)
    svc = gpu.LayerCaches([mk(*d) for d in data], "tiny")
    ref = [mk(*d) for d in data]
    total = 0
    for s in range(steps):
        kn = np.stack([np.stack([d[0][b, :, lens[b] + s] for b in range(Bn)]) for d in data])
        vn = np.stack([np.stack([d[1][b, :, lens[b] + s] for b in range(Bn)]) for d in data])
        n = svc.step(kn, vn)
        moves = [r.append(kn[l], vn[l], profile="tiny") for l, r in enumerate(ref)]
        assert sum(len(m) for m in moves) == n
        total += n
        q = synth.queries(81, Bn, Hq, step=s)
        for l in range(L):
            a, b = svc.caches[l], ref[l]
            assert list(a.lengths()) == list(b.lengths()) == [t + s + 1 for t in lens]
            np.testing.assert_array_equal(a.level_host, b.level_host)
            np.testing.assert_array_equal(a.koff_host, b.koff_host)
            np.testing.assert_array_equal(a.voff_host, b.voff_host)
            assert all(a.pool.used(x) == b.pool.used(x) for x in gpu.LEVELS)
            assert torch.equal(a.decode(q), b.decode(q))
    assert total > 0
