"""Host-side checks of the C ABI (no GPU needed): exported symbols, ladder,
ladder crossings, slab pool, accounting, the packed-record decoder and argument
validation.  Expected values come from the oracle or from the layout as the
header documents it."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import accounting as oacc, fp16 as ofp16, ladder as olad, quant as oquant
from paper_2608_23599_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gkv.h")


@pytest.fixture(scope="module")
def B():
    from paper_2608_23599_amd import binding
    return binding


def test_library_exports_every_declared_symbol(B):
    text = open(HEADER).read()
    decl = set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]*?\b(gkv_\w+)\s*\(", text, re.M))
    assert len(decl) >= 20
    for name in decl:
        assert hasattr(B.lib, name), name
    assert decl == set(B.EXPORTED)


def test_f64_to_f16_matches_single_rounding(B):
    r = np.random.default_rng(5)
    xs = np.concatenate([
        r.standard_normal(3000) * 10.0 ** r.integers(-9, 5, 3000),
        (r.integers(-2048, 2048, 500) + 0.5) * 2.0 ** r.integers(-24, 6, 500),
        [1 + 2.0 ** -11 + 2.0 ** -40, 1 + 2.0 ** -11, 65519.9, 65520.0, 2.0 ** -25, 2.0 ** -25 * 1.0001, 0.0],
    ])
    want = xs.astype(np.float16).view(np.uint16)
    got = np.array([B.f64_to_f16(x) for x in xs], dtype=np.uint16)
    assert np.array_equal(got, want)
    assert B.f64_to_f16(-0.0) == 0x8000  # the raw conversion keeps the sign; stores canonicalise


@pytest.mark.parametrize("profile,T", [("tiny", 2048), ("tiny", 1000), ("graded", 16384), ("graded", 131072),
                                       ("graded", 1048576 + 64), ("graded", 5000), ("exact", 300),
                                       ("rdv2", 131072), ("rdv2", 700)])
def test_ladder_matches_oracle(B, profile, T):
    assert np.array_equal(B.ladder_levels(profile, T), olad.ladder(profile, T))


def test_block_bytes(B):
    for L in B.LEVELS:
        assert B.block_bytes(L) * 8 == oacc.block_bits(L)
    assert B.block_bytes(3) == 0


def _host_cache(B, Bn, Hkv, Hq, T, levels, page=0, nres=0):
    """A gkv_cache whose device pointers are host buffers (host-only calls never
    dereference them)."""
    nblk = (T + 63) // 64
    keep = {}
    c = B.CacheStruct()
    c.B, c.Hkv, c.Hq, c.D, c.T, c.nblk_cap = Bn, Hkv, Hq, 128, T, nblk + 4
    lv = np.zeros((Bn, Hkv, nblk + 4), dtype=np.int8)
    lv[:, :, :nblk] = levels
    keep["lv"] = lv
    for name in ("level", "koff", "voff", "arena"):
        a = np.zeros(64, dtype=np.int64)
        keep[name] = a
        setattr(c, name, a.ctypes.data)
    c.arena_bytes = 1 << 30
    c.level_host = lv.ctypes.data
    if page:
        bx = np.zeros(16, dtype=np.int64)
        keep["boxes"] = bx
        c.page, c.npage_cap, c.boxes = page, ((T // page) + 63) // 64 * 64 + 64, bx.ctypes.data
    if nres:
        for name in ("res_idx", "res_rows", "res_mask", "res_off"):
            a = np.zeros(8, dtype=np.int64)
            keep[name] = a
            setattr(c, name, a.ctypes.data)
        c.nres = c.nres_cap = nres
    return c, keep


@pytest.mark.parametrize("T,page,nres,sel", [(2048, 0, 0, None), (16384, 0, 0, None), (131072, 0, 2621, None),
                                             (32768, 16, 0, 128), (5000, 16, 0, 40), (16384, 64, 0, 32)])
def test_account_matches_oracle(B, T, page, nres, sel):
    prof = "tiny" if T == 2048 else "graded"
    lv = olad.ladder(prof, T)
    c, keep = _host_cache(B, 1, 2, 8, T, lv, page=page, nres=nres)
    pages = None
    if sel:
        r = np.random.default_rng(T)
        cur = (T - 1) // page
        pages = np.full((1, 2, sel), -1, dtype=np.int32)
        for h in range(2):
            pick = np.sort(r.choice(cur, size=min(sel, cur), replace=False))
            pages[0, h, :len(pick)] = pick
    rates = B.Rates()
    st = B._account(ctypes.byref(c), B._np_ptr(pages) if pages is not None else None, sel or 0, None,
                    ctypes.byref(rates))
    assert st == 0
    res, rd = 0, 0
    for h in range(2):
        o = oacc.unit_rates(lv, T, page=page or None, nres=nres, pages=None if pages is None else pages[0, h])
        res += o["resident_bits"]
        rd += o["read_bits"]
    assert rates.resident_bits == res and rates.read_bits == rd
    assert rates.values == 2 * T * 2 * 128


def test_ladder_crossings_and_monotone_rejection(B):
    T = 36 * 64
    lv = olad.ladder("graded", T)
    c, keep = _host_cache(B, 1, 2, 8, T, lv)
    jobs = np.zeros(3 * 64, dtype=np.int32)
    to = np.zeros(64, dtype=np.int8)
    n = B._ladder_crossings(ctypes.byref(c), 1, T + 1, B._np_ptr(jobs), B._np_ptr(to), 64)
    want = olad.crossings("graded", T, T + 1)
    assert n == 2 * len(want) and n > 0
    got = sorted((int(jobs[3 * i + 2]), int(to[i])) for i in range(n) if jobs[3 * i + 1] == 0)
    assert got == sorted((b, new) for b, old, new in want)
    # a ladder that would promote a block is rejected
    keep["lv"][:, :, 0] = olad.CENTROID
    keep["lv"][:, :, 1:36] = olad.INT2
    n = B._ladder_crossings(ctypes.byref(c), 2, T + 1, B._np_ptr(jobs), B._np_ptr(to), 64)
    assert n == -3


def test_demote_validation_runs_before_launch(B):
    T = 2048
    lv = olad.ladder("tiny", T)
    c, keep = _host_cache(B, 1, 1, 4, T, lv)
    jobs = np.array([0, 0, 31], dtype=np.int32)       # block 31 is exact
    nk = np.array([0], dtype=np.int64)
    for to, want in ((16, -3), (8, None)):
        t = np.array([to], dtype=np.int8)
        st = B._demote(ctypes.byref(c), 1, B._np_ptr(jobs), B._np_ptr(t), B._np_ptr(nk), B._np_ptr(nk), None)
        if want is not None:
            assert st == want
    j2 = np.array([0, 0, 0], dtype=np.int32)          # block 0 is int2: int4 would promote
    t = np.array([4], dtype=np.int8)
    assert B._demote(ctypes.byref(c), 1, B._np_ptr(j2), B._np_ptr(t), B._np_ptr(nk), B._np_ptr(nk), None) == -3
    c.D = 64
    assert B._demote(ctypes.byref(c), 1, B._np_ptr(j2), B._np_ptr(t), B._np_ptr(nk), B._np_ptr(nk), None) == -2


def test_call_validation_errors(B):
    T = 2048
    c, keep = _host_cache(B, 1, 2, 8, T, olad.ladder("tiny", T), page=16)
    ws = np.zeros(8, dtype=np.int64)
    q = np.zeros(8 * 128, dtype=np.uint16)
    pages = np.zeros(16, dtype=np.int32)
    out = np.zeros(8 * 128, dtype=np.float32)
    # top-k of zero, null pointers, undersized workspace
    assert B._quest_select(B._np_ptr(q), ctypes.byref(c), 0, B._np_ptr(pages), B._np_ptr(ws), 64, None) == -1
    assert B._quest_select(None, ctypes.byref(c), 4, B._np_ptr(pages), B._np_ptr(ws), 64, None) == -1
    assert B._quest_select(B._np_ptr(q), ctypes.byref(c), 4, B._np_ptr(pages), B._np_ptr(ws), 64, None) == -4
    assert B._attn(B._np_ptr(q), ctypes.byref(c), None, 0, B._np_ptr(out), B._np_ptr(ws), 64, None) == -4
    # quantize: an int block may not extend past the source rows
    src = np.zeros(16, dtype=np.uint16)
    assert B._quantize_block(ctypes.byref(c), 0, B._np_ptr(src), 1000, 0, 32, None) == -2
    # residual selection: source rows must be 16-byte aligned
    cr, keep_r = _host_cache(B, 1, 2, 8, T, olad.ladder("tiny", T), nres=64)
    rows = np.zeros(2 * T * 128 + 8, dtype=np.uint16)
    mass = np.zeros(2 * T, dtype=np.float32)
    wsr = np.zeros(16, dtype=np.int64)
    base = rows.ctypes.data + (-rows.ctypes.data) % 16
    for kp, vp in ((base + 2, base), (base, base + 8)):
        assert B._rd(ctypes.byref(cr), kp, vp, B._np_ptr(mass), 16, B._np_ptr(wsr), 1 << 40, None) == -1
    # aligned rows pass that check and meet the workspace check after it
    assert B._rd(ctypes.byref(cr), base, base, B._np_ptr(mass), 16, B._np_ptr(wsr), 8, None) == -4
    # G > 16 and a non-dividing head count
    c.Hq = 34
    assert B._attn(B._np_ptr(q), ctypes.byref(c), None, 0, B._np_ptr(out), B._np_ptr(ws), 1 << 30, None) == -2
    c.Hq = 64
    assert B._attn(B._np_ptr(q), ctypes.byref(c), None, 0, B._np_ptr(out), B._np_ptr(ws), 1 << 30, None) == -2


def test_pool_slots(B):
    p = B.Pool({16: 2, 8: 3, 1: 1, 0: 2})
    offs = [p.alloc(8) for _ in range(3)]
    assert len(set(offs)) == 3 and all(o % 16 == 0 for o in offs)
    with pytest.raises(B.GkvError):
        p.alloc(8)
    p.free(8, offs[1])
    assert p.alloc(8) == offs[1]
    with pytest.raises(B.GkvError):
        p.free(8, offs[0] + 1)
    assert p.used(8) == 3 and p.used(16) == 0
    e = [p.alloc(16), p.alloc(16)]
    c = p.alloc(1)
    mm = [p.alloc(0), p.alloc(0)]
    assert p.used(0) == 2 and all(o % 16 == 0 for o in mm)
    spans = sorted([(o, o + B.block_bytes(8)) for o in offs] + [(o, o + 16384) for o in e] + [(c, c + 1040)]
                   + [(o, o + 256) for o in mm])
    assert all(a[1] <= b[0] for a, b in zip(spans, spans[1:]))
    assert p.bytes >= spans[-1][1]


# ---------------------------------------------------------------- record layout
def _pack(level, tensor, rec):
    """Pack an oracle record into the byte layout the header documents
    (independent of the library's own packer)."""
    out = bytearray(B_bytes(level))

    def coord(pg, l, n):
        kg, m = l >> 4, l & 15
        if tensor == 0:
            return 16 * pg + m, 32 * (n >> 3) + 8 * kg + (n & 7)
        return 16 * pg + 4 * kg + (n & 3), 16 * (n >> 2) + m

    if level == 16:
        a = np.frombuffer(out, dtype=np.uint16) if False else np.zeros(8192, dtype=np.uint16)
        for pg in range(4):
            for l in range(64):
                for n in range(32):
                    t, ch = coord(pg, l, n)
                    a[(pg * 64 + l) * 32 + n] = rec.exact[t, ch]
        return a.tobytes()
    if level in (8, 4, 2):
        bits = level
        per_token = getattr(rec, "per_token", False)
        pos4 = [4, 20, 12, 28, 0, 16, 8, 24]
        pos2 = [8, 24, 14, 30, 6, 22, 12, 28, 4, 20, 10, 26, 0, 16, 2, 18]
        sz = np.zeros(256, dtype=np.uint16)
        if per_token:  # scale[64], zero[64] in token order, then 256 zero bytes
            sz[:64] = rec.s16
            sz[64:128] = rec.z16
        for e in range(128 if not per_token else 0):
            kg, n = e >> 5, e & 31
            ch = 32 * (n >> 3) + 8 * kg + (n & 7) if tensor == 0 else 16 * (n >> 2) + 4 * kg + (n & 3)
            sz[e] = rec.s16[ch]
            sz[128 + e] = rec.z16[ch]
        words = np.zeros(256 * bits, dtype=np.uint32)
        for pg in range(4):
            for l in range(64):
                for n in range(32):
                    t, ch = coord(pg, l, n)
                    c = int(rec.codes[t, ch])
                    if bits == 8:
                        w, p = n >> 2, 8 * (n & 3)
                    elif bits == 4:
                        w, p = n >> 3, pos4[n & 7]
                    else:
                        w, p = n >> 4, pos2[n & 15]
                    words[(pg * 64 + l) * bits + w] |= np.uint32(c << p)
        return sz.tobytes() + words.tobytes()
    if level == 0:  # one row of 128 fp16 values in channel order
        return np.asarray(rec.cent16[0], dtype=np.uint16).tobytes()
    cen = np.zeros(512, dtype=np.uint16)
    for k in range(4):
        for d in range(128):
            idx = k * 128 + d if tensor == 0 else ((d & 15) * 8 + (d >> 4)) * 4 + k
            cen[idx] = rec.cent16[k, d]
    ids = np.zeros(16, dtype=np.uint8)
    for t in range(64):
        ids[t >> 2] |= np.uint8(int(rec.ids[t]) << (2 * (t & 3)))
    return cen.tobytes() + ids.tobytes()


def B_bytes(level):
    return oacc.block_bits(level) // 8


@pytest.mark.parametrize("level", [16, 8, 4, 2, 1, 0])
@pytest.mark.parametrize("tensor", [0, 1])
def test_decode_record_reads_documented_layout(B, level, tensor):
    k, v = synth.kv_unit(300 + level, 0, 0, 64)
    rec = oquant.encode_fp16(level, k if tensor == 0 else v)
    raw = _pack(level, tensor, rec)
    assert len(raw) == B.block_bytes(level)
    d = B.decode_record(level, tensor, raw)
    np.testing.assert_array_equal(d["values"], oquant.decode(rec))
    if level in (8, 4, 2):
        np.testing.assert_array_equal(d["codes"], rec.codes)
        np.testing.assert_array_equal(d["s16"], rec.s16)
        np.testing.assert_array_equal(d["z16"], rec.z16)
    if level in (1, 0):
        np.testing.assert_array_equal(d["ids"], rec.ids)
        np.testing.assert_array_equal(d["cent16"], rec.cent16)


@pytest.mark.parametrize("level", [8, 4, 2])
def test_decode_per_token_value_record(B, level):
    """A value record grouped per token (scale and zero per token, token order)."""
    _, v = synth.kv_unit(310 + level, 0, 0, 64)
    rec = oquant.encode_fp16(level, v, per_token=True)
    raw = _pack(level, 1, rec)
    assert len(raw) == B.block_bytes(level)
    d = B.decode_record(level, B.VALUES_PER_TOKEN, raw)
    np.testing.assert_array_equal(d["values"], oquant.decode(rec))
    np.testing.assert_array_equal(d["codes"], rec.codes)
    np.testing.assert_array_equal(d["s16"], rec.s16)
    np.testing.assert_array_equal(d["z16"], rec.z16)


def test_layers_step_full_pool_changes_nothing(B):
    """gkv_layers_step takes every slot before enqueueing: with a pool that cannot
    hold the step's new exact blocks, it fails with GKV_E_POOL and leaves the caches,
    pools and offset mirrors as they were (host-only: nothing reaches the GPU)."""
    import ctypes
    T = 64 * 30  # the next token opens block 30 of every (b, h)
    lv = olad.ladder("graded", T)
    caches, keeps, pools, kos, vos = [], [], [], [], []
    for layer in range(2):
        c, keep = _host_cache(B, 1, 2, 8, T, lv)
        caches.append(c)
        keeps.append(keep)
        pools.append(B.Pool({16: 1 if layer else 8, 8: 8, 4: 8, 2: 8, 1: 8}))  # layer 1: one exact slot
        kos.append(np.arange(2 * 34, dtype=np.int64).reshape(1, 2, 34))
        vos.append(kos[-1] + 1000)
    before = [(k.copy(), v.copy(), kp["lv"].copy()) for k, v, kp in zip(kos, vos, keeps)]
    used = [[p.used(L) for L in B.LEVELS] for p in pools]
    arr = lambda xs: (ctypes.c_void_p * 2)(*xs)
    kn = np.zeros((2, 1, 2, 128), dtype=np.uint16)
    st = B._layers_step(arr([ctypes.addressof(c) for c in caches]), arr([p.h for p in pools]),
                        arr([k.ctypes.data for k in kos]), arr([v.ctypes.data for v in vos]), 2,
                        B.PROFILES["graded"], kn.ctypes.data, kn.ctypes.data, None)
    assert st == -7  # GKV_E_POOL
    for (k0, v0, l0), k, v, kp, c in zip(before, kos, vos, keeps, caches):
        assert np.array_equal(k0, k) and np.array_equal(v0, v) and np.array_equal(l0, kp["lv"])
        assert c.T == T
    assert used == [[p.used(L) for L in B.LEVELS] for p in pools]


def test_account_graded_quest_by_hand(B):
    """The library's read accounting on the hand-computed graded Compressed-Quest
    cases of the oracle's pin (section 3.5, R_read equation)."""
    from tests.test_oracle_quest_attn import GRADED_QUEST_CASES
    for case in GRADED_QUEST_CASES:
        T, lv = case["T"], np.array(case["levels"], dtype=np.int8)
        c, keep = _host_cache(B, 1, 1, 4, T, lv, page=16)
        pages = np.array(case["pages"], dtype=np.int32).reshape(1, 1, -1)
        rates = B.Rates()
        assert B._account(ctypes.byref(c), B._np_ptr(pages), pages.shape[-1], None, ctypes.byref(rates)) == 0
        assert rates.read_bits == case["read_bits"]
        if case["resident_bits"] is not None:
            assert rates.resident_bits == case["resident_bits"]


def _layers_setup(B, T, levels_per_layer, pool_caps, arena_bytes=None):
    caches, keeps, pools, kos, vos = [], [], [], [], []
    for lv, caps in zip(levels_per_layer, pool_caps):
        c, keep = _host_cache(B, 1, 2, 8, T, lv)
        if arena_bytes is not None:
            c.arena_bytes = arena_bytes
        caches.append(c)
        keeps.append(keep)
        pools.append(B.Pool(caps))
        nb = c.nblk_cap
        kos.append(np.arange(2 * nb, dtype=np.int64).reshape(1, 2, nb))
        vos.append(kos[-1] + 1000)
    return caches, keeps, pools, kos, vos


def _layers_call(B, caches, pools, kos, vos):
    L = len(caches)
    arr = lambda xs: (ctypes.c_void_p * L)(*xs)
    kn = np.zeros((L, 1, 2, 128), dtype=np.uint16)
    return B._layers_step(arr([ctypes.addressof(c) for c in caches]), arr([p.h for p in pools]),
                          arr([k.ctypes.data for k in kos]), arr([v.ctypes.data for v in vos]), L,
                          B.PROFILES["graded"], kn.ctypes.data, kn.ctypes.data, None)


def _unchanged(B, before, used, caches, keeps, pools, kos, vos, T):
    for (k0, v0, l0), k, v, kp, c in zip(before, kos, vos, keeps, caches):
        assert np.array_equal(k0, k) and np.array_equal(v0, v) and np.array_equal(l0, kp["lv"])
        assert c.T == T
    assert used == [[p.used(L) for L in B.LEVELS] for p in pools]


def test_layers_step_rejects_a_layer_the_ladder_would_raise(B):
    """Each layer's crossings come from its own levels: a layer holding a block below
    the level the profile gives it at T + 1 (here one int8-band block at int2) makes
    the call fail with GKV_E_NOT_MONOTONE before any slot is taken, leaving every
    cache, pool and mirror as it was; layer 0 alone would step."""
    T = 64 * 40 + 5
    lv = olad.ladder("graded", T)
    lv1 = lv.copy()
    i8 = int(np.flatnonzero(lv == 8)[0])
    lv1[i8] = 2
    caps = {16: 8, 8: 8, 4: 8, 2: 8, 1: 8}
    caches, keeps, pools, kos, vos = _layers_setup(B, T, [lv, lv1], [caps, caps])
    before = [(k.copy(), v.copy(), kp["lv"].copy()) for k, v, kp in zip(kos, vos, keeps)]
    used = [[p.used(L) for L in B.LEVELS] for p in pools]
    assert _layers_call(B, caches, pools, kos, vos) == -3  # GKV_E_NOT_MONOTONE
    _unchanged(B, before, used, caches, keeps, pools, kos, vos, T)


def test_layers_step_rejects_slots_past_the_arena(B):
    """A pool whose slots lie past a layer's arena_bytes: the step takes its slots,
    finds one outside the arena, gives every slot back and returns GKV_E_ARG with
    nothing changed."""
    T = 64 * 30  # the next token opens block 30 of every (b, h)
    lv = olad.ladder("graded", T)
    caps = {16: 8, 8: 8, 4: 8, 2: 8, 1: 8}
    caches, keeps, pools, kos, vos = _layers_setup(B, T, [lv, lv], [caps, caps], arena_bytes=4 * 16384)
    before = [(k.copy(), v.copy(), kp["lv"].copy()) for k, v, kp in zip(kos, vos, keeps)]
    used = [[p.used(L) for L in B.LEVELS] for p in pools]
    assert _layers_call(B, caches, pools, kos, vos) == -1  # GKV_E_ARG
    _unchanged(B, before, used, caches, keeps, pools, kos, vos, T)


def test_binding_append_with_full_pool_changes_nothing(B):
    """GradedCache.append takes the new block's slots all or none: with room for one
    exact slot where a new block needs two per (b, h), it raises before the library
    is called, and the pool and the offset mirrors are as they were (host-only: the
    tables live in host memory and nothing is enqueued)."""
    c = B.GradedCache(1, 2, 8, 64, 4, {16: 1}, device="cpu")
    ko, vo = c.koff_host.copy(), c.voff_host.copy()
    used = [c.pool.used(L) for L in B.LEVELS]
    with pytest.raises(B.GkvError):
        c.append(np.zeros((1, 2, 128), np.uint16), np.zeros((1, 2, 128), np.uint16))
    assert [c.pool.used(L) for L in B.LEVELS] == used
    assert np.array_equal(c.koff_host, ko) and np.array_equal(c.voff_host, vo)
    assert c.T == 64


def test_account_quest_with_residual_by_hand(B):
    """The library's Compressed-Quest read accounting with residual rows equals the
    oracle's hand-computed pin (rows of residual tokens in the read set plus one mask
    per touched block); without the residual tokens the call is refused."""
    from tests.test_oracle_quest_attn import GRADED_QUEST_CASES
    case = GRADED_QUEST_CASES[1]
    T, lv = case["T"], np.array(case["levels"], dtype=np.int8)
    res = np.array([5, 40, 52, 100, 150, 200, 250, 255], dtype=np.int32)
    c, keep = _host_cache(B, 1, 1, 4, T, lv, page=16, nres=len(res))
    pages = np.array(case["pages"] + [3], dtype=np.int32).reshape(1, 1, -1)  # page 3 listed twice
    rates = B.Rates()
    assert B._account(ctypes.byref(c), B._np_ptr(pages), pages.shape[-1], B._np_ptr(res), ctypes.byref(rates)) == 0
    assert rates.read_bits == 163840 + 5 * (2 * 128 * 16 + 32) + 3 * 64
    o = oacc.unit_rates(lv, T, page=16, nres=len(res), pages=pages[0, 0], res_idx=res)
    assert rates.read_bits == o["read_bits"] and rates.resident_bits == o["resident_bits"]
    assert B._account(ctypes.byref(c), B._np_ptr(pages), pages.shape[-1], None, ctypes.byref(rates)) == -1


def _ragged_cache(B, lens, Hkv=2, page=0):
    """A host-only cache of sequences of different lengths (levels: each sequence's
    own graded ladder)."""
    T = int(max(lens))
    nb = (T + 63) // 64
    lv = np.zeros((len(lens), Hkv, nb), np.int8)
    for b, t in enumerate(lens):
        if t > 0:
            lv[b, :, :(t + 63) // 64] = olad.ladder("graded", t)
    c, keep = _host_cache(B, len(lens), Hkv, 4 * Hkv, T, lv, page=page)
    sl = np.array(lens, np.int64)
    keep["sl"], keep["sld"] = sl, np.zeros(len(lens), np.int64)
    c.seq_len_host, c.seq_len = sl.ctypes.data, keep["sld"].ctypes.data
    return c, keep


def test_ragged_lengths_validation_crossings_and_accounting(B):
    """Per-sequence lengths: T must be the largest length and every length in
    [-1, T]; the crossings of one more token are each sequence's own (the oracle's
    ladder at its length + 1, a retired sequence none); the accounting counts every
    sequence at its own length and a retired one not at all."""
    lens = [64 * 40, 64 * 25 + 7, -1, 64 * 33]
    c, keep = _ragged_cache(B, lens)
    jobs = np.zeros(3 * 256, np.int32)
    to = np.zeros(256, np.int8)
    n = B._ladder_crossings(ctypes.byref(c), 1, c.T + 1, B._np_ptr(jobs), B._np_ptr(to), 256)
    want = []
    for b, t in enumerate(lens):
        if t < 0:
            continue
        for blk, old, new in olad.crossings("graded", t, t + 1):
            want += [(b, h, blk, new) for h in range(2)]
    assert n == len(want) and n > 0
    got = sorted((int(jobs[3 * i]), int(jobs[3 * i + 1]), int(jobs[3 * i + 2]), int(to[i])) for i in range(n))
    assert got == sorted(want)
    # the last block of sequence 1 (7 of its 64 tokens) stays exact although the block
    # ends below T: demoting it is rejected before anything is enqueued
    assert int(keep["lv"][1, 0, 25]) == 16
    nk = np.zeros(1, np.int64)
    j1, t8 = np.array([1, 0, 25], np.int32), np.array([8], np.int8)
    assert B._demote(ctypes.byref(c), 1, B._np_ptr(j1), B._np_ptr(t8), B._np_ptr(nk), B._np_ptr(nk), None) == -2
    rates = B.Rates()
    assert B._account(ctypes.byref(c), None, 0, None, ctypes.byref(rates)) == 0
    res = sum(2 * oacc.unit_rates(olad.ladder("graded", t), t)["resident_bits"] for t in lens if t > 0)
    assert rates.resident_bits == res and rates.read_bits == res
    assert rates.values == sum(2 * t * 2 * 128 for t in lens if t > 0)
    keep["sl"][0] = c.T + 1  # longer than T
    assert B._account(ctypes.byref(c), None, 0, None, ctypes.byref(rates)) == -2
    keep["sl"][0] = 5  # T no longer the largest length
    assert B._account(ctypes.byref(c), None, 0, None, ctypes.byref(rates)) == -2
    keep["sl"][0] = -2
    assert B._account(ctypes.byref(c), None, 0, None, ctypes.byref(rates)) == -2


def test_retire_checks_every_slot_before_anything_changes(B):
    """gkv_retire_sequence refuses (before any device work) a retired sequence, a
    cache without per-sequence lengths, and a sequence whose offsets are not used
    slots of the pool, leaving the pool and the lengths unchanged."""
    lens = [64 * 3, 64 * 2 + 5]
    c, keep = _ragged_cache(B, lens, Hkv=1)
    pool = B.Pool({L: 16 for L in B.LEVELS})
    nb = c.nblk_cap
    ko = np.zeros((2, 1, nb), np.int64)
    vo = np.zeros((2, 1, nb), np.int64)
    for b, t in enumerate(lens):
        for i in range((t + 63) // 64):
            L = int(keep["lv"][b, 0, i])
            ko[b, 0, i], vo[b, 0, i] = pool.alloc(L), pool.alloc(L)
    used = [pool.used(L) for L in B.LEVELS]
    retire = lambda b: B._retire(ctypes.byref(c), pool.h, B._np_ptr(ko), B._np_ptr(vo), b, None)
    ko[1, 0, 1] += 7  # not a slot boundary
    assert retire(1) == -1
    ko[1, 0, 1] -= 7
    vo[1, 0, 0] = ko[1, 0, 0]  # one slot listed twice
    assert retire(1) == -1
    keep["sl"][1] = -1
    c.T = 64 * 3
    assert retire(1) == -1  # already retired
    assert [pool.used(L) for L in B.LEVELS] == used
    assert list(keep["sl"]) == [64 * 3, -1]
    c2, _ = _host_cache(B, 1, 1, 4, 128, olad.ladder("exact", 128))
    assert B._retire(ctypes.byref(c2), pool.h, B._np_ptr(ko), B._np_ptr(vo), 0, None) == -1


def test_pool_occupancy_equals_the_accounted_graded_bits(B):
    """The resident rate measured from the slab pool (slots in use x record sizes)
    equals the accounting's graded bits exactly: every block holds one K and one V
    record of its level, and the record sizes are the accounting's block bits (the
    paper compares a measured packed format with its accounting, section 5.7)."""
    for prof, T in (("graded", 131072), ("tiny", 2048), ("rdv2", 5000)):
        lv = olad.ladder(prof, T)
        c, keep = _host_cache(B, 2, 2, 8, T, lv)
        pool = B.Pool({L: 2 * 2 * 2 * int((lv == L).sum()) for L in B.LEVELS})
        for _ in range(2 * 2):
            for L in lv:
                pool.alloc(int(L))
                pool.alloc(int(L))
        measured = sum(pool.used(L) * B.block_bytes(L) for L in B.LEVELS) * 8
        rates = B.Rates()
        assert B._account(ctypes.byref(c), None, 0, None, ctypes.byref(rates)) == 0
        assert measured == rates.resident_bits
