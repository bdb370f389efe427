"""The no-allocation attention entry point (gkv_graded_decode_attn_noalloc): the
library's own device scratch array as workspace, for callers that cannot allocate.
Its output equals gkv_graded_decode_attn's (same kernels, same plan) bit for bit on
two calls in a row, the second with a smaller input, and meets the oracle's
tolerance; a Compressed-Quest read too; a call needing more than the array is
refused before anything is enqueued."""
import ctypes

import numpy as np
import pytest

from oracle import cache as ocache, ladder as olad
from paper_2608_23599_amd import synth
from tests._util import TOL, kv_all, max_err, q_group

pytestmark = pytest.mark.gpu


def _build(gpu, ks, vs, Hq, levels, **kw):
    return gpu.GradedCache.build(ks, vs, Hq=Hq, levels=levels, device="cuda", **kw)


def _noalloc(gpu, cache, q, out, pages=None):
    topk = 0 if pages is None else int(pages.shape[-1])
    return gpu._attn_noalloc(gpu._dptr(gpu._as_bits(q, "cuda")), ctypes.byref(cache.c), gpu._dptr(pages), topk,
                             gpu._dptr(out), gpu._stream())


def test_noalloc_matches_workspace_call(gpu):
    import torch
    assert gpu._noalloc_bytes() == 32 << 20
    # call 1: 32 query / 8 KV heads, 16384 tokens (graded ladder with centroid blocks)
    # and a 2% residual; call 2: 8 query / 2 KV heads, 2048 tokens (tiny ladder)
    cases = [(2, 32, 8, 16384, "graded", 327), (1, 8, 2, 2048, "tiny", 0)]
    for wl, Hq, Hkv, T, prof, nres in cases:
        ks, vs = kv_all(wl, 1, Hkv, T)
        lv = olad.ladder(prof, T)
        cache = _build(gpu, ks, vs, Hq, lv, nres_cap=nres)
        mass = np.stack([synth.mass_unit(wl, 0, h, T) for h in range(Hkv)])[None]
        if nres:
            cache.rd_residual_select(ks, vs, mass, nres)
        q = synth.queries(wl, 1, Hq)
        want = cache.decode(q)
        out = torch.full_like(want, float("nan"))
        assert _noalloc(gpu, cache, q, out) == 0
        torch.cuda.synchronize()
        assert torch.equal(out, want), (wl, T)
        o = out.cpu().numpy()
        G = Hq // Hkv
        for h in (0, Hkv - 1):
            uc = ocache.UnitCache(ks[0, h], vs[0, h], lv)
            if nres:
                uc.select_residual(ks[0, h], vs[0, h], mass[0, h], nres)
            assert max_err(o[0, h * G:(h + 1) * G], uc.decode_dense(q_group(q, 0, h, G))) <= TOL


def test_noalloc_quest_read(gpu):
    import torch
    T, Hq, Hkv, topk = 4001, 8, 2, 64
    ks, vs = kv_all(3, 1, Hkv, T)
    cache = _build(gpu, ks, vs, Hq, olad.ladder("graded", T), page=16)
    q = synth.queries(3, 1, Hq)
    pages = cache.quest_select(q, topk)
    want = cache.decode(q, pages=pages)
    out = torch.empty_like(want)
    assert _noalloc(gpu, cache, q, out, pages) == 0
    torch.cuda.synchronize()
    assert torch.equal(out, want)


def test_noalloc_refuses_a_call_beyond_the_array(gpu):
    import torch
    ks, vs = kv_all(1, 1, 1, 128)
    cache = _build(gpu, ks, vs, 4, olad.ladder("exact", 128))
    big = gpu.CacheStruct.from_buffer_copy(cache.c)
    big.B, big.nblk_cap = 64, 1 << 14  # a workspace far beyond 32 MiB; nothing is launched
    out = torch.empty((1, 4, 128), dtype=torch.float32, device="cuda")
    q = synth.queries(1, 1, 4)
    st = gpu._attn_noalloc(gpu._dptr(gpu._as_bits(q, "cuda")), ctypes.byref(big), None, 0, gpu._dptr(out),
                           gpu._stream())
    assert st == -4  # GKV_E_WORKSPACE
