"""Pins for the decode-time attention error certificate (section 3.6, Eq. certificate)
as the oracle keeps it: per-block error numbers measured at encode time, carried
through demotions by the triangle inequality, and the bound evaluated from them."""
import numpy as np

from oracle import fp16, certificate, cache, attention
from oracle.ladder import ladder, EXACT, INT8
from paper_2608_23599_amd import synth


def _exact_error(uc, k, v, q):
    """||o - o_hat|| per head: exact attention vs the cache's graded attention (fp64)."""
    kf, vf = fp16.to_f64(k), fp16.to_f64(v)
    kh, vh = uc.khat_vhat()
    qf = fp16.to_f64(q)
    return np.sqrt(((attention.attend(qf, kf, vf) - attention.attend(qf, kh, vh)) ** 2).sum(axis=1))


def test_bound_holds_on_graded_caches():
    for prof, T, seed in (("tiny", 2048, 301), ("graded", 4096, 302)):
        k, v = synth.kv_unit(seed, 0, 0, T)
        uc = cache.UnitCache(k, v, ladder(prof, T))
        q = synth.queries(seed, 1, 8)[0]
        bnd = uc.certificate(q)
        err = _exact_error(uc, k, v, q)
        assert np.all(err <= bnd) and np.all(err > 0)


def test_bound_is_informative_for_int8():
    """All int8 blocks: logit errors stay small, so the bound sits well below the
    universal cap of 2 max||v||."""
    T = 1024
    k, v = synth.kv_unit(303, 0, 0, T)
    uc = cache.UnitCache(k, v, np.full(T // 64, INT8, np.int8))
    q = synth.queries(303, 1, 4)[0]
    bnd = uc.certificate(q)
    err = _exact_error(uc, k, v, q)
    assert np.all(err <= bnd)
    assert np.all(bnd < 0.5 * 2 * max(uc.vmax))


def test_all_exact_cache_has_zero_bound():
    T = 700
    k, v = synth.kv_unit(304, 0, 0, T)
    uc = cache.UnitCache(k, v, np.full((T + 63) // 64, EXACT, np.int8))
    assert np.all(uc.certificate(synth.queries(304, 1, 2)[0]) == 0.0)


def test_single_block_closed_form():
    """One int8 block: every weight is in the block, so the bound is
    verr + min(2, 2 sinh(2 eps)) vmax with eps = ||q|| kerr / sqrt(D)."""
    k, v = synth.kv_unit(305, 0, 0, 64)
    uc = cache.UnitCache(k, v, [INT8])
    q = synth.queries(305, 1, 3)[0]
    qf = fp16.to_f64(q)
    for g in range(3):
        eps = np.sqrt((qf[g] ** 2).sum()) * uc.kerr[0] / np.sqrt(128.0)
        want = uc.verr[0] + min(2.0, 2.0 * np.sinh(2.0 * eps)) * uc.vmax[0]
        assert abs(uc.certificate(q)[g] - want) <= 1e-12 * want


def test_demotion_carries_an_upper_bound_of_the_error():
    """After appends that demote blocks down the ladder, every block's carried error
    is at least its direct error against the exact rows, and the bound still holds."""
    T0 = 64 * 40
    k, v = synth.kv_unit(306, 0, 0, T0 + 130)
    uc = cache.UnitCache(k[:T0], v[:T0], ladder("graded", T0))
    moves = 0
    for t in range(T0, T0 + 130):
        moves += len(uc.append(k[t], v[t], "graded"))
    assert moves > 0
    kh, vh = uc.khat_vhat()
    kf, vf = fp16.to_f64(k[: uc.T]), fp16.to_f64(v[: uc.T])
    for b in range(len(uc.levels)):
        rows = slice(b * 64, min((b + 1) * 64, uc.T))
        ke, _ = certificate.block_numbers(kf[rows], kh[rows])
        ve, vn = certificate.block_numbers(vf[rows], vh[rows])
        assert uc.kerr[b] >= ke * (1 - 1e-12) and uc.verr[b] >= ve * (1 - 1e-12)
        assert abs(uc.vmax[b] - vn) <= 1e-12 * max(vn, 1.0)
    q = synth.queries(306, 1, 4)[0]
    assert np.all(_exact_error(uc, k[: uc.T], v[: uc.T], q) <= uc.certificate(q))


def test_residual_rows_count_as_exact():
    T = 1024
    k, v = synth.kv_unit(307, 0, 0, T)
    uc = cache.UnitCache(k, v, ladder("tiny", T))
    q = synth.queries(307, 1, 4)[0]
    before = uc.certificate(q)
    uc.select_residual(k, v, synth.mass_unit(307, 0, 0, T), 20)
    after = uc.certificate(q)
    assert np.all(_exact_error(uc, k, v, q) <= after)
    assert not np.array_equal(before, after)
