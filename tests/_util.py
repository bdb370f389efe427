"""Shared helpers for the GPU parity tests: build the same seeded workload for the
HIP path (through the C ABI) and for the CPU oracle."""
import numpy as np

from oracle import cache as ocache, fp16 as ofp16, quant as oquant
from paper_2608_23599_amd import synth

TOL = 2e-3  # max-abs attention tolerance on unit-scale outputs


def kv_all(wl, B, Hkv, T):
    ks = np.empty((B, Hkv, T, 128), dtype=np.uint16)
    vs = np.empty((B, Hkv, T, 128), dtype=np.uint16)
    for b in range(B):
        for h in range(Hkv):
            ks[b, h], vs[b, h] = synth.kv_unit(wl, b, h, T)
    return ks, vs


def oracle_units(ks, vs, levels):
    B, Hkv = ks.shape[:2]
    return {(b, h): ocache.UnitCache(ks[b, h], vs[b, h], levels) for b in range(B) for h in range(Hkv)}


def compare_record(gpu_cache, uc, b, h, blk, tensor):
    """Bit-exact comparison of one GPU record against the oracle record."""
    d = gpu_cache.record(b, h, blk, tensor)
    rec = (uc.k_recs if tensor == 0 else uc.v_recs)[blk]
    assert d["level"] == rec.level, (b, h, blk, tensor)
    if rec.level == 16:
        got = ofp16.from_f64(d["values"])  # exact level: raw bits round-trip (no -0 inputs here)
        np.testing.assert_array_equal(d["values"], ofp16.to_f64(rec.exact))
    elif rec.level in (8, 4, 2):
        np.testing.assert_array_equal(d["codes"], rec.codes, err_msg=f"codes {b} {h} {blk} {tensor}")
        np.testing.assert_array_equal(d["s16"], rec.s16, err_msg=f"scale {b} {h} {blk} {tensor}")
        np.testing.assert_array_equal(d["z16"], rec.z16, err_msg=f"zero {b} {h} {blk} {tensor}")
    else:
        np.testing.assert_array_equal(d["cent16"], rec.cent16, err_msg=f"centroids {b} {h} {blk} {tensor}")
        np.testing.assert_array_equal(d["ids"], rec.ids, err_msg=f"ids {b} {h} {blk} {tensor}")
    return d


def q_group(q, b, h, G):
    return q[b, h * G:(h + 1) * G]


def max_err(out, ref):
    return float(np.abs(np.asarray(out, dtype=np.float64) - ref).max())


def decode_oracle_record(rec):
    return oquant.decode(rec)
