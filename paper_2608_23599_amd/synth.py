"""Seeded synthetic inputs for the graded-KV decode workloads.

This module holds NO arithmetic of the method: it only draws random tensors.
Both the HIP path (through the tests and the benchmark) and the CPU oracle are fed
from it, so the two see identical inputs.

Recipe (the paper measures on activations of real checkpoints over WikiText-2
and PG-19; those are not available, and these draws stand in for them):

* every (workload, stream, sequence b, KV head h) has its own generator
  ``numpy.random.default_rng(SeedSequence([2608, 23599, workload, stream, b, h]))``;
  streams: 0 keys, 1 values, 2 queries, 3 outlier channels, 4 attention mass,
  5 appended tokens;
* keys and values are standard normal in fp32; for each (layer, KV head) four
  distinct key channels are drawn without replacement and multiplied by 10 in
  fp32 (outlier channels); both are then rounded to fp16;
* queries are standard normal rounded to fp16, layout [B][Hq][D];
* attention mass for residual selection is one Dirichlet(0.1 * 1_T) draw per
  (sequence, KV head), stored as fp32.
"""
import numpy as np

SEED = (2608, 23599)
S_KEYS, S_VALUES, S_QUERY, S_OUTLIER, S_MASS, S_APPEND = 0, 1, 2, 3, 4, 5


def rng(workload, stream, *unit):
    return np.random.default_rng(np.random.SeedSequence([*SEED, int(workload), int(stream), *[int(u) for u in unit]]))


def outlier_channels(workload, b, h, D=128, n=4):
    return np.sort(rng(workload, S_OUTLIER, b, h).choice(D, size=n, replace=False))


def kv_unit(workload, b, h, T, D=128, n_outlier=4, scale=10.0):
    """Keys and values of one (sequence, KV head): fp16 bit patterns [T][D] each."""
    k = rng(workload, S_KEYS, b, h).standard_normal((T, D), dtype=np.float32)
    ch = outlier_channels(workload, b, h, D, n_outlier)
    k[:, ch] *= np.float32(scale)
    v = rng(workload, S_VALUES, b, h).standard_normal((T, D), dtype=np.float32)
    return k.astype(np.float16).view(np.uint16), v.astype(np.float16).view(np.uint16)


def kv_rows(workload, b, h, T, rows, D=128):
    """Selected rows of ``kv_unit`` without keeping the whole unit (rows sorted)."""
    k, v = kv_unit(workload, b, h, T, D)
    return k[rows], v[rows]


def queries(workload, B, Hq, D=128, step=0):
    q = rng(workload, S_QUERY, step).standard_normal((B, Hq, D), dtype=np.float32)
    return q.astype(np.float16).view(np.uint16)


def mass_unit(workload, b, h, T, alpha=0.1):
    m = rng(workload, S_MASS, b, h).dirichlet(np.full(T, alpha))
    return m.astype(np.float32)


def append_tokens(workload, step, B, Hkv, D=128):
    """Key/value rows appended at decode step ``step``: fp16 bits [B][Hkv][D]."""
    r = rng(workload, S_APPEND, step)
    k = r.standard_normal((B, Hkv, D), dtype=np.float32)
    v = r.standard_normal((B, Hkv, D), dtype=np.float32)
    return k.astype(np.float16).view(np.uint16), v.astype(np.float16).view(np.uint16)
