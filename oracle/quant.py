"""Block quantizers of the precision ladder, their decoders, and demotion.

Method, section 3.2: levels 8, 4 and 2 are packed scalar quantizers with block
scale overhead; level 1 is a centroid state; once a block leaves the recent
window it can only be demoted, in place, re-encoding its current representation
(the original dense values are gone).

A block of one tensor (keys or values) is a [P=64 tokens][D=128 channels] array.

Readings (the paper gives no rounding mode, scale precision or degenerate case;
these are chosen because both sides can reproduce them exactly in fp64):

* Scalar level b, asymmetric, one group per channel over the block's 64 tokens,
  for keys AND values (the workloads fix per-block-per-channel groups); the
  paper's own text groups values per token instead (one group per token over its
  128 channels), which `per_token=True` selects for a value block, with the same
  formulas along the other axis:
      z16 = f16(min),  s16 = f16((max - min) / (2^b - 1)),
      code = 0 if s16 == 0 else clamp(rint((x - z16) / s16), 0, 2^b - 1),
  with fp64 arithmetic, IEEE division, rint = round-half-even, and one RNE
  rounding to fp16.  x - z16 is exact in fp64 (both are multiples of 2^-24
  below 2^17), and so is the decode  x_hat = code * s16 + z16.
* Centroid state: k = 4 centroids per block per tensor (keys and values
  clustered separately), deterministic Lloyd iteration in fp64:
  initial centroids = rows 0, 16, 32, 48; squared distance accumulated over
  channels in ascending order with separate multiply and add; ties go to the
  lower centroid; update = ascending-token sum / count, an empty cluster keeps
  its centroid; at most 10 rounds, stopping when an assignment repeats; then
  centroids are rounded to fp16 and every token is re-assigned against the
  stored fp16 centroids (what is stored is what is decoded).
  Parity of the centroid choices themselves is unpinned by the paper (no worked
  example); the invariants in the tests pin the implementation.
* One-centroid state (level 0): the same iteration with k = 1 (initial centroid
  row 0).  Every token is assigned to it, so one update gives the ascending-token
  fp64 mean and the next round repeats the assignment: the state is the fp16 of
  the block mean, which is the value centroid of Eq. rdscore.  A sum of 64 fp16
  values is exact in fp64, so this is the correctly rounded mean.
"""
import numpy as np

from . import fp16
from .ladder import EXACT, INT8, INT4, INT2, CENTROID, MEAN, ORDER

P, D = 64, 128
KCENT = 4


class Record:
    """One encoded tensor block.

    level      one of 16, 8, 4, 2, 1, 0
    exact      uint16 [P][D] fp16 bits              (level 16)
    codes      int32  [P][D] in [0, 2^b - 1]        (levels 8/4/2)
    s16, z16   uint16 [D] fp16 bits                 (levels 8/4/2)
    cent16     uint16 [KCENT][D] fp16 bits          (level 1; [1][D] at level 0)
    ids        int32  [P] in [0, KCENT)             (level 1; all 0 at level 0)
    per_token  s16, z16 are [P] (one group per token) instead of [D]
    """

    def __init__(self, level, **kw):
        self.level = int(level)
        self.exact = kw.get("exact")
        self.codes = kw.get("codes")
        self.s16 = kw.get("s16")
        self.z16 = kw.get("z16")
        self.cent16 = kw.get("cent16")
        self.ids = kw.get("ids")
        self.per_token = bool(kw.get("per_token", False))


# ---------------------------------------------------------------- scalar levels
def quantize_scalar(x, bits):
    """x: float64 [P][D] -> (codes int32 [P][D], s16 bits [D], z16 bits [D])."""
    x = np.asarray(x, dtype=np.float64)
    qmax = (1 << bits) - 1
    mn = x.min(axis=0)
    mx = x.max(axis=0)
    z16 = fp16.from_f64(mn)
    s16 = fp16.from_f64((mx - mn) / float(qmax))
    z = fp16.to_f64(z16)
    s = fp16.to_f64(s16)
    # every element is independent: one IEEE subtraction, division and rint each
    nz = s != 0.0
    safe = np.where(nz, s, 1.0)
    t = np.rint((x - z[None, :]) / safe[None, :])
    t = np.where(nz[None, :], t, 0.0)  # constant channel: every code is 0
    codes = np.clip(t, 0, qmax).astype(np.int32)
    return codes, s16, z16


def dequant_scalar(codes, s16, z16):
    """Exact fp64 decode code * s16 + z16."""
    return codes.astype(np.float64) * fp16.to_f64(s16)[None, :] + fp16.to_f64(z16)[None, :]


def quantize_scalar_per_token(x, bits):
    """One group per token (row): the per-channel quantizer of the transpose."""
    codes, s16, z16 = quantize_scalar(np.asarray(x, dtype=np.float64).T, bits)
    return codes.T.copy(), s16, z16


def dequant_scalar_per_token(codes, s16, z16):
    return codes.astype(np.float64) * fp16.to_f64(s16)[:, None] + fp16.to_f64(z16)[:, None]


# ---------------------------------------------------------------- centroid level
def _sq_dist(x, c):
    """[n][D] x [k][D] -> [n][k]; channel-ascending sum of (x - c)^2, no FMA."""
    acc = np.zeros((x.shape[0], c.shape[0]), dtype=np.float64)
    for d in range(x.shape[1]):
        diff = x[:, d][:, None] - c[:, d][None, :]
        sq = diff * diff
        acc = acc + sq
    return acc


def _assign(x, c):
    return np.argmin(_sq_dist(x, c), axis=1).astype(np.int32)  # first minimum = lower index


def kmeans_centroids(x, k=KCENT, iters=10):
    """x: float64 [P][D] -> (cent16 bits [k][D], ids int32 [P])."""
    x = np.asarray(x, dtype=np.float64)
    n = x.shape[0]
    init_rows = [i * (n // k) for i in range(k)]
    c = x[init_rows].copy()
    prev = None
    for _ in range(iters):
        a = _assign(x, c)
        if prev is not None and np.array_equal(a, prev):
            break
        prev = a
        for kk in range(k):
            members = np.nonzero(a == kk)[0]  # ascending token order
            if len(members) == 0:
                continue
            acc = np.zeros(x.shape[1], dtype=np.float64)
            for j in members:
                acc = acc + x[j]
            c[kk] = acc / float(len(members))
    cent16 = fp16.from_f64(c)
    ids = _assign(x, fp16.to_f64(cent16))
    return cent16, ids


def dequant_centroid(cent16, ids):
    return fp16.to_f64(cent16)[ids]


# ---------------------------------------------------------------- records
def encode(level, x, per_token=False):
    """Encode float64 block x [P][D] at ``level``.  For level 16 x must be
    fp16-representable (it is stored as-is).  per_token groups a scalar level per
    token (value blocks read the paper's way); other levels ignore it."""
    level = int(level)
    if level == EXACT:
        bits = fp16.from_f64(x)
        assert np.array_equal(fp16.to_f64(bits), np.asarray(x, np.float64)), "exact level needs fp16 values"
        return Record(EXACT, exact=bits)
    if level in (INT8, INT4, INT2):
        if per_token:
            codes, s16, z16 = quantize_scalar_per_token(x, level)
            return Record(level, codes=codes, s16=s16, z16=z16, per_token=True)
        codes, s16, z16 = quantize_scalar(x, level)
        return Record(level, codes=codes, s16=s16, z16=z16)
    if level == CENTROID:
        cent16, ids = kmeans_centroids(x)
        return Record(CENTROID, cent16=cent16, ids=ids)
    if level == MEAN:
        cent16, ids = kmeans_centroids(x, k=1)
        return Record(MEAN, cent16=cent16, ids=ids)
    raise ValueError(level)


def encode_fp16(level, bits, per_token=False):
    """Encode a block given as fp16 bit patterns [P][D]."""
    bits = np.asarray(bits, dtype=np.uint16)
    if int(level) == EXACT:
        return Record(EXACT, exact=bits.copy(), per_token=per_token)
    return encode(level, fp16.to_f64(bits), per_token)


def decode(rec):
    """Exact fp64 reconstruction of a record."""
    if rec.level == EXACT:
        return fp16.to_f64(rec.exact)
    if rec.level in (INT8, INT4, INT2):
        if rec.per_token:
            return dequant_scalar_per_token(rec.codes, rec.s16, rec.z16)
        return dequant_scalar(rec.codes, rec.s16, rec.z16)
    if rec.level in (CENTROID, MEAN):
        return dequant_centroid(rec.cent16, rec.ids)
    raise ValueError(rec.level)


class NotMonotone(ValueError):
    pass


def demote(rec, to_level):
    """Re-encode a record at a strictly lower level, directly from its current
    representation (section 3.2: demotion only, never promotion)."""
    if ORDER[int(to_level)] >= ORDER[rec.level]:
        raise NotMonotone(f"demote {rec.level} -> {to_level} is not a demotion")
    out = encode(to_level, decode(rec), rec.per_token)
    out.per_token = rec.per_token  # the grouping is a property of the tensor, kept down the ladder
    return out
