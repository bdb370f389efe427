"""Causal attention-mass observer, its EMA, and the analytic bit allocation
(Method, section 3.1: Eq. 1-2 and the EMA update, GQA aggregation; section 3.3:
Eq. allocation and its closed-form bit depth b*).

Test infrastructure: this is the oracle the GPU observer and allocator are
checked against; nothing in the product imports it.

Readings (the paper fixes the formulas but not these details; listed with the
others in the design notes):

* Observed queries are the last n_obs prompt positions T - n_obs .. T - 1, and
  query i sees keys 0 .. T - n_obs + i (causal prefill).
* w = softmax(q . k / sqrt(D)) over the visible keys, in fp64 (max-subtracted).
* GQA aggregation: a KV head's block mass is the mean over the group's query
  heads and the observed queries, so the masses of one KV head sum to 1.
* EMA: m = (1 - alpha) * m_old + alpha * m_new; alpha = 0.1 is the paper's
  update, alpha = 1 sets the mass from one observation.
* Error proxy e_b: the block's key range, max over channels of
  (max_t k - min_t k) over its tokens; the step of a b-bit scalar quantizer of
  that block is e_b / (2^b - 1).
* ||q||: the largest norm among the group's observed queries (fp64, channel-
  ascending sum of squares, then the square root).
* N_b: the number of blocks of the prefix, ceil(T / 64).
* b* = ceil(log2(x + 1)) with x = c * ||q|| * e_b * N_b * m_b / (2 * tau)
  (eps_t = tau / (N_b m_b) substituted), x formed left to right in fp64 from
  the fp32 mass.  b* (an integer) maps to a ladder level in one of two ways:
  - "up" (the default): the smallest level L in {1, 2, 4, 8} with b* <= L, else
    16, so that the level's step meets the tolerance eps_t;
  - "nearest": the level of {1, 2, 4, 8, 16} nearest to b*, ties to the larger
    level (the literal "nearest available discrete level" of section 3.3; b*
    = 3, 6 and 12 are the ties).
  Both are evaluated on x without a logarithm: b* <= n is exactly x <= 2^n - 1,
  so "up" has thresholds 1, 3, 15, 255 and "nearest" 1, 3, 31, 2047 (b* <= 5
  gives 4, b* <= 11 gives 8).  m_b = 0 gives b* = 0 and the centroid level
  (the clamp).
* e_b is the range of whatever fp16 tensor is passed: the keys (the default,
  matching the ||q|| factor, which bounds a logit error by ||q|| ||k - k_hat||)
  or the values (Fig. 1 labels e_b(L) a value error radius).
* The newest `window` blocks, and a partial last block, stay exact (the recent
  window of section 3.2).

The constants c and tau are not published; the tests pin the structure of the
formula (thresholds, monotonicity, window) rather than particular values.
"""
import numpy as np

from . import fp16
from .ladder import EXACT, INT8, INT4, INT2, CENTROID

P = 64


def _softmax_rows(s):
    """fp64 row softmax of logits with -inf for invisible keys."""
    m = np.max(s, axis=1, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=1, keepdims=True)


def observe_mass(q_bits, k_bits):
    """Eq. 1-2 for one KV head.

    q_bits : fp16 bits [n_obs][G][D], the group's queries at positions
             T - n_obs .. T - 1
    k_bits : fp16 bits [T][D], exact keys
    Returns m [nblk] fp64: mean over (query, head) of the softmax mass per block.
    """
    q = fp16.to_f64(np.asarray(q_bits, dtype=np.uint16))
    k = fp16.to_f64(np.asarray(k_bits, dtype=np.uint16))
    n_obs, G, D = q.shape
    T = k.shape[0]
    nblk = (T + P - 1) // P
    rows = q.reshape(n_obs * G, D)
    s = rows @ k.T / np.sqrt(D)  # [n_obs*G][T]
    pos = T - n_obs + np.repeat(np.arange(n_obs), G)  # position of each row's query
    s[np.arange(T)[None, :] > pos[:, None]] = -np.inf  # keys after the query
    w = _softmax_rows(s)
    per_blk = np.zeros((w.shape[0], nblk))
    for b in range(nblk):
        per_blk[:, b] = w[:, b * P:(b + 1) * P].sum(axis=1)
    return per_blk.mean(axis=0)


def ema(m_old, m_new, alpha=0.1):
    """Causal EMA of the mass (alpha = 1: the new observation alone)."""
    m_new = np.asarray(m_new, dtype=np.float64)
    if alpha == 1.0:
        return m_new.copy()
    return (1.0 - alpha) * np.asarray(m_old, dtype=np.float64) + alpha * m_new


def key_range(k_bits):
    """e_b for every block: max over channels of the range over the block's tokens
    (a partial last block over the tokens it has) of the fp16 tensor given, keys
    or values.  Exact in fp64."""
    k = fp16.to_f64(np.asarray(k_bits, dtype=np.uint16))
    T = k.shape[0]
    nblk = (T + P - 1) // P
    e = np.empty(nblk)
    for b in range(nblk):
        x = k[b * P:min((b + 1) * P, T)]
        e[b] = (x.max(axis=0) - x.min(axis=0)).max()
    return e


def query_norm(q_bits):
    """Largest ||q|| over the observed queries of one group (fp64, channel order)."""
    q = fp16.to_f64(np.asarray(q_bits, dtype=np.uint16)).reshape(-1, np.asarray(q_bits).shape[-1])
    best = 0.0
    for row in q:
        acc = 0.0
        for x in row:
            acc = acc + x * x
        best = max(best, float(np.sqrt(acc)))
    return best


# x <= 2^n - 1 is b* <= n: "up" takes n = L (the level itself); "nearest" takes the
# largest b* that is still nearer to L than to the next level (ties go up): 1, 2, 5, 11
_THRESH = {"up": ((CENTROID, 1.0), (INT2, 3.0), (INT4, 15.0), (INT8, 255.0)),
           "nearest": ((CENTROID, 1.0), (INT2, 3.0), (INT4, 31.0), (INT8, 2047.0))}


def bit_level(x, rounding="up"):
    """Ladder level of one block from x = c ||q|| e N m / (2 tau), b* = ceil(log2(x + 1)):
    "up" is the smallest L with b* <= L (x <= 2^L - 1), 16 above 255; "nearest" the
    level nearest to b*, ties up (thresholds 1, 3, 31, 2047)."""
    for lv, t in _THRESH[rounding]:
        if x <= t:
            return lv
    return EXACT


def allocate(m_f32, e, qn, T, c, tau, window, rounding="up"):
    """Levels per block (index 0 oldest) from the fp32 masses m_f32, the block
    ranges e and the query norm qn (section 3.3 closed form, read as above)."""
    m = np.asarray(m_f32, dtype=np.float32).astype(np.float64)
    nblk = (int(T) + P - 1) // P
    lv = np.empty(nblk, dtype=np.int8)
    for b in range(nblk):
        if b >= nblk - window or (b + 1) * P > T:
            lv[b] = EXACT
            continue
        x = float(c) * qn
        x = x * float(e[b])
        x = x * float(nblk)
        x = x * float(m[b])
        x = x / (2.0 * float(tau))
        lv[b] = bit_level(x, rounding)
    return lv
