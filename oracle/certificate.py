"""Attention error certificate (Method, section 3.6, Eq. certificate).

For exact keys/values k, v and their reconstructions k_hat, v_hat, with
compressed-cache weights a_hat and exact weights a, the output error splits as
    o - o_hat = sum_j a_hat_j (v_j - v_hat_j) + sum_j (a_j - a_hat_j) v_j
and is bounded by
    ||o - o_hat|| <= sum_b a_hat_b delta_b + min(2, M+/M- - M-/M+) * max_j ||v_j||,
    M+- = sum_b a_hat_b exp(+-eps_b),
with eps_b a bound on the logit error and delta_b on the value error of block b
(the second term is capped by the l1 distance of two distributions, 2).

``bound`` takes eps_b and delta_b from the exact keys and values (a pin: the
oracle's graded attention must satisfy it against its own exact attention).

At decode time the exact rows are gone, so the decode-time certificate
(``decode_bound``) works from per-block numbers kept with the cache:

    kerr_b = max_t ||k_t - k_hat_t||,  verr_b = max_t ||v_t - v_hat_t||,
    vmax_b = max_t ||v_t||  (over the block's 64 rows, exact rows as stored),

measured when a block is encoded, and carried through a demotion by the triangle
inequality (kerr_new = kerr_old + max_t ||k_hat_old,t - k_hat_new,t||, the same for
verr).  Then eps_b = ||q|| kerr_b / sqrt(D) bounds every logit error of the block
(Cauchy-Schwarz), delta_b = verr_b, and max_j ||v_j|| <= max_b vmax_b.  Tokens read
from the exact residual have eps = delta = 0.
"""
import numpy as np


def bound(q, k, v, khat, vhat, P=64):
    """q fp64 [D]; k, v, khat, vhat fp64 [T][D] -> (bound, ||o - o_hat||)."""
    Dd = q.shape[0]
    sc = 1.0 / np.sqrt(float(Dd))
    lg = (k @ q) * sc
    lh = (khat @ q) * sc
    a = np.exp(lg - lg.max())
    a /= a.sum()
    ah = np.exp(lh - lh.max())
    ah /= ah.sum()
    o = a @ v
    oh = ah @ vhat
    T = k.shape[0]
    nb = (T + P - 1) // P
    first = 0.0
    Mp = 0.0
    Mm = 0.0
    for b in range(nb):
        sl = slice(b * P, min((b + 1) * P, T))
        eps = np.max(np.abs(lg[sl] - lh[sl]))
        dlt = np.max(np.sqrt(((v[sl] - vhat[sl]) ** 2).sum(axis=1)))
        ab = ah[sl].sum()
        first += ab * dlt
        Mp += ab * np.exp(eps)
        Mm += ab * np.exp(-eps)
    second = min(2.0, Mp / Mm - Mm / Mp) * np.max(np.sqrt((v ** 2).sum(axis=1)))
    return first + second, float(np.sqrt(((o - oh) ** 2).sum()))


def block_numbers(x_exact, x_hat):
    """(max_t ||x_t - x_hat_t||, max_t ||x_t||) over the rows of one block (fp64)."""
    x_exact = np.asarray(x_exact, dtype=np.float64)
    x_hat = np.asarray(x_hat, dtype=np.float64)
    return float(np.sqrt(((x_exact - x_hat) ** 2).sum(axis=1)).max()), float(np.sqrt((x_exact ** 2).sum(axis=1)).max())


def demote_increment(x_hat_old, x_hat_new):
    """max_t ||x_hat_old,t - x_hat_new,t||: what a demotion adds to a block's error."""
    d = np.asarray(x_hat_old, dtype=np.float64) - np.asarray(x_hat_new, dtype=np.float64)
    return float(np.sqrt((d ** 2).sum(axis=1)).max())


def decode_bound(q, khat, kerr_tok, verr_tok, vmax):
    """Decode-time certificate for one query head.

    q fp64 [D]; khat fp64 [n][D] (the read set as decoded); kerr_tok, verr_tok [n] the
    per-token kerr and verr of the token's block (0 for exact rows); vmax the bound on
    every ||v_j||.  Returns sum_b a_hat_b delta_b + min(2, M+/M- - M-/M+) vmax."""
    q = np.asarray(q, dtype=np.float64)
    Dd = q.shape[0]
    lh = (khat @ q) / np.sqrt(float(Dd))
    ah = np.exp(lh - lh.max())
    ah /= ah.sum()
    eps = np.sqrt((q ** 2).sum()) * np.asarray(kerr_tok, dtype=np.float64) / np.sqrt(float(Dd))
    first = float((ah * np.asarray(verr_tok, dtype=np.float64)).sum())
    Mp = float((ah * np.exp(eps)).sum())
    Mm = float((ah * np.exp(-eps)).sum())
    return first + min(2.0, Mp / Mm - Mm / Mp) * float(vmax)
