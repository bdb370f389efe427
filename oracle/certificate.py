"""Attention error certificate (Method, section 3.6, Eq. certificate).

For exact keys/values k, v and their reconstructions k_hat, v_hat, with
compressed-cache weights a_hat and exact weights a, the output error splits as
    o - o_hat = sum_j a_hat_j (v_j - v_hat_j) + sum_j (a_j - a_hat_j) v_j
and is bounded by
    ||o - o_hat|| <= sum_b a_hat_b delta_b + min(2, M+/M- - M-/M+) * max_j ||v_j||,
    M+- = sum_b a_hat_b exp(+-eps_b),
with eps_b a bound on the logit error and delta_b on the value error of block b
(the second term is capped by the l1 distance of two distributions, 2).

Used only as a pin: the oracle's graded attention must satisfy the bound against
its own exact attention on every query head.
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
