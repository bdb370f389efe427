"""Rate-distortion exact residual (Method, section 3.4, Eq. rdscore).

Each prompt token j gets the score  s_j = a_j * ||v_j - v_bar_j||^2  where a_j is
its attention mass and the second factor its value distortion; the tokens with
the highest scores, up to a fixed exact fraction, are kept in fp16.  Selection
uses prompt activations only.

Readings (listed in the design notes):

* v_bar_j is the token's value as the graded cache reconstructs it at its
  block's level (the workloads define the error as ||v - dequant(v)||^2; for a
  centroid block this is exactly the equation's block value centroid).
* e_j = sum over channels, ascending, of fl(fl(v_jd - v_hat_jd)^2) in fp64 with
  separate multiply and add (v - v_hat is exact in fp64);
  s_j = fl(a_j * e_j) with a_j the fp32 mass widened to fp64.
* n = floor(frac * T) tokens per (sequence, KV head) are kept (frac a ratio of
  integers, floored once): the first n of the
  order (s descending, token index ascending), reported ascending.
"""
import numpy as np


def distortion(v_exact, v_hat):
    """fp64 [T][D] x [T][D] -> fp64 [T], channel-sequential, no FMA."""
    v_exact = np.asarray(v_exact, dtype=np.float64)
    v_hat = np.asarray(v_hat, dtype=np.float64)
    acc = np.zeros(v_exact.shape[0], dtype=np.float64)
    for d in range(v_exact.shape[1]):
        diff = v_exact[:, d] - v_hat[:, d]
        sq = diff * diff
        acc = acc + sq
    return acc


def scores(v_exact, v_hat, mass_f32):
    a = np.asarray(mass_f32, dtype=np.float32).astype(np.float64)
    return a * distortion(v_exact, v_hat) + 0.0


def n_keep(T, frac=2, den=100):
    """Rows kept for an exact fraction frac / den (2% by default; RD-V2 keeps
    102 / 1000)."""
    return (int(frac) * int(T)) // int(den)


def select(s, n):
    """First n of (score desc, index asc), ascending."""
    s = np.asarray(s, dtype=np.float64)
    order = np.lexsort((np.arange(s.shape[0]), -s))
    return np.sort(order[:n]).astype(np.int32)
