"""Compressed-Quest: exact per-page key boxes and box upper-bound page ranking.

Method, section 3.5: before quantization, the exact fp16 per-channel minimum and
maximum of the keys of each closed page are stored; a query ranks all closed
pages by the box upper bound and reads the top-ranked pages plus the current
partial page, which is always read; every other page is hard-masked.  The bound
is the one of Quest (related work): for a page with box [kmin, kmax],
    UB(q) = sum_d max(q_d * kmin_d, q_d * kmax_d) >= q . k   for every key k in the page.

Readings (listed in the design notes):

* Pages are 16 tokens (the workloads' page size); page p covers tokens
  [16p, 16p + 16).  The current page is cur = floor((T - 1) / 16); it is always
  read and never ranked; pages 0 .. cur-1 are ranked.
* The paper fixes no precision for the bound; it is evaluated in fp32 as a
  channel-ascending running sum acc <- acc + q_d * (q_d >= 0 ? kmax_d : kmin_d).
  Every product of two fp16 values is exact in fp32 (at most 22 significant
  bits, magnitudes between 2^-48 and 2^32, so no denormal and no overflow), so
  each step rounds once, on the add, with or without a fused multiply-add.  A -0
  result is canonicalised to +0.  No 1/sqrt(d) scale (it cannot change the
  order).  Because the terms satisfy term_d >= q_d * k_d for every key k of the
  page and round-to-nearest addition is monotone, the fp32 bound is never below
  the same channel-ascending fp32 sum for any of the page's keys.
* GQA: the KV head's page score is the maximum of the bound over the query
  heads of its group (the tightest bound on any group head's best logit).
* Selection: the first k pages of the order (score descending, page index
  ascending), reported in ascending page order, padded with -1 when fewer than
  k pages are ranked.
"""
import numpy as np

from . import fp16

PAGE = 16


def current_page(T, page=PAGE):
    return (int(T) - 1) // page


def page_boxes(k_bits, page=PAGE):
    """k_bits: uint16 [T][D] exact fp16 keys -> (kmin bits, kmax bits), each
    [npages_closed][D] for the pages whose tokens are all present."""
    k = fp16.to_f64(k_bits)
    T = k.shape[0]
    n = T // page
    kmin = np.empty((n, k.shape[1]), dtype=np.uint16)
    kmax = np.empty((n, k.shape[1]), dtype=np.uint16)
    for p in range(n):
        blk = k[p * page:(p + 1) * page]
        kmin[p] = fp16.from_f64(blk.min(axis=0))
        kmax[p] = fp16.from_f64(blk.max(axis=0))
    return kmin, kmax


def box_upper_bounds(q_bits, kmin_bits, kmax_bits):
    """q_bits [G][D], boxes [N][D] -> fp32 [G][N] channel-sequential bounds."""
    q = fp16.to_f64(q_bits).astype(np.float32)  # fp16 values are exact in fp32
    lo = fp16.to_f64(kmin_bits).astype(np.float32)
    hi = fp16.to_f64(kmax_bits).astype(np.float32)
    G, Dd = q.shape
    N = lo.shape[0]
    acc = np.zeros((G, N), dtype=np.float32)
    for d in range(Dd):
        qd = q[:, d][:, None]
        bound = np.where(qd >= 0.0, hi[:, d][None, :], lo[:, d][None, :])
        acc = acc + qd * bound  # float32 throughout: the product is exact, the add rounds
    assert acc.dtype == np.float32
    return acc


def page_scores(q_bits, kmin_bits, kmax_bits):
    """GQA page score: max over the group's query heads; -0 -> +0."""
    ub = box_upper_bounds(q_bits, kmin_bits, kmax_bits)
    s = ub.max(axis=0) if ub.shape[1] else np.zeros(0)
    return s + 0.0


def select_top(scores, k):
    """First k of the order (score desc, index asc), returned ascending, -1 padded."""
    scores = np.asarray(scores, dtype=np.float64)
    n = scores.shape[0]
    order = np.lexsort((np.arange(n), -scores))
    chosen = np.sort(order[:k]).astype(np.int32)
    out = np.full(k, -1, dtype=np.int32)
    out[:len(chosen)] = chosen
    return out


def quest_select(q_bits, kmin_bits, kmax_bits, T, k, page=PAGE):
    """Pages selected for one (sequence, KV head): ranked pages are 0 .. cur-1."""
    cur = current_page(T, page)
    s = page_scores(q_bits, kmin_bits[:cur], kmax_bits[:cur])
    return select_top(s, k)


def read_tokens(pages, T, page=PAGE):
    """Token indices read by a Quest step: selected pages plus the current page."""
    cur = current_page(T, page)
    toks = []
    for p in list(p for p in pages if p >= 0) + [cur]:
        toks.extend(range(p * page, min((p + 1) * page, T)))
    return np.array(sorted(set(toks)), dtype=np.int64)
