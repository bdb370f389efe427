"""Single-query (Q = 1) GQA decode attention over a graded read set.

Method, section 3.7: dequantization happens inside an online-softmax attention
loop over all KV heads of the layer; section 3.1: the KV representation is held
once per KV head and shared by the query heads of its group.  The oracle is the
plain definition, in fp64:

    l_gj = (q_g . k_hat_j) / sqrt(D),   p_g = softmax_j(l_g),   o_g = sum_j p_gj v_hat_j

over the read set (all tokens j < T for a dense read; the selected pages plus the
current page for Compressed-Quest, section 3.5).  k_hat, v_hat come from each
token's block level; a token held in the exact residual (section 3.4) reads its
exact fp16 key and value instead of the graded copy (reading: the residual
overrides the graded entry; its block was quantized with all 64 tokens).

The order of summation is free here: the GPU result is compared under a tolerance.
"""
import numpy as np

from . import fp16


def attend(q, khat, vhat):
    """q: fp64 [G][D]; khat, vhat: fp64 [n][D] -> fp64 [G][D]."""
    q = np.asarray(q, dtype=np.float64)
    if khat.shape[0] == 0:
        raise ValueError("empty read set")
    Dd = q.shape[1]
    logits = (q @ khat.T) / np.sqrt(float(Dd))
    m = logits.max(axis=1, keepdims=True)
    p = np.exp(logits - m)
    return (p @ vhat) / p.sum(axis=1, keepdims=True)


def attend_bruteforce(q, khat, vhat):
    """Independent scalar-loop formula (used to pin ``attend`` on tiny inputs)."""
    import math
    G, Dd = len(q), len(q[0])
    n = len(khat)
    out = [[0.0] * Dd for _ in range(G)]
    for g in range(G):
        ls = []
        for j in range(n):
            s = 0.0
            for d in range(Dd):
                s += float(q[g][d]) * float(khat[j][d])
            ls.append(s / math.sqrt(Dd))
        mx = max(ls)
        ws = [math.exp(x - mx) for x in ls]
        tot = math.fsum(ws)
        for d in range(Dd):
            out[g][d] = math.fsum(ws[j] * float(vhat[j][d]) for j in range(n)) / tot
    return np.array(out)


def unit_decode(q_bits_group, khat, vhat, read_idx=None):
    """One (sequence, KV head) unit: q_bits_group uint16 [G][D]; khat/vhat fp64
    [T][D] (already carrying residual overrides); read_idx = token indices read
    (None = all)."""
    q = fp16.to_f64(q_bits_group)
    if read_idx is not None:
        khat = khat[read_idx]
        vhat = vhat[read_idx]
    return attend(q, khat, vhat)
