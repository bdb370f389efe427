"""Resident and read bits per value (Method, section 3.5 rate equations; section
4.4 metrics: bits of resident data per K or V value including overhead, and
bits read per value per query).

Per tensor block of P = 64 tokens x D = 128 channels:

    exact     P * D * 16
    int b     P * D * b + D * 2 * 16          (fp16 scale and zero per channel)
    centroid  K * D * 16 + P * log2(K)        (K = 4 fp16 centroids, 2-bit ids)
    mean      D * 16                          (one fp16 centroid, no ids)

Compressed-Quest adds 2 * D * 16 bits of exact box per closed page
(R_resident = R_graded + sum of boxes) and reads, per query, all stored boxes
plus the graded data of the selected pages and the current page
(R_read = R_boxes + sum over S(q) and the current page of R_b; R_boxes is the
same term in both equations).  A page read
from a block costs its rows of codes (or ids) plus the block's scale/zero (or
centroids) once per block touched.

The exact residual (section 3.4) costs, per kept token, 2 * D * 16 bits of
exact key and value plus a 32-bit token index, and the cache keeps one 64-bit
override mask per block while a residual exists.  A dense read reads all of it.
A Compressed-Quest read of a cache with a residual (the paper prices the two
separately; this is the reading used here) reads the residual rows of the tokens
in its read set (2 * D * 16 + 32 bits each) and the override mask of every block
it touches; the graded rows of those tokens are still counted with their pages.

Values are normalised by B * Hkv * T * 2 * D (keys and values).  The newest
block is always fully allocated, so a partial block counts whole.
"""
from .ladder import EXACT, INT8, INT4, INT2, CENTROID, MEAN

P, D = 64, 128
KCENT = 4
IDBITS = 2


def block_bits(level, P=P, D=D):
    level = int(level)
    if level == EXACT:
        return P * D * 16
    if level in (INT8, INT4, INT2):
        return P * D * level + D * 2 * 16
    if level == CENTROID:
        return KCENT * D * 16 + P * IDBITS
    if level == MEAN:
        return D * 16
    raise ValueError(level)


def block_overhead_bits(level, D=D):
    """Per-block side data read once per block touched (scale/zero or centroids)."""
    level = int(level)
    if level in (INT8, INT4, INT2):
        return D * 2 * 16
    if level == CENTROID:
        return KCENT * D * 16
    if level == MEAN:
        return D * 16
    return 0


def row_bits(level, D=D):
    """Bits of one token row of codes / ids / exact values."""
    level = int(level)
    if level == EXACT:
        return D * 16
    if level in (INT8, INT4, INT2):
        return D * level
    if level == CENTROID:
        return IDBITS
    if level == MEAN:
        return 0
    raise ValueError(level)


BOX_BITS = 2 * D * 16
RES_ROW_BITS = 2 * D * 16 + 32
MASK_BITS = 64


def unit_rates(levels, T, page=None, nres=0, pages=None, res_idx=None, P=P, D=D):
    """Bits for one (sequence, KV head) unit.

    levels  : per-block levels (index 0 oldest)
    page    : Quest page size in tokens, or None when no boxes are kept
    nres    : exact residual rows kept
    pages   : selected page indices for one query (Quest read), or None (dense)
    res_idx : the residual rows' tokens (needed for a Quest read with nres > 0)
    Returns dict(resident_bits, read_bits, values).
    """
    nblk = len(levels)
    graded = 2 * sum(block_bits(lv, P, D) for lv in levels)
    boxes = 0
    if page is not None:
        boxes = (int(T) // page) * BOX_BITS
    res = 0
    if nres:
        res = nres * RES_ROW_BITS + nblk * MASK_BITS
    resident = graded + boxes + res
    if pages is None:
        read = graded + res
    else:
        cur = (int(T) - 1) // page
        read = boxes  # R_boxes: all stored summaries, as in the resident equation
        touched = set()
        tokens = set()
        for p in sorted(set(int(x) for x in pages if x >= 0) | {cur}):
            t0 = p * page
            t1 = min(t0 + page, int(T))
            for t in range(t0, t1):
                b = t // P
                read += 2 * row_bits(levels[b], D)
                touched.add(b)
                tokens.add(t)
        for b in touched:
            read += 2 * block_overhead_bits(levels[b], D)
        if nres:
            if res_idx is None:
                raise ValueError("a Compressed-Quest read with a residual needs the residual tokens")
            read += sum(1 for t in set(int(x) for x in res_idx[:nres]) if t in tokens) * RES_ROW_BITS
            read += len(touched) * MASK_BITS
    return dict(resident_bits=resident, read_bits=read, values=int(T) * 2 * D)


def bpv(bits, values):
    return bits / float(values)
