"""Monotone precision ladder by block age (Method, section 3.2).

The cache is cut into blocks of P = 64 tokens; each block holds one level of
{16 (exact fp16), 8, 4, 2 (packed scalar codes), 1 (centroid state with 4
centroids), 0 (one-centroid state: the block mean, no per-token code)}.  A block
only ever moves down the ladder as it ages: there is no promotion, because once
demoted its dense data no longer exists.

The paper's own allocator (section 3.3) needs attention statistics from a real
model; the workloads here use fixed age ladders instead, with the band sizes
below.  Reading of the paper (listed with the others in the design notes): the
int8/int4 band boundaries are taken as floors of CUMULATIVE fractions of the
non-exact blocks (25% and 25%+35% = 60%).  At every workload size this gives the
same band sizes as flooring 25% and 35% separately, and unlike that alternative
each boundary moves by at most one block when one block is appended, which is
what keeps the ladder monotone as the context grows.

Levels are returned per block, index 0 = oldest block.
"""
import numpy as np

EXACT, INT8, INT4, INT2, CENTROID, MEAN = 16, 8, 4, 2, 1, 0
LEVELS = (EXACT, INT8, INT4, INT2, CENTROID, MEAN)
BLOCK = 64

# rank of a level on the ladder: larger = more precise
ORDER = {MEAN: 0, CENTROID: 1, INT2: 2, INT4: 3, INT8: 4, EXACT: 5}


def n_blocks(T, P=BLOCK):
    return (int(T) + P - 1) // P


def tiny_ladder(nblk):
    """Small workload: newest 4 blocks exact, next 8 int8, next 12 int4, rest int2.

    At T = 2048 this is 256 exact / 512 int8 / 768 int4 / 512 int2 tokens.
    """
    lv = np.empty(nblk, dtype=np.int8)
    for i in range(nblk):
        r = nblk - 1 - i  # age rank, 0 = newest
        if r < 4:
            lv[i] = EXACT
        elif r < 12:
            lv[i] = INT8
        elif r < 24:
            lv[i] = INT4
        else:
            lv[i] = INT2
    return lv


def graded_ladder(nblk, exact_blocks=16, pct8=25, pct84=60, pct_centroid=10):
    """Long-context ladder: newest ``exact_blocks`` exact, then int8 / int4 / int2
    bands of 25% / 35% / 40% of the remaining blocks, with the oldest 10% of ALL
    blocks held as centroids (taken out of the int2 band).
    """
    R = max(nblk - exact_blocks, 0)
    b8 = exact_blocks + (pct8 * R) // 100
    b4 = exact_blocks + (pct84 * R) // 100
    nc = (pct_centroid * nblk) // 100
    lv = np.empty(nblk, dtype=np.int8)
    for i in range(nblk):
        r = nblk - 1 - i
        if r < exact_blocks:
            lv[i] = EXACT
        elif i < nc:
            lv[i] = CENTROID
        elif r < b8:
            lv[i] = INT8
        elif r < b4:
            lv[i] = INT4
        else:
            lv[i] = INT2
    return lv


def rdv2_ladder(nblk, exact_blocks=16):
    """Low-rate RD-V2 base (section 3.4; its base is almost all centroid state):
    the newest ``exact_blocks`` blocks exact, every older block in the
    one-centroid state.  The exact residual (about 10.2% of the tokens) is kept on
    top of it.
    """
    lv = np.full(nblk, MEAN, dtype=np.int8)
    lv[max(nblk - exact_blocks, 0):] = EXACT
    return lv


def ladder(profile, T):
    nblk = n_blocks(T)
    if profile == "tiny":
        return tiny_ladder(nblk)
    if profile == "graded":
        return graded_ladder(nblk)
    if profile == "rdv2":
        return rdv2_ladder(nblk)
    if profile == "exact":
        return np.full(nblk, EXACT, dtype=np.int8)
    raise ValueError(profile)


def crossings(profile, T_old, T_new):
    """Blocks whose level changes when the context grows from T_old to T_new.

    Returns a list of (block, old_level, new_level); blocks that did not exist
    at T_old are not listed (they are born at their level).
    """
    old = ladder(profile, T_old)
    new = ladder(profile, T_new)
    out = []
    for i in range(len(old)):
        if old[i] != new[i]:
            out.append((i, int(old[i]), int(new[i])))
    return out
