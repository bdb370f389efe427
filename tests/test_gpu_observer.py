"""GPU parity of the causal mass observer, the query norms and the closed-form
level allocation (sections 3.1 and 3.3) against the oracle, through the C ABI.
Masses within 1e-4 relative (+1e-7 absolute: fp32 softmax against fp64); query
norms and levels exact (both sides decide the levels in fp64 from the same fp32
masses and fp64 norms)."""
import numpy as np
import pytest

from oracle import observer as oobs
from paper_2608_23599_amd import synth
from tests._util import kv_all

pytestmark = pytest.mark.gpu


def _obs_queries(wl, B, n_obs, Hq):
    return np.stack([synth.queries(wl, B, Hq, step=i) for i in range(n_obs)], axis=1)  # [B][n_obs][Hq][128]


def _group(q_obs, b, h, G):
    return q_obs[b, :, h * G:(h + 1) * G]


def _mass_close(got, want):
    assert np.all(np.abs(got - want) <= 1e-4 * want + 1e-7), np.max(np.abs(got - want))


@pytest.mark.parametrize("B,Hq,Hkv,T,n_obs", [(2, 8, 2, 1000, 16), (1, 28, 4, 4133, 64), (1, 32, 4, 2048, 64),
                                              (1, 4, 1, 70, 70), (1, 16, 1, 5000, 1)])
def test_observer_mass_matches_oracle(gpu, B, Hq, Hkv, T, n_obs):
    """Eq. 1-2 with causal rows and the GQA mean; n_obs * G = 512 is the largest
    supported row count; T = 70 with n_obs = T makes every key hidden from some row."""
    ks, _ = kv_all(61, B, Hkv, T)
    q_obs = _obs_queries(61, B, n_obs, Hq)
    got = gpu.observe_mass(q_obs, ks).cpu().numpy()
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hkv):
            want = oobs.observe_mass(_group(q_obs, b, h, G), ks[b, h])
            _mass_close(got[b, h], want)
            assert abs(got[b, h].sum() - 1.0) < 1e-5


def _extreme_inputs(kind, T=64 * 40 + 9, n_obs=8, Hq=4):
    """fp16 bits of queries [1][n_obs][Hq][128] and keys [1][1][T][128] whose block sums
    leave [2^-64, 2^64] against a reference of 0, so that the kernel's general path
    (reference moved to the block maximum) runs: 'scaled' multiplies the queries by 8
    (block sums up to about 2^134); 'cold' points the first three blocks' keys away
    from a direction the queries share (their sums near 2^-92 while the row has no
    earlier block), and the later blocks then lie about 2^100 above that reference."""
    from oracle import fp16
    ks, _ = kv_all(66, 1, 1, T)
    q = _obs_queries(66, 1, n_obs, Hq)
    qf = fp16.to_f64(np.asarray(q, dtype=np.uint16))
    kf = fp16.to_f64(np.asarray(ks, dtype=np.uint16))
    if kind == "scaled":
        qf = qf * 8.0
    else:
        d = np.ones(128) / np.sqrt(128)
        qf = qf * 0.25 + 4.0 * d
        kf[0, 0, :192] = -192.0 * d
    return qf.astype(np.float16).view(np.uint16), kf.astype(np.float16).view(np.uint16)


@pytest.mark.parametrize("kind", ["scaled", "cold"])
def test_observer_mass_extreme_logits(gpu, kind):
    """Block sums far outside [2^-64, 2^64] of the running reference: fp32 logits of
    up to about 130 (log2 units) stay within the same tolerance (an fp32 simulation
    of these inputs lands below a tenth of it)."""
    q_obs, ks = _extreme_inputs(kind)
    got = gpu.observe_mass(q_obs, ks).cpu().numpy()
    want = oobs.observe_mass(q_obs[0], ks[0, 0])
    _mass_close(got[0, 0], want)
    assert abs(got[0, 0].sum() - 1.0) < 1e-5


def test_observer_ema_update(gpu):
    B, Hq, Hkv, T, n_obs = 1, 8, 2, 1500, 8
    ks, _ = kv_all(62, B, Hkv, T)
    qa = _obs_queries(62, B, n_obs, Hq)
    qb = _obs_queries(63, B, n_obs, Hq)
    mass = gpu.observe_mass(qa, ks)
    gpu.observe_mass(qb, ks, alpha=0.1, mass=mass)
    got = mass.cpu().numpy()
    G = Hq // Hkv
    for h in range(Hkv):
        ma = oobs.observe_mass(_group(qa, 0, h, G), ks[0, h])
        mb = oobs.observe_mass(_group(qb, 0, h, G), ks[0, h])
        _mass_close(got[0, h], oobs.ema(ma, mb, 0.1))


def test_query_norms_exact(gpu):
    q_obs = _obs_queries(64, 2, 5, 12)
    got = gpu.query_norms(q_obs, 3).cpu().numpy()
    for b in range(2):
        for h in range(3):
            assert got[b, h] == oobs.query_norm(_group(q_obs, b, h, 4))


@pytest.mark.parametrize("T,window,rounding,tensor", [(64 * 300 + 17, 16, "up", 0), (64 * 40, 0, "up", 0),
                                                     (64 * 300 + 17, 16, "nearest", 0), (64 * 40, 0, "nearest", 1)])
def test_allocation_levels_exact(gpu, T, window, rounding, tensor):
    """Levels from the same fp32 masses and query norms are identical, for both
    roundings of b* and for e_b taken over the keys (tensor 0) or the values (1).
    The masses are seeded log-uniform over 4.5 decades (observed masses of random
    keys are too even to reach every level), and tau puts the median block at x = 6,
    so that the blocks spread over the whole ladder."""
    torch = pytest.importorskip("torch")
    B, Hq, Hkv, n_obs = 1, 8, 2, 8
    ks, vs = kv_all(65, B, Hkv, T)
    if tensor:
        ks = vs  # e_b from the value ranges
    q_obs = _obs_queries(65, B, n_obs, Hq)
    G = Hq // Hkv
    nb = (T + 63) // 64
    m = np.zeros((B, Hkv, nb), np.float32)
    for b in range(B):
        for h in range(Hkv):
            r = np.random.default_rng([65, b, h])
            m[b, h] = (10.0 ** r.uniform(-4.5, 0.0, nb) / nb).astype(np.float32)
    qn = np.array([[oobs.query_norm(_group(q_obs, b, h, G)) for h in range(Hkv)] for b in range(B)])
    e = oobs.key_range(ks[0, 0])
    nblk = len(e)
    c = 1.0
    xmed = 6.0 if rounding == "up" else 40.0  # nearest: int8 covers x up to 2047
    tau = float(np.median(c * qn[0, 0] * e * nblk * m[0, 0].astype(np.float64))) / (2.0 * xmed)
    got = gpu.allocate_levels(ks, torch.from_numpy(m), torch.from_numpy(qn), c, tau, window,
                              rounding=rounding).cpu().numpy()
    seen = set()
    for b in range(B):
        for h in range(Hkv):
            want = oobs.allocate(m[b, h], oobs.key_range(ks[b, h]), qn[b, h], T, c, tau, window, rounding=rounding)
            np.testing.assert_array_equal(got[b, h], want)
            seen |= set(int(x) for x in want)
    assert {1, 2, 4, 8, 16} <= seen
    # the GPU's own query norms give the same levels
    got2 = gpu.allocate_levels(ks, torch.from_numpy(m), gpu.query_norms(q_obs, Hkv), c, tau, window,
                               rounding=rounding).cpu().numpy()
    np.testing.assert_array_equal(got2, got)


def test_observer_rejects_bad_arguments(gpu):
    ks, _ = kv_all(66, 1, 1, 256)
    with pytest.raises(gpu.GkvError):
        gpu.observe_mass(_obs_queries(66, 1, 65, 8), ks)   # 65 * 8 rows > 512
    with pytest.raises(gpu.GkvError):
        gpu.observe_mass(_obs_queries(66, 1, 4, 8), ks, alpha=0.0)
    with pytest.raises(gpu.GkvError):
        gpu.observe_mass(_obs_queries(66, 1, 300, 1), ks)  # more observed queries than tokens


def test_observer_128k_full_size_sampled(gpu):
    """The observer at the 128k decode workload's shape (B = 8, 28 query / 4 KV
    heads, T = 131072) with the last 64 prompt positions observed (448 rows per KV
    head).  Units (0, 0) and (7, 3) hold their own seeded keys and are checked
    against the oracle; the other units repeat them."""
    from paper_2608_23599_amd import workloads
    wl = workloads.RD128K
    B, Hq, Hkv, T, n_obs = wl.B, wl.Hq, wl.Hkv, wl.T, 64
    samp = [(0, 0), (B - 1, Hkv - 1)]
    keys = {u: synth.kv_unit(wl.id, *u, T)[0] for u in samp}
    ks = np.empty((B, Hkv, T, 128), np.uint16)
    for b in range(B):
        for h in range(Hkv):
            ks[b, h] = keys[samp[(b * Hkv + h) % 2]]
    q_obs = _obs_queries(wl.id, B, n_obs, Hq)
    got = gpu.observe_mass(q_obs, ks).cpu().numpy()
    G = Hq // Hkv
    for b, h in samp:
        _mass_close(got[b, h], oobs.observe_mass(_group(q_obs, b, h, G), ks[b, h]))
