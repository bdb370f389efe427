"""Thin ctypes binding over libgkv's C ABI (include/gkv.h).

torch supplies device memory and the current HIP stream; every step of the decode
path runs in the library's HIP kernels.  The library must be built
(``__graft_entry__.build()``); importing this module without it raises.

The function names mirror the C calls (``quantize_block``, ``demote``,
``page_boxes``, ``quest_select``, ``graded_decode_attn``, ``rd_residual_select``,
``append``); ``GradedCache`` owns the device tables and the slab arena of one
layer's cache and marshals them into the ``gkv_cache`` descriptor.
"""
import ctypes
import os

import numpy as np
import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "_lib", "libgkv.so")
if not os.path.exists(_LIB_PATH):
    raise ImportError(f"{_LIB_PATH} is not built; run __graft_entry__.build()")
lib = ctypes.CDLL(_LIB_PATH)

EXACT, INT8, INT4, INT2, CENTROID, MEAN = 16, 8, 4, 2, 1, 0
LEVELS = (EXACT, INT8, INT4, INT2, CENTROID, MEAN)
KEYS, VALUES, VALUES_PER_TOKEN = 0, 1, 2
PROFILES = {"tiny": 0, "graded": 1, "exact": 2, "rdv2": 3}
P, D = 64, 128

_vp, _i32, _i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64


class CacheStruct(ctypes.Structure):
    _fields_ = [
        ("B", _i32), ("Hkv", _i32), ("Hq", _i32), ("D", _i32),
        ("T", _i64), ("nblk_cap", _i32),
        ("level", _vp), ("koff", _vp), ("voff", _vp), ("arena", _vp), ("arena_bytes", _i64),
        ("level_host", _vp),
        ("page", _i32), ("npage_cap", _i64), ("boxes", _vp),
        ("nres", _i32), ("nres_cap", _i32), ("res_idx", _vp), ("res_rows", _vp), ("res_mask", _vp),
        ("res_off", _vp),
        ("cert", _vp),
        ("v_per_token", _i32),
        ("version", ctypes.c_uint64),
        ("seq_len", _vp), ("seq_len_host", _vp),
    ]


class Rates(ctypes.Structure):
    _fields_ = [("resident_bits", _i64), ("read_bits", _i64), ("values", _i64)]


def _sig(name, res, args):
    f = getattr(lib, name)
    f.restype = res
    f.argtypes = args
    return f


_P = ctypes.POINTER
_strerror = _sig("gkv_strerror", ctypes.c_char_p, [_i32])
_block_bytes = _sig("gkv_block_bytes", _i64, [_i32])
_ladder_levels = _sig("gkv_ladder_levels", _i32, [_i32, _i64, _vp, _i32])
_ladder_crossings = _sig("gkv_ladder_crossings", _i32, [_P(CacheStruct), _i32, _i64, _vp, _vp, _i32])
_pool_create = _sig("gkv_pool_create", _vp, [_vp])
_pool_bytes = _sig("gkv_pool_bytes", _i64, [_vp])
_pool_alloc = _sig("gkv_pool_alloc", _i64, [_vp, _i32])
_pool_free = _sig("gkv_pool_free", _i32, [_vp, _i32, _i64])
_pool_used = _sig("gkv_pool_used", _i64, [_vp, _i32])
_pool_destroy = _sig("gkv_pool_destroy", None, [_vp])
_account = _sig("gkv_account", _i32, [_P(CacheStruct), _vp, _i32, _vp, _P(Rates)])
_decode_record = _sig("gkv_decode_record", _i32, [_i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp])
_f64_to_f16 = _sig("gkv_f64_to_f16", ctypes.c_uint16, [ctypes.c_double])
_workspace_bytes = _sig("gkv_workspace_bytes", _i64, [_P(CacheStruct), _i32, _i32])
_quantize_block = _sig("gkv_quantize_block", _i32, [_P(CacheStruct), _i32, _vp, _i64, _i32, _i32, _vp])
_demote = _sig("gkv_demote", _i32, [_P(CacheStruct), _i32, _vp, _vp, _vp, _vp, _vp])
_page_boxes = _sig("gkv_page_boxes", _i32, [_P(CacheStruct), _vp, _i64, _i64, _i64, _vp])
_append = _sig("gkv_append", _i32, [_P(CacheStruct), _vp, _vp, _vp, _vp, _vp])
_quest_select = _sig("gkv_quest_select", _i32, [_vp, _P(CacheStruct), _i32, _vp, _vp, _i64, _vp])
_attn = _sig("gkv_graded_decode_attn", _i32, [_vp, _P(CacheStruct), _vp, _i32, _vp, _vp, _i64, _vp])
_attn_bound = _sig("gkv_graded_decode_attn_bound", _i32, [_vp, _P(CacheStruct), _vp, _vp, _vp, _i64, _vp])
_attn_plan = _sig("gkv_attn_plan", _i32, [_P(CacheStruct), _vp, _i32, _vp, _i64, _vp])
_attn_partials = _sig("gkv_attn_partials", _i32, [_vp, _P(CacheStruct), _vp, _i32, _vp, _i64, _vp])
_attn_merge = _sig("gkv_attn_merge", _i32, [_P(CacheStruct), _vp, _i32, _vp, _vp, _i64, _vp])
_rd = _sig("gkv_rd_residual_select", _i32, [_P(CacheStruct), _vp, _vp, _vp, _i32, _vp, _i64, _vp])
_cache_changed = _sig("gkv_cache_changed", None, [_P(CacheStruct)])
_retire = _sig("gkv_retire_sequence", _i32, [_P(CacheStruct), _vp, _vp, _vp, _i32, _vp])
_admit = _sig("gkv_admit_sequence", _i32, [_P(CacheStruct), _i32, _vp])
_stream_probe = _sig("gkv_stream_read_probe", _i32, [_vp, _i64, _vp, _i32, _vp])
_attn_noalloc = _sig("gkv_graded_decode_attn_noalloc", _i32, [_vp, _P(CacheStruct), _vp, _i32, _vp, _vp])
_noalloc_bytes = _sig("gkv_noalloc_scratch_bytes", _i64, [])
_layers_step = _sig("gkv_layers_step", _i32, [_vp, _vp, _vp, _vp, _i32, _i32, _vp, _vp, _vp])
_observe_ws = _sig("gkv_observe_ws_bytes", _i64, [_i32, _i32, _i32, _i64, _i32])
_observe = _sig("gkv_observe_mass", _i32,
                [_vp, _i32, _vp, _i32, _i32, _i32, _i64, ctypes.c_float, _vp, _vp, _i64, _vp])
_query_norms = _sig("gkv_query_norms", _i32, [_vp, _i32, _i32, _i32, _i32, _vp, _vp])
_allocate = _sig("gkv_allocate_levels", _i32,
                 [_vp, _vp, _vp, _i32, _i32, _i64, ctypes.c_double, ctypes.c_double, _i32, _i32, _vp, _vp])
ROUNDING = {"up": 0, "nearest": 1}

EXPORTED = [
    "gkv_strerror", "gkv_block_bytes", "gkv_ladder_levels", "gkv_ladder_crossings", "gkv_pool_create",
    "gkv_pool_bytes", "gkv_pool_alloc", "gkv_pool_free", "gkv_pool_used", "gkv_pool_destroy", "gkv_account",
    "gkv_decode_record", "gkv_f64_to_f16", "gkv_workspace_bytes", "gkv_quantize_block", "gkv_demote",
    "gkv_page_boxes", "gkv_append", "gkv_quest_select", "gkv_graded_decode_attn", "gkv_rd_residual_select",
    "gkv_attn_plan", "gkv_attn_partials", "gkv_attn_merge", "gkv_graded_decode_attn_bound",
    "gkv_observe_ws_bytes", "gkv_observe_mass", "gkv_query_norms", "gkv_allocate_levels", "gkv_layers_step",
    "gkv_cache_changed", "gkv_graded_decode_attn_noalloc", "gkv_noalloc_scratch_bytes", "gkv_retire_sequence",
    "gkv_admit_sequence", "gkv_stream_read_probe",
]


class GkvError(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__(f"{what}: {_strerror(status).decode()} ({status})")


def _check(st, what):
    if st != 0:
        raise GkvError(st, what)


def _np_ptr(a):
    return ctypes.c_void_p(a.ctypes.data)


def _dptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def block_bytes(level):
    return int(_block_bytes(level))


def _fp16_dev(x, device="cuda"):
    """fp16 bit patterns (numpy uint16 or a 16-bit tensor) as a contiguous device tensor."""
    if isinstance(x, np.ndarray):
        x = torch.from_numpy(np.ascontiguousarray(x).view(np.int16))
    return x.to(device).contiguous()


def observe_ws_bytes(B, Hkv, Hq, T, n_obs):
    nb = int(_observe_ws(B, Hkv, Hq, T, n_obs))
    if nb < 0:
        raise GkvError(-2, "observe_ws_bytes")
    return nb


def observe_mass(q_obs, k, alpha=1.0, mass=None, ws=None):
    """gkv_observe_mass: q_obs [B][n_obs][Hq][128], k [B][Hkv][T][128] fp16 bits.
    Returns the fp32 mass [B][Hkv][ceil(T/64)] (updated in place when given)."""
    q_obs, k = _fp16_dev(q_obs), _fp16_dev(k)
    B, n_obs, Hq, _ = q_obs.shape
    Hkv, T = k.shape[1], k.shape[2]
    nblk = (T + P - 1) // P
    if mass is None:
        mass = torch.empty((B, Hkv, nblk), dtype=torch.float32, device=k.device)
    nb = int(_observe_ws(B, Hkv, Hq, T, n_obs))
    if nb < 0:
        raise GkvError(-2, "observe_ws_bytes")
    if ws is None or ws.numel() < nb:
        ws = torch.empty(nb, dtype=torch.uint8, device=k.device)
    _check(_observe(_dptr(q_obs), n_obs, _dptr(k), B, Hkv, Hq, T, float(alpha), _dptr(mass), _dptr(ws), ws.numel(),
                    _stream()), "observe_mass")
    return mass


def query_norms(q_obs, Hkv):
    """gkv_query_norms: the largest query norm of each group, fp64 [B][Hkv]."""
    q_obs = _fp16_dev(q_obs)
    B, n_obs, Hq, _ = q_obs.shape
    qn = torch.empty((B, Hkv), dtype=torch.float64, device=q_obs.device)
    _check(_query_norms(_dptr(q_obs), n_obs, B, Hkv, Hq, _dptr(qn), _stream()), "query_norms")
    return qn


def allocate_levels(k, mass, qn, c, tau, window, rounding="up"):
    """gkv_allocate_levels: int8 levels [B][Hkv][ceil(T/64)] on the device.  e_b is
    the block range of the tensor passed as k (keys, or values for the value-range
    reading); rounding is "up" or "nearest"."""
    k = _fp16_dev(k)
    B, Hkv, T = k.shape[0], k.shape[1], k.shape[2]
    mass = mass.to(k.device, torch.float32).contiguous()
    qn = qn.to(k.device, torch.float64).contiguous()
    lv = torch.empty((B, Hkv, (T + P - 1) // P), dtype=torch.int8, device=k.device)
    _check(_allocate(_dptr(k), _dptr(mass), _dptr(qn), B, Hkv, T, float(c), float(tau), int(window),
                     ROUNDING[rounding], _dptr(lv), _stream()), "allocate_levels")
    return lv


def stream_read_probe(buf, sink):
    """gkv_stream_read_probe: one streaming read of a device buffer (measurement)."""
    _check(_stream_probe(_dptr(buf), buf.numel() * buf.element_size(), _dptr(sink), sink.numel(), _stream()),
           "stream_read_probe")


def f64_to_f16(x):
    return int(_f64_to_f16(float(x)))


def ladder_levels(profile, T):
    nblk = (int(T) + P - 1) // P
    out = np.empty(nblk, dtype=np.int8)
    _check(_ladder_levels(PROFILES.get(profile, profile), int(T), _np_ptr(out), nblk), "ladder_levels")
    return out


def decode_record(level, tensor, rec):
    """Host decode of one record (bytes / uint8 array) -> dict of numpy arrays."""
    rec = np.ascontiguousarray(np.frombuffer(bytes(rec), dtype=np.uint8))
    vals = np.empty((P, D), dtype=np.float64)
    codes = np.empty((P, D), dtype=np.int32)
    s = np.empty(D, dtype=np.uint16)
    z = np.empty(D, dtype=np.uint16)
    ids = np.empty(P, dtype=np.int32)
    cent = np.empty((4, D), dtype=np.uint16)
    _check(_decode_record(level, tensor, _np_ptr(rec), _np_ptr(vals), _np_ptr(codes), _np_ptr(s), _np_ptr(z),
                          _np_ptr(ids), _np_ptr(cent)), "decode_record")
    out = {"values": vals}
    if level in (INT8, INT4, INT2):
        g = P if tensor == VALUES_PER_TOKEN else D  # groups: tokens or channels
        out.update(codes=codes, s16=s[:g].copy(), z16=z[:g].copy())
    if level == CENTROID:
        out.update(ids=ids, cent16=cent)
    if level == MEAN:
        out.update(ids=ids, cent16=cent[:1].copy())
    return out


class Pool:
    """Per-level slab pools inside one arena (host bookkeeping in the library)."""

    def __init__(self, caps):
        arr = np.array([int(caps.get(lv, 0)) for lv in LEVELS], dtype=np.int64)
        self._caps = arr
        self.h = _pool_create(_np_ptr(arr))
        if not self.h:
            raise GkvError(-1, "pool_create")

    @property
    def bytes(self):
        return int(_pool_bytes(self.h))

    def alloc(self, level):
        off = int(_pool_alloc(self.h, level))
        if off < 0:
            raise GkvError(-1, f"pool exhausted for level {level}")
        return off

    def free(self, level, off):
        _check(_pool_free(self.h, level, int(off)), "pool_free")

    def used(self, level):
        return int(_pool_used(self.h, level))

    def __del__(self, _destroy=_pool_destroy):
        # the destroy function is bound at definition: at interpreter exit the module's
        # globals may already be gone when the last pools are collected
        if getattr(self, "h", None):
            _destroy(self.h)
            self.h = None


def _as_bits(t, device):
    """fp16 bit patterns as an int16 device tensor."""
    if isinstance(t, torch.Tensor) and t.dtype == torch.int16 and t.device == device and t.is_contiguous():
        return t  # already in place: no conversion or copy (the decode loop's case)
    if isinstance(t, np.ndarray):
        t = torch.from_numpy(np.ascontiguousarray(t).view(np.int16))
    if t.dtype == torch.float16:
        t = t.view(torch.int16)
    return t.to(device).contiguous()


class GradedCache:
    """One layer's graded KV cache in device memory (section 3.2 ladder, optional
    Compressed-Quest boxes and exact residual)."""

    def __init__(self, B, Hkv, Hq, T, nblk_cap, caps, page=0, npage_cap=0, nres_cap=0, device="cuda",
                 v_per_token=False, seq_lens=None):
        self.device = torch.device(device)
        # sequences of different lengths (-1: retired): host and device copies
        if seq_lens is not None:
            self.seq_len_host = np.ascontiguousarray(np.array(seq_lens, dtype=np.int64).reshape(B))
            self.seq_len = torch.from_numpy(self.seq_len_host.copy()).to(self.device)
            T = int(self.seq_len_host.max(initial=0))
        else:
            self.seq_len_host = self.seq_len = None
        self.v_per_token = bool(v_per_token)
        self.B, self.Hkv, self.Hq = B, Hkv, Hq
        self.units = B * Hkv
        self.nblk_cap = nblk_cap
        self.pool = Pool(caps)
        self.arena = torch.empty(max(self.pool.bytes, 256), dtype=torch.uint8, device=self.device)
        self._dev = self.arena.device  # the concrete device (with its index), for the inputs' fast path
        self.level = torch.zeros((B, Hkv, nblk_cap), dtype=torch.int8, device=self.device)
        self.koff = torch.zeros((B, Hkv, nblk_cap), dtype=torch.int64, device=self.device)
        self.voff = torch.zeros((B, Hkv, nblk_cap), dtype=torch.int64, device=self.device)
        self.level_host = np.zeros((B, Hkv, nblk_cap), dtype=np.int8)
        self.koff_host = np.zeros((B, Hkv, nblk_cap), dtype=np.int64)
        self.voff_host = np.zeros((B, Hkv, nblk_cap), dtype=np.int64)
        self.page = page
        self.npage_cap = npage_cap
        self.boxes = (torch.zeros((B, Hkv, npage_cap * 2 * D), dtype=torch.int16, device=self.device)
                      if page else None)
        self.nres_cap = nres_cap
        nrb = (nres_cap + P - 1) // P
        if nres_cap:
            self.res_idx = torch.zeros((B, Hkv, nres_cap), dtype=torch.int32, device=self.device)
            self.res_rows = torch.zeros((B, Hkv, nrb * 2 * 16384), dtype=torch.uint8, device=self.device)
            self.res_mask = torch.zeros((B, Hkv, nblk_cap), dtype=torch.int64, device=self.device)
            self.res_off = torch.zeros((B, Hkv, nblk_cap + 1), dtype=torch.int32, device=self.device)
        else:
            self.res_idx = self.res_rows = self.res_mask = self.res_off = None
        # per-block certificate numbers {kerr, verr, vmax, 0}
        self.cert = torch.zeros((B, Hkv, nblk_cap, 4), dtype=torch.float32, device=self.device)
        self.c = CacheStruct()
        self._bind(T, 0)
        self._ws = {}

    def _bind(self, T, nres):
        c = self.c
        c.B, c.Hkv, c.Hq, c.D = self.B, self.Hkv, self.Hq, D
        c.T = T
        c.nblk_cap = self.nblk_cap
        c.level = self.level.data_ptr()
        c.koff = self.koff.data_ptr()
        c.voff = self.voff.data_ptr()
        c.arena = self.arena.data_ptr()
        c.arena_bytes = self.arena.numel()
        c.level_host = self.level_host.ctypes.data
        c.page = self.page
        c.npage_cap = self.npage_cap
        c.boxes = self.boxes.data_ptr() if self.boxes is not None else None
        c.nres = nres
        c.nres_cap = self.nres_cap
        c.res_idx = self.res_idx.data_ptr() if self.nres_cap else None
        c.res_rows = self.res_rows.data_ptr() if self.nres_cap else None
        c.res_mask = self.res_mask.data_ptr() if self.nres_cap else None
        c.res_off = self.res_off.data_ptr() if self.nres_cap else None
        c.cert = self.cert.data_ptr()
        c.v_per_token = int(self.v_per_token)
        c.seq_len = self.seq_len.data_ptr() if self.seq_len is not None else None
        c.seq_len_host = self.seq_len_host.ctypes.data if self.seq_len_host is not None else None
        _cache_changed(ctypes.byref(c))  # new tables: a fresh version stamp

    def clone(self):
        """A read-only copy in separate device memory (same layout and offsets), for
        benchmarks that rotate identical caches; it cannot append or demote."""
        new = object.__new__(GradedCache)
        new.__dict__.update(self.__dict__)
        for name in ("arena", "level", "koff", "voff", "boxes", "res_idx", "res_rows", "res_mask", "res_off", "cert"):
            t = getattr(self, name)
            setattr(new, name, t.clone() if t is not None else None)
        new.level_host = self.level_host.copy()
        new.koff_host = self.koff_host.copy()
        new.voff_host = self.voff_host.copy()
        if self.seq_len is not None:
            new.seq_len = self.seq_len.clone()
            new.seq_len_host = self.seq_len_host.copy()
        new.pool = None
        new.c = CacheStruct()
        new._bind(self.T, int(self.c.nres))
        new._ws = {}
        return new

    # ------------------------------------------------------------ construction
    @classmethod
    def build(cls, k, v, Hq, levels, page=0, nres_cap=0, device="cuda", extra_blocks=0, slack=None,
              v_per_token=False, seq_lens=None):
        """k, v: fp16 bits [B][Hkv][T][128] (numpy uint16 or torch int16/float16).
        levels: per-block levels, [nblk] (shared) or [B][Hkv][nblk].  Encodes every
        block at its level (gkv_quantize_block) and, with page > 0, writes the page
        boxes from the exact keys (gkv_page_boxes).  seq_lens: per-sequence lengths
        (<= T; k and v are padded to T), blocks past a sequence's end take no slot."""
        kd = _as_bits(k, device)
        vd = _as_bits(v, device)
        B, Hkv, T, Dd = kd.shape
        assert Dd == D
        nblk = (T + P - 1) // P
        lv = np.asarray(levels, dtype=np.int8)
        if lv.ndim == 1:
            lv = np.broadcast_to(lv, (B, Hkv, nblk))
        assert lv.shape == (B, Hkv, nblk)
        nblk_cap = nblk + extra_blocks
        lens = np.full(B, T, np.int64) if seq_lens is None else np.asarray(seq_lens, np.int64)
        owned = np.arange(nblk)[None, :] < ((np.maximum(lens, 0) + P - 1) // P)[:, None]  # [B][nblk]
        owned = np.broadcast_to(owned[:, None, :], (B, Hkv, nblk))
        # one slot per tensor block (keys and values separately), plus slack for
        # demotions and appended blocks
        caps = {L: 2 * int(((lv == L) & owned).sum()) for L in LEVELS}
        for L, n in (slack or {}).items():
            caps[L] += 2 * n
        npage_cap = 0
        if page:
            npage_cap = (((T + extra_blocks * P) // page) + 63) // 64 * 64
        self = cls(B, Hkv, Hq, T, nblk_cap, caps, page=page, npage_cap=npage_cap, nres_cap=nres_cap, device=device,
                   v_per_token=v_per_token, seq_lens=seq_lens)
        for b in range(B):
            for h in range(Hkv):
                for i in range(nblk):
                    if not owned[b, h, i]:
                        continue
                    L = int(lv[b, h, i])
                    self.level_host[b, h, i] = L
                    self.koff_host[b, h, i] = self.pool.alloc(L)
                    self.voff_host[b, h, i] = self.pool.alloc(L)
        self._upload_tables()
        self.quantize_block(KEYS, kd, 0, nblk)
        self.quantize_block(VALUES, vd, 0, nblk)
        if page:
            self.page_boxes(kd, 0, T // page)
        return self

    def _upload_tables(self):
        self.level.copy_(torch.from_numpy(self.level_host))
        self.koff.copy_(torch.from_numpy(self.koff_host))
        self.voff.copy_(torch.from_numpy(self.voff_host))
        _cache_changed(ctypes.byref(self.c))  # the tables were written from here

    @property
    def T(self):
        return int(self.c.T)

    def lengths(self):
        """Tokens of every sequence (-1: retired)."""
        if self.seq_len_host is not None:
            return self.seq_len_host.copy()
        return np.full(self.B, self.T, np.int64)

    def retire(self, b):
        """gkv_retire_sequence: sequence b's slots go back to the pool."""
        _check(_retire(ctypes.byref(self.c), self.pool.h, _np_ptr(self.koff_host), _np_ptr(self.voff_host), int(b),
                       _stream()), "retire_sequence")

    def admit(self, b):
        """gkv_admit_sequence: retired slot b becomes an empty sequence."""
        _check(_admit(ctypes.byref(self.c), int(b), _stream()), "admit_sequence")

    def workspace(self, op, topk=0):
        """The workspace of call `op` (and top-k), allocated once: its size depends on the
        cache's capacities only, which do not change."""
        key = (op, topk)
        ws = self._ws.get(key)
        if ws is not None:
            return ws
        n = int(_workspace_bytes(ctypes.byref(self.c), op, topk))
        if n < 0:
            raise GkvError(-1, "workspace_bytes")
        ws = torch.zeros(max(n, 16), dtype=torch.uint8, device=self.device)
        self._ws[key] = ws
        return ws

    # ------------------------------------------------------------ the six calls (+ append)
    def quantize_block(self, which, src, blk_begin, blk_end):
        src = _as_bits(src, self._dev)
        _check(_quantize_block(ctypes.byref(self.c), which, _dptr(src), src.shape[2], blk_begin, blk_end, _stream()),
               "quantize_block")

    def page_boxes(self, k_src, page_begin, page_end):
        k_src = _as_bits(k_src, self._dev)
        _check(_page_boxes(ctypes.byref(self.c), _dptr(k_src), k_src.shape[2], page_begin, page_end, _stream()),
               "page_boxes")

    def _take(self, levels):
        """Slots of the given levels from the pool, all or none (a full pool gives back
        what was taken and raises)."""
        got = []
        try:
            for L in levels:
                got.append((L, self.pool.alloc(L)))
        except GkvError:
            for L, off in got:
                self.pool.free(L, off)
            raise
        return np.array([off for _, off in got], dtype=np.int64)

    def demote(self, jobs, to_levels):
        """jobs: [(b, h, blk)], to_levels: levels; allocates the new slots, demotes,
        and frees the old ones (stream-ordered reuse)."""
        n = len(jobs)
        if n == 0:
            return
        J = np.ascontiguousarray(np.array(jobs, dtype=np.int32).reshape(n, 3))
        to = np.ascontiguousarray(np.array(to_levels, dtype=np.int8))
        old = [(int(self.level_host[b, h, i]), int(self.koff_host[b, h, i]), int(self.voff_host[b, h, i]))
               for b, h, i in J]
        # K and V slots of one block side by side, so that demoted one-centroid blocks
        # keep forming runs of back-to-back records
        kv = self._take([int(t) for t in np.repeat(to, 2)])
        nk, nv = kv[0::2].copy(), kv[1::2].copy()
        st = _demote(ctypes.byref(self.c), n, _np_ptr(J), _np_ptr(to), _np_ptr(nk), _np_ptr(nv), _stream())
        if st != 0:
            for t, a, bb in zip(to, nk, nv):
                self.pool.free(int(t), int(a))
                self.pool.free(int(t), int(bb))
            raise GkvError(st, "demote")
        for (b, h, i), (L, ko, vo), t, a, bb in zip(J, old, to, nk, nv):
            self.pool.free(L, ko)
            self.pool.free(L, vo)
            self.koff_host[b, h, i] = a
            self.voff_host[b, h, i] = bb

    def append(self, k_new, v_new, profile=None):
        """Append one token per (b,h) (k_new, v_new fp16 bits [B][Hkv][128]); then,
        with a ladder profile, demote every block whose level the profile lowers.
        Returns the demotions [(b, h, blk, old, new)]."""
        kd = _as_bits(k_new, self._dev)
        vd = _as_bits(v_new, self._dev)
        lens = self.lengths()
        opens = [b for b in range(self.B) if lens[b] >= 0 and lens[b] % P == 0]
        nk = nv = None
        if opens:
            # K and V slots of one block side by side (the order gkv_layers_step takes
            # them), for the units whose sequence opens a block
            kv = self._take([EXACT] * (2 * self.Hkv * len(opens)))
            nk = np.full(self.units, -1, np.int64)
            nv = np.full(self.units, -1, np.int64)
            i = 0
            for b in opens:
                for h in range(self.Hkv):
                    nk[b * self.Hkv + h], nv[b * self.Hkv + h] = kv[i], kv[i + 1]
                    i += 2
        st = _append(ctypes.byref(self.c), _dptr(kd), _dptr(vd), _np_ptr(nk) if nk is not None else None,
                     _np_ptr(nv) if nv is not None else None, _stream())
        if st != 0:
            if nk is not None:
                for off in kv:
                    self.pool.free(EXACT, int(off))
            raise GkvError(st, "append")
        for b in opens:  # the mirrors follow the library only once the call succeeded
            blk = int(lens[b]) // P
            self.koff_host[b, :, blk] = nk[b * self.Hkv:(b + 1) * self.Hkv]
            self.voff_host[b, :, blk] = nv[b * self.Hkv:(b + 1) * self.Hkv]
        moves = []
        if profile is not None:
            jobs = np.empty(3 * 64, dtype=np.int32)
            to = np.empty(64, dtype=np.int8)
            n = _ladder_crossings(ctypes.byref(self.c), PROFILES.get(profile, profile), self.T, _np_ptr(jobs),
                                  _np_ptr(to), 64)
            if n < 0:
                raise GkvError(n, "ladder_crossings")
            if n > 64:
                jobs = np.empty(3 * n, dtype=np.int32)
                to = np.empty(n, dtype=np.int8)
                n = _ladder_crossings(ctypes.byref(self.c), PROFILES.get(profile, profile), self.T, _np_ptr(jobs),
                                      _np_ptr(to), n)
            J = jobs[: 3 * n].reshape(n, 3)
            olds = [int(self.level_host[b, h, i]) for b, h, i in J]
            self.demote([tuple(x) for x in J], to[:n])
            moves = [(int(b), int(h), int(i), o, int(t)) for (b, h, i), o, t in zip(J, olds, to[:n])]
        return moves

    def quest_select(self, q, topk, out=None):
        q = _as_bits(q, self._dev)
        if out is None:
            out = torch.empty((self.B, self.Hkv, topk), dtype=torch.int32, device=self.device)
        ws = self.workspace(0)
        _check(_quest_select(_dptr(q), ctypes.byref(self.c), topk, _dptr(out), _dptr(ws), ws.numel(), _stream()),
               "quest_select")
        return out

    def graded_decode_attn(self, q, pages=None, out=None):
        q = _as_bits(q, self._dev)
        topk = int(pages.shape[-1]) if pages is not None else 0
        if out is None:
            out = torch.empty((self.B, self.Hq, D), dtype=torch.float32, device=self.device)
        ws = self.workspace(1, topk)
        _check(_attn(_dptr(q), ctypes.byref(self.c), _dptr(pages), topk, _dptr(out), _dptr(ws), ws.numel(),
                     _stream()), "graded_decode_attn")
        return out

    decode = graded_decode_attn

    def graded_decode_attn_noalloc(self, q, pages=None, out=None):
        """gkv_graded_decode_attn_noalloc: the same read with the library's own device
        scratch array as workspace (no workspace argument; out must be given by a
        caller that cannot allocate)."""
        q = _as_bits(q, self._dev)
        topk = int(pages.shape[-1]) if pages is not None else 0
        if out is None:
            out = torch.empty((self.B, self.Hq, D), dtype=torch.float32, device=self.device)
        _check(_attn_noalloc(_dptr(q), ctypes.byref(self.c), _dptr(pages), topk, _dptr(out), _stream()),
               "graded_decode_attn_noalloc")
        return out

    def decode_bound(self, q, out=None, bound=None):
        """Dense decode plus the attention error certificate per query head:
        returns (out [B][Hq][128] fp32, bound [B][Hq] fp32)."""
        q = _as_bits(q, self._dev)
        if out is None:
            out = torch.empty((self.B, self.Hq, D), dtype=torch.float32, device=self.device)
        if bound is None:
            bound = torch.empty((self.B, self.Hq), dtype=torch.float32, device=self.device)
        ws = self.workspace(1, 0)
        _check(_attn_bound(_dptr(q), ctypes.byref(self.c), _dptr(out), _dptr(bound), _dptr(ws), ws.numel(),
                           _stream()), "graded_decode_attn_bound")
        return out, bound

    # the three stages of graded_decode_attn (same result when called in order)
    def attn_plan(self, pages=None):
        topk = int(pages.shape[-1]) if pages is not None else 0
        ws = self.workspace(1, topk)
        _check(_attn_plan(ctypes.byref(self.c), _dptr(pages), topk, _dptr(ws), ws.numel(), _stream()), "attn_plan")

    def attn_partials(self, q, pages=None):
        q = _as_bits(q, self._dev)
        topk = int(pages.shape[-1]) if pages is not None else 0
        ws = self.workspace(1, topk)
        _check(_attn_partials(_dptr(q), ctypes.byref(self.c), _dptr(pages), topk, _dptr(ws), ws.numel(), _stream()),
               "attn_partials")

    def attn_merge(self, out, pages=None):
        topk = int(pages.shape[-1]) if pages is not None else 0
        ws = self.workspace(1, topk)
        _check(_attn_merge(ctypes.byref(self.c), _dptr(pages), topk, _dptr(out), _dptr(ws), ws.numel(), _stream()),
               "attn_merge")

    def rd_residual_select(self, k_src, v_src, mass, nkeep):
        kd = _as_bits(k_src, self._dev)
        vd = _as_bits(v_src, self._dev)
        if isinstance(mass, np.ndarray):
            mass = torch.from_numpy(np.ascontiguousarray(mass, dtype=np.float32))
        md = mass.to(self.device, torch.float32).contiguous()
        ws = self.workspace(2)
        _check(_rd(ctypes.byref(self.c), _dptr(kd), _dptr(vd), _dptr(md), nkeep, _dptr(ws), ws.numel(), _stream()),
               "rd_residual_select")

    # ------------------------------------------------------------ inspection
    def pool_bits(self):
        """Bits of the arena slots in use (the K and V records of every block), as the
        slab pool counts them."""
        return sum(self.pool.used(L) * block_bytes(L) for L in LEVELS) * 8

    def account(self, pages=None):
        r = Rates()
        if pages is not None:
            ph = np.ascontiguousarray(pages.cpu().numpy() if torch.is_tensor(pages) else pages, dtype=np.int32)
            ri = None
            if int(self.c.nres):  # a Compressed-Quest read also reads the residual rows in its read set
                ri = np.ascontiguousarray(self.res_idx.cpu().numpy(), dtype=np.int32)
            _check(_account(ctypes.byref(self.c), _np_ptr(ph), ph.shape[-1], _np_ptr(ri) if ri is not None else None,
                            ctypes.byref(r)), "account")
        else:
            _check(_account(ctypes.byref(self.c), None, 0, None, ctypes.byref(r)), "account")
        return dict(resident_bits=r.resident_bits, read_bits=r.read_bits, values=r.values,
                    resident_bpv=r.resident_bits / r.values, read_bpv=r.read_bits / r.values)

    def record_bytes(self, b, h, blk, tensor):
        L = int(self.level_host[b, h, blk])
        off = int((self.koff_host if tensor == KEYS else self.voff_host)[b, h, blk])
        n = block_bytes(L)
        return L, self.arena[off:off + n].cpu().numpy().tobytes()

    def record(self, b, h, blk, tensor):
        L, raw = self.record_bytes(b, h, blk, tensor)
        d = decode_record(L, VALUES_PER_TOKEN if tensor == VALUES and self.v_per_token else tensor, raw)
        d["level"] = L
        return d

    def boxes_host(self, b, h, npages):
        """Boxes of (b,h) as (kmin bits [npages][D], kmax bits [npages][D])."""
        raw = self.boxes[b, h].cpu().numpy().view(np.uint16)
        g = raw.reshape(-1, D, 64, 2)
        kmin = g[..., 0].transpose(0, 2, 1).reshape(-1, D)[:npages]
        kmax = g[..., 1].transpose(0, 2, 1).reshape(-1, D)[:npages]
        return kmin, kmax


class LayerCaches:
    """The graded caches of L layers stepped together (gkv_layers_step): one call per
    decode step appends every layer's token and demotes what the ladder lowers."""

    def __init__(self, caches, profile):
        self.caches = list(caches)
        self.profile = PROFILES.get(profile, profile)
        L = len(self.caches)
        ptr = lambda xs: (ctypes.c_void_p * L)(*xs)
        self._c = ptr([ctypes.addressof(c.c) for c in self.caches])
        self._p = ptr([c.pool.h for c in self.caches])
        self._ko = ptr([c.koff_host.ctypes.data for c in self.caches])
        self._vo = ptr([c.voff_host.ctypes.data for c in self.caches])

    def step(self, k_new, v_new):
        """k_new, v_new: [L][B][Hkv][128] fp16 bits (device tensors or numpy).
        Returns the number of blocks demoted over all layers."""
        k_new = _fp16_dev(k_new, self.caches[0].device)
        v_new = _fp16_dev(v_new, self.caches[0].device)
        n = int(_layers_step(self._c, self._p, self._ko, self._vo, len(self.caches), self.profile, _dptr(k_new),
                             _dptr(v_new), _stream()))
        if n < 0:
            raise GkvError(n, "layers_step")
        return n
