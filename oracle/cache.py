"""A whole graded cache for one (sequence, KV head) unit, built from the oracle's
per-block functions, and the three flows of the hot path on it:

* dense graded decode (Method, sections 3.2 and 3.7),
* graded decode with the exact residual (section 3.4),
* Compressed-Quest decode (section 3.5),

plus the monotone per-step append-and-demote update (section 3.2).
"""
import numpy as np

from . import fp16, quant, quest, attention, residual, certificate
from .ladder import EXACT, ORDER, ladder

P = 64


class UnitCache:
    def __init__(self, k_bits, v_bits, levels, v_per_token=False):
        """k_bits, v_bits: uint16 [T][D] exact fp16; levels per block (oldest first);
        v_per_token groups the values' scalar levels per token (section 3.2 text)."""
        self.T = k_bits.shape[0]
        self.D = k_bits.shape[1]
        self.levels = np.array(levels, dtype=np.int8)
        self.v_per_token = bool(v_per_token)
        self.k_recs = []
        self.v_recs = []
        # decode-time certificate numbers per block (see certificate.decode_bound)
        self.kerr, self.verr, self.vmax = [], [], []
        for b, lv in enumerate(self.levels):
            rows = slice(b * P, min((b + 1) * P, self.T))
            kb = np.zeros((P, self.D), dtype=np.uint16)
            vb = np.zeros((P, self.D), dtype=np.uint16)
            kb[: rows.stop - rows.start] = k_bits[rows]
            vb[: rows.stop - rows.start] = v_bits[rows]
            if rows.stop - rows.start < P and lv != EXACT:
                raise ValueError("only an exact block may be partial")
            self.k_recs.append(quant.encode_fp16(lv, kb))
            self.v_recs.append(quant.encode_fp16(lv, vb, v_per_token))
            ke, _ = certificate.block_numbers(fp16.to_f64(kb), quant.decode(self.k_recs[-1]))
            ve, vn = certificate.block_numbers(fp16.to_f64(vb), quant.decode(self.v_recs[-1]))
            self.kerr.append(ke)
            self.verr.append(ve)
            self.vmax.append(vn)
        self.res_idx = np.zeros(0, dtype=np.int32)
        self.res_k = None
        self.res_v = None

    # ------------------------------------------------------------ reconstruction
    def khat_vhat(self):
        kh = np.concatenate([quant.decode(r) for r in self.k_recs])[: self.T]
        vh = np.concatenate([quant.decode(r) for r in self.v_recs])[: self.T]
        if len(self.res_idx):
            kh = kh.copy()
            vh = vh.copy()
            kh[self.res_idx] = fp16.to_f64(self.res_k)
            vh[self.res_idx] = fp16.to_f64(self.res_v)
        return kh, vh

    # ------------------------------------------------------------ residual
    def select_residual(self, k_bits, v_bits, mass, n):
        """Section 3.4: score every token against its graded value, keep top n exact."""
        vh = np.concatenate([quant.decode(r) for r in self.v_recs])[: self.T]
        s = residual.scores(fp16.to_f64(v_bits), vh, mass)
        idx = residual.select(s, n)
        self.res_idx = idx
        self.res_k = np.asarray(k_bits)[idx].copy()
        self.res_v = np.asarray(v_bits)[idx].copy()
        return idx, s

    # ------------------------------------------------------------ decode
    def decode_dense(self, q_bits_group):
        kh, vh = self.khat_vhat()
        return attention.unit_decode(q_bits_group, kh, vh)

    def certificate(self, q_bits_group):
        """Decode-time certificate of a dense read, per query head of the group."""
        kh, _ = self.khat_vhat()
        kerr = np.repeat(np.asarray(self.kerr), P)[: self.T]
        verr = np.repeat(np.asarray(self.verr), P)[: self.T]
        if len(self.res_idx):
            kerr = kerr.copy()
            verr = verr.copy()
            kerr[self.res_idx] = 0.0
            verr[self.res_idx] = 0.0
        q = fp16.to_f64(q_bits_group)
        vmax = max(self.vmax)
        return np.array([certificate.decode_bound(q[g], kh, kerr, verr, vmax) for g in range(q.shape[0])])

    def decode_quest(self, q_bits_group, pages, page=quest.PAGE):
        kh, vh = self.khat_vhat()
        idx = quest.read_tokens(pages, self.T, page)
        return attention.unit_decode(q_bits_group, kh, vh, idx)

    # ------------------------------------------------------------ append / demote
    def append(self, k_row_bits, v_row_bits, profile):
        """Append one token (section 3.2: incremental append, monotone demotion).

        The new token lands in the newest block (a new exact block when T is a
        multiple of P); then the ladder is re-evaluated at the new length and
        every block whose level drops is re-encoded from its current record.
        Returns the list of (block, old, new) demotions."""
        t = self.T
        if t % P == 0:
            z = np.zeros((P, self.D), dtype=np.uint16)
            self.k_recs.append(quant.Record(EXACT, exact=z.copy()))
            self.v_recs.append(quant.Record(EXACT, exact=z.copy(), per_token=self.v_per_token))
            self.levels = np.append(self.levels, np.int8(EXACT))
            self.kerr.append(0.0)
            self.verr.append(0.0)
            self.vmax.append(0.0)
        b = t // P
        assert self.k_recs[b].level == EXACT
        self.k_recs[b].exact[t % P] = k_row_bits
        self.v_recs[b].exact[t % P] = v_row_bits
        self.vmax[b] = max(self.vmax[b], float(np.sqrt((fp16.to_f64(np.asarray(v_row_bits)) ** 2).sum())))
        self.T = t + 1
        new_lv = ladder(profile, self.T)
        moves = []
        for i, (old, new) in enumerate(zip(self.levels, new_lv)):
            if old != new:
                if ORDER[int(new)] > ORDER[int(old)]:
                    raise quant.NotMonotone(f"block {i}: {old} -> {new}")
                kold, vold = self.k_recs[i], self.v_recs[i]
                self.k_recs[i] = quant.demote(kold, new)
                self.v_recs[i] = quant.demote(vold, new)
                self.kerr[i] += certificate.demote_increment(quant.decode(kold), quant.decode(self.k_recs[i]))
                self.verr[i] += certificate.demote_increment(quant.decode(vold), quant.decode(self.v_recs[i]))
                moves.append((i, int(old), int(new)))
        self.levels = np.array(new_lv, dtype=np.int8)
        return moves
