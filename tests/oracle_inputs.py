"""Builds oracle-side state from the seeded workload (tests only).

The workload module draws raw values; this helper turns them into NumPy
arrays and runs the oracle's own append to fill a poisoned host pool.  No
value here comes from the GPU path.
"""
from __future__ import annotations

import numpy as np

import workload
from oracle import paged

POISON = {"f32": np.float32(np.nan), "bf16": np.uint16(0x7FC0), "fp8": np.uint8(0x7F)}


def to_numpy(t):
    """torch tensor -> numpy: float32 stays float32, bfloat16 becomes its
    uint16 bit patterns."""
    import torch

    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype == torch.float32:
        return t.numpy()
    if t.dtype == torch.uint8:
        return t.numpy()
    raise TypeError(t.dtype)


def q_to_f64(q_np, q_dtype):
    from oracle import formats

    if q_dtype == "bf16":
        return formats.bf16_bits_to_f64(q_np)
    return np.asarray(q_np, dtype=np.float32).astype(np.float64)


class OracleState:
    """Host pools for a workload, filled the way a server would have filled
    them: every sequence's resident tokens appended at set-up."""

    def __init__(self, wl: workload.Workload, sids=None, device="cpu", raw=None):
        cfg = wl.cfg
        self.wl = wl
        self.cfg = cfg
        self.sids = list(range(len(wl.seqs))) if sids is None else list(sids)
        self.in_dtype = workload.kv_dtype_in(cfg)
        self.raw = {}
        for sid in self.sids:
            if raw is not None and sid in raw:
                k, v = raw[sid]
            else:
                k, v = workload.sequence_kv(wl, sid, device)
            self.raw[sid] = (k, v)
        shape = (wl.num_pages, cfg.num_kv_heads, cfg.page_size, cfg.head_dim)
        dt = paged.POOL_NP_DTYPE[cfg.kv_dtype]
        self.pool_k = np.full(shape, POISON[cfg.kv_dtype], dtype=dt)
        self.pool_v = np.full(shape, POISON[cfg.kv_dtype], dtype=dt)
        self.k_scale = self.v_scale = None
        if cfg.kv_dtype == "fp8":
            self.k_scale = np.full((wl.num_pages, cfg.num_kv_heads), np.nan, np.float32)
            self.v_scale = np.full((wl.num_pages, cfg.num_kv_heads), np.nan, np.float32)
            for sid in self.sids:
                ks, vs = workload.page_scales(wl, sid, *self.raw[sid])
                pages = wl.seqs[sid].pages
                self.k_scale[pages] = ks.cpu().numpy()
                self.v_scale[pages] = vs.cpu().numpy()
        # set-up: resident tokens of every sequence
        for sid in self.sids:
            s = wl.seqs[sid]
            if s.resident == 0:
                continue
            k, v = self.raw[sid]
            self._append_rows(s.pages[None, :], [0], [s.resident],
                              to_numpy(k[:s.resident]), to_numpy(v[:s.resident]))

    def _append_rows(self, bt, ctx, n, k_np, v_np):
        kw = dict(page_size=self.cfg.page_size, kv_dtype=self.cfg.kv_dtype, in_dtype=self.in_dtype)
        paged.append(self.pool_k, bt, ctx, n, k_np, scale=self.k_scale, **kw)
        paged.append(self.pool_v, bt, ctx, n, v_np, scale=self.v_scale, **kw)

    # ---- step inputs ---------------------------------------------------
    def prefill_new_kv(self, rows=None):
        """Packed raw new-turn K, V of the prefill batch (rows: subset of b)."""
        import torch

        b_all = range(self.wl.prefill.num_seqs) if rows is None else rows
        ks, vs = [], []
        for b in b_all:
            sid = int(self.wl.prefill.seq_ids[b])
            P = int(self.wl.prefill.ctx_lens[b])
            n = int(self.wl.prefill.q_lens[b])
            k, v = self.raw[sid]
            ks.append(k[P:P + n])
            vs.append(v[P:P + n])
        return torch.cat(ks), torch.cat(vs)

    def decode_new_kv(self, rows=None):
        import torch

        b_all = range(self.wl.decode.num_seqs) if rows is None else rows
        ks, vs = [], []
        for b in b_all:
            sid = int(self.wl.decode.seq_ids[b])
            c = int(self.wl.decode.ctx_lens[b])  # c_b - 1: position of the decode token
            k, v = self.raw[sid]
            ks.append(k[c:c + 1])
            vs.append(v[c:c + 1])
        return torch.cat(ks), torch.cat(vs)

    def append_prefill(self, rows=None):
        pf = self.wl.prefill
        idx = list(range(pf.num_seqs)) if rows is None else list(rows)
        k, v = self.prefill_new_kv(idx)
        self._append_rows(pf.block_table[idx], pf.ctx_lens[idx], pf.q_lens[idx], to_numpy(k), to_numpy(v))

    def append_decode(self, rows=None):
        dc = self.wl.decode
        idx = list(range(dc.num_seqs)) if rows is None else list(rows)
        k, v = self.decode_new_kv(idx)
        self._append_rows(dc.block_table[idx], dc.ctx_lens[idx], dc.q_lens[idx], to_numpy(k), to_numpy(v))

    def kwargs(self):
        return dict(page_size=self.cfg.page_size, kv_dtype=self.cfg.kv_dtype,
                    softmax_scale=self.cfg.softmax_scale, k_scale=self.k_scale, v_scale=self.v_scale)
