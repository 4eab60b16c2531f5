"""Builds oracle-side state from the seeded workload (tests only).

The workload module draws raw values; this helper turns them into NumPy
arrays and runs the oracle's own append to fill a poisoned host pool that
holds only the selected sequences' pages (a compact copy: physical page p of
the real pool is page page_map[p] here).  No value here comes from the GPU
path: raw values are regenerated from their seeds on `device` (the same
generator the GPU harness used) and copied to the host.
"""
from __future__ import annotations

import numpy as np

import workload
from oracle import formats, paged

POISON = {"f32": np.float32(np.nan), "bf16": np.uint16(0x7FC0), "fp8": np.uint8(0x7F)}


def to_numpy(t):
    """torch tensor -> numpy: float32 stays float32, bfloat16 becomes its
    uint16 bit patterns, uint8 stays uint8."""
    import torch

    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype in (torch.float32, torch.uint8, torch.int32):
        return t.numpy()
    raise TypeError(t.dtype)


def q_to_f64(q_np, q_dtype):
    if q_dtype == "bf16":
        return formats.bf16_bits_to_f64(q_np)
    return np.asarray(q_np, dtype=np.float32).astype(np.float64)


class OracleState:
    """Host pools for the selected sequences of a workload, filled the way a
    server would have filled them: each sequence's resident tokens appended
    at set-up (by the oracle's append)."""

    def __init__(self, wl: workload.Workload, sids=None, device="cpu"):
        cfg = wl.cfg
        self.wl, self.cfg, self.device = wl, cfg, device
        self.sids = list(range(len(wl.seqs))) if sids is None else sorted(set(int(s) for s in sids))
        self.in_dtype = workload.kv_dtype_in(cfg)
        self.pages = np.concatenate([wl.seqs[s].pages for s in self.sids]).astype(np.int64)
        self.page_map = np.full(wl.num_pages, -1, np.int64)
        self.page_map[self.pages] = np.arange(len(self.pages))
        self.raw = {sid: workload.sequence_kv(wl, sid, device) for sid in self.sids}
        shape = (len(self.pages), cfg.num_kv_heads, cfg.page_size, cfg.head_dim)
        dt = paged.POOL_NP_DTYPE[cfg.kv_dtype]
        self.pool_k = np.full(shape, POISON[cfg.kv_dtype], dtype=dt)
        self.pool_v = np.full(shape, POISON[cfg.kv_dtype], dtype=dt)
        self.k_scale = self.v_scale = None
        if cfg.kv_dtype == "fp8":
            self.k_scale = np.full(shape[:2], np.nan, np.float32)
            self.v_scale = np.full(shape[:2], np.nan, np.float32)
            for sid in self.sids:
                ks, vs = workload.page_scales(wl, sid, *self.raw[sid])
                idx = self.page_map[wl.seqs[sid].pages]
                self.k_scale[idx] = ks.cpu().numpy()
                self.v_scale[idx] = vs.cpu().numpy()
        for sid in self.sids:
            s = wl.seqs[sid]
            if s.resident == 0:
                continue
            k, v = self.raw[sid]
            self._append(self.page_map[s.pages][None, :], [0], [s.resident],
                         to_numpy(k[:s.resident]), to_numpy(v[:s.resident]))

    def _append(self, bt, ctx, n, k_np, v_np):
        kw = dict(page_size=self.cfg.page_size, kv_dtype=self.cfg.kv_dtype, in_dtype=self.in_dtype)
        paged.append(self.pool_k, bt, ctx, n, k_np, scale=self.k_scale, **kw)
        paged.append(self.pool_v, bt, ctx, n, v_np, scale=self.v_scale, **kw)

    def rows_of(self, batch, rows=None):
        idx = [b for b in range(batch.num_seqs) if int(batch.seq_ids[b]) in self.sids]
        if rows is not None:
            idx = [b for b in idx if b in set(rows)]
        return idx

    def table(self, batch, rows):
        """Block-table rows remapped to the compact pool (unused entries -> 0)."""
        bt = self.page_map[batch.block_table[rows]]
        return np.where(bt < 0, 0, bt)

    def _new_rows(self, batch, rows, decode):
        ks, vs = [], []
        for b in rows:
            k, v = self.raw[int(batch.seq_ids[b])]
            c = int(batch.ctx_lens[b])
            n = 1 if decode else int(batch.q_lens[b])
            ks.append(to_numpy(k[c:c + n]))
            vs.append(to_numpy(v[c:c + n]))
        return np.concatenate(ks), np.concatenate(vs)

    def append_prefill(self, rows=None):
        pf = self.wl.prefill
        rows = self.rows_of(pf, rows)
        k, v = self._new_rows(pf, rows, False)
        self._append(self.table(pf, rows), pf.ctx_lens[rows], pf.q_lens[rows], k, v)

    def append_decode(self, rows=None):
        dc = self.wl.decode
        rows = self.rows_of(dc, rows)
        k, v = self._new_rows(dc, rows, True)
        self._append(self.table(dc, rows), dc.ctx_lens[rows], dc.q_lens[rows], k, v)

    def kwargs(self):
        return dict(page_size=self.cfg.page_size, kv_dtype=self.cfg.kv_dtype,
                    softmax_scale=self.cfg.softmax_scale, k_scale=self.k_scale, v_scale=self.v_scale)

    def prefill(self, q_packed_np, rows, window=0, row_subsets=None):
        """Oracle prefill output for batch rows `rows`: {b: [len(t), H_q, D]}.
        q_packed_np holds the whole batch's packed queries (host copy of the
        generator's values)."""
        pf = self.wl.prefill
        cu = pf.cu_q_lens
        out = {}
        q64 = q_to_f64(q_packed_np, self.cfg.q_dtype)
        for b in rows:
            t = np.arange(int(pf.q_lens[b])) if row_subsets is None else np.asarray(row_subsets[b])
            if t.size == 0:
                out[b] = np.zeros((0,) + q64.shape[1:])
                continue
            qb = q64[cu[b]:cu[b + 1]]
            r = paged.prefix_prefill(qb, self.pool_k, self.pool_v, self.table(pf, [b]),
                                     pf.ctx_lens[[b]], pf.q_lens[[b]], window=window,
                                     rows={0: t}, **self.kwargs())
            out[b] = r[0]
        return out

    def decode(self, q_np, rows, window=0):
        dc = self.wl.decode
        q64 = q_to_f64(q_np, self.cfg.q_dtype)
        out = {}
        for b in rows:
            r = paged.paged_decode(q64[b:b + 1], self.pool_k, self.pool_v, self.table(dc, [b]),
                                   self.wl.decode_ctx[[b]], window=window, **self.kwargs())
            out[b] = r[0]
        return out
