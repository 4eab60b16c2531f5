"""Device-side set-up and stepping of a synthetic workload through libckv.

A DeviceWorkload owns one paged pool (poisoned: NaN patterns in every slot
that no sequence writes), uploads the block tables and lengths of a
prefix-reuse prefill batch and a decode batch, and fills the pool the way a
server would have: each sequence's resident tokens are appended with
kv_append at set-up, before any step.  A step is then

    kv_append(new turn)  ->  prefix_prefill_attn  ->
    kv_append(decode token)  ->  paged_decode_attn

All arithmetic happens in libckv's kernels; this module only allocates,
uploads and calls.
"""
from __future__ import annotations

import numpy as np
import torch

import workload

from . import ckv

POISON_BYTES = {"f32": (torch.float32, float("nan")), "bf16": (torch.bfloat16, float("nan")),
                "fp8": (torch.uint8, 0x7F)}
_TORCH = {"f32": torch.float32, "bf16": torch.bfloat16}


def _i32(x, device):
    return torch.as_tensor(np.ascontiguousarray(x, dtype=np.int32), device=device)


class DeviceWorkload:
    def __init__(self, wl: workload.Workload, device="cuda", window: int = 0, keep_raw=()):
        cfg = wl.cfg
        self.wl, self.cfg, self.device, self.window = wl, cfg, device, window
        shape = (wl.num_pages, cfg.num_kv_heads, cfg.page_size, cfg.head_dim)
        dt, fill = POISON_BYTES[cfg.kv_dtype]
        k = torch.full(shape, fill, dtype=dt, device=device)
        v = torch.full(shape, fill, dtype=dt, device=device)
        ks = vs = None
        if cfg.kv_dtype == "fp8":
            ks = torch.full(shape[:2], float("nan"), dtype=torch.float32, device=device)
            vs = torch.full(shape[:2], float("nan"), dtype=torch.float32, device=device)
        self.pool = ckv.Pool(k, v, ks, vs)
        pf, dc = wl.prefill, wl.decode
        # host-side contract check before anything is launched
        for batch, decode in ((pf, False), (dc, True)):
            if batch.num_seqs:
                ctx = batch.ctx_lens + (1 if decode else 0)
                ckv.validate_batch(wl.num_pages, cfg.page_size, batch.block_table, ctx,
                                   None if decode else batch.cu_q_lens, batch.max_q_len,
                                   int(ctx.max()), decode)
        self.prefill = ckv.Batch(_i32(pf.block_table, device), _i32(pf.ctx_lens, device),
                                 _i32(pf.cu_q_lens, device), pf.total_q, pf.max_q_len, pf.max_ctx_len)
        # decode token append: ctx = c_b - 1 rows of 1
        self.decode_append = ckv.Batch(_i32(dc.block_table, device), _i32(dc.ctx_lens, device),
                                       _i32(dc.cu_q_lens, device), dc.total_q, dc.max_q_len,
                                       dc.max_ctx_len)
        dctx = wl.decode_ctx
        self.decode = ckv.Batch(_i32(dc.block_table, device), _i32(dctx, device), None, dc.num_seqs,
                                1, int(dctx.max()) if dc.num_seqs else 0)
        self.raw = {}
        self._setup(set(keep_raw))
        # step inputs
        qdt = _TORCH[cfg.q_dtype]
        self.q_prefill = (workload.concat_rows(pf, lambda b: workload.prefill_q(wl, b, device))
                          if pf.num_seqs else torch.empty((0, cfg.num_q_heads, cfg.head_dim), dtype=qdt,
                                                          device=device))
        self.q_decode = (workload.concat_rows(dc, lambda b: workload.decode_q(wl, b, device))
                         if dc.num_seqs else None)
        self.out_prefill = torch.empty_like(self.q_prefill)
        self.out_decode = torch.empty_like(self.q_decode) if self.q_decode is not None else None
        nws = ckv.decode_workspace_bytes(self.pool, self.decode, cfg.num_q_heads) if dc.num_seqs else 0
        self.ws_decode = torch.empty(max(nws, 1), dtype=torch.uint8, device=device)
        torch.cuda.synchronize()

    def _setup(self, keep_raw):
        wl, cfg, dev = self.wl, self.cfg, self.device
        pf, dc = wl.prefill, wl.decode
        new_k = [None] * pf.num_seqs
        new_v = [None] * pf.num_seqs
        dec_k = [None] * dc.num_seqs
        dec_v = [None] * dc.num_seqs
        pf_rows = {int(s): b for b, s in enumerate(pf.seq_ids)}
        dc_rows = {int(s): b for b, s in enumerate(dc.seq_ids)}
        for sid, s in enumerate(wl.seqs):
            k, v = workload.sequence_kv(wl, sid, dev)
            if sid in keep_raw:
                self.raw[sid] = (k, v)
            if cfg.kv_dtype == "fp8":
                ksc, vsc = workload.page_scales(wl, sid, k, v)
                pages = torch.as_tensor(s.pages.astype(np.int64), device=dev)
                self.pool.k_scale[pages] = ksc
                self.pool.v_scale[pages] = vsc
            if s.resident:
                one = ckv.Batch(_i32(s.pages[None, :], dev), _i32([0], dev), _i32([0, s.resident], dev),
                                s.resident, s.resident, 0)
                ckv.kv_append(self.pool, one, k[:s.resident].contiguous(), v[:s.resident].contiguous())
            if sid in pf_rows:
                b = pf_rows[sid]
                P, n = int(pf.ctx_lens[b]), int(pf.q_lens[b])
                new_k[b], new_v[b] = k[P:P + n].clone(), v[P:P + n].clone()
            if sid in dc_rows:
                b = dc_rows[sid]
                c1 = int(dc.ctx_lens[b])
                dec_k[b], dec_v[b] = k[c1:c1 + 1].clone(), v[c1:c1 + 1].clone()
            del k, v
        shape_empty = (0, cfg.num_kv_heads, cfg.head_dim)
        kdt = _TORCH[workload.kv_dtype_in(cfg)]
        self.k_new = torch.cat(new_k) if new_k else torch.empty(shape_empty, dtype=kdt, device=dev)
        self.v_new = torch.cat(new_v) if new_v else torch.empty(shape_empty, dtype=kdt, device=dev)
        self.k_dec = torch.cat(dec_k) if dec_k else torch.empty(shape_empty, dtype=kdt, device=dev)
        self.v_dec = torch.cat(dec_v) if dec_v else torch.empty(shape_empty, dtype=kdt, device=dev)

    # ---- the hot path ----------------------------------------------------
    def append_prefill(self):
        ckv.kv_append(self.pool, self.prefill, self.k_new, self.v_new)

    def run_prefill(self, window=None):
        w = self.window if window is None else window
        return ckv.prefix_prefill_attn(self.pool, self.prefill, self.q_prefill, self.cfg.softmax_scale,
                                       w, out=self.out_prefill)

    def append_decode(self):
        ckv.kv_append(self.pool, self.decode_append, self.k_dec, self.v_dec)

    def run_decode(self, window=None, kv_split_len=0, out=None, workspace=None):
        w = self.window if window is None else window
        if kv_split_len:
            nws = ckv.decode_workspace_bytes(self.pool, self.decode, self.cfg.num_q_heads, kv_split_len)
            workspace = torch.empty(max(nws, 1), dtype=torch.uint8, device=self.device)
        return ckv.paged_decode_attn(self.pool, self.decode, self.q_decode, self.cfg.softmax_scale, w,
                                     kv_split_len, out=self.out_decode if out is None else out,
                                     workspace=self.ws_decode if workspace is None else workspace)

    def step(self):
        if self.wl.prefill.num_seqs:
            self.append_prefill()
            self.run_prefill()
        if self.wl.decode.num_seqs:
            self.append_decode()
            self.run_decode()
