"""Offline profile on one MI355X (one attention layer): host-link page
throughput and prefill time against context length.

Continuum's cost model needs the time to rebuild a request's KV cache when
its TTL has expired (Prefill-Reload(r), Sec. 4.1): a reload from host memory
when CPU offloading is on, else a new prefill.  The paper gets both from a
short offline profile per (hardware, model) (Sec. 5.2, "Offline Profile"):
(1) the GPU-CPU throughput of offloading, and (2) prefill for a ladder of
context sizes up to the maximum context, then a quadratic fit of time
against context length.  (1) here times kv_pages_offload / kv_pages_reload
on whole pages of the model's pool layout, beside a plain pinned-memory
copy of the same bytes (the link's practical rate).  For (2), serving engines prefill in
chunks (the paper's vLLM baseline uses 2048-token chunks, Sec. 6.1), so the
profile here measures both

  full      one prefill of L tokens (retained prefix P = 0, n = L), and
  chunked   the same L tokens as consecutive chunks of C tokens, each a
            prefix-reuse prefill over the chunks before it (P = kC, n = C),

with the library's own prefix_prefill_attn, and fits
t(L) = a L^2 + b L + c to each series.  Only the attention layer is timed:
the model's linear layers (projections, MLP) add a term linear in L that
this library does not run.

    python -m paper_2511_02230_amd.offline_profile --config llama3.1-70b \
        --max-len 65536 --chunks 256 512 1024 2048 4096
    python -m paper_2511_02230_amd.offline_profile --config llama3.1-70b --transfer

One sequence of max-len tokens is appended to the pool once; every timed
call is a view of it (block table, ctx_lens = P, cu_q_lens = [0, n]).
"""
from __future__ import annotations

import argparse
import json
import sys
from typing import Dict, List, Sequence, Tuple

import numpy as np


def length_ladder(max_len: int, first: int = 1000) -> List[int]:
    """first, 2 first, 4 first, ... below max_len, then max_len (the
    paper's {1000, 2000, 4000, ..., max_context_length})."""
    if max_len < 1:
        raise ValueError("max_len must be positive")
    out, x = [], first
    while x < max_len:
        out.append(x)
        x *= 2
    out.append(max_len)
    return out


def chunk_plan(length: int, chunk: int) -> List[Tuple[int, int]]:
    """(P, n) of every chunk when `length` tokens are prefilled `chunk` at a
    time: P = k chunk, n = min(chunk, length - P)."""
    if length < 0 or chunk < 1:
        raise ValueError("length >= 0 and chunk >= 1")
    return [(p, min(chunk, length - p)) for p in range(0, length, chunk)]


def fit_quadratic(lengths: Sequence[float], times: Sequence[float]) -> Dict[str, float]:
    """Least-squares t = a L^2 + b L + c; also R^2 of the fit."""
    x = np.asarray(lengths, dtype=np.float64)
    y = np.asarray(times, dtype=np.float64)
    if x.size < 3:
        raise ValueError("a quadratic needs at least three points")
    A = np.stack([x * x, x, np.ones_like(x)], axis=1)
    (a, b, c), *_ = np.linalg.lstsq(A, y, rcond=None)
    resid = y - A @ np.array([a, b, c])
    ss_tot = float(((y - y.mean()) ** 2).sum())
    r2 = 1.0 - float((resid ** 2).sum()) / ss_tot if ss_tot > 0 else 1.0
    return {"a": float(a), "b": float(b), "c": float(c), "r2": r2}


def fit_linear(sizes: Sequence[float], times: Sequence[float]) -> Dict[str, float]:
    """Least-squares t = t0 + x / bw for transfer sizes x (bytes) and times t
    (ms): bw in GB/s, t0 in microseconds, and R^2 of the fit."""
    x = np.asarray(sizes, dtype=np.float64)
    y = np.asarray(times, dtype=np.float64)
    if x.size < 2:
        raise ValueError("a line needs at least two points")
    A = np.stack([x, np.ones_like(x)], axis=1)
    (slope, t0), *_ = np.linalg.lstsq(A, y, rcond=None)
    resid = y - A @ np.array([slope, t0])
    ss_tot = float(((y - y.mean()) ** 2).sum())
    r2 = 1.0 - float((resid ** 2).sum()) / ss_tot if ss_tot > 0 else 1.0
    return {"gbps": float(1e-6 / slope) if slope > 0 else float("inf"), "t0_us": float(t0 * 1e3),
            "r2": r2}


def attention_flops(P: int, n: int, num_q_heads: int, head_dim: int, window: int = 0) -> float:
    """4 D H_q per visible (row, key) pair, rows at positions P .. P+n-1."""
    i = P + np.arange(n, dtype=np.int64)
    cnt = i + 1 if window <= 0 else np.minimum(i + 1, window)
    return 4.0 * head_dim * num_q_heads * float(cnt.sum())


class PrefillTimer:
    """One resident sequence of max_len tokens; times prefix_prefill_attn on
    (P, n) views of it."""

    def __init__(self, cfg, max_len: int, device="cuda", window: int = 0):
        import torch

        import workload
        from . import ckv
        from .harness import DeviceWorkload

        self.torch, self.ckv, self.cfg, self.window = torch, ckv, cfg, window
        self.wl = workload.make_workload(cfg, prefill=[(0, max_len)], decode=[])
        self.dw = DeviceWorkload(self.wl, device, window=window)
        self.dw.append_prefill()  # all max_len tokens resident
        torch.cuda.synchronize()
        self.bt = self.dw.prefill.block_table
        self.q = self.dw.q_prefill
        self.out = torch.empty_like(self.q)
        self.max_len = max_len

    def _batch(self, P: int, n: int):
        torch = self.torch
        dev = self.q.device
        return self.ckv.Batch(self.bt, torch.tensor([P], dtype=torch.int32, device=dev),
                              torch.tensor([0, n], dtype=torch.int32, device=dev), n, n, P)

    def time(self, pairs: Sequence[Tuple[int, int]], reps: int = 3, warmup: int = 1) -> float:
        """Milliseconds for the calls (P, n) back to back (median over reps)."""
        torch = self.torch
        batches = [(self._batch(P, n), n) for P, n in pairs if n > 0]
        for P, n in pairs:
            if P + n > self.max_len:
                raise ValueError("view beyond the resident sequence")
        for _ in range(warmup):
            for bt, n in batches:
                self.ckv.prefix_prefill_attn(self.dw.pool, bt, self.q[:n], self.cfg.softmax_scale,
                                             self.window, out=self.out[:n])
        times = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for bt, n in batches:
                self.ckv.prefix_prefill_attn(self.dw.pool, bt, self.q[:n], self.cfg.softmax_scale,
                                             self.window, out=self.out[:n])
            e1.record()
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1))
        return float(np.median(times))


class TransferTimer:
    """Pool of the model's page layout, pinned host pages and staging for up
    to max_pages pages; times offload and reload of n pages named by a
    shuffled page list, and a plain pinned copy of the same bytes."""

    def __init__(self, cfg, max_pages: int, pool_pages: int = 0, device="cuda", seed: int = 0):
        import torch

        from . import ckv

        self.torch, self.ckv, self.cfg = torch, ckv, cfg
        pool_pages = pool_pages or 4 * max_pages
        dt = {"f32": torch.float32, "bf16": torch.bfloat16, "fp8": torch.uint8}[cfg.kv_dtype]
        shape = (pool_pages, cfg.num_kv_heads, cfg.page_size, cfg.head_dim)
        g = torch.Generator(device=device).manual_seed(seed)
        k = torch.randint(0, 256, shape + (torch.finfo(dt).bits // 8 if dt.is_floating_point else 1,),
                          dtype=torch.uint8, device=device, generator=g).view(dt).view(shape)
        v = k.roll(1, 0).contiguous()
        ks = vs = None
        if cfg.kv_dtype == "fp8":
            ks = torch.rand(shape[:2], device=device, generator=g) + 0.5
            vs = ks.flip(0).contiguous()
        self.pool = ckv.Pool(k, v, ks, vs)
        self.pages = torch.randperm(pool_pages, device=device, generator=g)[:max_pages].to(torch.int32)
        self.page_shape, self.dt = shape[1:], dt
        self.host_buf = torch.empty(ckv.pages_staging_bytes(self.pool, max_pages), dtype=torch.uint8,
                                    pin_memory=True)
        self.staging = torch.empty(ckv.pages_staging_bytes(self.pool, max_pages), dtype=torch.uint8,
                                   device=device)
        self.dev_flat = torch.empty(2 * k[0].numel() * k.element_size() * max_pages, dtype=torch.uint8,
                                    device=device)
        self.host_flat = torch.empty(self.dev_flat.numel(), dtype=torch.uint8, pin_memory=True)
        self.max_pages = max_pages

    def host_views(self, n: int):
        """K pages, V pages and fp8 scales of n pages, back to back in one
        pinned buffer (the layout that moves as a single copy)."""
        torch = self.torch
        nb = n * int(np.prod(self.page_shape)) * self.pool.k.element_size()
        sb = n * self.cfg.num_kv_heads * 4 if self.cfg.kv_dtype == "fp8" else 0
        b = self.host_buf
        hk = b[:nb].view(self.dt).view((n,) + self.page_shape)
        hv = b[nb:2 * nb].view(self.dt).view((n,) + self.page_shape)
        if not sb:
            return hk, hv, None, None
        return (hk, hv, b[2 * nb:2 * nb + sb].view(torch.float32).view(n, -1),
                b[2 * nb + sb:2 * nb + 2 * sb].view(torch.float32).view(n, -1))

    def page_bytes(self, n: int) -> int:
        """K + V (+ fp8 scales) bytes of n pages."""
        b = 2 * n * self.pool.k[0].numel() * self.pool.k.element_size()
        if self.cfg.kv_dtype == "fp8":
            b += 2 * n * self.cfg.num_kv_heads * 4
        return b

    def _time(self, fn, reps: int, warmup: int) -> float:
        torch = self.torch
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        times = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1))
        return float(np.median(times))

    def time(self, n: int, reps: int = 5, warmup: int = 2) -> Dict[str, float]:
        """Milliseconds for offload, reload and a plain copy each way of n pages."""
        if not 0 < n <= self.max_pages:
            raise ValueError("n must lie in [1, max_pages]")
        ckv, pg = self.ckv, self.pages[:n]
        hk, hv, hks, hvs = self.host_views(n)
        nb = self.page_bytes(n) - (2 * n * self.cfg.num_kv_heads * 4 if self.cfg.kv_dtype == "fp8" else 0)
        d, h = self.dev_flat[:nb], self.host_flat[:nb]
        return {
            "offload": self._time(lambda: ckv.kv_pages_offload(self.pool, pg, hk, hv, hks, hvs,
                                                               staging=self.staging), reps, warmup),
            "reload": self._time(lambda: ckv.kv_pages_reload(self.pool, pg, hk, hv, hks, hvs,
                                                             staging=self.staging), reps, warmup),
            "copy_d2h": self._time(lambda: h.copy_(d, non_blocking=True), reps, warmup),
            "copy_h2d": self._time(lambda: d.copy_(h, non_blocking=True), reps, warmup),
        }


def transfer_profile(cfg, page_counts: Sequence[int], reps: int = 5) -> dict:
    """GB/s of offload / reload per page count (the paper's item (1)), with
    the plain pinned copy of the same bytes alongside."""
    timer = TransferTimer(cfg, max(page_counts))
    res = {"config": cfg.name, "page_counts": list(page_counts), "bytes": [], "ms": {}, "gbps": {}}
    for n in page_counts:
        t = timer.time(n, reps=reps)
        nb = timer.page_bytes(n)
        res["bytes"].append(nb)
        for key, ms in t.items():
            res["ms"].setdefault(key, []).append(ms)
            res["gbps"].setdefault(key, []).append(nb / (ms * 1e-3) / 1e9)
        print(f"[transfer] pages={n:6d} ({nb / 2**20:8.1f} MiB): " +
              "  ".join(f"{k} {nb / (v * 1e-3) / 1e9:6.1f} GB/s" for k, v in t.items()),
              file=sys.stderr, flush=True)
    res["fit"] = {key: fit_linear(res["bytes"], ms) for key, ms in res["ms"].items()}
    for key, f in res["fit"].items():
        print(f"[transfer] fit {key:8s}: {f['gbps']:6.1f} GB/s + {f['t0_us']:6.1f} us  (R^2 {f['r2']:.6f})",
              file=sys.stderr, flush=True)
    return res


def profile(cfg, max_len: int, chunks: Sequence[int], first: int = 1000, reps: int = 3,
            window: int = 0) -> dict:
    timer = PrefillTimer(cfg, max_len, window=window)
    lengths = length_ladder(max_len, first)
    res = {"config": cfg.name, "window": window, "lengths": lengths, "series": {}}
    series = [("full", None)] + [(f"chunk{c}", c) for c in chunks]
    for name, c in series:
        ts, fl = [], []
        for L in lengths:
            pairs = [(0, L)] if c is None else chunk_plan(L, c)
            ts.append(timer.time(pairs, reps=reps))
            fl.append(sum(attention_flops(P, n, cfg.num_q_heads, cfg.head_dim, window) for P, n in pairs))
            print(f"[profile] {name:10s} L={L:6d}: {ts[-1]:9.3f} ms  "
                  f"{fl[-1] / (ts[-1] * 1e-3) / 1e12:7.1f} TFLOP/s", file=sys.stderr, flush=True)
        res["series"][name] = {"ms": ts, "tflops": [f / (t * 1e-3) / 1e12 for f, t in zip(fl, ts)],
                               "fit_ms": fit_quadratic(lengths, ts)}
    return res


def main(argv=None):
    import workload

    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--config", default="llama3.1-70b", choices=sorted(workload.CONFIGS))
    ap.add_argument("--max-len", type=int, default=65536)
    ap.add_argument("--first", type=int, default=1000)
    ap.add_argument("--chunks", type=int, nargs="*", default=[256, 512, 1024, 2048, 4096])
    ap.add_argument("--window", type=int, default=0)
    ap.add_argument("--reps", type=int, default=3)
    ap.add_argument("--transfer", action="store_true",
                    help="profile host-link page offload/reload instead of prefill")
    ap.add_argument("--pages", type=int, nargs="*", default=[16, 64, 256, 1024, 4096, 16384])
    args = ap.parse_args(argv)
    cfg = workload.CONFIGS[args.config]
    if args.transfer:
        print(json.dumps(transfer_profile(cfg, args.pages, max(args.reps, 3))))
        return
    print(json.dumps(profile(cfg, args.max_len, args.chunks, args.first, args.reps, args.window)))


if __name__ == "__main__":
    main()
