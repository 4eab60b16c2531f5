"""Offline prefill-vs-context profile on one MI355X (one attention layer).

Continuum's cost model needs the time to rebuild a request's KV cache when
its TTL has expired (Prefill-Reload(r), Sec. 4.1).  The paper gets it from a
short offline profile per (hardware, model): prefill for a ladder of context
sizes up to the maximum context, then a quadratic fit of time against
context length (Sec. 5.2, "Offline Profile").  Serving engines prefill in
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
    args = ap.parse_args(argv)
    cfg = workload.CONFIGS[args.config]
    print(json.dumps(profile(cfg, args.max_len, args.chunks, args.first, args.reps, args.window)))


if __name__ == "__main__":
    main()
