"""Seeded agent-serving simulation driving the TTL control plane.

Programs (tool-calling agents) arrive as a Poisson process at `jps` jobs per
second.  Each runs N turns: a turn prefills its new tokens (tool output +
next prompt) over the program's context, decodes its output tokens, and,
unless it is the last, calls a tool whose duration is drawn from that tool's
distribution (Sec. 3.1 describes such traces).  The library's C++ scheduler
(Alg. 1, include/ckv_ttl.h) decides which request runs and whether the
program's pages stay pinned across the tool call; a hit reuses the retained
prefix, a miss rebuilds it (new prefill of the whole context, or a reload
from host memory when offloading is on).

Service times come from `CostModel` (one GPU, all layers), or, with
`GpuLayer`, from running kv_append + prefix_prefill_attn of one attention
layer on the GPU through block tables over the pages the scheduler kept,
scaled to the model's layer count.  Running requests do not slow each other
down here: the simulation exercises the control plane, memory and the
kernels of a turn, not batching.

    python -m paper_2511_02230_amd.serve_sim --programs 200 --jps 0.3 --policy ttl
    python -m paper_2511_02230_amd.serve_sim --programs 200 --jps 0.3 --policy none
"""
from __future__ import annotations

import argparse
import dataclasses
import heapq
import json
import math
import sys
from typing import Dict, List, Optional, Tuple

import numpy as np

from .ttl import Scheduler


# ------------------------------------------------------------------- traces

@dataclasses.dataclass
class Program:
    arrival: float
    turns: List[Tuple[int, int, int]]  # (new tokens, output tokens, tool called after it)
    tool_s: List[float]                # duration of the tool after turn k (last unused)


def make_trace(seed: int, num_programs: int, jps: float, mean_turns: float = 8.0,
               turns_law: str = "fixed", tool_means=(0.5, 2.0, 8.0), first_tokens=(2000, 0.5),
               turn_tokens=(600, 0.8), out_tokens=(200, 0.5), max_context: int = 60000) -> List[Program]:
    """Poisson arrivals; turn counts fixed or geometric with the given mean;
    lognormal token counts (median, sigma); tool k's duration ~ Exp(mean k).
    Contexts are capped at max_context tokens by ending the program early."""
    rng = np.random.default_rng(seed)
    t, out = 0.0, []
    for _ in range(num_programs):
        t += rng.exponential(1.0 / jps)
        if turns_law == "fixed":
            N = max(1, int(round(mean_turns)))
        elif turns_law == "geometric":
            N = int(rng.geometric(1.0 / mean_turns))
        else:
            raise ValueError(turns_law)
        turns, tools, ctx = [], [], 0
        for k in range(N):
            med, sig = first_tokens if k == 0 else turn_tokens
            n = max(1, int(rng.lognormal(math.log(med), sig)))
            o = max(1, int(rng.lognormal(math.log(out_tokens[0]), out_tokens[1])))
            if ctx + n + o > max_context:
                break
            f = int(rng.integers(len(tool_means)))
            turns.append((n, o, f))
            tools.append(float(rng.exponential(tool_means[f])))
            ctx += n + o
        if not turns:
            turns, tools = [(1, 1, 0)], [0.0]
        out.append(Program(t, turns, tools))
    return out


# --------------------------------------------------------------- cost model

@dataclasses.dataclass
class CostModel:
    """Seconds per turn on one GPU for a whole model.

    Attention: the per-layer full-prefill fit t(L) = a L^2 + b L + c (ms) of
    the offline profile, so a prefix-reuse prefill of n tokens over P costs
    layers * (a ((P+n)^2 - P^2) + b n + c).  Linear layers: a per-token
    cost; decode: a per-output-token cost; reload: KV bytes over the host
    link.  The defaults are the Llama-3.1-70B layer measured on one MI355X
    (attention fit; host link 56 GB/s) plus estimates for the parts this
    library does not run: 2 * 70e9 flop per token at 1.2 PFLOP/s for the
    linear layers, 20 ms per decode step."""

    layers: int = 80
    attn_ms: Tuple[float, float, float] = (1.3906e-08, 6.9167e-06, 7.7587e-02)
    linear_s_per_token: float = 2 * 70e9 / 1.2e15
    decode_s_per_token: float = 0.020
    kv_bytes_per_token: int = 80 * 2 * 8 * 128 * 2
    offload_gbps: float = 0.0  # > 0: evicted caches are reloaded from host memory
    page_size: int = 16

    def prefill_s(self, P: int, n: int) -> float:
        a, b, c = self.attn_ms
        attn = a * ((P + n) ** 2 - P ** 2) + b * n + c
        return self.layers * attn * 1e-3 + self.linear_s_per_token * n

    def reload_s(self, L: int) -> float:
        return L * self.kv_bytes_per_token / (self.offload_gbps * 1e9)

    def rebuild_s(self, L: int) -> float:
        """Prefill-Reload(r): rebuilding L tokens of KV cache (Sec. 4.1)."""
        if L <= 0:
            return 0.0
        if self.offload_gbps > 0:
            return min(self.reload_s(L), self.prefill_s(0, L))
        return self.prefill_s(0, L)

    def pages(self, tokens: int) -> int:
        return -(-tokens // self.page_size)


# ------------------------------------------------------------ GPU layer

class GpuLayer:
    """One attention layer's pool on the GPU; runs each issued turn's
    kv_append + prefix_prefill_attn through the block table of the pages
    the program holds, and times them.  K/V of program p at position j and
    the queries of each turn come from fixed seeds, so a rebuilt prefix
    holds exactly the values it held before eviction."""

    def __init__(self, cfg, capacity_pages: int, max_context: int, num_programs: int, seed: int = 0,
                 check: bool = False):
        import torch

        from . import ckv

        self.torch, self.ckv, self.cfg, self.check = torch, ckv, cfg, check
        dt = torch.bfloat16
        shape = (capacity_pages, cfg.num_kv_heads, cfg.page_size, cfg.head_dim)
        self.pool = ckv.Pool(torch.zeros(shape, dtype=dt, device="cuda"),
                             torch.zeros(shape, dtype=dt, device="cuda"))
        self.free = list(range(capacity_pages - 1, -1, -1))
        self.pages: Dict[int, List[int]] = {}
        self.seed, self.max_context = seed, max_context
        self.kv_cache: Dict[int, tuple] = {}
        self.checked = 0
        self.max_err = 0.0

    def _kv(self, p: int):
        torch = self.torch
        if p not in self.kv_cache:
            g = torch.Generator(device="cuda").manual_seed(self.seed * 1000003 + p)
            shp = (self.max_context, self.cfg.num_kv_heads, self.cfg.head_dim)
            self.kv_cache[p] = (torch.randn(shp, generator=g, device="cuda").to(torch.bfloat16),
                                torch.randn(shp, generator=g, device="cuda").to(torch.bfloat16))
        return self.kv_cache[p]

    def _q(self, p: int, turn: int, n: int):
        torch = self.torch
        g = torch.Generator(device="cuda").manual_seed(self.seed * 7919 + p * 131 + turn)
        return torch.randn((n, self.cfg.num_q_heads, self.cfg.head_dim), generator=g,
                           device="cuda").to(torch.bfloat16)

    def release(self, p: int):
        self.free.extend(reversed(self.pages.pop(p, [])))

    def _batch(self, p: int, P: int, n: int):
        torch = self.torch
        pages = self.pages[p]
        bt = torch.tensor([pages], dtype=torch.int32, device="cuda")
        return self.ckv.Batch(bt, torch.tensor([P], dtype=torch.int32, device="cuda"),
                              torch.tensor([0, n], dtype=torch.int32, device="cuda"), n, n, P)

    def run_turn(self, p: int, turn: int, held: bool, ctx: int, n: int, o: int, npages: int) -> float:
        """Milliseconds of this layer's GPU work for the turn.  held: the
        program's pages (its first ctx tokens) are still resident."""
        torch, ckv = self.torch, self.ckv
        if not held:
            self.release(p)
        have = self.pages.setdefault(p, [])
        while len(have) < npages:
            have.append(self.free.pop())
        k, v = self._kv(p)
        P = ctx if held else 0          # what stays resident vs what is rebuilt
        rows = ctx + n - P
        q_new = self._q(p, turn, n)
        q = q_new if held else torch.cat([self._q(p, -1 - turn, ctx), q_new]) if ctx else q_new
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        ckv.kv_append(self.pool, self._batch(p, P, rows), k[P:P + rows].contiguous(),
                      v[P:P + rows].contiguous())
        out = ckv.prefix_prefill_attn(self.pool, self._batch(p, P, rows), q, 1.0 / math.sqrt(self.cfg.head_dim))
        e1.record()
        # the turn's output tokens join the context (their K/V appended; decode is modeled)
        ckv.kv_append(self.pool, self._batch(p, ctx + n, o), k[ctx + n:ctx + n + o].contiguous(),
                      v[ctx + n:ctx + n + o].contiguous())
        torch.cuda.synchronize()
        if self.check and held and ctx > 0:
            # a hit must give what a rebuild would: the program's K/V regenerated
            # into a scratch pool, prefilled from position 0; this also shows
            # that no other program wrote into the pinned pages meanwhile
            L = ctx + n
            npg = -(-L // self.cfg.page_size)
            shp = (npg,) + tuple(self.pool.k.shape[1:])
            scratch = ckv.Pool(torch.zeros(shp, dtype=torch.bfloat16, device="cuda"),
                               torch.zeros(shp, dtype=torch.bfloat16, device="cuda"))
            bt = torch.arange(npg, dtype=torch.int32, device="cuda")[None]
            b0 = ckv.Batch(bt, torch.zeros(1, dtype=torch.int32, device="cuda"),
                           torch.tensor([0, L], dtype=torch.int32, device="cuda"), L, L, 0)
            ckv.kv_append(scratch, b0, k[:L].contiguous(), v[:L].contiguous())
            q_all = torch.cat([self._q(p, -1 - turn, ctx), q_new])
            full = ckv.prefix_prefill_attn(scratch, b0, q_all, 1.0 / math.sqrt(self.cfg.head_dim))
            torch.cuda.synchronize()
            err = (full[ctx:].float() - out.float()).abs().max().item()
            self.max_err = max(self.max_err, err)
            self.checked += 1
        return e0.elapsed_time(e1)


# ------------------------------------------------------------- simulation

def simulate(trace: List[Program], cost: CostModel, capacity_pages: int, policy: str = "ttl",
             min_records: int = 100, gpu: Optional[GpuLayer] = None) -> dict:
    """Run the trace; policy 'ttl' (Eq. 2), 'none' (retain nothing) or
    'static:<seconds>'."""
    fixed = None if policy == "ttl" else 0.0 if policy == "none" else float(policy.split(":")[1])
    sched = Scheduler(capacity_pages, min_records=min_records, fixed_ttl_s=fixed)
    events: list = []
    seq = 0

    def push(t, kind, payload):
        nonlocal seq
        heapq.heappush(events, (t, seq, kind, payload))
        seq += 1

    for p, prog in enumerate(trace):
        push(prog.arrival, "arrive", (p, 0))
    ctx = [0] * len(trace)               # resident tokens after each finished turn
    req_of: Dict[int, Tuple[int, int]] = {}
    end = [0.0] * len(trace)
    rid = 0
    hits = misses = rebuilt = 0
    gpu_ms = 0.0
    pinned_by_us: set = set()
    while events:
        now = events[0][0]
        while events and events[0][0] <= now:
            _, _, kind, payload = heapq.heappop(events)
            if kind == "arrive":
                p, k = payload
                n, o, _ = trace[p].turns[k]
                rid += 1
                req_of[rid] = (p, k)
                sched.arrive(rid, p, cost.pages(ctx[p] + n + o), now)
            else:
                r = payload
                p, k = req_of.pop(r)
                n, o, f = trace[p].turns[k]
                ctx[p] += n + o
                last = k == len(trace[p].turns) - 1
                tau = sched.finish(r, now, last=last, next_tool=f, prefill_reload_s=cost.rebuild_s(ctx[p]))
                if last:
                    end[p] = now
                    if gpu:
                        gpu.release(p)
                else:
                    if tau > 0:
                        pinned_by_us.add(p)
                    elif gpu:
                        gpu.release(p)
                    push(now + trace[p].tool_s[k], "arrive", (p, k + 1))
        issued = sched.schedule(now)
        # pins the scheduler dropped (expired, or victims of the deadlock
        # breaker) give their pages back before the issued turns take pages
        reused = {iss.program for iss in issued if iss.reused}
        for p in [p for p in pinned_by_us if p not in reused and sched.pin_expiry(p) < 0]:
            pinned_by_us.discard(p)
            if gpu:
                gpu.release(p)
        for iss in issued:
            p, k = req_of[iss.request]
            n, o, _ = trace[p].turns[k]
            pinned_by_us.discard(p)
            if iss.reused:
                hits += 1
                svc = cost.prefill_s(ctx[p], n)
            else:
                if k > 0:
                    misses += 1
                    rebuilt += ctx[p]
                svc = (cost.rebuild_s(ctx[p]) + cost.prefill_s(ctx[p], n)) if cost.offload_gbps > 0 \
                    else cost.prefill_s(0, ctx[p] + n)
            if gpu:
                gpu_ms += gpu.run_turn(p, k, iss.reused, ctx[p], n, o, cost.pages(ctx[p] + n + o))
            push(now + svc + cost.decode_s_per_token * o, "done", iss.request)
    jct = np.array([end[p] - trace[p].arrival for p in range(len(trace))])
    st = sched.stats()
    res = {"policy": policy, "programs": len(trace), "mean_jct_s": float(jct.mean()),
           "p50_jct_s": float(np.percentile(jct, 50)), "p90_jct_s": float(np.percentile(jct, 90)),
           "makespan_s": float(max(end)), "hits": hits, "misses": misses, "rebuilt_tokens": rebuilt,
           "eta": st["eta"], "mean_wait_s": st["mean_wait_s"], "tool_records": st["tool_records"],
           "leftover": {"waiting": st["waiting"], "running": st["running"], "pinned": st["pinned"]}}
    if gpu:
        res["gpu_attention_ms_one_layer"] = gpu_ms
        res["gpu_checked_hits"] = gpu.checked
        res["gpu_hit_vs_rebuild_max_abs_diff"] = gpu.max_err
    sched.close()
    return res


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--programs", type=int, default=200)
    ap.add_argument("--jps", type=float, default=0.3)
    ap.add_argument("--turns", type=float, default=8.0)
    ap.add_argument("--turns-law", default="fixed", choices=["fixed", "geometric"])
    ap.add_argument("--policy", nargs="+", default=["ttl", "none", "static:2", "static:10"])
    ap.add_argument("--kv-gb", type=float, default=60.0, help="HBM for the KV cache (all layers)")
    ap.add_argument("--offload-gbps", type=float, default=0.0)
    ap.add_argument("--seed", type=int, default=0)
    args = ap.parse_args(argv)
    cost = CostModel(offload_gbps=args.offload_gbps)
    cap = int(args.kv_gb * 1e9 // (cost.kv_bytes_per_token * cost.page_size))
    trace = make_trace(args.seed, args.programs, args.jps, args.turns, args.turns_law)
    for pol in args.policy:
        r = simulate(trace, cost, cap, pol)
        print(json.dumps(r), flush=True)
        print(f"[sim] {pol:10s} mean JCT {r['mean_jct_s']:8.1f} s  p90 {r['p90_jct_s']:8.1f} s  "
              f"hits {r['hits']:5d}  misses {r['misses']:5d}  eta {r['eta']:.2f}", file=sys.stderr)


if __name__ == "__main__":
    main()
