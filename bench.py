"""Benchmark of the paged-KV hot path on one MI355X.

A step is one pass of the whole hot path over one batch of the Llama-3.1-70B
attention-layer workload (64 query heads, 8 KV heads, head_dim 128, bf16,
page 16; 8 agent sequences at a random turn with retained prefixes and new
turns; a 128-sequence decode batch):

    kv_append(new turn) -> prefix_prefill_attn -> kv_append(decode token)
    -> paged_decode_attn

and the same step as one mixed launch (both appends, then mixed_attn: the
prefill's row tiles and the decode's partitions in one grid) is timed after
it and reported as "mixed_step".

Inputs are synthetic and already resident in HBM when timing starts.  The
headline value is prefix_prefill_attn's throughput in algorithmic TFLOP/s
(4 * D * H_q per visible (query row, key) pair); the decode kernel's
algorithmic GB/s and kv_append's GB/s are reported beside it, each with its
roofline.  The CPU baseline is the fp64 oracle timed on a bounded sample.

    python bench.py [--steps K] [--warmup W] [--config NAME] [--window W]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
E = {"f32": 4, "bf16": 2, "fp8": 1}


def visible_pairs(P, n, window):
    """sum over new rows t < n of |{j : j <= P + t, (W == 0 or P + t - j < W)}|"""
    i = P + np.arange(n, dtype=np.int64)
    cnt = i + 1
    if window > 0:
        cnt = np.minimum(cnt, window)
    return int(cnt.sum())


def prefill_flops(wl, window):
    cfg = wl.cfg
    pf = wl.prefill
    pairs = sum(visible_pairs(int(pf.ctx_lens[b]), int(pf.q_lens[b]), window) for b in range(pf.num_seqs))
    return 4.0 * cfg.head_dim * cfg.num_q_heads * pairs


def decode_bytes(wl, window):
    cfg = wl.cfg
    c = wl.decode_ctx.astype(np.int64)
    keys = np.minimum(c, window) if window > 0 else c
    ekv = E[cfg.kv_dtype]
    kv = keys * cfg.num_kv_heads * cfg.head_dim * 2 * ekv
    qo = cfg.num_q_heads * cfg.head_dim * 2 * E[cfg.q_dtype]
    tables = 4 * (-(-c // cfg.page_size))
    scales = 8 * cfg.num_kv_heads * (-(-keys // cfg.page_size)) if cfg.kv_dtype == "fp8" else 0
    return float((kv + qo + tables + scales).sum())


def append_bytes(wl, rows):
    cfg = wl.cfg
    e_in = 4 if cfg.kv_dtype == "f32" else 2
    return float(rows * cfg.num_kv_heads * cfg.head_dim * 2 * (e_in + E[cfg.kv_dtype]))


def measured_traffic(kernel_key):
    """HBM bytes per launch that rocprofv3 measured for this kernel
    (FETCH_SIZE / WRITE_SIZE passes scaled by a plain copy's readings, kept in
    profiles/traffic.json), or None when there is no measurement or the
    code of the kernel's sources (comments aside) has changed since it was
    taken."""
    import hashlib

    try:
        with open(os.path.join(ROOT, "profiles", "traffic.json")) as f:
            entry = json.load(f).get(kernel_key)
    except (OSError, ValueError):
        return None
    if not entry:
        return None
    h = hashlib.sha256()
    for src in entry["sources"]:
        with open(os.path.join(ROOT, "paper_2511_02230_amd", "csrc", src)) as f:
            h.update(code_text(f.read()).encode())
    if h.hexdigest()[:16] != entry["code_sha256_16"]:
        return None
    return float(entry["bytes"])


def code_text(src):
    """A source file's code without its comments and with runs of whitespace
    made one space: what the traffic entries' hashes cover, so that editing a
    comment does not void a measurement while any change to the code does."""
    import re

    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    return re.sub(r"\s+", " ", src).strip()


def cpu_baseline(wl, window, budget_s=30.0):
    """Time the fp64 oracle on a bounded sample of the same workload: new-turn
    rows of the longest prefill sequence (prefill TFLOP/s of the sample)."""
    from threadpoolctl import threadpool_info

    from tests.oracle_inputs import OracleState, to_numpy
    import torch
    import workload

    cfg = wl.cfg
    pf = wl.prefill
    b = int(np.argmax(pf.ctx_lens + pf.q_lens))
    P, n = int(pf.ctx_lens[b]), int(pf.q_lens[b])
    st = OracleState(wl, sids=[int(pf.seq_ids[b])], device="cuda")
    st.append_prefill([b])
    q = to_numpy(workload.concat_rows(pf, lambda r: workload.prefill_q(wl, r, "cuda")))
    # size the sample from a 16-row probe so that it takes about budget_s
    probe = np.linspace(0, n - 1, min(n, 16)).astype(np.int64)
    st.prefill(q, [b], window, {b: probe[:2]})  # warm caches / BLAS threads
    t0 = time.perf_counter()
    st.prefill(q, [b], window, {b: probe})
    per_row = (time.perf_counter() - t0) / len(probe)
    rows = int(max(1, min(n, budget_s / max(per_row, 1e-4))))
    sel = np.linspace(0, n - 1, rows).astype(np.int64)
    t0 = time.perf_counter()
    st.prefill(q, [b], window, {b: sel})
    dt = time.perf_counter() - t0
    i = P + sel
    cnt = np.minimum(i + 1, window) if window > 0 else i + 1
    flops = 4.0 * cfg.head_dim * cfg.num_q_heads * float(cnt.sum())
    threads = sum(int(x.get("num_threads", 0)) for x in threadpool_info() if x.get("user_api") == "blas")
    del torch
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": max(threads, 1), "kind": "oracle",
            "sample": f"prefix_prefill rows of sequence {b} (P={P}, n={n}): {rows} of {n} rows, "
                      f"{flops / 1e9:.1f} GFLOP fp64 in {dt:.1f} s; affinity {len(os.sched_getaffinity(0))} cpus"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="llama3.1-70b")
    ap.add_argument("--window", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="after timing, run one 512 MiB device-to-device copy (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the kernels run on one device's share of the work "
              "(sharding by sequence or KV head needs no exchange); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    import workload
    from paper_2511_02230_amd.harness import DeviceWorkload

    cfg = workload.CONFIGS[args.config]
    wl = workload.make_workload(cfg)
    print(f"[bench] setting up {cfg.name}: {wl.prefill.num_seqs} prefills "
          f"(T_new={wl.prefill.total_q}), {wl.decode.num_seqs} decodes, pool {wl.num_pages} pages",
          file=sys.stderr, flush=True)
    dw = DeviceWorkload(wl, "cuda", window=args.window)
    stream = torch.cuda.current_stream()

    for _ in range(args.warmup):
        dw.step()
    torch.cuda.synchronize()
    print("[bench] warmup done", file=sys.stderr, flush=True)

    names = ["kv_append_prefill", "prefix_prefill_attn", "kv_append_decode", "paged_decode_attn"]
    calls = [dw.append_prefill, dw.run_prefill, dw.append_decode, dw.run_decode]
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(calls) + 1)] for _ in range(args.steps)]
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for k in range(args.steps):
        ev[k][0].record(stream)
        for i, fn in enumerate(calls):
            fn()
            ev[k][i + 1].record(stream)
    end.record(stream)
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(end) / args.steps
    per = {nm: float(np.mean([ev[k][i].elapsed_time(ev[k][i + 1]) for k in range(args.steps)]))
           for i, nm in enumerate(names)}

    # the same step as one mixed launch: both appends, then prefill and decode
    # work items in one grid (decode partitions of the mixed launch's own
    # length), timed the same way
    from paper_2511_02230_amd import ckv

    mixed = None
    if cfg.q_dtype == "bf16" and wl.prefill.num_seqs and wl.decode.num_seqs:
        mws_n = ckv.mixed_workspace_bytes(dw.pool, dw.prefill, dw.decode, cfg.num_q_heads)
        mws = torch.empty(max(1, mws_n), dtype=torch.uint8, device="cuda")
        op, od = torch.empty_like(dw.out_prefill), torch.empty_like(dw.out_decode)

        def mixed_step():
            dw.append_prefill()
            dw.append_decode()
            ckv.mixed_attn(dw.pool, dw.prefill, dw.q_prefill, dw.decode, dw.q_decode, cfg.softmax_scale,
                           args.window, out_prefill=op, out_decode=od, workspace=mws)

        def time_steps(fn):
            for _ in range(args.warmup):
                fn()
            torch.cuda.synchronize()
            m0 = torch.cuda.Event(enable_timing=True)
            m1 = torch.cuda.Event(enable_timing=True)
            m0.record(stream)
            for _ in range(args.steps):
                fn()
            m1.record(stream)
            torch.cuda.synchronize()
            return m0.elapsed_time(m1) / args.steps

        mixed_ms = time_steps(mixed_step)
        mixed = {"ms_per_step": mixed_ms, "sequential_ms_per_step": ms_step, "speedup": ms_step / mixed_ms,
                 "launch": "kv_append x2 + mixed_attn (prefill row tiles and decode partitions in one grid)"}
        if cfg.kv_dtype == "bf16":
            # the whole step in one launch: mixed_attn given the new rows
            # writes them into the pool itself (the same pool contents)
            def fused_step():
                ckv.mixed_attn(dw.pool, dw.prefill, dw.q_prefill, dw.decode, dw.q_decode, cfg.softmax_scale,
                               args.window, out_prefill=op, out_decode=od, workspace=mws,
                               k_prefill=dw.k_new, v_prefill=dw.v_new, k_decode=dw.k_dec, v_decode=dw.v_dec)

            mixed["fused_append_ms_per_step"] = time_steps(fused_step)
            mixed["fused_append_launch"] = "mixed_attn given the new K/V rows (the appends inside the same launch)"

    w = args.window
    # the stored traffic was measured on the default workload only
    default_cfg = args.config == "llama3.1-70b" and w == 0
    if mixed is not None:
        mixed["traffic"] = measured_traffic("mixed_attn") if default_cfg else None
    flops = prefill_flops(wl, w)
    dbytes = decode_bytes(wl, w)
    abytes = append_bytes(wl, wl.prefill.total_q)
    adbytes = append_bytes(wl, wl.decode.num_seqs)
    tflops = flops / (per["prefix_prefill_attn"] * 1e-3) / 1e12
    dec_gbs = dbytes / (per["paged_decode_attn"] * 1e-3) / 1e9
    app_gbs = abytes / (per["kv_append_prefill"] * 1e-3) / 1e9
    rooflines = {
        "prefix_prefill_attn": {"bound": "mfma", "achieved": tflops, "peak": PEAK_BF16_TFLOPS,
                                "unit": "TFLOP/s", "frac": tflops / PEAK_BF16_TFLOPS,
                                "traffic": measured_traffic("prefix_prefill_attn") if default_cfg else None,
                                "ms": per["prefix_prefill_attn"], "work": flops},
        "paged_decode_attn": {"bound": "hbm", "achieved": dec_gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                              "frac": dec_gbs / PEAK_HBM_GBS,
                              "traffic": measured_traffic("paged_decode_attn") if default_cfg else None,
                              "ms": per["paged_decode_attn"], "work": dbytes},
        "kv_append": {"bound": "hbm", "achieved": app_gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                      "frac": app_gbs / PEAK_HBM_GBS,
                      "traffic": measured_traffic("kv_append") if default_cfg else None,
                      "ms": per["kv_append_prefill"],
                      "work": abytes},
        "kv_append_decode": {"bound": "hbm", "ms": per["kv_append_decode"], "work": adbytes},
    }
    if args.calibrate_copy:
        src = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        cpu = cpu_baseline(wl, w)
    line = {
        "metric": "prefix-prefill attn TFLOP/s (% MFMA peak); paged decode attn GB/s (% HBM)",
        "value": tflops,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.kv_dtype != "f32" else "f32",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name} attention layer: prefix-reuse turn + decode batch",
                   "num_q_heads": cfg.num_q_heads, "num_kv_heads": cfg.num_kv_heads,
                   "head_dim": cfg.head_dim, "page_size": cfg.page_size, "kv_dtype": cfg.kv_dtype,
                   "window": w, "prefill_seqs": wl.prefill.num_seqs, "new_turn_tokens": wl.prefill.total_q,
                   "decode_seqs": wl.decode.num_seqs,
                   "decode_context_tokens": int(wl.decode_ctx.sum()), "seed": cfg.seed},
        "decode_gbs": dec_gbs,
        "decode_frac_hbm": dec_gbs / PEAK_HBM_GBS,
        "roofline": rooflines["prefix_prefill_attn"],
        "rooflines": rooflines,
        "cpu_baseline": cpu,
        "mixed_step": mixed,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
