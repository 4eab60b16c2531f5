"""The benchmark's algorithmic work and bytes, pinned by independent counts
(CPU only): the headline TFLOP/s and GB/s divide these by measured time."""
import os
import subprocess
import sys

import numpy as np
import pytest

import bench
import workload
from oracle import paged

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("P, n, W", [(0, 1, 0), (0, 7, 0), (5, 9, 0), (40, 13, 0), (40, 13, 8), (3, 20, 1),
                                     (100, 3, 1000), (0, 0, 0)])
def test_visible_pairs_equals_brute_force(P, n, W):
    brute = sum(1 for t in range(n) for j in range(P + t + 1) if paged.visible(P + t, j, W))
    assert bench.visible_pairs(P, n, W) == brute


def test_prefill_flops_counts_every_visible_pair():
    wl = workload.make_workload(workload.TINY)
    cfg, pf = wl.cfg, wl.prefill
    for W in (0, 17):
        pairs = 0
        for b in range(pf.num_seqs):
            P, n = int(pf.ctx_lens[b]), int(pf.q_lens[b])
            pairs += sum(1 for t in range(n) for j in range(P + t + 1) if paged.visible(P + t, j, W))
        assert bench.prefill_flops(wl, W) == 4.0 * cfg.head_dim * cfg.num_q_heads * pairs


def test_decode_bytes_by_hand():
    # one bf16 sequence of 40 tokens, page 16, H_kv 2, D 64, H_q 4:
    # K and V 40*2*64*2 B each, q and out 4*64*2 B each, 3 block-table entries
    wl = workload.make_workload(workload.Config("hand", 3, 4, 2, 64, 16, "bf16", "bf16"),
                                prefill=[], decode=[40])
    assert list(wl.decode_ctx) == [40]
    kv = 2 * 40 * 2 * 64 * 2
    qo = 2 * 4 * 64 * 2
    assert bench.decode_bytes(wl, 0) == kv + qo + 3 * 4
    # a window of 20 keys reads 20 rows of K and V; the table is still walked to c
    assert bench.decode_bytes(wl, 20) == 2 * 20 * 2 * 64 * 2 + qo + 3 * 4


def test_fp8_decode_bytes_add_one_scale_pair_per_page_and_head():
    wl = workload.make_workload(workload.Config("hand8", 4, 8, 2, 128, 64, "bf16", "fp8"),
                                prefill=[], decode=[100])
    c = 100
    kv = 2 * c * 2 * 128 * 1
    qo = 2 * 8 * 128 * 2
    pages = 2
    assert bench.decode_bytes(wl, 0) == kv + qo + 4 * pages + 8 * 2 * pages


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_traffic_entry_follows_the_code_not_its_comments(tmp_path, monkeypatch):
    """A stored HBM-traffic measurement stays valid when only comments or
    spacing of its kernel's sources change, and is dropped when code does."""
    import hashlib
    import json
    import shutil

    src = "__global__ void k(int *p) {\n  p[0] = 1;  // one store\n}\n"
    (tmp_path / "paper_2511_02230_amd" / "csrc").mkdir(parents=True)
    (tmp_path / "profiles").mkdir()
    kfile = tmp_path / "paper_2511_02230_amd" / "csrc" / "k.hip"
    kfile.write_text(src)
    h = hashlib.sha256(bench.code_text(src).encode()).hexdigest()[:16]
    (tmp_path / "profiles" / "traffic.json").write_text(
        json.dumps({"k": {"sources": ["k.hip"], "code_sha256_16": h, "bytes": 1234}}))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("k") == 1234.0
    kfile.write_text("/* a kernel */\n__global__ void k(int *p) {\n    p[0] = 1;   // a store\n}\n")
    assert bench.measured_traffic("k") == 1234.0
    kfile.write_text("__global__ void k(int *p) {\n  p[0] = 2;  // one store\n}\n")
    assert bench.measured_traffic("k") is None
    assert bench.measured_traffic("missing") is None
    shutil.rmtree(tmp_path / "profiles")
    assert bench.measured_traffic("k") is None
