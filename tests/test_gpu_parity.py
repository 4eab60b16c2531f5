"""GPU parity of libckv against the fp64 oracle (needs an MI355X).

Every case runs the HIP kernels through the C ABI (via the ctypes binding)
on seeded synthetic inputs and compares with the oracle on the same inputs:
  kv_append            bit-exact, pool page by page (poisoned slots must
                       stay poisoned)
  attention, f32       max |err| <= 1e-5
  attention, bf16      max |err| <= 2e-2 and mean |err| <= 2e-3
  attention, fp8 KV    max |err| <= 3e-2 and mean |err| <= 2e-3
and, for bf16 and fp8, every output row within 2 % (mean |err|) of the
oracle row's RMS and 10 % (max |err|) of its largest value, which keeps
the check able to fail at long context (tests/parity.py).
Small cases compare every output; the full-size configurations (in the
launch configuration the benchmark times) compare sampled sequences / rows.
"""
import dataclasses
import sys

import numpy as np
import pytest
import torch

import workload
from oracle import formats
from tests import parity
from tests.oracle_inputs import OracleState, to_numpy

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2511_02230_amd import ckv  # noqa: F401  (fails loudly if libckv.so is missing)


def out_f64(t):
    x = to_numpy(t)
    return formats.bf16_bits_to_f64(x) if x.dtype == np.uint16 else x.astype(np.float64)


def check_close(got, ref, cfg, what):
    bad, summary = parity.failures(got, ref, parity.kind_of(cfg))
    say(f"  {what}: {summary}")
    assert not bad, f"{what}: " + "; ".join(bad)


def check_pool(dw, st, what):
    """GPU pool pages of the oracle's sequences equal the oracle's bytes."""
    pages = torch.as_tensor(st.pages, device="cuda")
    for name, gpu, ref in (("K", dw.pool.k, st.pool_k), ("V", dw.pool.v, st.pool_v)):
        g = to_numpy(gpu.index_select(0, pages))
        assert g.view(np.uint8).tobytes() == ref.view(np.uint8).tobytes(), f"{what}: {name} pool differs"


def check_unused_pages_poisoned(dw, used):
    mask = torch.ones(dw.wl.num_pages, dtype=torch.bool, device="cuda")
    mask[torch.as_tensor(np.asarray(used, np.int64), device="cuda")] = False
    for t in (dw.pool.k, dw.pool.v):
        rest = t[mask]
        if t.dtype == torch.uint8:
            assert bool((rest == 0x7F).all())
        else:
            assert bool(torch.isnan(rest.float()).all())


def run_case(wl, window=0, prefill_rows=None, decode_rows=None, row_subsets=None, split_lens=(0,)):
    from paper_2511_02230_amd.harness import DeviceWorkload

    cfg = wl.cfg
    pf, dc = wl.prefill, wl.decode
    pf_rows = list(range(pf.num_seqs)) if prefill_rows is None else list(prefill_rows)
    dc_rows = list(range(dc.num_seqs)) if decode_rows is None else list(decode_rows)
    sids = sorted(set(int(pf.seq_ids[b]) for b in pf_rows) | set(int(dc.seq_ids[b]) for b in dc_rows))
    say(f"case {cfg.name} D={cfg.head_dim} ps={cfg.page_size} G={cfg.group} kv={cfg.kv_dtype} "
        f"W={window} prefill={pf.num_seqs} decode={dc.num_seqs}")
    dw = DeviceWorkload(wl, "cuda", window=window)
    st = OracleState(wl, sids=sids, device="cuda")
    check_pool(dw, st, "set-up append")
    if pf.num_seqs:
        dw.append_prefill()
        torch.cuda.synchronize()
        st.append_prefill(pf_rows)
        check_pool(dw, st, "new-turn append")
        out = dw.run_prefill()
        torch.cuda.synchronize()
        got = out_f64(out)
        ref = st.prefill(to_numpy(dw.q_prefill), [b for b in pf_rows if b in st.rows_of(pf)], window,
                         row_subsets)
        cu = pf.cu_q_lens
        for b, r in ref.items():
            t = np.arange(int(pf.q_lens[b])) if row_subsets is None else np.asarray(row_subsets[b])
            check_close(got[cu[b] + t], r, cfg, f"prefill seq {b} (P={pf.ctx_lens[b]}, n={pf.q_lens[b]})")
    if dc.num_seqs:
        dw.append_decode()
        torch.cuda.synchronize()
        st.append_decode(dc_rows)
        check_pool(dw, st, "decode-token append")
        ref = st.decode(to_numpy(dw.q_decode), st.rows_of(dc, dc_rows), window)
        for split in split_lens:
            out = dw.run_decode(kv_split_len=split)
            torch.cuda.synchronize()
            got = out_f64(out)
            for b, r in ref.items():
                check_close(got[b], r, cfg, f"decode seq {b} (c={wl.decode_ctx[b]}, split={split})")
    return dw, st


# --------------------------------------------------------------- Tiny

def test_tiny_config_whole_pool():
    wl = workload.make_workload(workload.TINY)
    dw, st = run_case(wl)
    check_unused_pages_poisoned(dw, st.pages)


# ------------------------------------------------------- small shapes

def cfg_of(name, hq, hkv, d, ps, kv, q="bf16", seed=11):
    return workload.Config(name, seed, hq, hkv, d, ps, q, kv)


SMALL = [
    # (config, prefill [(P, n)], decode [c], window)
    (cfg_of("c1", 8, 1, 128, 16, "bf16"), [(0, 1), (5, 40), (130, 67), (0, 300)], [1, 17, 64, 65, 700], 0),
    (cfg_of("c2", 32, 8, 128, 16, "bf16"), [(100, 33), (1, 1), (257, 130)], [300, 2, 1000], 0),
    (cfg_of("c3", 16, 8, 256, 16, "bf16"), [(64, 64), (3, 90)], [129, 513], 0),
    (cfg_of("c4", 4, 4, 64, 64, "bf16"), [(200, 100), (0, 64)], [63, 64, 65], 0),
    (cfg_of("c5", 96, 8, 128, 64, "fp8"), [(300, 20), (64, 70), (0, 5)], [1, 200, 700], 0),
    (cfg_of("c6", 12, 1, 128, 16, "fp8"), [(40, 50)], [33, 99], 0),
    (cfg_of("c7", 20, 1, 64, 16, "bf16"), [(10, 13)], [77], 0),
    (cfg_of("w1", 16, 8, 256, 16, "bf16"), [(100, 60), (0, 200), (1500, 40)], [300, 1200, 5], 17),
    (cfg_of("w2", 8, 2, 128, 16, "bf16"), [(50, 50)], [90, 3], 1),
    (cfg_of("w3", 8, 2, 128, 64, "fp8"), [(500, 100)], [400], 100),
    # rows whose window starts within the first keys of a block, while other
    # rows of the same wave already see keys in earlier blocks
    (cfg_of("w4", 16, 8, 128, 16, "bf16"), [(100, 60), (97, 70)], [130], 40),
    # head_dim 256 on 64-token pages; a sequence with no new-turn rows in the
    # prefill batch
    (cfg_of("e1", 8, 2, 256, 64, "bf16"), [(100, 0), (64, 33), (0, 5)], [1, 130], 0),
    (cfg_of("e2", 8, 2, 256, 64, "bf16"), [(200, 70)], [333], 50),
    (cfg_of("e3", 16, 8, 64, 64, "fp8"), [(0, 40), (130, 0), (70, 17)], [1, 64, 129], 0),
    # few row tiles over long prefixes: the prefill splits each tile's keys
    # into partitions and merges them
    (cfg_of("s1", 32, 8, 128, 16, "bf16"), [(6000, 300)], [6300], 0),
    (cfg_of("s2", 16, 8, 256, 16, "bf16"), [(5000, 100)], [5100], 700),
    (cfg_of("s3", 24, 2, 128, 64, "fp8"), [(4000, 64), (100, 20)], [4064], 0),
    # a handful of tiles over a 40k / 70k prefix: 20 and 32 partitions (the most)
    (cfg_of("s4", 8, 1, 128, 16, "bf16"), [(40000, 64)], [40064], 0),
    (cfg_of("s5", 16, 2, 128, 64, "fp8"), [(70000, 32)], [70032], 0),
    # a group of 20 query heads: prefill row tiles cut tokens mid-group, and
    # decode covers the group in two head chunks, the second one ragged
    (cfg_of("g1", 40, 2, 128, 16, "bf16"), [(90, 33), (0, 7)], [1, 77, 300], 0),
    (cfg_of("g2", 40, 2, 128, 64, "fp8"), [(150, 21)], [64, 129], 0),
    # three KV heads: the append's index math without power-of-two shifts
    (cfg_of("h3", 6, 3, 128, 16, "bf16"), [(40, 20), (3, 30)], [50, 17], 0),
    (cfg_of("h3f8", 12, 3, 128, 64, "fp8"), [(70, 9)], [80], 0),
    (cfg_of("f1", 4, 2, 64, 16, "f32", "f32"), [(30, 20), (0, 3)], [19, 50], 0),
    (cfg_of("f2", 4, 1, 128, 64, "f32", "f32"), [(70, 9)], [129], 5),
]


@pytest.mark.parametrize("case", SMALL, ids=lambda c: c[0].name)
def test_small_shapes(case):
    cfg, pf, dc, w = case
    wl = workload.make_workload(cfg, prefill=pf, decode=dc)
    dw, st = run_case(wl, window=w, split_lens=(0, 64, 128) if cfg.q_dtype == "bf16" else (0,))
    check_unused_pages_poisoned(dw, st.pages)


# ----------------------------------------------------------- full size

def _sample_rows(wl, rng, k_pf=3, k_dc=4):
    pf, dc = wl.prefill, wl.decode
    lens = pf.ctx_lens + pf.q_lens
    pf_rows = sorted(set([int(np.argmax(lens)), int(np.argmin(pf.q_lens))] +
                         [int(x) for x in rng.choice(pf.num_seqs, k_pf, replace=False)]))[:k_pf + 1]
    dctx = wl.decode_ctx
    dc_rows = sorted(set([int(np.argmax(dctx)), int(np.argmin(dctx))] +
                         [int(x) for x in rng.choice(dc.num_seqs, k_dc, replace=False)]))
    subsets = {}
    for b in pf_rows:
        n = int(pf.q_lens[b])
        P = int(pf.ctx_lens[b])
        ps = wl.cfg.page_size
        edge = [t for t in range(n) if (P + t) % ps in (0, ps - 1)][:8]
        t = sorted(set([0, n - 1] + edge + [int(x) for x in rng.choice(n, min(n, 12), replace=False)]))
        subsets[b] = np.array(t)
    return pf_rows, dc_rows, subsets


@pytest.mark.parametrize("name,window", [("llama3.1-8b", 0), ("gemma3-12b", 0), ("gemma3-12b", 1024),
                                         ("llama3.1-70b", 0), ("glm4.5-355b", 0)])
def test_full_config_sampled(name, window):
    cfg = workload.CONFIGS[name]
    wl = workload.make_workload(cfg)
    rng = np.random.default_rng([cfg.seed, window, 7])
    pf_rows, dc_rows, subsets = _sample_rows(wl, rng)
    run_case(wl, window, pf_rows, dc_rows, subsets)


# ----------------------------------------------------------- invariants

def _outputs(wl, window=0):
    from paper_2511_02230_amd.harness import DeviceWorkload

    dw = DeviceWorkload(wl, "cuda", window=window)
    dw.step()
    torch.cuda.synchronize()
    return dw.out_prefill.clone(), dw.out_decode.clone()


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
def test_page_shuffle_is_bit_identical(kv):
    cfg = cfg_of("shuf", 16, 2, 128, 16, kv)
    pf, dc = [(300, 100), (17, 250)], [1000, 33]
    a = _outputs(workload.make_workload(cfg, prefill=pf, decode=dc))
    b = _outputs(workload.make_workload(cfg, prefill=pf, decode=dc, slack_pages=37))
    for x, y in zip(a, b):
        assert torch.equal(x.view(torch.int16), y.view(torch.int16))


def test_decode_matches_one_row_prefill_on_gpu():
    """decode(c) and a one-row prefill at P = c - 1 give the same row: each
    within the bars of the oracle, and the two within the per-row bar of
    each other."""
    from paper_2511_02230_amd import ckv
    from paper_2511_02230_amd.harness import DeviceWorkload

    cfg = cfg_of("dvp", 32, 8, 128, 16, "bf16")
    wl = workload.make_workload(cfg, prefill=[], decode=[1000, 77, 4096, 20000])
    dw = DeviceWorkload(wl, "cuda")
    st = OracleState(wl, device="cuda")
    dw.append_decode()
    st.append_decode()
    dec = out_f64(dw.run_decode())
    dcx = wl.decode_ctx
    # the same queries as one-row prefills at P = c - 1
    bt = dw.decode.block_table
    ctx = torch.as_tensor((dcx - 1).astype(np.int32), device="cuda")
    cu = torch.arange(len(dcx) + 1, dtype=torch.int32, device="cuda")
    batch = ckv.Batch(bt, ctx, cu, len(dcx), 1, int(dcx.max()) - 1)
    pre = out_f64(ckv.prefix_prefill_attn(dw.pool, batch, dw.q_decode, cfg.softmax_scale))
    ref = st.decode(to_numpy(dw.q_decode), st.rows_of(wl.decode))
    for b, r in ref.items():
        check_close(dec[b], r, cfg, f"decode c={dcx[b]}")
        check_close(pre[b], r, cfg, f"one-row prefill P={dcx[b] - 1}")
        check_close(dec[b], pre[b], cfg, f"decode vs one-row prefill c={dcx[b]}")


def _plant_keys(dw, st, sid, upto, rng, every=2048):
    """In each `every`-key range of sequence `sid` below position `upto`,
    overwrite one key (all KV heads) with a large component on dimension 0
    and its value with a one-hot on dimension r (the range's index), in the
    GPU pool and the oracle's pool alike.  fp8 pages are re-encoded around
    the planted row with a new (page, head) scale.  Returns the planted
    positions."""
    cfg, wl = dw.cfg, dw.wl
    ps, D = cfg.page_size, cfg.head_dim
    seq = wl.seqs[sid]
    planted = []
    for r, r0 in enumerate(range(0, upto, every)):
        j = r0 + int(rng.integers(0, min(every, upto - r0)))
        planted.append(j)
        page = int(seq.pages[j // ps])
        comp = int(st.page_map[page])
        slot = j % ps
        kvec = np.zeros(D, np.float32)
        kvec[0] = 16.0
        vvec = np.zeros(D, np.float32)
        vvec[r % D] = 1.0
        for name, vec in (("k", kvec), ("v", vvec)):
            host = getattr(st, f"pool_{name}")
            if cfg.kv_dtype == "fp8":
                scale = getattr(st, f"{name}_scale")
                valid = np.arange(ps) + (j // ps) * ps < seq.length
                for g in range(cfg.num_kv_heads):
                    vals = formats.e4m3_to_f64(host[comp, g]) * np.float64(scale[comp, g])
                    vals[slot] = vec
                    vals = vals[valid].astype(np.float32)
                    sc = np.float32(np.abs(vals).max() / 448.0)
                    host[comp, g, valid] = formats.fp8_quantize(vals, sc)
                    scale[comp, g] = sc
                gpu_scale = getattr(dw.pool, f"{name}_scale")
                gpu_scale[page] = torch.as_tensor(scale[comp], device="cuda")
                getattr(dw.pool, name)[page] = torch.as_tensor(host[comp], device="cuda")
            else:
                bits = formats.bf16_bits_from_f32(vec)
                host[comp, :, slot, :] = bits
                getattr(dw.pool, name)[page, :, slot, :] = (
                    torch.from_numpy(bits.view(np.int16)).to("cuda").view(torch.bfloat16))
    torch.cuda.synchronize()
    return planted


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
def test_every_key_partition_carries_weight(kv):
    """Long prefixes cut into many key partitions (prefill: 20 of 2048 keys
    for bf16, 32 of 2240 for fp8; decode: the library's split and 2048),
    with one planted key per 2048-key range whose score (~11 in natural
    units, against ~5 for the largest of the others) gives it ~5 % of the
    weight: each range adds ~0.05 on its own output dimension, so a lost
    partition, block or merge weight breaks even the absolute bounds."""
    from paper_2511_02230_amd.harness import DeviceWorkload

    if kv == "bf16":
        cfg, P, n = cfg_of("plant16", 8, 1, 128, 16, "bf16"), 40000, 64
    else:
        cfg, P, n = cfg_of("plant8", 16, 2, 128, 64, "fp8"), 70000, 32
    wl = workload.make_workload(cfg, prefill=[(P, n)], decode=[P + n])
    say(f"case planted keys kv={kv} P={P} n={n}")
    dw = DeviceWorkload(wl, "cuda")
    st = OracleState(wl, device="cuda")
    dw.append_prefill()
    dw.append_decode()
    torch.cuda.synchronize()
    st.append_prefill()
    st.append_decode()
    rng = np.random.default_rng([P, 17])
    planted = []
    for sid in range(len(wl.seqs)):
        planted = _plant_keys(dw, st, sid, P, rng)
    dw.q_prefill[..., 0] = 8.0
    dw.q_decode[..., 0] = 8.0
    torch.cuda.synchronize()
    nr = len(planted)
    pf, dc = wl.prefill, wl.decode
    ref = st.prefill(to_numpy(dw.q_prefill), st.rows_of(pf))[0]
    # every range carries weight in the oracle's output
    assert float(ref[..., :nr].min()) > 0.02, float(ref[..., :nr].min())
    got = out_f64(dw.run_prefill())
    check_close(got, ref, cfg, f"prefill P={P} n={n}, {nr} planted keys")
    ref_d = st.decode(to_numpy(dw.q_decode), st.rows_of(dc))[0]
    assert float(ref_d[..., :nr].min()) > 0.02
    for split in (0, 2048):
        got = out_f64(dw.run_decode(kv_split_len=split))
        check_close(got[0], ref_d, cfg, f"decode c={P + n} split {split}")


def test_fp8_quantizer_every_bf16_value():
    """kv_append's bf16 -> E4M3FN encoder on every finite bf16 bit pattern
    and three scales, against the oracle's encoder."""
    from paper_2511_02230_amd import ckv

    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    vals = formats.bf16_bits_to_f64(bits)
    bits = bits[~np.isnan(vals)]
    n_tok = -(-len(bits) // 128)
    pad = n_tok * 128 - len(bits)
    bits = np.concatenate([bits, np.zeros(pad, np.uint16)])
    x = torch.from_numpy(bits.view(np.int16).reshape(n_tok, 1, 128)).view(torch.bfloat16).cuda()
    for scale in (1.0, 0.37, 3.1e-3):
        npages = -(-n_tok // 64)
        k = torch.full((npages, 1, 64, 128), 0x7F, dtype=torch.uint8, device="cuda")
        v = torch.full_like(k, 0x7F)
        ks = torch.full((npages, 1), scale, dtype=torch.float32, device="cuda")
        pool = ckv.Pool(k, v, ks, ks.clone())
        bt = torch.arange(npages, dtype=torch.int32, device="cuda")[None]
        batch = ckv.Batch(bt, torch.zeros(1, dtype=torch.int32, device="cuda"),
                          torch.tensor([0, n_tok], dtype=torch.int32, device="cuda"), n_tok, n_tok, 0)
        ckv.kv_append(pool, batch, x, x)
        torch.cuda.synchronize()
        got = k.reshape(-1)[:n_tok * 128].cpu().numpy()
        ref = formats.fp8_quantize(formats.bf16_bits_to_f32(bits), np.float32(scale))
        bad = np.nonzero(got != ref)[0]
        assert bad.size == 0, (scale, bad[:5], bits[bad[:5]], got[bad[:5]], ref[bad[:5]])


@pytest.mark.parametrize("ps, which, value", [(16, "kv", 0.0), (64, "kv", 0.0), (16, "k", 0.0), (64, "v", 0.0),
                                              (16, "v", 1e-39), (64, "kv", 1e-39)])
def test_fp8_pages_with_zero_scale(ps, which, value):
    """A page of zeros carries scale 0 (its codes then decode to 0 whatever
    they hold); a page of tiny values a subnormal scale.  Such key or value
    scales on some pages of the sequences: prefill and decode still match
    the oracle, which decodes with the same scales."""
    from paper_2511_02230_amd.harness import DeviceWorkload

    cfg = cfg_of(f"z{ps}{which}{value}", 16, 2, 128, ps, "fp8")
    wl = workload.make_workload(cfg, prefill=[(300, 70), (0, 40)], decode=[200, 513])
    say(f"case scale {value} on some pages ps={ps} which={which}")
    dw = DeviceWorkload(wl, "cuda")
    sids = sorted(set(int(x) for x in wl.prefill.seq_ids) | set(int(x) for x in wl.decode.seq_ids))
    st = OracleState(wl, sids=sids, device="cuda")
    dw.append_prefill()
    dw.append_decode()
    torch.cuda.synchronize()
    st.append_prefill()
    st.append_decode()
    zero = st.pages[::3]  # every third page of the selected sequences, both KV heads
    for name in which:
        getattr(dw.pool, f"{name}_scale")[torch.as_tensor(zero, device="cuda")] = value
        getattr(st, f"{name}_scale")[st.page_map[zero]] = np.float32(value)
    torch.cuda.synchronize()
    pf, dc = wl.prefill, wl.decode
    got = out_f64(dw.run_prefill())
    ref = st.prefill(to_numpy(dw.q_prefill), st.rows_of(pf))
    for b, r in ref.items():
        check_close(got[pf.cu_q_lens[b]:pf.cu_q_lens[b + 1]], r, cfg, f"prefill seq {b}")
    ref = st.decode(to_numpy(dw.q_decode), st.rows_of(dc))
    for split in (0, 64):
        got = out_f64(dw.run_decode(kv_split_len=split))
        for b, r in ref.items():
            check_close(got[b], r, cfg, f"decode seq {b} split {split}")


GROW = [(128, "bf16", 16, [(700, 90), (0, 130)]), (64, "bf16", 64, [(700, 90), (0, 130)]),
        (256, "bf16", 16, [(700, 90), (0, 130)]), (128, "fp8", 16, [(700, 90), (0, 130)]),
        # few row tiles over a long prefix: key partitions, each with its own
        # reference maximum, merged afterwards
        (128, "bf16", 16, [(5000, 40)]), (128, "fp8", 64, [(5000, 40)])]


@pytest.mark.parametrize("d, kv, ps, prefill", GROW, ids=lambda c: str(c) if not isinstance(c, list) else f"P{c[0][0]}")
def test_scores_growing_along_the_keys(d, kv, ps, prefill):
    """Keys scaled by a factor that grows with their position, so that nearly
    every block's maximum exceeds the reference by more than the lazy-rescale
    slack: the kernels' reduced path (row maximum, rescale, moved fold) runs
    on most blocks instead of a few.  bf16 pools: row t of K times 1 + t / 32
    (rounded to bf16 in both pools); fp8 pools: the key scale of the
    sequence's i-th page times 1 + i."""
    from paper_2511_02230_amd.harness import DeviceWorkload

    cfg = cfg_of(f"grow{d}{kv}{ps}", 8, 2, d, ps, kv)
    wl = workload.make_workload(cfg, prefill=prefill, decode=[900, 70])
    say(f"case growing scores d={d} kv={kv} ps={ps} prefill={prefill}")
    dw = DeviceWorkload(wl, "cuda")
    sids = sorted(set(int(x) for x in wl.prefill.seq_ids) | set(int(x) for x in wl.decode.seq_ids))
    st = OracleState(wl, sids=sids, device="cuda")
    dw.append_prefill()
    dw.append_decode()
    torch.cuda.synchronize()
    st.append_prefill()
    st.append_decode()
    for sid in sids:
        pages = np.asarray(wl.seqs[sid].pages, np.int64)
        comp = st.page_map[pages]
        if kv == "fp8":
            f = (1.0 + np.arange(len(pages))).astype(np.float32)[:, None]
            st.k_scale[comp] = st.k_scale[comp] * f
            dw.pool.k_scale[torch.as_tensor(pages, device="cuda")] = torch.as_tensor(st.k_scale[comp], device="cuda")
        else:
            tok = np.arange(len(pages))[:, None] * ps + np.arange(ps)[None, :]  # [page, slot]
            f = (1.0 + tok / 32.0).astype(np.float32)[:, None, :, None]       # [page, 1, slot, 1]
            bits = formats.bf16_bits_from_f32(formats.bf16_bits_to_f32(st.pool_k[comp]) * f)
            st.pool_k[comp] = bits
            dw.pool.k[torch.as_tensor(pages, device="cuda")] = (
                torch.from_numpy(bits.view(np.int16)).to("cuda").view(torch.bfloat16))
    torch.cuda.synchronize()
    pf, dc = wl.prefill, wl.decode
    got = out_f64(dw.run_prefill())
    ref = st.prefill(to_numpy(dw.q_prefill), st.rows_of(pf))
    for b, r in ref.items():
        check_close(got[pf.cu_q_lens[b]:pf.cu_q_lens[b + 1]], r, cfg, f"prefill seq {b}")
    ref = st.decode(to_numpy(dw.q_decode), st.rows_of(dc))
    for split in (0, 128):
        got = out_f64(dw.run_decode(kv_split_len=split))
        for b, r in ref.items():
            check_close(got[b], r, cfg, f"decode seq {b} split {split}")


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
def test_loose_host_bounds(kv):
    """max_q_len and max_ctx_len are upper bounds: looser ones launch more
    row tiles and key partitions, the extra ones empty, and the results still
    match the oracle."""
    from paper_2511_02230_amd import ckv
    from paper_2511_02230_amd.harness import DeviceWorkload

    cfg = cfg_of(f"loose{kv}", 16, 2, 128, 16, kv)
    wl = workload.make_workload(cfg, prefill=[(300, 40), (20, 5)], decode=[100, 260])
    say(f"case loose bounds kv={kv}")
    dw = DeviceWorkload(wl, "cuda")
    sids = sorted(set(int(x) for x in wl.prefill.seq_ids) | set(int(x) for x in wl.decode.seq_ids))
    st = OracleState(wl, sids=sids, device="cuda")
    dw.append_prefill()
    dw.append_decode()
    torch.cuda.synchronize()
    st.append_prefill()
    st.append_decode()
    pf, dc = wl.prefill, wl.decode
    cap = int(dw.prefill.block_table.shape[1]) * cfg.page_size
    loose = dataclasses.replace(dw.prefill, max_q_len=min(cap, 3 * dw.prefill.max_q_len), max_ctx_len=cap)
    got = out_f64(ckv.prefix_prefill_attn(dw.pool, loose, dw.q_prefill, cfg.softmax_scale, 0))
    ref = st.prefill(to_numpy(dw.q_prefill), st.rows_of(pf))
    for b, r in ref.items():
        check_close(got[pf.cu_q_lens[b]:pf.cu_q_lens[b + 1]], r, cfg, f"prefill seq {b}")
    dcap = int(dw.decode.block_table.shape[1]) * cfg.page_size
    loose_d = dataclasses.replace(dw.decode, max_ctx_len=dcap)
    ref = st.decode(to_numpy(dw.q_decode), st.rows_of(dc))
    for split in (0, 64):
        got = out_f64(ckv.paged_decode_attn(dw.pool, loose_d, dw.q_decode, cfg.softmax_scale, 0, split))
        for b, r in ref.items():
            check_close(got[b], r, cfg, f"decode seq {b} split {split}")


def test_empty_and_degenerate_batches():
    from paper_2511_02230_amd import ckv

    cfg = cfg_of("deg", 8, 2, 128, 16, "bf16")
    wl = workload.make_workload(cfg, prefill=[(20, 0), (0, 1), (16, 16)], decode=[1])
    run_case(wl)
    # an empty launch is a no-op
    dw_pool = ckv.Pool(torch.zeros(1, 2, 16, 128, dtype=torch.bfloat16, device="cuda"),
                       torch.zeros(1, 2, 16, 128, dtype=torch.bfloat16, device="cuda"))
    empty = ckv.Batch(torch.zeros((0, 1), dtype=torch.int32, device="cuda"),
                      torch.zeros(0, dtype=torch.int32, device="cuda"),
                      torch.zeros(1, dtype=torch.int32, device="cuda"), 0, 0, 0)
    q = torch.zeros((0, 8, 128), dtype=torch.bfloat16, device="cuda")
    ckv.kv_append(dw_pool, empty, torch.zeros((0, 2, 128), dtype=torch.bfloat16, device="cuda"),
                  torch.zeros((0, 2, 128), dtype=torch.bfloat16, device="cuda"))
    ckv.prefix_prefill_attn(dw_pool, empty, q, 0.1)
    torch.cuda.synchronize()


# ------------------------------------------------- mixed prefill + decode

MIXED = [
    (cfg_of("m1", 32, 8, 128, 16, "bf16"), [(300, 70), (0, 200), (1000, 33)], [1, 700, 2049, 64], 0),
    (cfg_of("m2", 48, 4, 128, 64, "fp8"), [(500, 40), (64, 64)], [200, 3000, 65], 0),
    (cfg_of("m3", 16, 8, 256, 16, "bf16"), [(100, 60), (1500, 40)], [300, 1200], 17),
    (cfg_of("m4", 8, 2, 64, 16, "bf16"), [(40, 30)], [90, 3, 17], 0),
    # a prefill batch small enough to split its keys into partitions
    (cfg_of("m5", 8, 1, 128, 16, "bf16"), [(6000, 64)], [6100, 100], 0),
    # one of the two batches empty
    (cfg_of("m6", 16, 2, 128, 16, "bf16"), [(200, 50)], [], 0),
    (cfg_of("m7", 16, 2, 128, 16, "bf16"), [], [300, 5], 0),
]


@pytest.mark.parametrize("case", MIXED, ids=lambda c: c[0].name)
def test_mixed_launch_equals_the_separate_calls(case):
    """mixed_attn returns the separate calls' bits for every interleaving of
    the two kinds of work, and those match the oracle.  (The decode batches
    here are small enough that the mixed launch's own partition length, the
    decode's capped at 2048 keys, is the decode's.)"""
    from paper_2511_02230_amd import ckv
    from paper_2511_02230_amd.harness import DeviceWorkload

    cfg, pf, dc, w = case
    wl = workload.make_workload(cfg, prefill=pf, decode=dc)
    say(f"case mixed {cfg.name} prefill={pf} decode={dc} W={w}")
    dw = DeviceWorkload(wl, "cuda", window=w)
    st = OracleState(wl, device="cuda")
    if wl.prefill.num_seqs:
        dw.append_prefill()
        st.append_prefill()
    if wl.decode.num_seqs:
        dw.append_decode()
        st.append_decode()
    torch.cuda.synchronize()
    H, D = cfg.num_q_heads, cfg.head_dim
    qp = dw.q_prefill if wl.prefill.num_seqs else torch.empty((0, H, D), dtype=torch.bfloat16, device="cuda")
    qd = dw.q_decode if wl.decode.num_seqs else torch.empty((0, H, D), dtype=torch.bfloat16, device="cuda")
    empty = ckv.Batch(torch.zeros((0, 1), dtype=torch.int32, device="cuda"),
                      torch.zeros(0, dtype=torch.int32, device="cuda"),
                      torch.zeros(1, dtype=torch.int32, device="cuda"), 0, 0, 0)
    pbatch = dw.prefill if wl.prefill.num_seqs else empty
    dbatch = dw.decode if wl.decode.num_seqs else empty
    for split in (0, 128):
        ref_p = dw.run_prefill().clone() if wl.prefill.num_seqs else None
        ref_d = dw.run_decode(kv_split_len=split).clone() if wl.decode.num_seqs else None
        for inter in (0, 1, 2, 5, 32, 1000):
            op, od = ckv.mixed_attn(dw.pool, pbatch, qp, dbatch, qd, cfg.softmax_scale, w, split, inter)
            torch.cuda.synchronize()
            if ref_p is not None:
                assert torch.equal(op.view(torch.int16), ref_p.view(torch.int16)), (split, inter)
            if ref_d is not None:
                assert torch.equal(od.view(torch.int16), ref_d.view(torch.int16)), (split, inter)
        if ref_p is not None:
            ref = st.prefill(to_numpy(dw.q_prefill), st.rows_of(wl.prefill), w)
            got = out_f64(op)
            cu = wl.prefill.cu_q_lens
            for b, r in ref.items():
                check_close(got[cu[b]:cu[b + 1]], r, cfg, f"mixed prefill seq {b}")
        if ref_d is not None:
            ref = st.decode(to_numpy(dw.q_decode), st.rows_of(wl.decode), w)
            got = out_f64(od)
            for b, r in ref.items():
                check_close(got[b], r, cfg, f"mixed decode seq {b} split {split}")


def _empty_batch(ckv):
    return ckv.Batch(torch.zeros((0, 1), dtype=torch.int32, device="cuda"),
                     torch.zeros(0, dtype=torch.int32, device="cuda"),
                     torch.zeros(1, dtype=torch.int32, device="cuda"), 0, 0, 0)


def _pools_equal(a, b):
    return (torch.equal(a.pool.k.view(torch.int16), b.pool.k.view(torch.int16))
            and torch.equal(a.pool.v.view(torch.int16), b.pool.v.view(torch.int16)))


MIXED_APPEND = [c for c in MIXED if c[0].kv_dtype == "bf16"] + [
    # one query head per KV head: a tile owns 128 tokens, more rows than one
    # batch of the workgroup's copy
    (cfg_of("a1", 2, 2, 128, 16, "bf16"), [(100, 300), (0, 129)], [5, 1], 0),
    (cfg_of("a2", 4, 2, 256, 64, "bf16"), [(70, 150), (0, 1)], [64, 65], 0),
    # key partitions under a window: partition 0 of the late tiles is empty,
    # and its workgroup still writes its tokens
    (cfg_of("a3", 8, 1, 128, 16, "bf16"), [(6000, 64)], [6100, 100], 100),
]


@pytest.mark.parametrize("case", MIXED_APPEND, ids=lambda c: c[0].name)
def test_mixed_launch_with_the_append_fused(case):
    """Given the new K/V rows, mixed_attn leaves the whole pool exactly as
    kv_append does (every other slot keeps its poison) and returns the bits
    of the same launch over the appended pool, for the rows of both batches
    at once or of one batch (the other appended beforehand), at several
    interleavings; outputs within the bars of the oracle."""
    from paper_2511_02230_amd import ckv
    from paper_2511_02230_amd.harness import DeviceWorkload

    cfg, pf, dc, w = case
    wl = workload.make_workload(cfg, prefill=pf, decode=dc)
    say(f"case mixed+append {cfg.name} prefill={pf} decode={dc} W={w}")
    H, D = cfg.num_q_heads, cfg.head_dim
    has_p, has_d = wl.prefill.num_seqs > 0, wl.decode.num_seqs > 0
    ref = DeviceWorkload(wl, "cuda", window=w)
    if has_p:
        ref.append_prefill()
    if has_d:
        ref.append_decode()
    empty = _empty_batch(ckv)
    qp = ref.q_prefill if has_p else torch.empty((0, H, D), dtype=torch.bfloat16, device="cuda")
    qd = ref.q_decode if has_d else torch.empty((0, H, D), dtype=torch.bfloat16, device="cuda")
    pbatch = ref.prefill if has_p else empty
    dbatch = ref.decode if has_d else empty
    rp, rd = ckv.mixed_attn(ref.pool, pbatch, qp, dbatch, qd, cfg.softmax_scale, w)
    torch.cuda.synchronize()
    for mode in ("both", "prefill", "decode"):
        dw = DeviceWorkload(wl, "cuda", window=w)
        fuse_p, fuse_d = has_p and mode != "decode", has_d and mode != "prefill"
        if has_p and not fuse_p:
            dw.append_prefill()
        if has_d and not fuse_d:
            dw.append_decode()
        rows = dict(k_prefill=dw.k_new if fuse_p else None, v_prefill=dw.v_new if fuse_p else None,
                    k_decode=dw.k_dec if fuse_d else None, v_decode=dw.v_dec if fuse_d else None)
        for inter in (0, 1, 32):
            op, od = ckv.mixed_attn(dw.pool, dw.prefill if has_p else empty, dw.q_prefill if has_p else qp,
                                    dw.decode if has_d else empty, dw.q_decode if has_d else qd,
                                    cfg.softmax_scale, w, 0, inter, **rows)
            torch.cuda.synchronize()
            assert _pools_equal(dw, ref), (mode, inter)
            if has_p:
                assert torch.equal(op.view(torch.int16), rp.view(torch.int16)), (mode, inter)
            if has_d:
                assert torch.equal(od.view(torch.int16), rd.view(torch.int16)), (mode, inter)
        del dw
    st = OracleState(wl, device="cuda")
    if has_p:
        st.append_prefill()
        ref_o = st.prefill(to_numpy(ref.q_prefill), st.rows_of(wl.prefill), w)
        got = out_f64(op)
        cu = wl.prefill.cu_q_lens
        for b, r in ref_o.items():
            check_close(got[cu[b]:cu[b + 1]], r, cfg, f"fused-append prefill seq {b}")
    if has_d:
        st.append_decode()
        ref_o = st.decode(to_numpy(ref.q_decode), st.rows_of(wl.decode), w)
        got = out_f64(od)
        for b, r in ref_o.items():
            check_close(got[b], r, cfg, f"fused-append decode seq {b}")


def test_mixed_launch_with_the_append_fused_full_config():
    """The benchmark's whole Llama-3.1-70B step in one launch: the pool and
    both outputs equal kv_append x2 followed by mixed_attn, bit for bit."""
    from paper_2511_02230_amd import ckv
    from paper_2511_02230_amd.harness import DeviceWorkload

    cfg = workload.CONFIGS["llama3.1-70b"]
    wl = workload.make_workload(cfg)
    say("case mixed+append full llama3.1-70b")
    ref = DeviceWorkload(wl, "cuda")
    ref.append_prefill()
    ref.append_decode()
    rp, rd = ckv.mixed_attn(ref.pool, ref.prefill, ref.q_prefill, ref.decode, ref.q_decode, cfg.softmax_scale)
    torch.cuda.synchronize()
    dw = DeviceWorkload(wl, "cuda")
    op, od = ckv.mixed_attn(dw.pool, dw.prefill, dw.q_prefill, dw.decode, dw.q_decode, cfg.softmax_scale,
                            k_prefill=dw.k_new, v_prefill=dw.v_new, k_decode=dw.k_dec, v_decode=dw.v_dec)
    torch.cuda.synchronize()
    assert _pools_equal(dw, ref)
    assert torch.equal(op.view(torch.int16), rp.view(torch.int16))
    assert torch.equal(od.view(torch.int16), rd.view(torch.int16))


@pytest.mark.parametrize("name", ["llama3.1-70b", "glm4.5-355b"])
def test_mixed_launch_full_config(name):
    """The benchmark's mixed step at full size (decode partitions of 2048
    keys, the mixed launch's own choice there): bit-identical to the
    separate calls at that length, and sampled rows within the bars of the
    oracle."""
    from paper_2511_02230_amd import ckv
    from paper_2511_02230_amd.harness import DeviceWorkload

    cfg = workload.CONFIGS[name]
    wl = workload.make_workload(cfg)
    rng = np.random.default_rng([cfg.seed, 0, 11])
    pf_rows, dc_rows, subsets = _sample_rows(wl, rng)
    say(f"case mixed full {name}")
    dw = DeviceWorkload(wl, "cuda")
    dw.append_prefill()
    dw.append_decode()
    ref_p = dw.run_prefill().clone()
    ref_d = dw.run_decode(kv_split_len=2048).clone()
    op, od = ckv.mixed_attn(dw.pool, dw.prefill, dw.q_prefill, dw.decode, dw.q_decode, cfg.softmax_scale)
    torch.cuda.synchronize()
    assert torch.equal(op.view(torch.int16), ref_p.view(torch.int16))
    assert torch.equal(od.view(torch.int16), ref_d.view(torch.int16))
    op2, od2 = ckv.mixed_attn(dw.pool, dw.prefill, dw.q_prefill, dw.decode, dw.q_decode, cfg.softmax_scale,
                              kv_split_len=2048, interleave=32)
    torch.cuda.synchronize()
    assert torch.equal(op2.view(torch.int16), ref_p.view(torch.int16))
    assert torch.equal(od2.view(torch.int16), ref_d.view(torch.int16))
    sids = sorted(set(int(wl.prefill.seq_ids[b]) for b in pf_rows) | set(int(wl.decode.seq_ids[b]) for b in dc_rows))
    st = OracleState(wl, sids=sids, device="cuda")
    st.append_prefill(pf_rows)
    st.append_decode(dc_rows)
    ref = st.prefill(to_numpy(dw.q_prefill), [b for b in pf_rows if b in st.rows_of(wl.prefill)], 0, subsets)
    got = out_f64(op)
    cu = wl.prefill.cu_q_lens
    for b, r in ref.items():
        check_close(got[cu[b] + subsets[b]], r, cfg, f"mixed prefill seq {b}")
    ref = st.decode(to_numpy(dw.q_decode), st.rows_of(wl.decode, dc_rows))
    got = out_f64(od)
    for b, r in ref.items():
        check_close(got[b], r, cfg, f"mixed decode seq {b}")
