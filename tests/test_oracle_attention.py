"""Pins of the fp64 attention oracle (CPU only).

Each test ties the oracle to something other than itself: hand-derived
closed forms (tests/golden), a pure-Python brute force with explicit page
walks, torch's scaled_dot_product_attention in float64, and invariants the
definition implies (prefix reuse equals the tail of a full recomputation,
page placement does not matter, decode is a one-row prefill, GQA equals MHA
with repeated KV heads, split-and-merge of the softmax equals the whole).
"""
import json
import os

import numpy as np
import pytest
import torch

from oracle import brute, paged

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def dense_to_pool(k, v, page_size, rng, extra_pages=3):
    """Scatter dense [L, H, D] K/V into a float64 pool at random pages;
    unused slots hold NaN.  Returns pool_k, pool_v, block-table row."""
    L, H, D = k.shape
    npg = -(-L // page_size)
    num_pages = npg + extra_pages
    pages = rng.permutation(num_pages)[:npg].astype(np.int32)
    pk = np.full((num_pages, H, page_size, D), np.nan)
    pv = np.full((num_pages, H, page_size, D), np.nan)
    j = np.arange(L)
    pk[pages[j // page_size], :, j % page_size, :] = k
    pv[pages[j // page_size], :, j % page_size, :] = v
    return pk, pv, pages


def pool_f32(pk):
    return pk.astype(np.float32)


def run_prefill(q, pk, pv, bt, P, n, ps, scale, window):
    return paged.prefix_prefill(q, pk, pv, bt, np.array(P), np.array(n), page_size=ps,
                                kv_dtype="f32", softmax_scale=scale, window=window)


@pytest.mark.parametrize("case", json.load(open(os.path.join(GOLD, "attention_closed_forms.json")))["cases"],
                         ids=lambda c: c["name"])
def test_golden_closed_forms(case):
    k = np.array(case["k"], np.float64)[:, None, :]
    v = np.array(case["v"], np.float64)[:, None, :]
    q = np.array(case["q"], np.float64)[None, None, :]
    i = case["q_pos"]
    out = paged.attend(q, np.array([i]), k[:i + 1], v[:i + 1], case["scale"], case["window"])
    assert np.allclose(out[0, 0], case["out"], rtol=0, atol=1e-13)
    # the same through a paged pool and the prefill entry (P = i, n = 1)
    rng = np.random.default_rng(0)
    pk, pv, pages = dense_to_pool(k[:i + 1], v[:i + 1], case["page_size"], rng)
    o2 = run_prefill(q, pk, pv, pages[None], [i], [1], case["page_size"], case["scale"], case["window"])
    # an f32 pool stores the logs of the weights rounded to binary32
    assert np.allclose(o2[0, 0], case["out"], rtol=0, atol=1e-6)


def _random_case(rng):
    Hkv = int(rng.choice([1, 2]))
    Hq = Hkv * int(rng.choice([1, 2, 4]))
    D = int(rng.choice([4, 8, 64]))
    ps = int(rng.choice([1, 2, 16]))
    B = int(rng.integers(1, 3))
    P = [int(rng.integers(0, 41)) for _ in range(B)]
    n = [int(rng.integers(1, 9)) for _ in range(B)]
    W = int(rng.choice([0, 1, 3, 17]))
    return Hq, Hkv, D, ps, P, n, W


@pytest.mark.parametrize("seed", range(12))
def test_oracle_matches_brute_force(seed):
    rng = np.random.default_rng(100 + seed)
    Hq, Hkv, D, ps, P, n, W = _random_case(rng)
    B = len(P)
    lens = [p + m for p, m in zip(P, n)]
    npg = [-(-L // ps) for L in lens]
    num_pages = sum(npg) + 2
    perm = rng.permutation(num_pages).astype(np.int32)
    bt = np.zeros((B, max(npg)), np.int32)
    off = 0
    for b in range(B):
        bt[b, :npg[b]] = perm[off:off + npg[b]]
        off += npg[b]
    pk = rng.standard_normal((num_pages, Hkv, ps, D)).astype(np.float32)
    pv = rng.standard_normal((num_pages, Hkv, ps, D)).astype(np.float32)
    q = rng.standard_normal((sum(n), Hq, D)).astype(np.float32)
    scale = 1.0 / np.sqrt(D)
    out = paged.prefix_prefill(q, pk, pv, bt, np.array(P), np.array(n), page_size=ps, kv_dtype="f32",
                               softmax_scale=scale, window=W)
    ref = brute.prefill(q.astype(np.float64).tolist(), pk.astype(np.float64).tolist(),
                        pv.astype(np.float64).tolist(), bt.tolist(), P, n, ps, scale, W)
    assert np.max(np.abs(out - np.array(ref))) <= 1e-12


def test_oracle_matches_brute_force_tiny_config():
    import workload
    from tests.oracle_inputs import OracleState, q_to_f64, to_numpy

    wl = workload.make_workload(workload.TINY)
    st = OracleState(wl)
    st.append_prefill()
    q = to_numpy(workload.concat_rows(wl.prefill, lambda b: workload.prefill_q(wl, b)))
    pf = wl.prefill
    bt = st.table(pf, [0])
    out = paged.prefix_prefill(q, st.pool_k, st.pool_v, bt, pf.ctx_lens, pf.q_lens,
                               page_size=16, kv_dtype="f32", softmax_scale=0.125)
    rows = [0, 7, 15]
    sel_q = q_to_f64(q, "f32")[rows]
    ref = brute.prefill(sel_q.tolist(), st.pool_k.astype(np.float64).tolist(),
                        st.pool_v.astype(np.float64).tolist(), [bt[0].tolist()] * 3,
                        [240 + r for r in rows], [1, 1, 1], 16, 0.125)
    assert np.max(np.abs(out[rows] - np.array(ref))) <= 1e-12


@pytest.mark.parametrize("W", [0, 5, 64])
def test_oracle_matches_torch_sdpa(W):
    rng = np.random.default_rng(7)
    Hq, Hkv, D, L, n = 8, 2, 32, 100, 20
    P = L - n
    k = rng.standard_normal((L, Hkv, D))
    v = rng.standard_normal((L, Hkv, D))
    q = rng.standard_normal((n, Hq, D))
    scale = 0.3
    out = paged.attend(q, P + np.arange(n), k, v, scale, W)
    G = Hq // Hkv
    kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(G, 0)[None]
    vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(G, 0)[None]
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]
    i = torch.arange(n)[:, None] + P
    j = torch.arange(L)[None, :]
    mask = j <= i
    if W:
        mask &= (i - j) < W
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=scale)
    ref = ref[0].permute(1, 0, 2).numpy()
    assert np.max(np.abs(out - ref)) <= 1e-12


def _dense_case(rng, L=77, Hq=4, Hkv=2, D=16):
    return (rng.standard_normal((L, Hkv, D)), rng.standard_normal((L, Hkv, D)),
            rng.standard_normal((L, Hq, D)))


@pytest.mark.parametrize("W", [0, 9])
def test_prefix_reuse_equals_tail_of_full_recompute(W):
    rng = np.random.default_rng(3)
    k, v, qall = _dense_case(rng)
    L = k.shape[0]
    ps = 4
    pk, pv, pages = dense_to_pool(k, v, ps, rng)
    for P in [0, 1, 30, 76]:
        n = L - P
        full = run_prefill(qall, pk, pv, pages[None], [0], [L], ps, 0.25, W)
        reuse = run_prefill(qall[P:], pk, pv, pages[None], [P], [n], ps, 0.25, W)
        assert np.max(np.abs(reuse - full[P:])) <= 1e-12


def test_page_shuffle_invariance():
    rng = np.random.default_rng(4)
    k, v, q = _dense_case(rng, L=50)
    ps = 8
    pk, pv, pages = dense_to_pool(k, v, ps, rng, extra_pages=5)
    a = run_prefill(q[40:], pk, pv, pages[None], [40], [10], ps, 0.2, 0)
    # move every page to a new physical slot and rewrite the block table
    perm = rng.permutation(pk.shape[0])
    pk2 = np.empty_like(pk)
    pv2 = np.empty_like(pv)
    pk2[perm] = pk
    pv2[perm] = pv
    b = run_prefill(q[40:], pk2, pv2, perm[pages][None], [40], [10], ps, 0.2, 0)
    assert np.array_equal(a, b)


def test_decode_equals_one_row_prefill():
    rng = np.random.default_rng(5)
    k, v, q = _dense_case(rng, L=61)
    ps = 16
    pk, pv, pages = dense_to_pool(k, v, ps, rng)
    for W in (0, 7):
        for c in (1, 16, 17, 61):
            d = paged.paged_decode(q[c - 1:c], pk, pv, pages[None], np.array([c]), page_size=ps,
                                   kv_dtype="f32", softmax_scale=0.5, window=W)
            p = run_prefill(q[c - 1:c], pk, pv, pages[None], [c - 1], [1], ps, 0.5, W)
            assert np.max(np.abs(d - p)) == 0.0


def test_gqa_equals_mha_with_repeated_kv():
    rng = np.random.default_rng(6)
    k, v, q = _dense_case(rng, L=40, Hq=8, Hkv=2)
    pos = np.arange(30, 40)
    gqa = paged.attend(q[30:], pos, k, v, 0.3, 0)
    mha = paged.attend(q[30:], pos, np.repeat(k, 4, axis=1), np.repeat(v, 4, axis=1), 0.3, 0)
    assert np.max(np.abs(gqa - mha)) == 0.0
    # and head h really reads KV head h // G (a transposed mapping would differ)
    wrong = paged.attend(q[30:], pos, np.tile(k, (1, 4, 1)), np.tile(v, (1, 4, 1)), 0.3, 0)
    assert np.max(np.abs(gqa - wrong)) > 1e-3


def test_uniform_weights_give_mean_of_visible_values():
    rng = np.random.default_rng(8)
    k, v, q = _dense_case(rng, L=33)
    q0 = np.zeros((3, 4, 16))
    pos = np.array([0, 10, 32])
    out = paged.attend(q0, pos, k, v, 1.0, 0)
    for r, i in enumerate(pos):
        for h in range(4):
            assert np.allclose(out[r, h], v[:i + 1, h // 2].mean(axis=0), atol=1e-13)
    # identical keys: any q gives the same mean
    kk = np.repeat(k[:1], 33, axis=0)
    out2 = paged.attend(q[:3], pos, kk, v, 1.0, 4)
    for r, i in enumerate(pos):
        lo = max(0, i - 3)
        for h in range(4):
            assert np.allclose(out2[r, h], v[lo:i + 1, h // 2].mean(axis=0), atol=1e-13)


def test_single_key_and_window_one():
    rng = np.random.default_rng(9)
    k, v, q = _dense_case(rng, L=20)
    out = paged.attend(q[:1], np.array([0]), k, v, 1.0, 0)
    assert np.array_equal(out[0], np.repeat(v[0], 2, axis=0).reshape(4, 16))
    out1 = paged.attend(q, np.arange(20), k, v, 1.0, 1)
    assert np.array_equal(out1, np.repeat(v, 2, axis=1))


def test_large_window_equals_global():
    rng = np.random.default_rng(10)
    k, v, q = _dense_case(rng, L=45)
    pos = np.arange(30, 45)
    a = paged.attend(q[30:], pos, k, v, 0.4, 0)
    b = paged.attend(q[30:], pos, k, v, 0.4, 45)
    assert np.array_equal(a, b)
    c = paged.attend(q[30:], pos, k, v, 0.4, 44)  # the first row still sees all 31
    assert np.array_equal(a[:1], c[:1]) and np.max(np.abs(a[-1] - c[-1])) > 0


@pytest.mark.parametrize("W", [0, 11])
def test_lse_merge_of_any_partition(W):
    rng = np.random.default_rng(12)
    k, v, q = _dense_case(rng, L=64)
    i = 63
    whole = paged.attend(q[i:i + 1], np.array([i]), k, v, 0.35, W)[0]
    for cuts in ([32], [5, 17, 40], [1, 2, 3, 62], [63]):
        edges = [0] + cuts + [64]
        parts = [paged.partial(q[i], i, k, v, 0.35, W, np.arange(a, b)) for a, b in zip(edges, edges[1:])]
        merged = paged.lse_merge(parts)
        assert np.max(np.abs(merged - whole)) <= 1e-12


def test_append_touches_only_addressed_slots():
    rng = np.random.default_rng(13)
    ps, H, D = 4, 2, 3
    pool = rng.standard_normal((9, H, ps, D)).astype(np.float32)
    before = pool.copy()
    bt = np.array([[3, 7, 1, 0], [5, 2, 8, 6]], np.int32)
    ctx = np.array([2, 7])
    n = np.array([5, 3])
    new = rng.standard_normal((8, H, D)).astype(np.float32)
    paged.append(pool, bt, ctx, n, new, page_size=ps, kv_dtype="f32", in_dtype="f32")
    expect = before.copy()
    r = 0
    for b in range(2):  # slot-by-slot restatement
        for t in range(n[b]):
            pos = ctx[b] + t
            for h in range(H):
                expect[bt[b][pos // ps], h, pos % ps, :] = new[r, h]
            r += 1
    assert np.array_equal(pool.view(np.uint32), expect.view(np.uint32))
    assert np.count_nonzero((pool != before).any(axis=3)) == 8 * H


def test_fp8_pool_decodes_with_page_head_scale():
    from oracle import formats

    rng = np.random.default_rng(14)
    ps, H, D = 2, 2, 4
    x = rng.standard_normal((3, H, D)).astype(np.float32)
    xb = formats.bf16_bits_from_f32(x)
    scale = np.array([[0.5, 2.0], [0.25, 1.0], [4.0, 8.0]], np.float32)
    pool = np.zeros((3, H, ps, D), np.uint8)
    bt = np.array([[2, 0]], np.int32)
    paged.append(pool, bt, np.array([0]), np.array([3]), xb, page_size=ps, kv_dtype="fp8",
                 in_dtype="bf16", scale=scale)
    got = paged.gather(pool, bt[0], 3, page_size=ps, kv_dtype="fp8", scale=scale)
    xv = formats.bf16_bits_to_f64(xb)
    for j in range(3):
        page = bt[0][j // ps]
        for h in range(H):
            code = formats.fp8_quantize(np.float32(xv[j, h, 0]), scale[page, h])
            assert got[j, h, 0] == formats.E4M3_TABLE[code] * float(scale[page, h])
    # relative error of the encode/decode round trip is bounded by 2^-4 for normals
    rel = np.abs(got - xv) / np.maximum(np.abs(xv), 1e-30)
    big = np.abs(xv) / scale[bt[0][np.arange(3) // ps]][:, :, None] >= 2 ** -6
    assert np.all(rel[big] <= 2 ** -4)
