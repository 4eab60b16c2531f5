"""Plain fp64 oracle of the paged-KV hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this.

What is computed (Continuum keeps a finished request's KV blocks resident,
Sec. 5.2 "Request Pinning", so the next turn's prefill only has to cover the
new tokens and reuses the retained pages, Sec. 1 and Sec. 5.2 "Offline
Profile"):

  append   every new-turn token t of sequence b lands at absolute position
           pos = P_b + t, i.e. in physical page bt[b][pos // ps] at slot
           pos % ps, head by head; nothing else in the pool changes.
  prefill  new-turn row t of head h (absolute position i = P_b + t) attends,
           with scaled dot-product softmax attention, to the keys j of its
           sequence with j <= i (and i - j < W for a window W > 0), read
           through the block table; query head h uses KV head h // G.
  decode   the same for one query at position c_b - 1 over c_b tokens.
  offload / reload
           whole pages copied to host memory and back, bit for bit, when
           CPU offloading is on (an evicted request's cache returns without
           a new prefill, Sec. 1 and Sec. 3.2).

The pool is [num_pages, H_kv, page_size, D] for K and for V, stored as
float32, bfloat16 bit patterns (uint16) or E4M3FN codes (uint8) with one
fp32 scale per (page, head).  Every value is decoded exactly to float64 and
the softmax is evaluated directly from its definition, per KV head, on the
gathered dense rows (no key tiling, no running maximum).
"""
from __future__ import annotations

import numpy as np

from . import formats

POOL_NP_DTYPE = {"f32": np.float32, "bf16": np.uint16, "fp8": np.uint8}


# --------------------------------------------------------------- append

def encode(x, kv_dtype: str, in_dtype: str, scale=None) -> np.ndarray:
    """Pool representation of raw values x.

    f32 -> f32 and bf16 -> bf16 are bit copies; bf16 -> fp8 divides by the
    (page, head) scale in binary32, clamps to +-448 and rounds to E4M3FN.
    x is float32 (f32 input) or uint16 bf16 bit patterns (bf16 input)."""
    if kv_dtype == in_dtype:
        return np.array(x, copy=True)
    if kv_dtype == "fp8" and in_dtype == "bf16":
        xf = formats.bf16_bits_to_f32(x)
        return formats.fp8_quantize(xf, scale)
    raise ValueError(f"unsupported encode {in_dtype} -> {kv_dtype}")


def append(pool, block_table, ctx_lens, q_lens, new, *, page_size, kv_dtype,
           in_dtype, scale=None):
    """Write new[cu_b + t, h, :] for t < q_lens[b] into the pool (in place).

    pool [num_pages, H, ps, D]; new [sum(q_lens), H, D]; scale [num_pages, H]
    (fp8 only).  Rows of the packed input follow the order of the batch."""
    cu = 0
    for b in range(len(q_lens)):
        n = int(q_lens[b])
        if n == 0:
            continue
        pos = int(ctx_lens[b]) + np.arange(n)
        pages = np.asarray(block_table[b])[pos // page_size]
        slots = pos % page_size
        rows = new[cu:cu + n]  # [n, H, D]
        sc = None
        if kv_dtype == "fp8":
            sc = np.asarray(scale)[pages][:, :, None]  # [n, H, 1]
        pool[pages, :, slots, :] = encode(rows, kv_dtype, in_dtype, sc)
        cu += n


# --------------------------------------------------------------- gather

def decode_values(stored, kv_dtype: str, scale=None) -> np.ndarray:
    """Exact float64 value of stored pool elements (scale broadcast by the
    caller for fp8)."""
    if kv_dtype == "f32":
        return np.asarray(stored, dtype=np.float32).astype(np.float64)
    if kv_dtype == "bf16":
        return formats.bf16_bits_to_f64(stored)
    if kv_dtype == "fp8":
        return formats.e4m3_to_f64(stored) * np.asarray(scale, dtype=np.float32).astype(np.float64)
    raise ValueError(kv_dtype)


def gather(pool, block_table_row, length: int, *, page_size, kv_dtype, scale=None):
    """Dense float64 [length, H, D] view of one sequence's tokens 0..length-1
    read through its block table."""
    j = np.arange(length)
    pages = np.asarray(block_table_row)[j // page_size]
    slots = j % page_size
    stored = pool[pages, :, slots, :]  # [L, H, D]
    sc = None
    if kv_dtype == "fp8":
        sc = np.asarray(scale)[pages][:, :, None]
    return decode_values(stored, kv_dtype, sc)


# ------------------------------------------------------------ attention

def visible(i, j, window: int):
    """Key j is visible to the query at absolute position i iff j <= i and,
    for a window W > 0, i - j < W (the query sees exactly W keys, itself
    included).

    Parity unpinned for the window edge: the paper has no sliding-window
    layer at all (the window comes from the Gemma-3 layer shapes this path
    is sized for), so "exactly W keys, self included" is a declared
    convention; the tests pin everything around it (W >= context equals
    global attention, W = 1 sees only itself) but not the edge itself."""
    ok = j <= i
    if window > 0:
        ok = ok & (i - j < window)
    return ok


def attend(q, pos, k, v, softmax_scale: float, window: int = 0, row_chunk=None):
    """softmax(scale * q k^T over visible keys) v, in float64.

    q [R, H_q, D], pos [R] absolute positions, k, v [L, H_kv, D];
    query head h reads KV head h // (H_q / H_kv).  Returns [R, H_q, D]."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    R, Hq, D = q.shape
    L, Hkv, _ = k.shape
    G = Hq // Hkv
    pos = np.asarray(pos, dtype=np.int64)
    out = np.empty((R, Hq, D), dtype=np.float64)
    if R == 0:
        return out
    if row_chunk is None:
        row_chunk = max(1, (1 << 24) // max(1, L * G))
    j = np.arange(L)
    for g in range(Hkv):
        kg = k[:, g, :]
        vg = v[:, g, :]
        for r0 in range(0, R, row_chunk):
            r1 = min(R, r0 + row_chunk)
            qg = q[r0:r1, g * G:(g + 1) * G, :].reshape(-1, D)  # [(r, hh), D]
            s = softmax_scale * (qg @ kg.T)  # [(r, hh), L]
            mask = visible(pos[r0:r1, None], j[None, :], window)  # [r, L]
            mask = np.repeat(mask, G, axis=0)
            s = np.where(mask, s, -np.inf)
            m = s.max(axis=1, keepdims=True)
            e = np.exp(s - m)
            o = (e @ vg) / e.sum(axis=1, keepdims=True)
            out[r0:r1, g * G:(g + 1) * G, :] = o.reshape(r1 - r0, G, D)
    return out


def prefix_prefill(q, pool_k, pool_v, block_table, ctx_lens, q_lens, *, page_size,
                   kv_dtype, softmax_scale, window=0, k_scale=None, v_scale=None,
                   rows=None):
    """Prefix-reuse prefill.  q [sum n_b, H_q, D] packed by row order.

    rows: optional {b: array of t} to evaluate only those new-turn rows
    (sampled checks); returns {b: [len(t), H_q, D]} then, else the packed
    [sum n_b, H_q, D] output."""
    q = np.asarray(q)
    cu = np.concatenate([[0], np.cumsum(np.asarray(q_lens, dtype=np.int64))])
    outs = {}
    for b in range(len(q_lens)):
        n = int(q_lens[b])
        if n == 0 or (rows is not None and b not in rows):
            continue
        P = int(ctx_lens[b])
        t = np.arange(n) if rows is None else np.asarray(rows[b], dtype=np.int64)
        L = P + int(t.max()) + 1
        k = gather(pool_k, block_table[b], L, page_size=page_size, kv_dtype=kv_dtype, scale=k_scale)
        vv = gather(pool_v, block_table[b], L, page_size=page_size, kv_dtype=kv_dtype, scale=v_scale)
        outs[b] = attend(q[cu[b] + t], P + t, k, vv, softmax_scale, window)
    if rows is not None:
        return outs
    total = int(cu[-1])
    Hq, D = q.shape[1], q.shape[2]
    out = np.zeros((total, Hq, D), dtype=np.float64)
    for b, o in outs.items():
        out[cu[b]:cu[b + 1]] = o
    return out


def paged_decode(q, pool_k, pool_v, block_table, context_lens, *, page_size, kv_dtype,
                 softmax_scale, window=0, k_scale=None, v_scale=None, rows=None):
    """Decode: q [B, H_q, D]; row b attends at position c_b - 1 over its
    c_b = context_lens[b] tokens.  rows: optional iterable of b to evaluate
    (others left as NaN)."""
    q = np.asarray(q)
    B, Hq, D = q.shape
    out = np.full((B, Hq, D), np.nan, dtype=np.float64)
    sel = range(B) if rows is None else rows
    for b in sel:
        c = int(context_lens[b])
        k = gather(pool_k, block_table[b], c, page_size=page_size, kv_dtype=kv_dtype, scale=k_scale)
        vv = gather(pool_v, block_table[b], c, page_size=page_size, kv_dtype=kv_dtype, scale=v_scale)
        out[b] = attend(q[b:b + 1], np.array([c - 1]), k, vv, softmax_scale, window)[0]
    return out


# ------------------------------------------------------------ LSE merge

def partial(q, pos, k, v, softmax_scale, window, keys):
    """Softmax state of one query row over a subset of keys: (m, l, o) with
    m = max score, l = sum exp(s - m), o = sum exp(s - m) v / l.  q [Hq, D]."""
    q = np.asarray(q, dtype=np.float64)
    Hq, D = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    keys = np.asarray(keys, dtype=np.int64)
    keys = keys[visible(pos, keys, window)]
    m = np.full(Hq, -np.inf)
    l = np.zeros(Hq)
    o = np.zeros((Hq, D))
    if keys.size == 0:
        return m, l, o
    for h in range(Hq):
        g = h // G
        s = softmax_scale * (k[keys, g, :] @ q[h])
        m[h] = s.max()
        e = np.exp(s - m[h])
        l[h] = e.sum()
        o[h] = (e @ v[keys, g, :]) / l[h]
    return m, l, o


def lse_merge(parts):
    """Combine softmax states of disjoint key sets: with M = max m_s,
    w_s = l_s exp(m_s - M), o = sum w_s o_s / sum w_s."""
    ms = np.stack([p[0] for p in parts])  # [S, Hq]
    ls = np.stack([p[1] for p in parts])
    os_ = np.stack([p[2] for p in parts])  # [S, Hq, D]
    M = ms.max(axis=0)
    w = np.where(np.isfinite(ms), ls * np.exp(ms - M), 0.0)
    return (w[:, :, None] * os_).sum(axis=0) / w.sum(axis=0)[:, None]


# ------------------------------------------------------- page offload/reload

def offload_pages(pool, pages, scale=None):
    """Host copy of pool pages: host page i is pool page pages[i], byte for
    byte, with its (page, head) scales for fp8.  An evicted request's pages
    leave the GPU this way when CPU offloading is on (Sec. 1; Sec. 3.2).
    Ids outside [0, num_pages) give an all-zero host page here; the library
    leaves such a page unspecified, so tests compare valid ids only."""
    num_pages = pool.shape[0]
    host = np.zeros((len(pages),) + pool.shape[1:], dtype=pool.dtype)
    host_scale = None if scale is None else np.zeros((len(pages), pool.shape[1]), dtype=scale.dtype)
    for i, p in enumerate(pages):
        if 0 <= p < num_pages:
            host[i] = pool[p]
            if scale is not None:
                host_scale[i] = scale[p]
    return host, host_scale


def reload_pages(pool, pages, host, scale=None, host_scale=None):
    """Write host page i into pool page pages[i] (in place), scales likewise:
    a TTL miss with offloading on brings the pages back instead of
    re-running prefill (Sec. 1; Sec. 3.2; Prefill-Reload(r), Sec. 4.1).
    Ids outside [0, num_pages) are skipped; every other pool page keeps its
    bytes."""
    num_pages = pool.shape[0]
    for i, p in enumerate(pages):
        if 0 <= p < num_pages:
            pool[p] = host[i]
            if scale is not None:
                scale[p] = host_scale[i]
