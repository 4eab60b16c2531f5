"""Pure-Python brute force of paged attention, for tiny inputs only.

TEST INFRASTRUCTURE ONLY.  An independent restatement used to pin the NumPy
oracle: explicit loops over pages and slots, math.exp with no maximum
subtraction, and the visibility rule written out (key j is seen by the query
at position i iff j <= i and, for a window W > 0, i - j < W).
"""
from __future__ import annotations

import math


def key_row(pool, block_table_row, page_size, j, h):
    """Values of token j, KV head h, as a list of Python floats."""
    page = int(block_table_row[j // page_size])
    slot = j % page_size
    return [float(x) for x in pool[page][h][slot]]


def attention_row(qrow, i, pool_k, pool_v, block_table_row, page_size, h_kv, scale, window):
    """One query vector at absolute position i attending through the block
    table to KV head h_kv; pools hold already-decoded float values."""
    num = None
    den = 0.0
    for j in range(i + 1):
        if window > 0 and i - j >= window:
            continue
        kr = key_row(pool_k, block_table_row, page_size, j, h_kv)
        vr = key_row(pool_v, block_table_row, page_size, j, h_kv)
        s = 0.0
        for a, b in zip(qrow, kr):
            s += float(a) * b
        w = math.exp(scale * s)
        den += w
        if num is None:
            num = [w * x for x in vr]
        else:
            num = [acc + w * x for acc, x in zip(num, vr)]
    return [x / den for x in num]


def prefill(q, pool_k, pool_v, block_table, ctx_lens, q_lens, page_size, scale, window=0):
    """q: nested lists [sum n][H_q][D]; returns the same shape."""
    hq = len(q[0]) if q else 0
    hkv = len(pool_k[0])
    G = hq // hkv
    out = []
    cu = 0
    for b in range(len(q_lens)):
        for t in range(int(q_lens[b])):
            i = int(ctx_lens[b]) + t
            out.append([attention_row(q[cu + t][h], i, pool_k, pool_v, block_table[b],
                                      page_size, h // G, scale, window) for h in range(hq)])
        cu += int(q_lens[b])
    return out
