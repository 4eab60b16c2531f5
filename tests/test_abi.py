"""The C-ABI library loads, exports every symbol include/ckv.h declares, and
rejects invalid host-side arguments before launching anything (CPU only:
no call here reaches a kernel)."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ckv.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def ckv():
    from paper_2511_02230_amd import ckv as mod

    return mod


def test_header_declares_the_three_calls():
    names = declared_functions()
    for fn in ("kv_append", "prefix_prefill_attn", "paged_decode_attn"):
        assert fn in names


def test_library_exports_every_declared_symbol(ckv):
    out = subprocess.run(["nm", "-D", "--defined-only", ckv.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(line.split()[-1] for line in out.splitlines() if " T " in line)
    for fn in declared_functions():
        assert fn in exported, fn
        assert getattr(ckv.LIB, fn) is not None
    assert set(ckv.EXPORTS) == set(declared_functions())


def test_status_strings_and_version(ckv):
    for code in range(5):
        assert ckv.status_string(code).startswith(ckv.STATUS[code])
    assert ckv.version() >= 100


def _pool(ckv, **kw):
    base = dict(k_pages=1, v_pages=1, k_scale=None, v_scale=None, num_pages=4, num_kv_heads=2,
                page_size=16, head_dim=128, kv_dtype=ckv.CKV_BF16)
    base.update(kw)
    return ckv.PoolT(**base)


def _batch(ckv, **kw):
    base = dict(num_seqs=1, max_pages_per_seq=2, block_table=1, ctx_lens=1, cu_q_lens=1,
                total_q_len=4, max_q_len=4, max_ctx_len=8)
    base.update(kw)
    return ckv.BatchT(**base)


def _append(ckv, pool, batch, k=1, v=1, in_dtype=1):
    return ckv.LIB.kv_append(ctypes.byref(pool) if pool is not None else None,
                             ctypes.byref(batch) if batch is not None else None, k, v, in_dtype, None)


def test_append_argument_checks(ckv):
    assert _append(ckv, None, _batch(ckv)) == 1
    assert _append(ckv, _pool(ckv, k_pages=None), _batch(ckv)) == 1
    assert _append(ckv, _pool(ckv, num_pages=0), _batch(ckv)) == 1
    assert _append(ckv, _pool(ckv, head_dim=96), _batch(ckv)) == 2
    assert _append(ckv, _pool(ckv, page_size=32), _batch(ckv)) == 2
    assert _append(ckv, _pool(ckv, kv_dtype=ckv.CKV_FP8_E4M3), _batch(ckv)) == 1  # no scales
    assert _append(ckv, _pool(ckv), _batch(ckv), in_dtype=0) == 2  # f32 into a bf16 pool
    assert _append(ckv, _pool(ckv), _batch(ckv, cu_q_lens=None)) == 1
    assert _append(ckv, _pool(ckv), _batch(ckv, max_ctx_len=40)) == 1  # beyond the table
    assert _append(ckv, _pool(ckv), _batch(ckv, max_q_len=33, total_q_len=4)) == 1
    assert _append(ckv, _pool(ckv), _batch(ckv), k=None) == 1
    assert _append(ckv, _pool(ckv), _batch(ckv, num_seqs=0)) == 0  # nothing to do
    assert _append(ckv, _pool(ckv), _batch(ckv, total_q_len=0)) == 0


def test_attention_argument_checks(ckv):
    P, B = _pool(ckv), _batch(ckv)
    f = ckv.LIB.prefix_prefill_attn
    assert f(ctypes.byref(P), ctypes.byref(B), 1, 1, 3, 0.1, 0, 1, None, 0, None) == 1  # 3 % 2
    assert f(ctypes.byref(P), ctypes.byref(B), 1, 0, 4, 0.1, 0, 1, None, 0, None) == 2  # f32 q, bf16 pool
    assert f(ctypes.byref(P), ctypes.byref(B), 1, 1, 4, float("nan"), 0, 1, None, 0, None) == 1
    # the softmax scale must be positive: the kernels mask with -inf scores
    for bad_scale in (0.0, -0.0, -0.1, float("inf")):
        assert f(ctypes.byref(P), ctypes.byref(B), 1, 1, 4, bad_scale, 0, 1, None, 0, None) == 1
    assert f(ctypes.byref(P), ctypes.byref(B), 1, 1, 4, 0.1, -1, 1, None, 0, None) == 1
    assert f(ctypes.byref(P), ctypes.byref(B), None, 1, 4, 0.1, 0, 1, None, 0, None) == 1
    d = ckv.LIB.paged_decode_attn
    DB = _batch(ckv, cu_q_lens=None, max_ctx_len=20000, max_pages_per_seq=2000)
    assert d(ctypes.byref(P), ctypes.byref(DB), 1, 1, 4, 0.1, 0, 100, 1, None, 0, None) == 1  # split % 64
    for bad_scale in (0.0, -1.0):
        assert d(ctypes.byref(P), ctypes.byref(DB), 1, 1, 4, bad_scale, 0, 0, 1, None, 0, None) == 1
    need = ckv.LIB.paged_decode_workspace_bytes(ctypes.byref(P), ctypes.byref(DB), 4, 0)
    assert need > 0
    assert d(ctypes.byref(P), ctypes.byref(DB), 1, 1, 4, 0.1, 0, 0, 1, None, 0, None) == 3
    assert d(ctypes.byref(P), ctypes.byref(DB), 1, 1, 4, 0.1, 0, 0, 1, 1, need - 1, None) == 3
    assert d(ctypes.byref(P), ctypes.byref(_batch(ckv, max_ctx_len=0)), 1, 1, 4, 0.1, 0, 0, 1, None,
             0, None) == 1


def test_decode_workspace_grows_with_splits(ckv):
    P = _pool(ckv)
    DB = _batch(ckv, cu_q_lens=None, max_ctx_len=4096, max_pages_per_seq=256)
    a = ckv.LIB.paged_decode_workspace_bytes(ctypes.byref(P), ctypes.byref(DB), 4, 512)
    b = ckv.LIB.paged_decode_workspace_bytes(ctypes.byref(P), ctypes.byref(DB), 4, 1024)
    assert a == 1 * 4 * 8 * (128 + 2) * 4 and b == 1 * 4 * 4 * (128 + 2) * 4
    assert ckv.LIB.paged_decode_workspace_bytes(ctypes.byref(P), ctypes.byref(DB), 4, 4096) == 0


def test_validate_batch(ckv):
    bt = np.array([[3, 1, 0], [2, 0, 0]], np.int32)
    ckv.validate_batch(4, 16, bt, [20, 5], [0, 10, 12], 10, 20, decode=False)
    ckv.validate_batch(4, 16, bt, [40, 16], None, 1, 40, decode=True, distinct_pages=False)
    with pytest.raises(ckv.CkvError):  # page id out of range
        ckv.validate_batch(3, 16, bt, [20, 5], [0, 10, 12], 10, 20, decode=False)
    with pytest.raises(ckv.CkvError):  # positions beyond the table
        ckv.validate_batch(4, 16, bt, [40, 5], [0, 10, 12], 10, 40, decode=False)
    with pytest.raises(ckv.CkvError):  # shared page across sequences
        ckv.validate_batch(4, 16, np.array([[3, 1], [1, 0]], np.int32), [20, 5], [0, 1, 2], 1, 20,
                           decode=False, distinct_pages=True)
    with pytest.raises(ckv.CkvError):  # decode context 0
        ckv.validate_batch(4, 16, bt, [0, 5], None, 1, 40, decode=True)
    with pytest.raises(ckv.CkvError):  # bound violated
        ckv.validate_batch(4, 16, bt, [20, 5], [0, 10, 12], 9, 20, decode=False)


def test_binding_rejects_cpu_tensors(ckv):
    import torch

    with pytest.raises(ValueError):
        ckv.Pool(torch.zeros(2, 1, 16, 64), torch.zeros(2, 1, 16, 64))


def test_size_limits_are_rejected_before_any_launch(ckv):
    P = _pool(ckv, num_pages=100000)
    # more sequences than a grid dimension holds
    assert _append(ckv, P, _batch(ckv, num_seqs=65536, total_q_len=4)) == 2
    # more query heads than the fp32 path's grid holds
    f = ckv.LIB.prefix_prefill_attn
    B = _batch(ckv)
    assert f(ctypes.byref(P), ctypes.byref(B), 1, 1, 65536 * 2, 0.1, 0, 1, None, 0, None) == 2
    # more prefill row tiles than grid.y holds: 1 048 576 new rows x 8 heads / 128
    big = _batch(ckv, max_pages_per_seq=70000, max_q_len=1048576, total_q_len=1048576, max_ctx_len=0)
    assert f(ctypes.byref(P), ctypes.byref(big), 1, 1, 16, 0.1, 0, 1, None, 0, None) == 2
    assert ckv.LIB.prefix_prefill_workspace_bytes(ctypes.byref(P), ctypes.byref(big), 16) == 0
    # one tile short of the limit is accepted by the checks (it fails later on the dummy pointers'
    # missing workspace only if one is needed, so ask for the size instead)
    ok = _batch(ckv, max_pages_per_seq=70000, max_q_len=65535 * 16, total_q_len=65535 * 16, max_ctx_len=0)
    assert ckv.LIB.prefix_prefill_workspace_bytes(ctypes.byref(P), ctypes.byref(ok), 16) == 0


@pytest.mark.parametrize("h_q,h_kv,d,n,prefix,splits", [
    (64, 8, 128, 256, 65280, 4),    # 128 row tiles on 512 slots: one full wave of quarter-length work
    (64, 8, 128, 768, 64768, 4),    # 384 tiles: three full waves instead of one 3/4-full wave
    (64, 8, 128, 1536, 64000, 2),   # 768 tiles: three half-length waves instead of two
    (64, 8, 128, 256, 3840, 2),     # a 4096-key context allows two partitions of >= 2048 keys
    (64, 8, 128, 4096, 61440, 1),   # 2048 tiles: four waves or more keep one partition
    (16, 8, 256, 256, 65280, 8),    # head_dim 256, one workgroup per CU: 32 tiles on 256 slots
])
def test_prefill_key_partitions(ckv, h_q, h_kv, d, n, prefix, splits):
    """Key partitions of small prefill batches, seen through the workspace size:
    total rows x query heads x partitions x (head_dim + 2) fp32 values, or 0 for one."""
    P = _pool(ckv, num_pages=100000, num_kv_heads=h_kv, head_dim=d)
    pages = (prefix + n + 15) // 16
    B = _batch(ckv, max_pages_per_seq=pages, total_q_len=n, max_q_len=n, max_ctx_len=prefix)
    got = ckv.LIB.prefix_prefill_workspace_bytes(ctypes.byref(P), ctypes.byref(B), h_q)
    assert got == (0 if splits == 1 else n * h_q * splits * (d + 2) * 4)


def test_noalloc_decode_checks_arguments_and_the_scratch_bound_on_the_host(ckv):
    """paged_decode_attn_noalloc rejects what paged_decode_attn rejects, and
    partials larger than its scratch, before touching the GPU."""
    P = _pool(ckv, num_pages=100000)
    f = ckv.LIB.paged_decode_attn_noalloc
    DB = _batch(ckv, cu_q_lens=None, max_ctx_len=20000, max_pages_per_seq=2000)
    assert f(ctypes.byref(P), ctypes.byref(DB), 1, 1, 3, 0.1, 0, 0, 1, None) == 1  # 3 % 2
    assert f(ctypes.byref(P), ctypes.byref(DB), 1, 1, 4, 0.0, 0, 0, 1, None) == 1  # scale
    assert f(ctypes.byref(P), ctypes.byref(DB), 1, 1, 4, 0.1, 0, 100, 1, None) == 1  # split % 64
    assert f(ctypes.byref(P), ctypes.byref(DB), 1, 1, 4, 0.1, 0, 0, None, None) == 1  # no out
    assert f(ctypes.byref(P), ctypes.byref(_batch(ckv, num_seqs=0)), 1, 1, 4, 0.1, 0, 0, 1, None) == 0
    big = _batch(ckv, num_seqs=4096, cu_q_lens=None, max_ctx_len=65536, max_pages_per_seq=4096)
    need = ckv.LIB.paged_decode_workspace_bytes(ctypes.byref(P), ctypes.byref(big), 64, 512)
    assert need > ckv.DECODE_SCRATCH_BYTES
    assert f(ctypes.byref(P), ctypes.byref(big), 1, 1, 64, 0.1, 0, 512, 1, None) == 3


def test_mixed_launch_checks_arguments_on_the_host(ckv):
    """mixed_attn applies both calls' checks before launching anything."""
    P = _pool(ckv, num_pages=100000)
    f = ckv.LIB.mixed_attn
    PB = _batch(ckv)
    DB = _batch(ckv, cu_q_lens=None, max_ctx_len=2000, max_pages_per_seq=200)
    E = _batch(ckv, num_seqs=0)

    def call(pb=PB, db=DB, qp=1, op=1, qd=1, od=1, qdt=1, hq=4, scale=0.1, w=0, split=0, inter=0,
             ws=1, wsb=1 << 30, kp=None, vp=None, kd=None, vd=None, pool=P):
        return f(ctypes.byref(pool), ctypes.byref(pb), qp, kp, vp, op, ctypes.byref(db), qd, kd, vd, od, qdt,
                 hq, scale, w, split, inter, ws, wsb, None)

    assert call(hq=3) == 1                 # 3 % 2
    assert call(qdt=0) == 2                # fp32 queries: no mixed kernel
    assert call(scale=0.0) == 1
    assert call(w=-1) == 1
    assert call(split=100) == 1            # not a multiple of 64
    assert call(inter=-1) == 1
    assert call(qp=None) == 1              # prefill rows without queries
    assert call(od=None) == 1              # decode rows without an output
    assert call(pb=E, db=E) == 0           # nothing to do
    need = ckv.LIB.mixed_attn_workspace_bytes(ctypes.byref(P), ctypes.byref(PB), ctypes.byref(DB), 4, 128)
    assert need > 0
    assert call(split=128, ws=None) == 3
    assert call(split=128, wsb=need - 1) == 3
    assert call(split=128, ws=1 << 20 | 16) == 1   # not 256-byte aligned
    # fused append: rows come in K / V pairs, for bf16 pools only
    assert call(kp=1) == 1
    assert call(vd=1) == 1
    F8 = _pool(ckv, num_pages=100000, kv_dtype=ckv.CKV_FP8_E4M3, k_scale=1, v_scale=1)
    assert call(pool=F8, kp=1, vp=1) == 2
    assert call(pool=F8, kd=1, vd=1) == 2
    assert call(pool=F8, pb=E, db=E, kp=1, vp=1) == 0  # nothing to append
