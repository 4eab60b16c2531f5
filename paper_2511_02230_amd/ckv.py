"""ctypes binding of libckv.so: argument marshalling only.

Every step of the hot path runs in the library's HIP kernels; this module
checks tensor dtypes / shapes / devices, fills the C structs of the C ABI
(include/ckv.h) and passes raw device pointers plus the current HIP stream.
It never computes anything itself and has no fallback: if libckv.so is
missing or fails to load, importing this module raises.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional

import numpy as np
import torch  # must be loaded first: libckv.so then binds to torch's HIP runtime

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libckv.so")

CKV_F32, CKV_BF16, CKV_FP8_E4M3 = 0, 1, 2
STATUS = {0: "CKV_OK", 1: "CKV_ERR_INVALID_ARG", 2: "CKV_ERR_UNSUPPORTED", 3: "CKV_ERR_WORKSPACE",
          4: "CKV_ERR_LAUNCH"}
EXPORTS = ("kv_append", "prefix_prefill_attn", "paged_decode_attn", "paged_decode_attn_noalloc",
           "mixed_attn", "mixed_attn_workspace_bytes", "prefix_prefill_workspace_bytes",
           "paged_decode_workspace_bytes", "kv_pages_reload", "kv_pages_offload",
           "kv_pages_staging_bytes", "ckv_validate_batch", "ckv_status_string", "ckv_version")


class CkvError(RuntimeError):
    def __init__(self, fn: str, code: int):
        super().__init__(f"{fn} failed: {STATUS.get(code, code)}")
        self.code = code


class PoolT(ctypes.Structure):
    _fields_ = [("k_pages", ctypes.c_void_p), ("v_pages", ctypes.c_void_p),
                ("k_scale", ctypes.c_void_p), ("v_scale", ctypes.c_void_p),
                ("num_pages", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("kv_dtype", ctypes.c_int)]


class BatchT(ctypes.Structure):
    _fields_ = [("num_seqs", ctypes.c_int32), ("max_pages_per_seq", ctypes.c_int32),
                ("block_table", ctypes.c_void_p), ("ctx_lens", ctypes.c_void_p),
                ("cu_q_lens", ctypes.c_void_p), ("total_q_len", ctypes.c_int32),
                ("max_q_len", ctypes.c_int32), ("max_ctx_len", ctypes.c_int32)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2511_02230_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P, B = ctypes.POINTER(PoolT), ctypes.POINTER(BatchT)
    vp, i32, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
    sig = {
        "kv_append": ([P, B, vp, vp, ctypes.c_int, vp], ctypes.c_int),
        "prefix_prefill_attn": ([P, B, vp, ctypes.c_int, i32, f32, i32, vp, vp, sz, vp], ctypes.c_int),
        "paged_decode_attn": ([P, B, vp, ctypes.c_int, i32, f32, i32, i32, vp, vp, sz, vp], ctypes.c_int),
        "paged_decode_attn_noalloc": ([P, B, vp, ctypes.c_int, i32, f32, i32, i32, vp, vp], ctypes.c_int),
        "mixed_attn": ([P, B, vp, vp, vp, vp, B, vp, vp, vp, vp, ctypes.c_int, i32, f32, i32, i32, i32, vp, sz,
                        vp],
                       ctypes.c_int),
        "mixed_attn_workspace_bytes": ([P, B, B, i32, i32], sz),
        "prefix_prefill_workspace_bytes": ([P, B, i32], sz),
        "paged_decode_workspace_bytes": ([P, B, i32, i32], sz),
        "kv_pages_reload": ([P, vp, i32, vp, vp, vp, vp, vp, sz, vp], ctypes.c_int),
        "kv_pages_offload": ([P, vp, i32, vp, vp, vp, vp, vp, sz, vp], ctypes.c_int),
        "kv_pages_staging_bytes": ([P, i32], sz),
        "ckv_validate_batch": ([P, i32, i32, vp, vp, vp, i32, i32, i32, i32], ctypes.c_int),
        "ckv_status_string": ([ctypes.c_int], ctypes.c_char_p),
        "ckv_version": ([], i32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


LIB = _load()

_KV_DTYPES = {torch.float32: CKV_F32, torch.bfloat16: CKV_BF16, torch.uint8: CKV_FP8_E4M3}
_Q_DTYPES = {torch.float32: CKV_F32, torch.bfloat16: CKV_BF16}


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _dev(t: torch.Tensor, name: str, dtype=None):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


@dataclasses.dataclass
class Pool:
    """Paged KV pool: k/v [num_pages, H_kv, page_size, D] (float32, bfloat16,
    or uint8 E4M3FN codes with float32 k_scale / v_scale [num_pages, H_kv])."""

    k: torch.Tensor
    v: torch.Tensor
    k_scale: Optional[torch.Tensor] = None
    v_scale: Optional[torch.Tensor] = None

    def __post_init__(self):
        _dev(self.k, "pool.k")
        _dev(self.v, "pool.v", self.k.dtype)
        if self.k.dim() != 4 or self.v.shape != self.k.shape:
            raise ValueError("pool tensors must be [num_pages, H_kv, page_size, D]")
        if self.k.dtype not in _KV_DTYPES:
            raise ValueError(f"unsupported pool dtype {self.k.dtype}")
        if self.k.dtype == torch.uint8:
            if self.k_scale is None or self.v_scale is None:
                raise ValueError("fp8 pool needs k_scale and v_scale")
            for nm, s in (("k_scale", self.k_scale), ("v_scale", self.v_scale)):
                _dev(s, nm, torch.float32)
                if tuple(s.shape) != tuple(self.k.shape[:2]):
                    raise ValueError(f"{nm} must be [num_pages, H_kv]")

    @property
    def kv_dtype(self) -> int:
        return _KV_DTYPES[self.k.dtype]

    def c(self) -> PoolT:
        n, h, ps, d = self.k.shape
        return PoolT(_ptr(self.k), _ptr(self.v), _ptr(self.k_scale), _ptr(self.v_scale), n, h, ps, d,
                     self.kv_dtype)


@dataclasses.dataclass
class Batch:
    """Block tables and lengths on the GPU (int32) plus host-side bounds."""

    block_table: torch.Tensor  # [B, max_pages] int32
    ctx_lens: torch.Tensor     # [B] int32
    cu_q_lens: Optional[torch.Tensor]  # [B+1] int32 (append / prefill)
    total_q_len: int
    max_q_len: int
    max_ctx_len: int

    def __post_init__(self):
        _dev(self.block_table, "block_table", torch.int32)
        _dev(self.ctx_lens, "ctx_lens", torch.int32)
        if self.cu_q_lens is not None:
            _dev(self.cu_q_lens, "cu_q_lens", torch.int32)

    @property
    def num_seqs(self) -> int:
        return int(self.ctx_lens.shape[0])

    def c(self) -> BatchT:
        return BatchT(self.num_seqs, int(self.block_table.shape[1]), _ptr(self.block_table),
                      _ptr(self.ctx_lens), _ptr(self.cu_q_lens), int(self.total_q_len),
                      int(self.max_q_len), int(self.max_ctx_len))


def _check(name: str, code: int):
    if code != 0:
        raise CkvError(name, code)


def kv_append(pool: Pool, batch: Batch, k_new: torch.Tensor, v_new: torch.Tensor, stream=None):
    """Write new-turn rows k_new / v_new [total_q_len, H_kv, D] into the pool."""
    _dev(k_new, "k_new")
    _dev(v_new, "v_new", k_new.dtype)
    if k_new.dtype not in _Q_DTYPES:
        raise ValueError(f"unsupported k_new dtype {k_new.dtype}")
    if tuple(k_new.shape) != (batch.total_q_len,) + tuple(pool.k.shape[1:2]) + tuple(pool.k.shape[3:]):
        raise ValueError("k_new must be [total_q_len, H_kv, D]")
    pc, bc = pool.c(), batch.c()
    _check("kv_append", LIB.kv_append(ctypes.byref(pc), ctypes.byref(bc), _ptr(k_new), _ptr(v_new),
                                      _Q_DTYPES[k_new.dtype], _stream(stream)))


def prefill_workspace_bytes(pool: Pool, batch: Batch, num_q_heads: int) -> int:
    pc, bc = pool.c(), batch.c()
    return int(LIB.prefix_prefill_workspace_bytes(ctypes.byref(pc), ctypes.byref(bc), num_q_heads))


def decode_workspace_bytes(pool: Pool, batch: Batch, num_q_heads: int, kv_split_len: int = 0) -> int:
    pc, bc = pool.c(), batch.c()
    return int(LIB.paged_decode_workspace_bytes(ctypes.byref(pc), ctypes.byref(bc), num_q_heads,
                                                kv_split_len))


def _out_like(q, out):
    if out is None:
        out = torch.empty_like(q)
    _dev(out, "out", q.dtype)
    if out.shape != q.shape:
        raise ValueError("out must have q's shape")
    return out


def _workspace(nbytes: int, workspace, device):
    if nbytes == 0:
        return None, 0
    if workspace is None:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)
    _dev(workspace, "workspace")
    return workspace, workspace.numel() * workspace.element_size()


def prefix_prefill_attn(pool: Pool, batch: Batch, q: torch.Tensor, softmax_scale: float,
                        window: int = 0, out=None, workspace=None, stream=None) -> torch.Tensor:
    """Causal GQA attention of the new-turn rows q [total_q_len, H_q, D]."""
    _dev(q, "q")
    if q.dtype not in _Q_DTYPES or q.dim() != 3 or q.shape[0] != batch.total_q_len:
        raise ValueError("q must be [total_q_len, H_q, D] float32 or bfloat16")
    out = _out_like(q, out)
    ws, wsb = _workspace(prefill_workspace_bytes(pool, batch, q.shape[1]), workspace, q.device)
    pc, bc = pool.c(), batch.c()
    _check("prefix_prefill_attn", LIB.prefix_prefill_attn(
        ctypes.byref(pc), ctypes.byref(bc), _ptr(q), _Q_DTYPES[q.dtype], q.shape[1],
        float(softmax_scale), int(window), _ptr(out), _ptr(ws), wsb, _stream(stream)))
    return out


def paged_decode_attn(pool: Pool, batch: Batch, q: torch.Tensor, softmax_scale: float,
                      window: int = 0, kv_split_len: int = 0, out=None, workspace=None,
                      stream=None) -> torch.Tensor:
    """Decode attention of q [B, H_q, D]; batch.ctx_lens holds c_b."""
    _dev(q, "q")
    if q.dtype not in _Q_DTYPES or q.dim() != 3 or q.shape[0] != batch.num_seqs:
        raise ValueError("q must be [num_seqs, H_q, D] float32 or bfloat16")
    out = _out_like(q, out)
    ws, wsb = _workspace(decode_workspace_bytes(pool, batch, q.shape[1], kv_split_len), workspace,
                         q.device)
    pc, bc = pool.c(), batch.c()
    _check("paged_decode_attn", LIB.paged_decode_attn(
        ctypes.byref(pc), ctypes.byref(bc), _ptr(q), _Q_DTYPES[q.dtype], q.shape[1],
        float(softmax_scale), int(window), int(kv_split_len), _ptr(out), _ptr(ws), wsb,
        _stream(stream)))
    return out


def mixed_workspace_bytes(pool: Pool, prefill: Batch, decode: Batch, num_q_heads: int,
                          kv_split_len: int = 0) -> int:
    pc, pb, db = pool.c(), prefill.c(), decode.c()
    return int(LIB.mixed_attn_workspace_bytes(ctypes.byref(pc), ctypes.byref(pb), ctypes.byref(db),
                                              num_q_heads, kv_split_len))


def _append_rows(pool: Pool, k, v, n: int, name: str):
    """The fused append's new rows: both None, or bf16 [n, H_kv, D] each."""
    if (k is None) != (v is None):
        raise ValueError(f"{name}: give both K and V rows, or neither")
    if k is None:
        return None, None
    for t, nm in ((k, "k"), (v, "v")):
        _dev(t, f"{nm}_{name}", torch.bfloat16)
        if tuple(t.shape) != (n, pool.k.shape[1], pool.k.shape[3]):
            raise ValueError(f"{nm}_{name} must be [{n}, H_kv, D]")
    return k, v


def mixed_attn(pool: Pool, prefill: Batch, q_prefill: torch.Tensor, decode: Batch, q_decode: torch.Tensor,
               softmax_scale: float, window: int = 0, kv_split_len: int = 0, interleave: int = 0,
               out_prefill=None, out_decode=None, workspace=None, stream=None,
               k_prefill=None, v_prefill=None, k_decode=None, v_decode=None):
    """Prefill over `prefill` (q_prefill [total_q_len, H_q, D]) and decode over
    `decode` (q_decode [num_seqs, H_q, D]) in one launch; returns
    (out_prefill, out_decode).  k_/v_prefill ([total_q_len, H_kv, D]) and
    k_/v_decode ([num_seqs, H_kv, D]), bf16 pools only: new rows that the
    launch appends to the pool itself (else the pool already holds them)."""
    _dev(q_prefill, "q_prefill", torch.bfloat16)
    _dev(q_decode, "q_decode", torch.bfloat16)
    if q_prefill.dim() != 3 or q_prefill.shape[0] != prefill.total_q_len:
        raise ValueError("q_prefill must be [total_q_len, H_q, D]")
    if q_decode.dim() != 3 or q_decode.shape[0] != decode.num_seqs or q_decode.shape[1:] != q_prefill.shape[1:]:
        raise ValueError("q_decode must be [num_seqs, H_q, D]")
    k_prefill, v_prefill = _append_rows(pool, k_prefill, v_prefill, prefill.total_q_len, "prefill")
    k_decode, v_decode = _append_rows(pool, k_decode, v_decode, decode.num_seqs, "decode")
    out_prefill = _out_like(q_prefill, out_prefill)
    out_decode = _out_like(q_decode, out_decode)
    h_q = q_prefill.shape[1]
    ws, wsb = _workspace(mixed_workspace_bytes(pool, prefill, decode, h_q, kv_split_len), workspace,
                         q_prefill.device)
    pc, pb, db = pool.c(), prefill.c(), decode.c()
    _check("mixed_attn", LIB.mixed_attn(
        ctypes.byref(pc), ctypes.byref(pb), _ptr(q_prefill), _ptr(k_prefill), _ptr(v_prefill),
        _ptr(out_prefill), ctypes.byref(db), _ptr(q_decode), _ptr(k_decode), _ptr(v_decode),
        _ptr(out_decode), CKV_BF16, h_q, float(softmax_scale), int(window), int(kv_split_len),
        int(interleave), _ptr(ws), wsb, _stream(stream)))
    return out_prefill, out_decode


DECODE_SCRATCH_BYTES = 64 << 20  # CKV_DECODE_SCRATCH_BYTES


def paged_decode_attn_noalloc(pool: Pool, batch: Batch, q: torch.Tensor, softmax_scale: float,
                              out: torch.Tensor, window: int = 0, kv_split_len: int = 0,
                              stream=None) -> torch.Tensor:
    """paged_decode_attn with its partials in the library's per-GPU scratch:
    nothing is allocated (out must be given)."""
    _dev(q, "q")
    if q.dtype not in _Q_DTYPES or q.dim() != 3 or q.shape[0] != batch.num_seqs:
        raise ValueError("q must be [num_seqs, H_q, D] float32 or bfloat16")
    _dev(out, "out", q.dtype)
    if out.shape != q.shape:
        raise ValueError("out must have q's shape")
    pc, bc = pool.c(), batch.c()
    _check("paged_decode_attn_noalloc", LIB.paged_decode_attn_noalloc(
        ctypes.byref(pc), ctypes.byref(bc), _ptr(q), _Q_DTYPES[q.dtype], q.shape[1],
        float(softmax_scale), int(window), int(kv_split_len), _ptr(out), _stream(stream)))
    return out


def pages_staging_bytes(pool: Pool, num_moved: int) -> int:
    pc = pool.c()
    return int(LIB.kv_pages_staging_bytes(ctypes.byref(pc), int(num_moved)))


def _host(t: torch.Tensor, name: str, dtype, shape):
    if t.is_cuda:
        raise ValueError(f"{name} must be a host tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.dtype != dtype or tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must be {dtype} {tuple(shape)}, got {t.dtype} {tuple(t.shape)}")


def _page_move_args(pool: Pool, pages: torch.Tensor, host, staging):
    _dev(pages, "pages", torch.int32)
    if pages.dim() != 1:
        raise ValueError("pages must be 1-D")
    n = int(pages.shape[0])
    page_shape = (n,) + tuple(pool.k.shape[1:])
    fp8 = pool.kv_dtype == CKV_FP8_E4M3
    names = ("host_k", "host_v", "host_k_scale", "host_v_scale")
    for i, t in enumerate(host):
        if i < 2:
            _host(t, names[i], pool.k.dtype, page_shape)
        elif fp8:
            _host(t, names[i], torch.float32, page_shape[:2])
    staging, sb = _workspace(pages_staging_bytes(pool, n), staging, pool.k.device)
    ptrs = [_ptr(t) for t in host[:2]] + [_ptr(t) if fp8 else None for t in host[2:]]
    return n, ptrs, staging, sb


def kv_pages_reload(pool: Pool, pages: torch.Tensor, host_k: torch.Tensor, host_v: torch.Tensor,
                    host_k_scale: Optional[torch.Tensor] = None,
                    host_v_scale: Optional[torch.Tensor] = None, staging=None, stream=None):
    """Copy host pages i (host_k / host_v [n, H_kv, page_size, D] in the pool's
    dtype, pinned for an asynchronous copy; fp8 scales [n, H_kv]) into pool
    pages pages[i] (int32 on the GPU).  Enqueued on the stream only."""
    host = (host_k, host_v, host_k_scale, host_v_scale)
    n, ptrs, st, sb = _page_move_args(pool, pages, host, staging)
    pc = pool.c()
    _check("kv_pages_reload", LIB.kv_pages_reload(ctypes.byref(pc), _ptr(pages), n, *ptrs, _ptr(st), sb,
                                                  _stream(stream)))


def kv_pages_offload(pool: Pool, pages: torch.Tensor, host_k=None, host_v=None, host_k_scale=None,
                     host_v_scale=None, staging=None, stream=None):
    """Copy pool pages pages[i] into host pages i.  Missing host buffers come
    from one pinned allocation laid out like the staging area (K pages, V
    pages, then fp8 scales), so the host side moves as a single copy.
    Returns (host_k, host_v, host_k_scale, host_v_scale); they hold the pages
    once the stream has passed the call."""
    n = int(pages.shape[0])
    shape = (n,) + tuple(pool.k.shape[1:])
    if host_k is None or host_v is None:
        fp8 = pool.kv_dtype == CKV_FP8_E4M3
        nb = n * pool.k[0].numel() * pool.k.element_size() if n else 0
        sb = n * pool.k.shape[1] * 4 if fp8 else 0
        buf = torch.empty(2 * nb + 2 * sb, dtype=torch.uint8, pin_memory=True)
        host_k = buf[:nb].view(pool.k.dtype).view(shape)
        host_v = buf[nb:2 * nb].view(pool.k.dtype).view(shape)
        if fp8:
            host_k_scale = buf[2 * nb:2 * nb + sb].view(torch.float32).view(shape[:2])
            host_v_scale = buf[2 * nb + sb:].view(torch.float32).view(shape[:2])
    elif pool.kv_dtype == CKV_FP8_E4M3 and (host_k_scale is None or host_v_scale is None):
        host_k_scale = torch.empty(shape[:2], dtype=torch.float32, pin_memory=True)
        host_v_scale = torch.empty(shape[:2], dtype=torch.float32, pin_memory=True)
    host = (host_k, host_v, host_k_scale, host_v_scale)
    n, ptrs, st, sb = _page_move_args(pool, pages, host, staging)
    pc = pool.c()
    _check("kv_pages_offload", LIB.kv_pages_offload(ctypes.byref(pc), _ptr(pages), n, *ptrs, _ptr(st), sb,
                                                    _stream(stream)))
    return host


def validate_batch(num_pages: int, page_size: int, block_table: np.ndarray, ctx_lens: np.ndarray,
                   cu_q_lens: Optional[np.ndarray], max_q_len: int, max_ctx_len: int, decode: bool,
                   distinct_pages: bool = False) -> None:
    """Host-side check (C ABI ckv_validate_batch) of block tables and lengths
    before a launch; raises CkvError on a violation."""
    bt = np.ascontiguousarray(block_table, dtype=np.int32)
    ctx = np.ascontiguousarray(ctx_lens, dtype=np.int32)
    cu = None if cu_q_lens is None else np.ascontiguousarray(cu_q_lens, dtype=np.int32)
    pc = PoolT(None, None, None, None, num_pages, 1, page_size, 64, CKV_BF16)
    code = LIB.ckv_validate_batch(ctypes.byref(pc), len(ctx), bt.shape[1] if bt.ndim == 2 else 0,
                                  bt.ctypes.data, ctx.ctypes.data,
                                  None if cu is None else cu.ctypes.data, max_q_len, max_ctx_len,
                                  1 if decode else 0, 1 if distinct_pages else 0)
    _check("ckv_validate_batch", code)


def status_string(code: int) -> str:
    return LIB.ckv_status_string(code).decode()


def version() -> int:
    return int(LIB.ckv_version())
