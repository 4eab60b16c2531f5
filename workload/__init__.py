"""Seeded synthetic multi-turn agent workloads for the paged-KV hot path.

When a tool-calling program's KV cache is kept resident between turns
(Continuum, Sec. 5.2 "Request Pinning"), the program's next turn arrives as a
retained prefix of P tokens plus n new-turn tokens (tool output + next
prompt, Sec. 5.1).  The paper's traces (SWE-Bench, BFCL, OpenHands; Table 2)
are not available, so this module draws stand-in workloads with the shapes
and length laws of five attention-layer configurations (Tiny, Llama-3.1-8B,
Gemma-3-12B, Llama-3.1-70B, GLM-4.5-355B).

What lives here, and only this:
  * length draws (retained prefix P, new-turn length n, decode context c),
  * physical page placement (a seeded permutation) and block tables,
  * raw Q/K/V values ~N(0,1), drawn per sequence from their own seeds,
  * the fp8 scale policy s = amax/448 per (page, head), with s = 1 for amax 0.

None of the method's arithmetic (append/quantize, attention, softmax) is
here; both the oracle and the GPU path consume what this module draws.
"""
from __future__ import annotations

import dataclasses
import hashlib
import math
from typing import List, Optional, Sequence, Tuple

import numpy as np

FP8_E4M3_MAX = 448.0

# ---------------------------------------------------------------------------
# Configurations
# ---------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class Config:
    """Shapes of one attention layer plus the length laws of its batches."""

    name: str
    seed: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    q_dtype: str  # "f32" or "bf16"
    kv_dtype: str  # "f32", "bf16" or "fp8"
    windows: Tuple[int, ...] = (0,)

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def softmax_scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)


TINY = Config("tiny", 0, 2, 1, 64, 16, "f32", "f32")
LLAMA8B = Config("llama3.1-8b", 1, 32, 8, 128, 16, "bf16", "bf16")
GEMMA12B = Config("gemma3-12b", 2, 16, 8, 256, 16, "bf16", "bf16", (0, 1024))
LLAMA70B = Config("llama3.1-70b", 3, 64, 8, 128, 16, "bf16", "bf16")
GLM355B = Config("glm4.5-355b", 4, 96, 8, 128, 64, "bf16", "fp8")

CONFIGS = {c.name: c for c in (TINY, LLAMA8B, GEMMA12B, LLAMA70B, GLM355B)}


# ---------------------------------------------------------------------------
# Sequences, batches, workload
# ---------------------------------------------------------------------------


@dataclasses.dataclass
class Sequence:
    """One program's resident KV history.

    length    tokens this sequence holds once the step's writes are done
    resident  tokens already in the pool before the step (written at set-up)
    pages     physical page ids of logical pages 0..ceil(length/ps)-1
    stream    seed tuple of this sequence's raw K/V values
    """

    sid: int
    length: int
    resident: int
    pages: np.ndarray
    stream: Tuple[int, ...]


@dataclasses.dataclass
class Batch:
    """A launch: per row b, sequence seq_ids[b] with ctx_lens[b] tokens
    before the call and q_lens[b] rows in the call."""

    seq_ids: np.ndarray  # int64 [B]
    ctx_lens: np.ndarray  # int32 [B]
    q_lens: np.ndarray  # int32 [B]
    block_table: np.ndarray  # int32 [B, max_pages]

    @property
    def num_seqs(self) -> int:
        return int(len(self.seq_ids))

    @property
    def cu_q_lens(self) -> np.ndarray:
        cu = np.zeros(self.num_seqs + 1, dtype=np.int32)
        np.cumsum(self.q_lens, out=cu[1:])
        return cu

    @property
    def total_q(self) -> int:
        return int(self.q_lens.sum())

    @property
    def max_q_len(self) -> int:
        return int(self.q_lens.max()) if self.num_seqs else 0

    @property
    def max_ctx_len(self) -> int:
        return int(self.ctx_lens.max()) if self.num_seqs else 0


@dataclasses.dataclass
class Workload:
    """A prefix-reuse turn (prefill batch) and a decode batch on one pool.

    prefill: ctx_lens = retained prefix P_b, q_lens = new-turn length n_b.
    decode:  ctx_lens = c_b - 1 tokens before the decode token is appended,
             q_lens = 1; the attention call sees c_b = ctx_lens + 1 tokens.
    """

    cfg: Config
    num_pages: int
    seqs: List[Sequence]
    prefill: Batch
    decode: Batch

    @property
    def decode_ctx(self) -> np.ndarray:
        return (self.decode.ctx_lens + 1).astype(np.int32)


def _mix(*parts: int) -> int:
    """64-bit seed from a tuple of integers (stable across platforms)."""
    h = hashlib.blake2b(digest_size=8)
    for p in parts:
        h.update(int(p).to_bytes(8, "little", signed=True))
    return int.from_bytes(h.digest(), "little") & ((1 << 63) - 1)


def _lognormal_int(rng, mu: float, sigma: float) -> int:
    return max(1, int(round(float(rng.lognormal(mu, sigma)))))


def _agent_trace_context(rng, cap: int) -> Tuple[int, int]:
    """Turn t ~ U{1..30}; prefix = sum of t-1 prior turn lengths, each
    lognormal with mean 1500 tokens (sigma_ln = 1), capped at `cap`;
    new-turn length n ~ U{64..4096}."""
    t = int(rng.integers(1, 31))
    mu = math.log(1500.0) - 0.5
    prefix = sum(_lognormal_int(rng, mu, 1.0) for _ in range(t - 1))
    prefix = min(prefix, cap)
    n = int(rng.integers(64, 4097))
    return prefix, n


def draw_lengths(cfg: Config):
    """Return (prefill [(P, n)], decode [c], shared_decode) for a config.

    shared_decode is True when the decode batch reuses the prefill batch's
    sequences (Tiny: one decode step over all P + n tokens).
    """
    rng = np.random.default_rng(cfg.seed)
    if cfg.name == "tiny":
        return [(240, 16)], [256], True
    if cfg.name == "llama3.1-8b":
        pf = [(int(rng.integers(2048, 16385)), int(rng.integers(128, 2049))) for _ in range(16)]
        dc = [int(rng.integers(4096, 32769)) for _ in range(64)]
        return pf, dc, False
    if cfg.name == "gemma3-12b":
        mu = math.log(8192.0)

        def one():
            p = min(_lognormal_int(rng, mu, 1.0), 32768)
            return p, int(rng.integers(256, 4097))

        pf = [one() for _ in range(32)]
        dc = [sum(one()) for _ in range(64)]
        return pf, dc, False
    if cfg.name == "llama3.1-70b":
        pf = [_agent_trace_context(rng, 65536) for _ in range(8)]
        dc = []
        for _ in range(128):
            p, n = _agent_trace_context(rng, 65536)
            dc.append(min(p + n, 65536))
        return pf, dc, False
    if cfg.name == "glm4.5-355b":
        budget = 8 * 1024 * 1024
        for attempt in range(1000):
            r = np.random.default_rng([cfg.seed, attempt])
            pf = [(int(r.integers(4096, 131073)), int(r.integers(256, 4097))) for _ in range(32)]
            dc = []
            for _ in range(224):
                p, n = _agent_trace_context(r, 131072)
                dc.append(min(p + n, 131072))
            if sum(p + n for p, n in pf) + sum(dc) <= budget:
                return pf, dc, False
        raise RuntimeError("no draw met the resident-token budget")
    raise KeyError(cfg.name)


def make_workload(
    cfg: Config,
    prefill: Optional[Sequence[Tuple[int, int]]] = None,
    decode: Optional[Sequence[int]] = None,
    shared_decode: Optional[bool] = None,
    slack_pages: Optional[int] = None,
    num_pages: Optional[int] = None,
) -> Workload:
    """Place every sequence's pages in one pool and build the block tables.

    Lengths default to the config's own law; tests pass explicit ones.
    The pool holds the needed pages plus at least 1/16 slack; physical ids
    come from a seeded permutation, so logical neighbours are scattered.
    """
    if prefill is None and decode is None:
        prefill, decode, shared = draw_lengths(cfg)
    else:
        prefill = list(prefill or [])
        decode = list(decode or [])
        shared = bool(shared_decode)
    if shared_decode is not None:
        shared = shared_decode
    ps = cfg.page_size
    lengths = [p + n for p, n in prefill]
    resident = [p for p, _ in prefill]
    if shared:
        # decode row b reads prefill sequence b after its new turn landed
        assert len(decode) <= len(prefill)
        for b, c in enumerate(decode):
            assert c <= lengths[b]
        dec_ids = list(range(len(decode)))
    else:
        dec_ids = list(range(len(prefill), len(prefill) + len(decode)))
        lengths += list(decode)
        resident += [c - 1 for c in decode]
    need = [-(-L // ps) for L in lengths]
    total = int(sum(need))
    rng = np.random.default_rng([cfg.seed, 0x9A6E])
    if num_pages is None:
        if cfg.name == "tiny" and slack_pages is None and total == 16:
            num_pages = 64
        else:
            slack = slack_pages if slack_pages is not None else max(1, total // 16)
            num_pages = total + slack
    assert num_pages >= total
    perm = rng.permutation(num_pages)[:total].astype(np.int32)
    seqs = []
    off = 0
    for sid, (L, r, k) in enumerate(zip(lengths, resident, need)):
        seqs.append(Sequence(sid, L, r, perm[off:off + k].copy(), (cfg.seed, 0x5E0, sid)))
        off += k

    def table(ids):
        mp = max([len(seqs[i].pages) for i in ids] + [1])
        bt = np.zeros((len(ids), mp), dtype=np.int32)
        for row, i in enumerate(ids):
            bt[row, :len(seqs[i].pages)] = seqs[i].pages
        return bt

    pf_ids = np.arange(len(prefill), dtype=np.int64)
    pf = Batch(pf_ids, np.array([p for p, _ in prefill], np.int32),
               np.array([n for _, n in prefill], np.int32), table(pf_ids))
    d_ids = np.array(dec_ids, dtype=np.int64)
    dc = Batch(d_ids, np.array([c - 1 for c in decode], np.int32),
               np.ones(len(decode), np.int32), table(d_ids))
    return Workload(cfg, int(num_pages), seqs, pf, dc)


# ---------------------------------------------------------------------------
# Values (torch generators; the device decides the bit stream)
# ---------------------------------------------------------------------------


def _torch():
    import torch

    return torch


def _dtype(name: str):
    torch = _torch()
    return {"f32": torch.float32, "bf16": torch.bfloat16}[name]


def _normal(seed: int, shape, device, out_dtype):
    torch = _torch()
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    return x.to(out_dtype)


def kv_dtype_in(cfg: Config) -> str:
    """dtype of raw (pre-pool) K/V: f32 for Tiny, bf16 otherwise."""
    return "f32" if cfg.kv_dtype == "f32" else "bf16"


def sequence_kv(wl: Workload, sid: int, device="cpu"):
    """Raw K, V of every token of sequence `sid`: [length, H_kv, D]."""
    cfg, s = wl.cfg, wl.seqs[sid]
    shape = (s.length, cfg.num_kv_heads, cfg.head_dim)
    dt = _dtype(kv_dtype_in(cfg))
    return (_normal(_mix(*s.stream, 1), shape, device, dt),
            _normal(_mix(*s.stream, 2), shape, device, dt))


def prefill_q(wl: Workload, b: int, device="cpu"):
    """Queries of prefill row b's new turn: [n_b, H_q, D]."""
    cfg = wl.cfg
    n = int(wl.prefill.q_lens[b])
    sid = int(wl.prefill.seq_ids[b])
    return _normal(_mix(*wl.seqs[sid].stream, 3), (n, cfg.num_q_heads, cfg.head_dim),
                   device, _dtype(cfg.q_dtype))


def decode_q(wl: Workload, b: int, device="cpu"):
    """Query of decode row b: [1, H_q, D]."""
    cfg = wl.cfg
    sid = int(wl.decode.seq_ids[b])
    return _normal(_mix(*wl.seqs[sid].stream, 4), (1, cfg.num_q_heads, cfg.head_dim),
                   device, _dtype(cfg.q_dtype))


def page_scales(wl: Workload, sid: int, k, v):
    """fp8 scale policy for sequence `sid`: per (logical page, head),
    s = amax/448 in fp32 over every value the page-head will hold, and
    s = 1 where amax is 0.  Returns (k_scale, v_scale) [pages, H_kv] fp32."""
    torch = _torch()
    ps = wl.cfg.page_size
    s = wl.seqs[sid]
    npg = len(s.pages)

    def one(x):
        pad = npg * ps - x.shape[0]
        xf = x.float().abs()
        if pad:
            xf = torch.cat([xf, xf.new_zeros((pad,) + tuple(xf.shape[1:]))])
        amax = xf.view(npg, ps, x.shape[1], x.shape[2]).amax(dim=(1, 3))
        sc = amax / torch.tensor(FP8_E4M3_MAX, dtype=torch.float32, device=x.device)
        return torch.where(amax > 0, sc, torch.ones_like(sc))

    return one(k), one(v)


def concat_rows(batch: Batch, per_row, device="cpu"):
    """Pack per-row tensors [q_len_b, ...] along dim 0 (cu_q_lens order)."""
    torch = _torch()
    parts = [per_row(b) for b in range(batch.num_seqs)]
    return torch.cat(parts) if parts else None
