"""Seeded workload generator: determinism and structural invariants (CPU)."""
import numpy as np
import pytest
import torch

import workload


@pytest.mark.parametrize("name", list(workload.CONFIGS))
def test_lengths_follow_the_config_laws(name):
    cfg = workload.CONFIGS[name]
    pf, dc, shared = workload.draw_lengths(cfg)
    P = np.array([p for p, _ in pf])
    n = np.array([m for _, m in pf])
    if name == "tiny":
        assert pf == [(240, 16)] and dc == [256] and shared
    elif name == "llama3.1-8b":
        assert len(pf) == 16 and len(dc) == 64
        assert P.min() >= 2048 and P.max() <= 16384 and n.min() >= 128 and n.max() <= 2048
        assert min(dc) >= 4096 and max(dc) <= 32768
    elif name == "gemma3-12b":
        assert len(pf) == 32 and len(dc) == 64
        assert P.max() <= 32768 and n.min() >= 256 and n.max() <= 4096
    elif name == "llama3.1-70b":
        assert len(pf) == 8 and len(dc) == 128
        assert P.max() <= 65536 and n.min() >= 64 and n.max() <= 4096 and max(dc) <= 65536
    elif name == "glm4.5-355b":
        assert len(pf) == 32 and len(dc) == 224
        assert P.max() <= 131072 and n.min() >= 256 and n.max() <= 4096 and max(dc) <= 131072
        assert int((P + n).sum()) + sum(dc) <= 8 * 1024 * 1024


@pytest.mark.parametrize("name", list(workload.CONFIGS))
def test_pages_are_distinct_and_in_range(name):
    wl = workload.make_workload(workload.CONFIGS[name])
    allp = np.concatenate([s.pages for s in wl.seqs])
    assert len(np.unique(allp)) == len(allp)
    assert allp.min() >= 0 and allp.max() < wl.num_pages
    assert wl.num_pages >= len(allp) + (0 if name == "tiny" else len(allp) // 16)
    for batch in (wl.prefill, wl.decode):
        for b in range(batch.num_seqs):
            s = wl.seqs[int(batch.seq_ids[b])]
            end = int(batch.ctx_lens[b] + batch.q_lens[b])
            assert end <= s.length
            npg = -(-end // wl.cfg.page_size)
            assert np.array_equal(batch.block_table[b, :npg], s.pages[:npg])


def test_tiny_pool_is_16_of_64_pages():
    wl = workload.make_workload(workload.TINY)
    assert wl.num_pages == 64 and len(wl.seqs) == 1 and len(wl.seqs[0].pages) == 16
    assert int(wl.decode_ctx[0]) == 256 and int(wl.decode.seq_ids[0]) == 0


def test_values_are_deterministic_and_per_sequence():
    wl = workload.make_workload(workload.LLAMA8B, prefill=[(40, 8), (30, 5)], decode=[17])
    k1, v1 = workload.sequence_kv(wl, 1)
    k1b, v1b = workload.sequence_kv(wl, 1)
    assert torch.equal(k1.view(torch.int16), k1b.view(torch.int16))
    k0, _ = workload.sequence_kv(wl, 0)
    assert not torch.equal(k0[:30].float(), k1.float())
    assert not torch.equal(k1.float(), v1.float())
    q = workload.prefill_q(wl, 0)
    assert q.shape == (8, 32, 128) and q.dtype == torch.bfloat16
    # roughly N(0, 1)
    x = k0.float()
    assert abs(float(x.mean())) < 0.05 and abs(float(x.std()) - 1) < 0.05


def test_fp8_scales_cover_page_head_amax():
    wl = workload.make_workload(workload.GLM355B, prefill=[(100, 50)], decode=[70])
    for sid in range(2):
        k, v = workload.sequence_kv(wl, sid)
        ks, vs = workload.page_scales(wl, sid, k, v)
        assert ks.shape == (len(wl.seqs[sid].pages), 8)
        x = k.float().abs()
        for pg in range(ks.shape[0]):
            amax = x[pg * 64:(pg + 1) * 64].amax(dim=(0, 2))
            assert torch.all(amax / ks[pg] <= 448.0 * (1 + 2 ** -23))
