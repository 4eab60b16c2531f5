"""paged_decode_attn_noalloc (needs an MI355X): the allocation-free decode
entry point, called through the C ABI, returns the same bits as
paged_decode_attn with a caller workspace, on two calls in a row (the second
with a smaller batch, so it reads partials the first call's larger ones were
written over), bf16 and fp8 pools, and both match the fp64 oracle.  Sizes
beyond the scratch are rejected before anything runs."""
import numpy as np
import pytest
import torch

import workload
from tests import parity
from tests.oracle_inputs import OracleState, to_numpy
from oracle import formats

pytestmark = pytest.mark.gpu


def _cfg(kv):
    if kv == "bf16":
        return workload.Config("na16", 21, 32, 8, 128, 16, "bf16", "bf16")
    return workload.Config("na8", 22, 48, 4, 128, 64, "bf16", "fp8")


def _out_f64(t):
    x = to_numpy(t)
    return formats.bf16_bits_to_f64(x)


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
def test_noalloc_decode_matches_the_workspace_entry_point(kv):
    from paper_2511_02230_amd import ckv
    from paper_2511_02230_amd.harness import DeviceWorkload

    cfg = _cfg(kv)
    calls = [[9000, 1, 4100, 777, 12000, 65, 3000, 2048],  # first call: many partitions
             [700, 5000, 33]]                              # second call: fewer, smaller
    for i, ctx in enumerate(calls):
        print(f"case noalloc kv={kv} call {i} contexts {ctx}", flush=True)
        wl = workload.make_workload(cfg, prefill=[], decode=ctx)
        dw = DeviceWorkload(wl, "cuda")
        dw.append_decode()
        st = OracleState(wl, device="cuda")
        st.append_decode()
        for split in (0, 512):
            need = ckv.decode_workspace_bytes(dw.pool, dw.decode, cfg.num_q_heads, split)
            assert 0 < need <= ckv.DECODE_SCRATCH_BYTES
            ref_out = dw.run_decode(kv_split_len=split).clone()
            na = torch.full_like(ref_out, float("nan"))
            ckv.paged_decode_attn_noalloc(dw.pool, dw.decode, dw.q_decode, cfg.softmax_scale, na,
                                          0, split)
            torch.cuda.synchronize()
            assert torch.equal(na.view(torch.int16), ref_out.view(torch.int16)), (kv, i, split)
            ref = st.decode(to_numpy(dw.q_decode), st.rows_of(wl.decode))
            got = _out_f64(na)
            for b, r in ref.items():
                bad, summary = parity.failures(got[b], r, parity.kind_of(cfg))
                assert not bad, (kv, i, split, b, summary, bad)


def test_noalloc_decode_rejects_partials_beyond_the_scratch():
    from paper_2511_02230_amd import ckv

    cfg = _cfg("bf16")
    pool = ckv.Pool(torch.zeros(4, 8, 16, 128, dtype=torch.bfloat16, device="cuda"),
                    torch.zeros(4, 8, 16, 128, dtype=torch.bfloat16, device="cuda"))
    B = 2048
    big = ckv.Batch(torch.zeros((B, 4096), dtype=torch.int32, device="cuda"),
                    torch.full((B,), 65536, dtype=torch.int32, device="cuda"), None, B, 1, 65536)
    need = ckv.decode_workspace_bytes(pool, big, cfg.num_q_heads, 512)
    assert need > ckv.DECODE_SCRATCH_BYTES
    q = torch.zeros((B, cfg.num_q_heads, 128), dtype=torch.bfloat16, device="cuda")
    out = torch.zeros_like(q)
    with pytest.raises(ckv.CkvError) as e:
        ckv.paged_decode_attn_noalloc(pool, big, q, cfg.softmax_scale, out, 0, 512)
    assert e.value.code == 3
    torch.cuda.synchronize()
    assert not bool(out.any())  # nothing ran
