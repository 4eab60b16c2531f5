"""Offline prefill-vs-context profile: host logic on the CPU, one small
sweep (with a parity check of a chunk view) on the GPU."""
import numpy as np
import pytest

from paper_2511_02230_amd import offline_profile as op


def test_length_ladder_doubles_up_to_the_maximum():
    assert op.length_ladder(65536) == [1000, 2000, 4000, 8000, 16000, 32000, 64000, 65536]
    assert op.length_ladder(1000) == [1000]
    assert op.length_ladder(3000, first=1000) == [1000, 2000, 3000]
    with pytest.raises(ValueError):
        op.length_ladder(0)


def test_chunk_plan_covers_every_token_once():
    for L, C in [(0, 16), (1, 16), (2048, 2048), (5000, 2048), (4096, 256)]:
        plan = op.chunk_plan(L, C)
        covered = [p + t for p, n in plan for t in range(n)]
        assert covered == list(range(L))
        assert all(n <= C for _, n in plan) and all(p % C == 0 for p, _ in plan)


def test_quadratic_fit_recovers_exact_coefficients():
    L = np.array([1000, 2000, 4000, 8000, 16000], dtype=np.float64)
    t = 3e-9 * L * L + 2e-5 * L + 0.7
    f = op.fit_quadratic(L, t)
    assert f["a"] == pytest.approx(3e-9, rel=1e-6)
    assert f["b"] == pytest.approx(2e-5, rel=1e-5)
    assert f["c"] == pytest.approx(0.7, rel=1e-5)
    assert f["r2"] == pytest.approx(1.0, abs=1e-12)
    with pytest.raises(ValueError):
        op.fit_quadratic([1, 2], [1, 2])


def test_attention_flops_counts_visible_pairs():
    # row at absolute position i sees i + 1 keys (min(i + 1, W) with a window)
    assert op.attention_flops(0, 3, 2, 4) == 4 * 4 * 2 * (1 + 2 + 3)
    assert op.attention_flops(10, 2, 1, 8) == 4 * 8 * 1 * (11 + 12)
    assert op.attention_flops(10, 2, 1, 8, window=5) == 4 * 8 * 1 * (5 + 5)
    # chunked prefill of L tokens does the same attention work as one prefill
    full = op.attention_flops(0, 5000, 8, 64)
    chunked = sum(op.attention_flops(p, n, 8, 64) for p, n in op.chunk_plan(5000, 1024))
    assert chunked == full


@pytest.mark.gpu
def test_small_sweep_on_gpu_and_chunk_view_parity():
    import torch

    import workload
    from tests.oracle_inputs import OracleState, to_numpy

    cfg = workload.Config("prof", 5, 16, 4, 128, 16, "bf16", "bf16")
    timer = op.PrefillTimer(cfg, 2048)
    # a chunk view (P = 512, n = 256) equals rows 512..767 of the full prefill
    bt = timer._batch(512, 256)
    out = timer.ckv.prefix_prefill_attn(timer.dw.pool, bt, timer.q[512:768].contiguous(),
                                        cfg.softmax_scale, 0)
    torch.cuda.synchronize()
    st = OracleState(timer.wl, device="cuda")
    st.append_prefill()
    ref = st.prefill(to_numpy(timer.q), [0], 0, {0: np.arange(512, 768)})[0]
    from oracle import formats
    got = formats.bf16_bits_to_f64(to_numpy(out))
    err = np.abs(got - ref)
    assert err.max() <= 2e-2 and err.mean() <= 2e-3
    # timings rise with context and follow a quadratic
    lengths = op.length_ladder(2048, first=256)
    ms = [timer.time([(0, L)], reps=3) for L in lengths]
    assert all(t > 0 for t in ms)
    assert ms[-1] > ms[0]
    assert op.fit_quadratic(lengths, ms)["r2"] > 0.9


@pytest.mark.gpu
def test_transfer_profile_small():
    import workload

    cfg = workload.Config("prof", 5, 16, 4, 128, 16, "bf16", "bf16")
    res = op.transfer_profile(cfg, [8, 64], reps=3)
    assert res["bytes"] == [2 * n * 4 * 16 * 128 * 2 for n in (8, 64)]
    for key in ("offload", "reload", "copy_d2h", "copy_h2d"):
        assert all(g > 0 for g in res["gbps"][key])


def test_linear_fit_recovers_bandwidth_and_fixed_cost():
    x = np.array([1e6, 4e6, 16e6, 64e6])
    t = 0.025 + x / 56e9 * 1e3  # ms: 25 us + bytes at 56 GB/s
    f = op.fit_linear(x, t)
    assert f["gbps"] == pytest.approx(56.0, rel=1e-9)
    assert f["t0_us"] == pytest.approx(25.0, rel=1e-9)
    assert f["r2"] == pytest.approx(1.0, abs=1e-12)
    with pytest.raises(ValueError):
        op.fit_linear([1.0], [1.0])
