"""Agent-serving simulation over the TTL control plane: host logic on the
CPU; on the GPU, real kv_append / prefix_prefill_attn turns through the
pages the scheduler kept, each TTL hit checked against a rebuild."""
import numpy as np
import pytest

from paper_2511_02230_amd import serve_sim as sim


def test_trace_is_seeded_and_bounded():
    a = sim.make_trace(3, 20, 0.5, mean_turns=5, max_context=8000)
    b = sim.make_trace(3, 20, 0.5, mean_turns=5, max_context=8000)
    assert [(p.arrival, p.turns) for p in a] == [(p.arrival, p.turns) for p in b]
    for p in a:
        assert 1 <= len(p.turns) <= 5
        assert sum(n + o for n, o, _ in p.turns) <= 8000
    arr = [p.arrival for p in a]
    assert arr == sorted(arr)
    g = sim.make_trace(4, 400, 0.5, mean_turns=4, turns_law="geometric")
    assert 3.0 < np.mean([len(p.turns) for p in g]) < 5.0


def test_cost_model_prefix_reuse_is_cheaper_than_rebuild():
    c = sim.CostModel()
    # a reuse prefill plus the prefix's own prefill covers the whole
    # context's attention, up to one extra per-call constant
    a, b, k = c.attn_ms
    whole = c.prefill_s(0, 12000)
    split = c.prefill_s(0, 10000) + c.prefill_s(10000, 2000)
    assert split == pytest.approx(whole + c.layers * k * 1e-3)
    assert c.prefill_s(10000, 2000) < c.prefill_s(0, 12000)
    c2 = sim.CostModel(offload_gbps=56.0)
    assert c2.rebuild_s(20000) == pytest.approx(20000 * c2.kv_bytes_per_token / 56e9)
    assert c.rebuild_s(0) == 0.0


@pytest.mark.parametrize("policy", ["ttl", "none", "static:3"])
def test_every_program_completes_and_nothing_leaks(policy):
    trace = sim.make_trace(5, 40, 0.5, mean_turns=4, max_context=20000)
    c = sim.CostModel()
    r = sim.simulate(trace, c, capacity_pages=4000, policy=policy, min_records=10)
    assert r["leftover"] == {"waiting": 0, "running": 0, "pinned": 0}
    assert r["hits"] + r["misses"] == sum(len(p.turns) - 1 for p in trace)
    if policy == "none":
        assert r["hits"] == 0


def test_pinning_for_longer_than_every_tool_hits_every_turn():
    trace = sim.make_trace(6, 30, 0.2, mean_turns=4, max_context=20000)
    longest = max(max(p.tool_s[:-1] or [0.0]) for p in trace)
    r = sim.simulate(trace, sim.CostModel(), capacity_pages=10 ** 7, policy=f"static:{longest + 1}")
    assert r["misses"] == 0 and r["rebuilt_tokens"] == 0
    none = sim.simulate(trace, sim.CostModel(), capacity_pages=10 ** 7, policy="none")
    assert none["mean_jct_s"] > r["mean_jct_s"]


@pytest.mark.gpu
def test_gpu_turns_hits_match_rebuilds():
    import workload

    print("[sim] gpu turns", flush=True)
    cfg = workload.LLAMA8B
    trace = sim.make_trace(7, 8, 2.0, mean_turns=4, first_tokens=(300, 0.3), turn_tokens=(120, 0.5),
                           out_tokens=(16, 0.3), tool_means=(0.2, 1.0, 3.0), max_context=2000)
    cost = sim.CostModel(decode_s_per_token=0.005)
    cap = 200  # pages: tight enough that some pins are dropped
    gpu = sim.GpuLayer(cfg, cap, max_context=2048, num_programs=len(trace), check=True)
    r = sim.simulate(trace, cost, cap, policy="static:1.5", min_records=5, gpu=gpu)
    assert r["leftover"] == {"waiting": 0, "running": 0, "pinned": 0}
    assert r["hits"] > 0 and r["gpu_checked_hits"] == r["hits"]
    assert r["gpu_hit_vs_rebuild_max_abs_diff"] <= 2e-2
    assert r["gpu_attention_ms_one_layer"] > 0
    assert sorted(gpu.free) == list(range(cap))  # every page came back
