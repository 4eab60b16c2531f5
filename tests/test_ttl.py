"""TTL control plane (host code, CPU only).

The oracle (oracle/ttl.py) is pinned to values worked out by hand from the
paper's definitions and to closed forms; the library's C++ scheduler is then
compared with it on hand-built scenarios and on random event traces."""
import math
import os
import re
import subprocess

import numpy as np
import pytest

from oracle import ttl as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def T():
    from paper_2511_02230_amd import ttl

    return ttl


# ----------------------------------------------------------------- ABI

def test_header_symbols_exported(T):
    text = open(os.path.join(ROOT, "include", "ckv_ttl.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    declared = set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M))
    from paper_2511_02230_amd import ckv

    out = subprocess.run(["nm", "-D", "--defined-only", ckv.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(line.split()[-1] for line in out.splitlines() if " T " in line)
    assert declared <= exported
    assert set(T.EXPORTS) == declared


def test_invalid_arguments(T):
    with pytest.raises(ValueError):
        T.Scheduler(0)
    s = T.Scheduler(10)
    s.arrive(1, 7, 4, 0.0)
    with pytest.raises(Exception):
        s.arrive(1, 8, 4, 0.0)      # duplicate request id
    with pytest.raises(Exception):
        s.arrive(2, 7, 4, 0.0)      # program already has a request waiting
    with pytest.raises(Exception):
        s.arrive(3, 9, 0, 0.0)      # no pages
    with pytest.raises(Exception):
        s.finish(1, 1.0)            # not running
    with pytest.raises(Exception):
        s.arrive(4, 10, 1, -1.0)    # time going backwards
    assert s.schedule(0.5)[0].request == 1
    with pytest.raises(Exception):
        s.finish(1, 1.0, next_tool=-1)


# ----------------------------------------------------------------- oracle pins

def test_oracle_eq2_worked_examples():
    # S = {1, 2, 3, 10}: candidate values with B = 5 are 0, 0.25, 0.5, 0.75, -5
    assert O.eq2_ttl([1.0, 2.0, 3.0, 10.0], 5.0) == 3.0
    # with B = 2 every positive candidate loses to tau = 0
    assert O.eq2_ttl([1.0, 2.0, 3.0, 10.0], 2.0) == 0.0
    # repeated durations raise the CDF step: {1, 1, 1, 4}, B = 2 -> 0.75*2-1 = 0.5 at tau = 1
    assert O.eq2_ttl([1.0, 1.0, 1.0, 4.0], 2.0) == 1.0
    # ties go to the smaller TTL: {2, 4}, B = 4 -> tau 2: 2-2 = 0 = tau 0
    assert O.eq2_ttl([2.0, 4.0], 4.0) == 0.0
    assert O.eq2_ttl([], 3.0) == 0.0


def test_oracle_cold_start_is_the_exp1_optimum():
    grid = np.linspace(0.0, 12.0, 120001)
    for B in [0.3, 1.0, 1.5, 2.0, math.e, 10.0, 1000.0]:
        obj = (1.0 - np.exp(-grid)) * B - grid
        assert O.cold_ttl(B) == pytest.approx(grid[np.argmax(obj)], abs=2e-4)
    assert O.cold_ttl(math.e) == pytest.approx(1.0)


def test_oracle_memoryfulness_closed_forms():
    assert O.memoryfulness([5] * 20) == pytest.approx(1.0, abs=1e-12)   # fixed N
    assert O.memoryfulness([1, 3]) == pytest.approx(5.0 / 11.0, abs=1e-12)  # worked by hand
    rng = np.random.default_rng(0)
    geo = rng.geometric(0.2, size=20000).tolist()                       # memoryless
    assert abs(O.memoryfulness(geo)) < 0.02
    assert O.memoryfulness([]) == 1.0 and O.memoryfulness([1]) == 1.0


def test_empirical_eq2_approaches_the_exp1_closed_form(T):
    """With many Exp(1) durations the empirical Eq. 2 optimum nears ln B."""
    rng = np.random.default_rng(1)
    S = rng.exponential(1.0, size=200000)
    for B in [2.0, 5.0, 20.0]:
        assert T.ttl_argmax(S, B) == pytest.approx(math.log(B), abs=0.08)


# ----------------------------------------------------------------- C++ vs oracle

def test_stateless_functions_match_the_oracle(T):
    rng = np.random.default_rng(2)
    for _ in range(300):
        n = int(rng.integers(1, 40))
        S = np.round(rng.exponential(2.0, size=n), int(rng.integers(0, 3)))  # ties, zeros
        B = float(rng.uniform(0.0, 10.0))
        got, ref = T.ttl_argmax(S, B), O.eq2_ttl(S.tolist(), B)
        val = lambda tau: O.cdf(S.tolist(), tau) * B - tau
        assert val(got) == pytest.approx(val(ref), abs=1e-12)
        assert T.ttl_cold(B) == pytest.approx(O.cold_ttl(B), abs=1e-15)
    for _ in range(50):
        Ns = rng.integers(1, 12, size=int(rng.integers(1, 30))).tolist()
        assert T.memoryfulness(Ns) == pytest.approx(O.memoryfulness(Ns), abs=1e-12)
    assert T.ttl_argmax([], 3.0) == 0.0


def _both(T, capacity, K=100, window=100, fixed=None):
    return T.Scheduler(capacity, K, window, fixed), O.Scheduler(capacity, K, window, fixed)


def _issued(s):
    return [(i.request, i.program, i.reused, i.held_pages) for i in s]


def _oissued(x):
    return [(a, b, c, d) for a, b, c, d, _ in x]


def test_pin_then_reuse_within_ttl(T):
    s, o = _both(T, 100)
    for x in (s, o):
        x.arrive(1, 1, 10, 0.0)
    assert _issued(s.schedule(0.0)) == _oissued(o.schedule(0.0)) == [(1, 1, False, 0)]
    # cold start: B = T + Prefill-Reload = 0 + e -> tau = ln e = 1
    assert s.finish(1, 1.0, next_tool=3, prefill_reload_s=math.e) == pytest.approx(1.0)
    assert o.finish(1, 1.0, next_tool=3, PR=math.e) == pytest.approx(1.0)
    assert s.pin_expiry(1) == pytest.approx(2.0)
    assert s.stats()["pinned_pages"] == 10 and s.stats()["free_pages"] == 90
    for x in (s, o):
        x.arrive(2, 1, 15, 1.5)  # the tool took 0.5 s
    assert s.stats()["tool_records"] == 1 and o.S == {3: [0.5]}
    assert _issued(s.schedule(1.5)) == _oissued(o.schedule(1.5)) == [(2, 1, True, 10)]
    assert s.stats()["running_pages"] == 15 and s.stats()["pinned_pages"] == 0


def test_expired_pin_is_kept_while_its_program_waits(T):
    for waiting in (False, True):
        s, o = _both(T, 100)
        for x in (s, o):
            x.arrive(1, 1, 10, 0.0)
            x.schedule(0.0)
        s.finish(1, 1.0, next_tool=0, prefill_reload_s=math.e)  # expires at 2
        o.finish(1, 1.0, next_tool=0, PR=math.e)
        for x in (s, o):
            x.arrive(5, 2, 5, 1.2)
            if waiting:
                x.arrive(2, 1, 12, 2.2)  # after the expiry, before the next step
        got, ref = s.schedule(2.5), o.schedule(2.5)
        assert _issued(got) == _oissued(ref)
        by = {i.request: i for i in got}
        if waiting:
            assert by[2].reused and by[2].held_pages == 10
        else:
            assert s.stats()["pinned"] == 0 and 2 not in by


def test_priority_order(T):
    s, o = _both(T, 1000)
    # program 1 arrives first but is not pinned; program 2 pinned; program 3 preempted
    for x in (s, o):
        x.arrive(10, 2, 5, 0.0)
        x.arrive(11, 3, 5, 0.1)
        x.schedule(0.1)
    s.finish(10, 0.5, next_tool=0, prefill_reload_s=100.0)
    o.finish(10, 0.5, next_tool=0, PR=100.0)
    s.preempt(11)
    o.preempt(11)
    for x in (s, o):
        x.arrive(12, 1, 5, 0.6)   # a new program
        x.arrive(13, 2, 6, 0.7)   # program 2 returns within its TTL
        x.arrive(14, 4, 5, 0.8)
    got = s.schedule(0.9)
    assert _issued(got) == _oissued(o.schedule(0.9))
    # preempted (11), pinned (13), then program arrival order: 12 (program 1
    # first seen at 0.6) before 14 (program 4 at 0.8)
    assert [i.request for i in got] == [11, 13, 12, 14]


def test_deadlock_breaker_unpins_latest_programs_first(T):
    s, o = _both(T, 30)
    for x in (s, o):
        for p in range(3):
            x.arrive(p, p, 10, float(p))
            x.schedule(float(p))
    for p in range(3):
        s.finish(p, 3.0 + p, next_tool=0, prefill_reload_s=100.0)
        o.finish(p, 3.0 + p, next_tool=0, PR=100.0)
    assert s.stats()["pinned_pages"] == 30 and s.stats()["free_pages"] == 0
    for x in (s, o):
        x.arrive(9, 9, 15, 6.0)
    got = s.schedule(6.0)
    assert _issued(got) == _oissued(o.schedule(6.0)) == [(9, 9, False, 0)]
    # programs 2 and 1 (latest arrivals) gave their pages; program 0 keeps its pin
    assert s.pin_expiry(0) > 0 and s.pin_expiry(1) < 0 and s.pin_expiry(2) < 0
    st = s.stats()
    assert st["pinned_pages"] == 10 and st["running_pages"] == 15 and st["free_pages"] == 5


def test_request_that_cannot_fit_stops_scheduling(T):
    s, o = _both(T, 10)
    for x in (s, o):
        x.arrive(1, 1, 8, 0.0)
        x.arrive(2, 2, 5, 0.0)
        x.arrive(3, 3, 1, 0.0)
    # 1 runs; 2 does not fit and stops the loop although 3 would fit (Alg. 1 break)
    assert _issued(s.schedule(0.0)) == _oissued(o.schedule(0.0)) == [(1, 1, False, 0)]
    assert s.stats()["waiting"] == 2


def test_cold_start_thresholds_and_queueing_delay(T):
    s = T.Scheduler(100, min_records=2, wait_window=2)
    o = O.Scheduler(100, K=2, window=2)
    # at most K records: cold start ln(T + PR)
    for d in (1.0, 3.0):
        s.record_tool(0, d)
        o.S.setdefault(0, []).append(d)
        o.S_all.append(d)
    assert s.ttl(0, 5.0) == pytest.approx(math.log(5.0)) == pytest.approx(o.ttl(0, 5.0))
    # K + 1 records in total, at most K for tool 1: the CDF of all tools
    s.record_tool(1, 2.0)
    o.S.setdefault(1, []).append(2.0)
    o.S_all.append(2.0)
    # S = {1, 2, 3}, B = 0 * eta + 5: values 0, 1/3*5-1, 2/3*5-2, 5-3 = 2 -> tau 3
    assert s.ttl(1, 5.0) == 3.0 == o.ttl(1, 5.0)
    # more than K for tool 0: its own CDF {1, 3, 2.5}
    s.record_tool(0, 2.5)
    o.S[0].append(2.5)
    o.S_all.append(2.5)
    # B = 1.2: tool 0 values: 1/3*1.2-1 < 0, ... -> tau 0; all tools: same
    assert s.ttl(0, 1.2) == 0.0 == o.ttl(0, 1.2)
    assert s.ttl(0, 9.0) == o.ttl(0, 9.0) == 3.0


def test_queueing_delay_window(T):
    s, o = _both(T, 5, K=100, window=2)
    # one program at a time fits; program 1's cache is never pinned (tau = 0)
    for x in (s, o):
        x.arrive(1, 1, 5, 0.0)
        x.schedule(0.0)
    delays = []
    t = 0.0
    for turn in range(4):
        # T + 0.5 stays below 1, so the cold-start TTL ln(T + 0.5) is 0: never pinned
        s.finish(1 + turn, t + 1.0, next_tool=0, prefill_reload_s=0.5)
        o.finish(1 + turn, t + 1.0, next_tool=0, PR=0.5)
        for x in (s, o):
            x.arrive(2 + turn, 1, 5, t + 2.0)
        wait = 0.1 * (turn + 1)
        got = s.schedule(t + 2.0 + wait)
        assert _issued(got) == _oissued(o.schedule(t + 2.0 + wait))
        delays.append(wait)
        assert s.stats()["mean_wait_s"] == pytest.approx(np.mean(delays[-2:]))
        t += 2.0 + wait


def _random_trace(seed):
    """Events of agent programs on a small pool: arrivals after tool calls,
    finishes after a service time, schedule steps in between."""
    rng = np.random.default_rng(seed)
    n_prog = int(rng.integers(3, 12))
    turns = {p: int(rng.integers(1, 6)) for p in range(n_prog)}
    events = []  # (time, kind, program)
    for p in range(n_prog):
        events.append((float(rng.uniform(0, 5)), "arrive", p))
    return rng, turns, sorted(events)


@pytest.mark.parametrize("seed", range(16))
def test_random_traces_match_the_oracle(T, seed):
    rng, turns, events = _random_trace(seed)
    cap = int(rng.integers(20, 80))
    K = int(rng.integers(0, 6))
    fixed = [None, None, 0.0, 1.5][seed % 4]  # Eq. 2, no retention, static TTL
    s, o = _both(T, cap, K=K, window=int(rng.integers(1, 5)), fixed=fixed)
    served = {p: 0 for p in turns}
    rid = 0
    queue = list(events)
    running = {}  # request -> (program, finish time)
    now = 0.0
    steps = 0
    while (queue or running) and steps < 2000:
        steps += 1
        nxt = min([e[0] for e in queue] + [f for _, f in running.values()])
        now = max(now, nxt)
        for e in [e for e in queue if e[0] <= now]:
            queue.remove(e)
            p = e[2]
            rid += 1
            pages = int(rng.integers(1, 12)) + 2 * served[p]
            s.arrive(rid, p, pages, now)
            o.arrive(rid, p, pages, now)
        for r, (p, f) in list(running.items()):
            if f <= now:
                del running[r]
                served[p] += 1
                last = served[p] == turns[p]
                tool = int(rng.integers(0, 3))
                pr = float(rng.uniform(0, 6))
                a = s.finish(r, now, last=last, next_tool=tool, prefill_reload_s=pr)
                b = o.finish(r, now, last=last, next_tool=tool, PR=pr)
                assert a == pytest.approx(b, abs=1e-12)
                if not last:
                    queue.append((now + float(rng.exponential(1.5)), "arrive", p))
        got = s.schedule(now)
        ref = o.schedule(now)
        assert _issued(got) == _oissued(ref)
        for i in got:
            running[i.request] = (i.program, now + float(rng.uniform(0.1, 2.0)))
        st = s.stats()
        assert st["pinned_pages"] == sum(q["pin_pages"] for q in o.prog.values() if q["pinned"])
        assert st["mean_wait_s"] == pytest.approx(o.T(), abs=1e-12)
        assert st["eta"] == pytest.approx(O.memoryfulness(o.finished_N), abs=1e-12)
    # every program ran to its end: pins never starve the pool (the breaker)
    assert not queue and not running
    assert s.stats()["waiting"] == 0 and s.stats()["pinned"] == 0 and not o.prog
