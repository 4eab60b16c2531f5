"""ctypes binding of the TTL control plane in libckv.so (include/ckv_ttl.h):
argument marshalling only.  Every decision is taken by the library's C++
scheduler; this module converts Python values and raises on error codes.
"""
from __future__ import annotations

import ctypes
import dataclasses
from typing import List, Sequence

import numpy as np

from .ckv import LIB, CkvError

EXPORTS = ("ckv_sched_create", "ckv_sched_destroy", "ckv_sched_arrive", "ckv_sched_finish",
           "ckv_sched_schedule", "ckv_sched_preempt", "ckv_sched_ttl", "ckv_sched_record_tool",
           "ckv_sched_stats", "ckv_sched_pin_expiry", "ckv_ttl_argmax", "ckv_ttl_cold",
           "ckv_memoryfulness")


class ConfigT(ctypes.Structure):
    _fields_ = [("min_records", ctypes.c_int32), ("wait_window", ctypes.c_int32),
                ("fixed_ttl_s", ctypes.c_double)]


class IssueT(ctypes.Structure):
    _fields_ = [("request", ctypes.c_int64), ("program", ctypes.c_int32), ("reused", ctypes.c_int32),
                ("held_pages", ctypes.c_int64), ("queue_delay_s", ctypes.c_double)]


class StatsT(ctypes.Structure):
    _fields_ = [("capacity_pages", ctypes.c_int64), ("free_pages", ctypes.c_int64),
                ("pinned_pages", ctypes.c_int64), ("running_pages", ctypes.c_int64),
                ("waiting", ctypes.c_int32), ("running", ctypes.c_int32), ("pinned", ctypes.c_int32),
                ("tool_records", ctypes.c_int64), ("mean_wait_s", ctypes.c_double),
                ("eta", ctypes.c_double)]


def _bind():
    vp, i32, i64, f64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    sig = {
        "ckv_sched_create": ([ctypes.POINTER(ConfigT), i64], vp),
        "ckv_sched_destroy": ([vp], None),
        "ckv_sched_arrive": ([vp, i64, i32, i64, i32, f64], ctypes.c_int),
        "ckv_sched_finish": ([vp, i64, i32, i32, f64, f64, ctypes.POINTER(f64)], ctypes.c_int),
        "ckv_sched_schedule": ([vp, f64, ctypes.POINTER(IssueT), i32], i32),
        "ckv_sched_preempt": ([vp, i64], ctypes.c_int),
        "ckv_sched_ttl": ([vp, i32, f64], f64),
        "ckv_sched_record_tool": ([vp, i32, f64], ctypes.c_int),
        "ckv_sched_stats": ([vp, ctypes.POINTER(StatsT)], None),
        "ckv_sched_pin_expiry": ([vp, i32], f64),
        "ckv_ttl_argmax": ([vp, i64, f64], f64),
        "ckv_ttl_cold": ([f64], f64),
        "ckv_memoryfulness": ([vp, i64], f64),
    }
    for name, (args, res) in sig.items():
        fn = getattr(LIB, name)
        fn.argtypes = args
        fn.restype = res


_bind()


def _check(name: str, code: int):
    if code != 0:
        raise CkvError(name, code)


@dataclasses.dataclass(frozen=True)
class Issue:
    request: int
    program: int
    reused: bool
    held_pages: int
    queue_delay_s: float


class Scheduler:
    """Alg. 1 over a pool of `capacity_pages` pages with a caller-driven clock.
    fixed_ttl_s None: the TTL of Eq. 2; a number: that TTL for every pin."""

    def __init__(self, capacity_pages: int, min_records: int = 100, wait_window: int = 100,
                 fixed_ttl_s=None):
        cfg = ConfigT(min_records, wait_window, -1.0 if fixed_ttl_s is None else float(fixed_ttl_s))
        self._h = LIB.ckv_sched_create(ctypes.byref(cfg), int(capacity_pages))
        if not self._h:
            raise ValueError("invalid scheduler configuration")

    def close(self):
        if self._h:
            LIB.ckv_sched_destroy(self._h)
            self._h = None

    def __del__(self):
        self.close()

    def arrive(self, request: int, program: int, pages: int, now: float, preempted: bool = False):
        _check("ckv_sched_arrive", LIB.ckv_sched_arrive(self._h, request, program, pages,
                                                        1 if preempted else 0, float(now)))

    def finish(self, request: int, now: float, last: bool = False, next_tool: int = 0,
               prefill_reload_s: float = 0.0) -> float:
        tau = ctypes.c_double(0.0)
        _check("ckv_sched_finish", LIB.ckv_sched_finish(self._h, request, 1 if last else 0, next_tool,
                                                        float(prefill_reload_s), float(now),
                                                        ctypes.byref(tau)))
        return tau.value

    def schedule(self, now: float, max_issued: int = 4096) -> List[Issue]:
        buf = (IssueT * max_issued)()
        n = LIB.ckv_sched_schedule(self._h, float(now), buf, max_issued)
        return [Issue(int(b.request), int(b.program), bool(b.reused), int(b.held_pages),
                      float(b.queue_delay_s)) for b in buf[:n]]

    def preempt(self, request: int):
        _check("ckv_sched_preempt", LIB.ckv_sched_preempt(self._h, request))

    def ttl(self, tool: int, prefill_reload_s: float) -> float:
        return float(LIB.ckv_sched_ttl(self._h, tool, float(prefill_reload_s)))

    def record_tool(self, tool: int, duration_s: float):
        _check("ckv_sched_record_tool", LIB.ckv_sched_record_tool(self._h, tool, float(duration_s)))

    def stats(self) -> dict:
        st = StatsT()
        LIB.ckv_sched_stats(self._h, ctypes.byref(st))
        return {name: getattr(st, name) for name, _ in StatsT._fields_}

    def pin_expiry(self, program: int) -> float:
        return float(LIB.ckv_sched_pin_expiry(self._h, program))


def ttl_argmax(durations: Sequence[float], benefit_s: float) -> float:
    d = np.ascontiguousarray(durations, dtype=np.float64)
    return float(LIB.ckv_ttl_argmax(d.ctypes.data if d.size else None, d.size, float(benefit_s)))


def ttl_cold(benefit_s: float) -> float:
    return float(LIB.ckv_ttl_cold(float(benefit_s)))


def memoryfulness(requests_per_program: Sequence[int]) -> float:
    n = np.ascontiguousarray(requests_per_program, dtype=np.int32)
    return float(LIB.ckv_memoryfulness(n.ctypes.data if n.size else None, n.size))
