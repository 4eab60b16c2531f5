"""Plain Python restatement of Continuum's TTL control plane.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this.

  cdf(S, tau)        empirical CDF of tool durations (Sec. 4.2)
  eq2_ttl(S, B)      Eq. 2: the candidate in {0} U S maximizing cdf * B - tau
                     (first of equal values, candidates ascending)
  cold_ttl(B)        the cold-start TTL: the optimum of Eq. 2 when durations
                     follow Exp(1) (cdf = 1 - e^-tau) and eta = 1 (Sec. 4.2)
  memoryfulness(Ns)  eta = -Corr(k, N - k) over the requests of finished
                     programs (Sec. 4.1)
  Scheduler          Alg. 1 with the Sec. 4.3 order and the Sec. 5.2 pin,
                     unpin and deadlock rules, with lists and linear scans
"""
from __future__ import annotations

import math


def cdf(S, tau):
    return sum(1 for t in S if t <= tau) / len(S)


def eq2_ttl(S, B):
    if not S:
        return 0.0
    best_tau, best = None, None
    for tau in [0.0] + sorted(set(S)):
        val = cdf(S, tau) * B - tau
        if best is None or val > best:
            best_tau, best = tau, val
    return best_tau


def cold_ttl(B):
    # d/dtau [(1 - e^-tau) B - tau] = B e^-tau - 1 vanishes at tau = ln B,
    # a maximum (second derivative -B e^-tau < 0); for B <= 1 the objective
    # decreases on tau >= 0, so tau = 0
    return math.log(B) if B > 1.0 else 0.0


def memoryfulness(Ns):
    ks, rs = [], []
    for N in Ns:
        for k in range(N):
            ks.append(k)
            rs.append(N - k)
    n = len(ks)
    if n < 2:
        return 1.0
    mk, mr = sum(ks) / n, sum(rs) / n
    ckr = sum((a - mk) * (b - mr) for a, b in zip(ks, rs))
    ckk = sum((a - mk) ** 2 for a in ks)
    crr = sum((b - mr) ** 2 for b in rs)
    if ckk <= 0 or crr <= 0:
        return 1.0
    return -ckr / math.sqrt(ckk * crr)


class Scheduler:
    def __init__(self, capacity, K=100, window=100, fixed=None):
        self.capacity, self.K, self.window, self.fixed = capacity, K, window, fixed
        self.S = {}          # tool -> durations
        self.S_all = []
        self.waits = []      # queueing delays of requests whose cache was gone
        self.finished_N = []  # request counts of finished programs
        self.waiting = []    # dicts: id, program, pages, arrival, preempted
        self.running = {}    # id -> request dict
        self.prog = {}       # program -> state dict

    # ---- statistics
    def T(self):
        w = self.waits[-self.window:]
        return sum(w) / len(w) if w else 0.0

    def ttl(self, tool, PR):
        if self.fixed is not None:
            return self.fixed
        if len(self.S_all) <= self.K:
            return cold_ttl(self.T() * 1.0 + PR)
        B = self.T() * memoryfulness(self.finished_N) + PR
        S = self.S.get(tool, [])
        return eq2_ttl(self.S_all if len(S) <= self.K else S, B)

    def used(self):
        return (sum(r["pages"] for r in self.running.values())
                + sum(p["pin_pages"] for p in self.prog.values() if p["pinned"]))

    # ---- Alg. 1
    def arrive(self, rid, program, pages, now, preempted=False):
        p = self.prog.get(program)
        if p is None:
            p = self.prog[program] = dict(first=now, served=0, pinned=False, expiry=0.0, pin_pages=0,
                                          tool=None, finish=0.0)
        if p["tool"] is not None:
            d = now - p["finish"]
            self.S.setdefault(p["tool"], []).append(d)
            self.S_all.append(d)
            p["tool"] = None
        self.waiting.append(dict(id=rid, program=program, pages=pages, arrival=now, preempted=preempted))

    def finish(self, rid, now, last=False, next_tool=0, PR=0.0):
        r = self.running.pop(rid)
        p = self.prog[r["program"]]
        p["served"] += 1
        if last:
            self.finished_N.append(p["served"])
            del self.prog[r["program"]]
            return 0.0
        tau = self.ttl(next_tool, PR)
        if tau > 0:
            p.update(pinned=True, expiry=now + tau, pin_pages=r["pages"])
        p.update(tool=next_tool, finish=now)
        return tau

    def preempt(self, rid):
        r = self.running.pop(rid)
        r["preempted"] = True
        self.waiting.append(r)

    def _key(self, r):
        p = self.prog[r["program"]]
        return (not r["preempted"], not p["pinned"], p["first"], r["arrival"], r["id"])

    def schedule(self, now):
        out = []
        while self.waiting:
            waiting_programs = {r["program"] for r in self.waiting}
            for pid, p in self.prog.items():
                if p["pinned"] and now > p["expiry"] and pid not in waiting_programs:
                    p.update(pinned=False, pin_pages=0)
            r = min(self.waiting, key=self._key)
            p = self.prog[r["program"]]
            own = p["pin_pages"] if p["pinned"] else 0
            need = max(r["pages"] - own, 0)
            while need > self.capacity - self.used():
                victims = [(q["first"], pid) for pid, q in self.prog.items()
                           if q["pinned"] and pid != r["program"]]
                if not victims:
                    break
                _, vid = max(victims)
                self.prog[vid].update(pinned=False, pin_pages=0)
            if need > self.capacity - self.used():
                break
            self.waiting.remove(r)
            reused = p["pinned"]
            if reused:
                p.update(pinned=False, pin_pages=0)
            elif p["served"] > 0 and not r["preempted"]:
                self.waits.append(now - r["arrival"])
            r["preempted"] = False
            self.running[r["id"]] = r
            out.append((r["id"], r["program"], reused, own, now - r["arrival"]))
        return out
