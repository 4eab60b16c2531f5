// KV-cache time-to-live control plane: tool statistics, Eq. 2 with its cold
// start, the TTL-aware queue order, pins and the deadlock breaker.  Host
// code only; the contract of every entry point is in include/ckv_ttl.h.
#include "../../include/ckv_ttl.h"

#include <algorithm>
#include <cmath>
#include <deque>
#include <limits>
#include <map>
#include <new>
#include <unordered_map>
#include <vector>

namespace {

// Sorted multiset of durations with a running count, for the empirical CDF.
struct Durations {
  std::vector<double> v;  // ascending
  void add(double d) { v.insert(std::upper_bound(v.begin(), v.end(), d), d); }
};

// Eq. 2 over sorted durations: candidates 0 and every distinct duration; the
// CDF at candidate c is the count of durations <= c over n.
double argmax_sorted(const std::vector<double> &d, double benefit) {
  const size_t n = d.size();
  if (n == 0) return 0.0;
  const double inv = 1.0 / (double)n;
  size_t at_zero = std::upper_bound(d.begin(), d.end(), 0.0) - d.begin();
  double best_tau = 0.0, best = (double)at_zero * inv * benefit;
  for (size_t i = 0; i < n;) {
    size_t j = i;
    while (j < n && d[j] == d[i]) ++j;  // d[i .. j) equal
    const double tau = d[i];
    if (tau > 0.0) {
      const double val = (double)j * inv * benefit - tau;
      if (val > best) {
        best = val;
        best_tau = tau;
      }
    }
    i = j;
  }
  return best_tau;
}

double cold_ttl(double benefit) { return benefit > 1.0 ? std::log(benefit) : 0.0; }

// -Corr(k, N - k) over k = 0 .. N_p - 1 of every program; 1 if undefined.
struct EtaAcc {
  double n = 0, sk = 0, sr = 0, skk = 0, srr = 0, skr = 0;
  void add_program(int64_t N) {
    for (int64_t k = 0; k < N; ++k) {
      const double x = (double)k, y = (double)(N - k);
      n += 1;
      sk += x;
      sr += y;
      skk += x * x;
      srr += y * y;
      skr += x * y;
    }
  }
  double eta() const {
    if (n < 2) return 1.0;
    const double ck = skk - sk * sk / n, cr = srr - sr * sr / n, c = skr - sk * sr / n;
    if (!(ck > 0) || !(cr > 0)) return 1.0;
    return -c / std::sqrt(ck * cr);
  }
};

enum class ReqState { Waiting, Running, Done };  // Done only until erased

struct Request {
  int32_t program;
  int64_t pages;
  double arrival;
  bool preempted;
  ReqState state;
};

struct Program {
  double first_arrival = 0;   // program-level arrival order
  int32_t served = 0;         // finished requests
  bool busy = false;          // a request waiting or running
  int64_t active = -1;        // that request
  bool pinned = false;
  double expiry = 0;
  int64_t pin_pages = 0;
  bool tool_pending = false;  // previous request finished with a tool call
  int32_t tool = -1;
  double finish_time = 0;
};

}  // namespace

struct ckv_sched {
  ckv_ttl_config_t cfg;
  int64_t capacity, running_pages = 0, pinned_pages = 0;
  double clock = -std::numeric_limits<double>::infinity();
  std::unordered_map<int64_t, Request> req;
  std::unordered_map<int32_t, Program> prog;
  std::vector<int64_t> waiting;  // request ids, arrival order
  int32_t running = 0, pinned = 0;
  std::map<int32_t, Durations> by_tool;
  Durations all;
  std::deque<double> waits;
  double wait_sum = 0;
  EtaAcc eta;

  double mean_wait() const { return waits.empty() ? 0.0 : wait_sum / (double)waits.size(); }

  void record_wait(double w) {
    waits.push_back(w);
    wait_sum += w;
    if ((int32_t)waits.size() > cfg.wait_window) {
      wait_sum -= waits.front();
      waits.pop_front();
    }
  }

  void record_tool(int32_t tool, double d) {
    by_tool[tool].add(d);
    all.add(d);
  }

  double ttl(int32_t tool, double prefill_reload) const {
    if (cfg.fixed_ttl_s >= 0) return cfg.fixed_ttl_s;
    const int64_t K = cfg.min_records;
    const int64_t total = (int64_t)all.v.size();
    if (total <= K) return cold_ttl(mean_wait() * 1.0 + prefill_reload);  // Exp(1), eta = 1
    const double B = mean_wait() * eta.eta() + prefill_reload;
    auto it = by_tool.find(tool);
    if (it == by_tool.end() || (int64_t)it->second.v.size() <= K) return argmax_sorted(all.v, B);
    return argmax_sorted(it->second.v, B);
  }

  void unpin(Program &p) {
    if (!p.pinned) return;
    p.pinned = false;
    pinned_pages -= p.pin_pages;
    p.pin_pages = 0;
    --pinned;
  }

  int64_t free_pages() const { return capacity - running_pages - pinned_pages; }

  // Sec. 4.3 order: true if request a goes before request b.
  bool before(int64_t a, int64_t b) const {
    const Request &ra = req.at(a), &rb = req.at(b);
    if (ra.preempted != rb.preempted) return ra.preempted;
    const Program &pa = prog.at(ra.program), &pb = prog.at(rb.program);
    if (pa.pinned != pb.pinned) return pa.pinned;
    if (pa.first_arrival != pb.first_arrival) return pa.first_arrival < pb.first_arrival;
    if (ra.arrival != rb.arrival) return ra.arrival < rb.arrival;
    return a < b;
  }
};

extern "C" {

ckv_sched_t *ckv_sched_create(const ckv_ttl_config_t *config, int64_t capacity_pages) {
  if (!config || capacity_pages <= 0 || config->min_records < 0 || config->wait_window < 1 ||
      std::isnan(config->fixed_ttl_s) || std::isinf(config->fixed_ttl_s))
    return nullptr;
  ckv_sched_t *s = new (std::nothrow) ckv_sched();
  if (!s) return nullptr;
  s->cfg = *config;
  s->capacity = capacity_pages;
  return s;
}

void ckv_sched_destroy(ckv_sched_t *s) { delete s; }

static bool advance(ckv_sched_t *s, double now) {
  if (!std::isfinite(now) || now < s->clock) return false;
  s->clock = now;
  return true;
}

ckv_status_t ckv_sched_arrive(ckv_sched_t *s, int64_t request, int32_t program, int64_t pages,
                              int32_t preempted, double now) {
  if (!s || pages <= 0 || s->req.count(request)) return CKV_ERR_INVALID_ARG;
  auto pit = s->prog.find(program);
  const bool is_new = pit == s->prog.end();
  if (!is_new && pit->second.busy) return CKV_ERR_INVALID_ARG;
  if (!advance(s, now)) return CKV_ERR_INVALID_ARG;
  Program &p = s->prog[program];  // may rehash: pit is not used below
  if (is_new) p.first_arrival = now;
  if (p.tool_pending) {  // the tool ran from the previous finish until now
    s->record_tool(p.tool, now - p.finish_time);
    p.tool_pending = false;
  }
  p.busy = true;
  p.active = request;
  s->req[request] = Request{program, pages, now, preempted != 0, ReqState::Waiting};
  s->waiting.push_back(request);
  return CKV_OK;
}

ckv_status_t ckv_sched_finish(ckv_sched_t *s, int64_t request, int32_t last, int32_t next_tool,
                              double prefill_reload_s, double now, double *ttl_out) {
  if (!s) return CKV_ERR_INVALID_ARG;
  auto it = s->req.find(request);
  if (it == s->req.end() || it->second.state != ReqState::Running) return CKV_ERR_INVALID_ARG;
  if (!last && (next_tool < 0 || !(prefill_reload_s >= 0) || !std::isfinite(prefill_reload_s)))
    return CKV_ERR_INVALID_ARG;
  if (!advance(s, now)) return CKV_ERR_INVALID_ARG;
  Request &r = it->second;
  const int32_t program = r.program;
  Program &p = s->prog[program];
  r.state = ReqState::Done;
  s->running_pages -= r.pages;
  --s->running;
  p.busy = false;
  p.active = -1;
  ++p.served;
  double tau = 0.0;
  if (last) {
    s->unpin(p);
    s->eta.add_program(p.served);
  } else {
    tau = s->ttl(next_tool, prefill_reload_s);
    if (tau > 0.0) {
      p.pinned = true;
      p.expiry = now + tau;
      p.pin_pages = r.pages;
      s->pinned_pages += r.pages;
      ++s->pinned;
    }
    p.tool_pending = true;
    p.tool = next_tool;
    p.finish_time = now;
  }
  s->req.erase(it);  // finished requests and programs leave no state behind
  if (last) s->prog.erase(program);
  if (ttl_out) *ttl_out = tau;
  return CKV_OK;
}

int32_t ckv_sched_schedule(ckv_sched_t *s, double now, ckv_issue_t *issued, int32_t max_issued) {
  if (!s || max_issued < 0 || (max_issued > 0 && !issued) || !advance(s, now)) return 0;
  int32_t count = 0;
  while (!s->waiting.empty() && count < max_issued) {
    // (1) expired pins of programs with nothing waiting
    for (auto &kv : s->prog) {
      Program &p = kv.second;
      if (p.pinned && now > p.expiry && !p.busy) s->unpin(p);
    }
    // (2) head of the TTL-aware order
    size_t hi = 0;
    for (size_t i = 1; i < s->waiting.size(); ++i)
      if (s->before(s->waiting[i], s->waiting[hi])) hi = i;
    const int64_t id = s->waiting[hi];
    Request &r = s->req[id];
    Program &p = s->prog[r.program];
    const int64_t own = p.pinned ? p.pin_pages : 0;
    const int64_t need = std::max<int64_t>(r.pages - own, 0);
    // (3) deadlock breaker: unpin others, latest program arrival first
    while (need > s->free_pages()) {
      Program *victim = nullptr;
      int32_t vid = 0;
      for (auto &kv : s->prog) {
        Program &q = kv.second;
        if (!q.pinned || &q == &p) continue;
        if (!victim || q.first_arrival > victim->first_arrival ||
            (q.first_arrival == victim->first_arrival && kv.first > vid)) {
          victim = &q;
          vid = kv.first;
        }
      }
      if (!victim) break;
      s->unpin(*victim);
    }
    if (need > s->free_pages()) break;
    // (4) issue
    s->waiting.erase(s->waiting.begin() + (std::ptrdiff_t)hi);
    ckv_issue_t out;
    out.request = id;
    out.program = r.program;
    out.reused = p.pinned ? 1 : 0;
    out.held_pages = own;
    out.queue_delay_s = now - r.arrival;
    if (p.pinned) {
      s->pinned_pages -= p.pin_pages;
      p.pin_pages = 0;
      p.pinned = false;
      --s->pinned;
    } else if (p.served > 0 && !r.preempted) {
      s->record_wait(out.queue_delay_s);  // its cache had been evicted (or never pinned)
    }
    s->running_pages += r.pages;
    ++s->running;
    r.state = ReqState::Running;
    r.preempted = false;
    issued[count++] = out;
  }
  return count;
}

ckv_status_t ckv_sched_preempt(ckv_sched_t *s, int64_t request) {
  if (!s) return CKV_ERR_INVALID_ARG;
  auto it = s->req.find(request);
  if (it == s->req.end() || it->second.state != ReqState::Running) return CKV_ERR_INVALID_ARG;
  Request &r = it->second;
  r.state = ReqState::Waiting;
  r.preempted = true;
  s->running_pages -= r.pages;
  --s->running;
  s->waiting.push_back(request);
  return CKV_OK;
}

double ckv_sched_ttl(const ckv_sched_t *s, int32_t tool, double prefill_reload_s) {
  if (!s || !(prefill_reload_s >= 0) || !std::isfinite(prefill_reload_s)) return 0.0;
  return s->ttl(tool, prefill_reload_s);
}

ckv_status_t ckv_sched_record_tool(ckv_sched_t *s, int32_t tool, double duration_s) {
  if (!s || tool < 0 || !(duration_s >= 0) || !std::isfinite(duration_s)) return CKV_ERR_INVALID_ARG;
  s->record_tool(tool, duration_s);
  return CKV_OK;
}

void ckv_sched_stats(const ckv_sched_t *s, ckv_sched_stats_t *out) {
  if (!s || !out) return;
  out->capacity_pages = s->capacity;
  out->free_pages = s->free_pages();
  out->pinned_pages = s->pinned_pages;
  out->running_pages = s->running_pages;
  out->waiting = (int32_t)s->waiting.size();
  out->running = s->running;
  out->pinned = s->pinned;
  out->tool_records = (int64_t)s->all.v.size();
  out->mean_wait_s = s->mean_wait();
  out->eta = s->eta.eta();
}

double ckv_sched_pin_expiry(const ckv_sched_t *s, int32_t program) {
  if (!s) return -1.0;
  auto it = s->prog.find(program);
  return it != s->prog.end() && it->second.pinned ? it->second.expiry : -1.0;
}

double ckv_ttl_argmax(const double *durations, int64_t n, double benefit_s) {
  if (!durations || n <= 0) return 0.0;
  std::vector<double> d(durations, durations + n);
  std::sort(d.begin(), d.end());
  return argmax_sorted(d, benefit_s);
}

double ckv_ttl_cold(double benefit_s) { return cold_ttl(benefit_s); }

double ckv_memoryfulness(const int32_t *requests_per_program, int64_t num_programs) {
  EtaAcc acc;
  for (int64_t i = 0; requests_per_program && i < num_programs; ++i)
    acc.add_program(requests_per_program[i]);
  return acc.eta();
}

}  // extern "C"
