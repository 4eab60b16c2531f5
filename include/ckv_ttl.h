/*
 * ckv_ttl.h -- host-side KV-cache time-to-live control plane (Continuum,
 * arXiv 2511.02230): tool-call statistics, the TTL of Eq. 2 with its cold
 * start, the TTL-aware waiting-queue order, pinning/unpinning and the
 * deadlock breaker, over a pool of KV pages.  Pure host code (no GPU); it
 * decides which requests run and whether their retained pages are reused,
 * while include/ckv.h runs the GPU work of each turn.
 *
 * Time is a caller-supplied clock in seconds ("now" arguments), so a
 * simulation can drive it with a fake clock.  Memory is counted in pool
 * pages.  Objects are not thread-safe; one scheduler per engine.
 *
 * Cost model (Sec. 4.1, Table 3 notation): pinning r for tau costs
 * MemUsage(r) / M * tau; a hit within the TTL saves
 * MemUsage(r) / M * (Prefill-Reload(r) + T * eta).  Dividing out
 * MemUsage(r) / M gives Eq. 2:
 *   tau* = argmax_tau P(tau, f) * B - tau,   B = T * eta + Prefill-Reload(r),
 * over tau in {0} and the distinct recorded durations of tool f (Sec. 4.2),
 * P being the empirical CDF of those durations.
 */
#ifndef CKV_TTL_H
#define CKV_TTL_H

#include <stdint.h>

#include "ckv.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  /* K of the cold start (Sec. 4.2): with at most K records in total the TTL
   * assumes Exp(1) tool durations and eta = 1, i.e. tau = max(0, ln B);
   * with more records in total but at most K for tool f it uses the CDF of
   * all tools.  The paper uses K = 100. */
  int32_t min_records;
  /* Length of the sliding window over which T, the mean queueing delay of
   * requests whose cache had been evicted, is averaged (Sec. 4.2; the paper
   * gives no length).  T starts at 0. */
  int32_t wait_window;
  /* < 0: the TTL of Eq. 2 (with its cold start).  >= 0: every pin lasts
   * this many seconds, the static-TTL ablation of the evaluation (Sec. 6);
   * 0 retains nothing, like an engine that frees a finished request's KV. */
  double fixed_ttl_s;
} ckv_ttl_config_t;

typedef struct ckv_sched ckv_sched_t;

/* One issued request, as Schedule() reports it. */
typedef struct {
  int64_t request;      /* request id */
  int32_t program;      /* its program */
  int32_t reused;       /* 1 if its program's pinned pages were still held */
  int64_t held_pages;   /* pages it reuses (its program's pinned pages), else 0 */
  double queue_delay_s; /* now - arrival */
} ckv_issue_t;

/* Create a scheduler over capacity_pages pool pages.  NULL on invalid
 * arguments (capacity <= 0, min_records < 0, wait_window < 1, fixed_ttl_s
 * not finite) or no memory. */
ckv_sched_t *ckv_sched_create(const ckv_ttl_config_t *config, int64_t capacity_pages);
void ckv_sched_destroy(ckv_sched_t *s);

/*
 * OnRequestArrive (Alg. 1): enqueue request `request` of program `program`
 * needing `pages` pool pages in total (retained prefix + new turn + decode
 * growth).  If the program's previous request finished with a tool call,
 * the interval since that finish is recorded as that tool's duration
 * (Sec. 5.1, "Recording the tool finish time").  preempted != 0 marks a
 * request re-queued after preemption (first in the priority order).
 * CKV_ERR_INVALID_ARG for a duplicate request id, pages <= 0, a program that
 * already has a request waiting or running, or time going backwards.
 */
ckv_status_t ckv_sched_arrive(ckv_sched_t *s, int64_t request, int32_t program, int64_t pages,
                              int32_t preempted, double now);

/*
 * OnRequestFinish (Alg. 1; Sec. 5.2, "Request Pinning"): the running request
 * finishes.  last != 0: the program ends; its pages are freed, any pin
 * dropped, and its request count recorded for eta.  Otherwise the program
 * next calls tool `next_tool` (>= 0) and its pages are pinned for
 * tau* = ckv_sched_ttl(s, next_tool, prefill_reload_s) seconds (freed at
 * once when tau* = 0).  *ttl_out (may be NULL) receives tau* (0 when last).
 * The request's id (and, when last, the program's id) may be used again
 * afterwards: a finished program keeps no state.
 */
ckv_status_t ckv_sched_finish(ckv_sched_t *s, int64_t request, int32_t last, int32_t next_tool,
                              double prefill_reload_s, double now, double *ttl_out);

/*
 * Schedule (Alg. 1; Sec. 4.3; Sec. 5.2): repeat while requests wait:
 *  (1) unpin every program whose TTL has expired (now > expiry) and that
 *      has no request waiting;
 *  (2) take the waiting request first in the order (preempted first, then
 *      programs holding a pin, then earlier program arrival, then earlier
 *      request arrival, then smaller id);
 *  (3) if its pages (minus its own program's pinned pages) exceed the free
 *      pages, unpin other programs, latest program arrival first, until it
 *      fits; if it still does not fit, stop;
 *  (4) issue it: its program's pin (if any) becomes part of the request.
 * Issued requests go to issued[0 .. max_issued-1] in order; returns their
 * count (at most max_issued; scheduling stops there), 0 also for invalid
 * arguments or time going backwards.  A request issued without its
 * program's pages after the program's first request (and not after a
 * preemption) counts its queueing delay into T.  Victims of (3) tie on
 * program arrival are taken larger program id first.
 */
int32_t ckv_sched_schedule(ckv_sched_t *s, double now, ckv_issue_t *issued, int32_t max_issued);

/* Preempt a running request: its pages are freed and it is re-queued with
 * the preempted mark (arrival time kept).  CKV_ERR_INVALID_ARG if it is
 * not running. */
ckv_status_t ckv_sched_preempt(ckv_sched_t *s, int64_t request);

/* The TTL a finish would set now: fixed_ttl_s when that is >= 0, else
 * Eq. 2 with the cold start for a request whose next tool is `tool`. */
double ckv_sched_ttl(const ckv_sched_t *s, int32_t tool, double prefill_reload_s);

/* Record a tool-call duration directly (e.g. statistics gathered offline
 * or during agent training, Sec. 4.2). */
ckv_status_t ckv_sched_record_tool(ckv_sched_t *s, int32_t tool, double duration_s);

/* State queries. */
typedef struct {
  int64_t capacity_pages, free_pages, pinned_pages, running_pages;
  int32_t waiting, running, pinned;
  int64_t tool_records;   /* |S| */
  double mean_wait_s;     /* T */
  double eta;             /* memoryfulness estimate (1 until defined) */
} ckv_sched_stats_t;
void ckv_sched_stats(const ckv_sched_t *s, ckv_sched_stats_t *out);
/* Expiry time of program's pin, or -1 when it holds none. */
double ckv_sched_pin_expiry(const ckv_sched_t *s, int32_t program);

/*
 * Stateless pieces, exposed for checking.
 * ckv_ttl_argmax: tau in {0} U durations[0..n) maximizing
 *   (#{d <= tau} / n) * benefit - tau; ties go to the smaller tau; 0 when n = 0.
 * ckv_ttl_cold: the Exp(1) / eta = 1 optimum max(0, ln benefit).
 * ckv_memoryfulness: eta = -Corr(k, N - k) over every request of the given
 *   finished programs (k = 0 .. N_p - 1 requests already served); 1 when the
 *   correlation is undefined (fewer than two samples or zero variance).
 */
double ckv_ttl_argmax(const double *durations, int64_t n, double benefit_s);
double ckv_ttl_cold(double benefit_s);
double ckv_memoryfulness(const int32_t *requests_per_program, int64_t num_programs);

#ifdef __cplusplus
}
#endif

#endif /* CKV_TTL_H */
