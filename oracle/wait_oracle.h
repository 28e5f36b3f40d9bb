/*
 * wait_oracle.h -- interface of the CPU oracle (test infrastructure only).
 *
 * The oracle is a plain, slow, event-driven simulation of the multi-stage
 * LLM-inference queueing model of "Optimizing LLM Inference: Fluid-Guided
 * Online Scheduling with Memory Constraints" (arXiv 2504.11320), Section 2,
 * under the WAIT policy (Algorithm 1), the Nested WAIT policy (Algorithm 2 and
 * its full event-driven form, Algorithm 4 of Appendix B.1) and the greedy FCFS
 * evict-on-overflow baseline (Section 4.1, made exact by the proof of
 * Proposition 3).  It keeps one record per request and re-derives every
 * decision from those records each iteration.
 *
 * Only tests, the smoke check and the CPU-baseline leg of the benchmark may
 * load this library.  It shares no code, header or constant with the GPU
 * library; the two agree only through the written model contract.
 */
#ifndef WAIT_ORACLE_H
#define WAIT_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define OR_WAIT 0
#define OR_NESTED 1
#define OR_FCFS 2
#define OR_WAIT_NOWAIT 3 /* WAIT's thresholds without waiting (appendix) */

#define OR_FLAG_CAPACITY 1u
#define OR_FLAG_STALL 2u
#define OR_FLAG_OVERFLOW 4u
#define OR_FLAG_THIN_LIMIT 8u /* 2^20 thinning rejections in a row */
#define OR_THIN_MAX (1u << 20)

typedef struct {
  int32_t m;                /* request types                                   */
  const int32_t *l;         /* prompt length l_j [m]                           */
  const double *lambda;     /* Poisson rate lambda_j per ms [m]                */
  const int32_t *lp;        /* known output length l'_j [m], or NULL           */
  int32_t out_cap;          /* output-length cap (distribution mode)           */
  const uint32_t *cdf;      /* [m][out_cap-1] u32 CDF thresholds               */
  double d0, d1;            /* iteration time d0 + d1 * tokens                 */
  int64_t C;                /* KV budget in tokens                             */
  const double *edges;      /* latency histogram edges [n_edges] or NULL       */
  int32_t n_edges;
  int64_t record_capacity;  /* external-queue capacity                         */
  const double *tr_time;    /* trace mode: arrival times [n_trace]             */
  const int32_t *tr_type;   /* trace mode: types [n_trace]                     */
  const int32_t *tr_L;      /* trace mode: output lengths [n_trace] or NULL    */
  int64_t n_trace;
  int32_t policy;           /* OR_WAIT / OR_NESTED / OR_FCFS / OR_WAIT_NOWAIT  */
  const int32_t *n;         /* thresholds: WAIT [m], NESTED [nseg]             */
  int32_t nseg;             /* NESTED: number of segments                      */
  const int32_t *seg_end;   /* NESTED: r_1 < ... < r_nseg                      */
  double reserve;           /* FCFS: admission reserve fraction of C           */
  /* time-varying arrivals (appendix, time-varying rates): intensity of type j
   * is lambda_j f_j(t), f_j piecewise linear through (rate_t[i],
   * rate_f[j * n_rate_pts + i]) and constant outside; n_rate_pts = 0 for
   * constant rates */
  int32_t n_rate_pts;
  const double *rate_t;
  const double *rate_f;
  int32_t chunk;            /* FCFS: prefill tokens per iteration (chunked
                               prefill), 0 = whole prefills                   */
  /* Per-stage caps (Section 6, "WAIT and Nested WAIT settings"), or NULL.
   * NESTED: stage_caps[s - 1] is the cap of decode stage s = 1..seg_end[nseg-1];
   * segment k's stages r_{k-1}+1..r_k hold its caps, taken in turn, one per
   * service of the segment, as the size of the entering cohort (NULL: every
   * service of segment k admits n[k-1]).  WAIT: per type j in turn, l'_j + 1
   * caps (its prefill and decode stages), taken in turn, one per service of
   * the type (NULL: n_j). */
  const int32_t *stage_caps;
} or_config;

typedef struct {
  int64_t batches, arrivals, completions, completed_tokens, evictions,
      evicted_tokens, fallback_evictions, batch_tokens_sum, peak_mem,
      waiting_end, resident_end, idle_waits;
  double t_end, busy_time, lat_area, ttft_area, lat_completed_sum, mem_area;
  uint32_t flags;
  uint32_t pad;
} or_result;

/* One record per batch, for hand-trace tests.  mplus: Nested WAIT's
 * projected resident memory M_res(Q+) after the pre-launch repair (0 for
 * the other policies). */
typedef struct {
  double t_launch, tau;
  int64_t tokens, prefills, selected, completions, evict_pre, evict_post,
      mem_after, waiting_after, resident_after, mplus;
} or_batch_rec;

/* Eviction kinds in the eviction log. */
#define OR_EV_POST 0          /* after the completion update, boundary/LIFO */
#define OR_EV_POST_FALLBACK 1 /* after the completion update, interior       */
#define OR_EV_PRE 2           /* before launch (Nested Q+), boundary         */
#define OR_EV_PRE_FALLBACK 3  /* before launch (Nested Q+), interior         */

/* Optional per-request log (request id = arrival order, 0-based) and
 * eviction log (one entry per eviction, in the order they happen). */
typedef struct {
  double *arr;   /* arrival time            [cap] */
  double *done;  /* completion time or -1   [cap] */
  double *first; /* first-token time or -1  [cap] */
  int64_t cap;
  int64_t *ev_id;    /* evicted request id            [ev_cap] */
  int64_t *ev_batch; /* batch index of the eviction   [ev_cap] */
  int32_t *ev_kind;  /* OR_EV_*                       [ev_cap] */
  int64_t ev_cap;
  int64_t n_ev;      /* evictions logged (written by the oracle) */
} or_req_log;

int oracle_run(const or_config *cfg, uint64_t seed, uint32_t replica_id,
               int64_t horizon, or_result *out, uint32_t *hist,
               or_batch_rec *btrace, int64_t btrace_cap, or_req_log *rlog);

int oracle_run_many(const or_config *cfg, uint64_t seed,
                    const uint32_t *replica_ids, int32_t n_replicas,
                    int64_t horizon, or_result *out, uint32_t *hist,
                    int32_t n_threads);

/* Building blocks, exported for the pinning tests. */
void oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2],
                          uint32_t out[4]);
double oracle_uniform(uint32_t w0, uint32_t w1);
double oracle_ln(double u);
/* First n arrival times (INFINITY once the type has stopped), output lengths
 * and Philox counters of one type's arrival process; returns result flags. */
int oracle_arrival_times(const or_config *cfg, uint64_t seed, uint32_t replica_id,
                         int32_t type, int64_t n, double *t, int32_t *L,
                         uint32_t *k);
void oracle_draw_w3(uint64_t seed, uint32_t replica_id, int32_t type, uint32_t k,
                    double lambda, const uint32_t *cdf_row, int32_t out_cap,
                    double *gap, int32_t *L, uint32_t *w3);
void oracle_draw(uint64_t seed, uint32_t replica_id, int32_t type,
                 uint32_t k, double lambda, const uint32_t *cdf_row,
                 int32_t out_cap, double *gap, int32_t *L);

#ifdef __cplusplus
}
#endif
#endif
