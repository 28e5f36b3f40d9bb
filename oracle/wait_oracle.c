/*
 * wait_oracle.c -- CPU oracle for the multi-stage LLM-inference queueing model.
 *
 * TEST INFRASTRUCTURE.  Only tests, the smoke check and the CPU-baseline leg of
 * the benchmark may load this file's library.  It shares no code with the GPU
 * path.  It is deliberately plain and slow: one record per request, and every
 * scheduling decision is re-derived from the records (sorting residents by
 * stage and admission order) at every iteration.
 *
 * What it follows (arXiv 2504.11320):
 *   - the model: Section 2 -- typed Poisson arrivals, prefill stage 0 and
 *     decode stages 1..l'_j, iteration time eq. (time_consump)
 *     tau = d0 + d1 * sum_{i in batch}(l_i + s_i), memory constraint
 *     eq. (memory_constraint) over GPU-resident prompts, LIFO eviction with
 *     restart from prefill, censored latency / TTFT metrics (Section 2.4);
 *   - WAIT: Algorithm 1 (Section 4.2), and its threshold-only variant
 *     WAIT-no-wait (appendix, threshold without waiting): a type is served
 *     whenever it has a waiting or resident prompt, admitting at most n_j
 *     waiting prompts, so the per-stage upper bound n_j is kept but service
 *     never waits for a full cohort;
 *   - Nested WAIT: Algorithm 2 (Section 5.1) in the event-driven form of
 *     Algorithm 4 (Appendix B.1), with coarse segments (Appendix A, segment
 *     design);
 *   - FCFS: Section 4.1, with the exact behaviour spelled out in the proof of
 *     Proposition 3; optionally with chunked prefill (the Sarathi-style
 *     baseline of Section 6: at most `chunk` prefill tokens per iteration,
 *     partial prefills interleaved with decodes).  Reading: the budget goes
 *     first to the partially prefilled prompt (at most one exists: it is the
 *     last one admitted), then to admissions from the queue head, each taking
 *     min(its remaining prompt, the budget left); admission still checks the
 *     whole prompt against C minus the reserve; a chunk that brings a prompt
 *     to p cached tokens charges p in the iteration time (the cache after it,
 *     as a whole prefill charges l); a partial prompt holds p tokens, is the
 *     most recently admitted for LIFO repair, and restarts from scratch when
 *     evicted; the prompt reaches stage 1 when its last chunk is processed.
 *
 * Readings of points the paper leaves open (they are the model contract and
 * are listed with their evidence in the design notes):
 *   charge of a resident at stage s >= 1 is l+s, a prefill being processed
 *   costs l, the external queue costs 0; a Nested boundary prompt is charged
 *   l+r_{k-1} and processed at stage r_{k-1}+1; the first output token is
 *   produced by the stage-1 processing; evicted prompts keep arrival time,
 *   type, output length and first-token flag and rejoin the tail of the
 *   external queue; selection inside a cell is FIFO; "most recently admitted"
 *   is the largest admission key (batch, position); WAIT and FCFS repair after
 *   the completion update with global LIFO; Nested repair evicts boundary
 *   prompts first and falls back to interior prompts (counted separately);
 *   horizon counts batches; arrivals at t <= t_end are handled before the
 *   decision at t_end.
 *
 * Time-varying arrivals (appendix, time-varying rates: independent
 * nonhomogeneous Poisson processes with continuous bounded intensities):
 * intensity lambda_j f_j(t), f_j piecewise linear through the profile points
 * and constant outside them, sampled by thinning (Lewis and Shedler, 1979):
 * candidates of the Poisson process at rate lambda_j max f_j drawn as above
 * (counter k = candidate index), candidate k kept when w3 max f_j < f_j(t_k)
 * 2^32 (w3 the candidate's fourth Philox word), its output length from its
 * w2.  A candidate inside a stretch where f_j is zero moves the clock to the
 * stretch's end; a type whose intensity is zero from the last point on, or
 * that rejects 2^20 candidates in a row (flagged), has no further arrivals.
 *
 * Randomness: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11) keyed by the
 * 64-bit seed, counter (k, type, replica, 0) for the k-th arrival of a type.
 * Uniform u = (2x+1) 2^-53 from 52 bits of (w0, w1); gap = -ln(u)/lambda with
 * ln built from IEEE basic operations only (atanh series); output length from
 * w2 against a u32 CDF table.
 *
 * Build with -ffp-contract=off and without fast-math.
 */
#include "wait_oracle.h"

#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>

static int is_wait(const or_config *c) {
  return c->policy == OR_WAIT || c->policy == OR_WAIT_NOWAIT;
}

/* ------------------------------------------------------------------ RNG -- */

void oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2],
                          uint32_t out[4]) {
  /* Philox4x32 with 10 rounds; multipliers and Weyl key increments from the
   * Philox paper (SC'11). */
  uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; round++) {
    if (round > 0) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)x0;
    uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)x2;
    uint32_t y0 = (uint32_t)(p1 >> 32) ^ x1 ^ k0;
    uint32_t y1 = (uint32_t)p1;
    uint32_t y2 = (uint32_t)(p0 >> 32) ^ x3 ^ k1;
    uint32_t y3 = (uint32_t)p0;
    x0 = y0;
    x1 = y1;
    x2 = y2;
    x3 = y3;
  }
  out[0] = x0;
  out[1] = x1;
  out[2] = x2;
  out[3] = x3;
}

double oracle_uniform(uint32_t w0, uint32_t w1) {
  uint64_t x = ((uint64_t)w0 << 20) | (uint64_t)(w1 >> 12); /* 52 bits */
  return (double)(2 * x + 1) * 0x1p-53;                     /* exact    */
}

/* sqrt(1/2) rounded to double, and ln 2 split so that e * LN2_HI is exact. */
static const double OR_SQRT_HALF = 0x1.6a09e667f3bcdp-1;
static const double OR_LN2_HI = 0x1.62e42fefa3800p-1;
static const double OR_LN2_LO = 0x1.ef35793c7673p-45;

double oracle_ln(double u) {
  /* ln u = e ln2 + ln f with u = f 2^e, f in [sqrt(1/2), sqrt(2)), and
   * ln f = 2 atanh(z) = 2z sum_i z^{2i}/(2i+1), z = (f-1)/(f+1). */
  int e = 0;
  double f = frexp(u, &e); /* exact: u = f 2^e, f in [1/2, 1) */
  if (f < OR_SQRT_HALF) {
    f = f + f;
    e = e - 1;
  }
  double z = (f - 1.0) / (f + 1.0);
  double w = z * z;
  double p = 1.0 / 23.0;
  p = p * w + 1.0 / 21.0;
  p = p * w + 1.0 / 19.0;
  p = p * w + 1.0 / 17.0;
  p = p * w + 1.0 / 15.0;
  p = p * w + 1.0 / 13.0;
  p = p * w + 1.0 / 11.0;
  p = p * w + 1.0 / 9.0;
  p = p * w + 1.0 / 7.0;
  p = p * w + 1.0 / 5.0;
  p = p * w + 1.0 / 3.0;
  p = p * w + 1.0;
  double lnf = (z + z) * p;
  double de = (double)e;
  return de * OR_LN2_HI + (de * OR_LN2_LO + lnf);
}

void oracle_draw_w3(uint64_t seed, uint32_t replica_id, int32_t type, uint32_t k,
                    double lambda, const uint32_t *cdf_row, int32_t out_cap,
                    double *gap, int32_t *L, uint32_t *w3) {
  uint32_t ctr[4] = {k, (uint32_t)type, replica_id, 0u};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t w[4];
  oracle_philox4x32_10(ctr, key, w);
  double u = oracle_uniform(w[0], w[1]);
  *gap = -oracle_ln(u) / lambda;
  if (cdf_row != NULL && L != NULL) {
    int32_t s = 1;
    while (s < out_cap && !(w[2] < cdf_row[s - 1])) s++;
    *L = s;
  }
  *w3 = w[3];
}

void oracle_draw(uint64_t seed, uint32_t replica_id, int32_t type, uint32_t k,
                 double lambda, const uint32_t *cdf_row, int32_t out_cap,
                 double *gap, int32_t *L) {
  uint32_t ctr[4] = {k, (uint32_t)type, replica_id, 0u};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t w[4];
  oracle_philox4x32_10(ctr, key, w);
  double u = oracle_uniform(w[0], w[1]);
  *gap = -oracle_ln(u) / lambda;
  if (cdf_row != NULL && L != NULL) {
    /* smallest s in 1..cap-1 with w2 < T[s], else cap (linear scan) */
    int32_t s = 1;
    while (s < out_cap && !(w[2] < cdf_row[s - 1])) s++;
    *L = s;
  }
}

/* ------------------------------------------------------- containers ---- */

typedef struct {
  int64_t *v;
  int64_t head, len, cap;
} dq_t;

static void dq_free(dq_t *d) { free(d->v); }

static void dq_grow(dq_t *d) {
  int64_t nc = d->cap ? d->cap * 2 : 64;
  int64_t *nv = (int64_t *)malloc((size_t)nc * sizeof(int64_t));
  for (int64_t i = 0; i < d->len; i++) nv[i] = d->v[(d->head + i) % d->cap];
  free(d->v);
  d->v = nv;
  d->head = 0;
  d->cap = nc;
}

static void dq_push(dq_t *d, int64_t x) {
  if (d->len == d->cap) dq_grow(d);
  d->v[(d->head + d->len) % d->cap] = x;
  d->len++;
}

static int64_t dq_at(const dq_t *d, int64_t i) {
  return d->v[(d->head + i) % d->cap];
}

static int64_t dq_pop_front(dq_t *d) {
  int64_t x = d->v[d->head];
  d->head = (d->head + 1) % d->cap;
  d->len--;
  return x;
}

static void dq_remove_at(dq_t *d, int64_t i) {
  for (int64_t k = i; k + 1 < d->len; k++)
    d->v[(d->head + k) % d->cap] = d->v[(d->head + k + 1) % d->cap];
  d->len--;
}

typedef struct {
  int64_t *v;
  int64_t len, cap;
} vec_t;

static void vec_push(vec_t *a, int64_t x) {
  if (a->len == a->cap) {
    a->cap = a->cap ? a->cap * 2 : 64;
    a->v = (int64_t *)realloc(a->v, (size_t)a->cap * sizeof(int64_t));
  }
  a->v[a->len++] = x;
}

/* ------------------------------------------------------------ state ---- */

enum { LOC_FREE = 0, LOC_QUEUE = 1, LOC_INT = 2, LOC_BND = 3, LOC_PRE = 4 };

typedef struct {
  double a;     /* arrival time                                  */
  int32_t j;    /* type                                          */
  int32_t L;    /* output length (decode tokens)                 */
  int32_t ft;   /* first output token produced                   */
  int32_t loc;  /* LOC_*                                         */
  int32_t s;    /* LOC_INT: stage s >= 1 (next processing stage) */
  int32_t seg;  /* Nested: segment (1-based) of LOC_INT/LOC_BND  */
  int32_t sel;  /* selected in the batch being formed            */
  int32_t sp;   /* processing stage when selected                */
  int32_t pp;   /* LOC_PRE: prompt tokens cached so far          */
  int32_t cq;   /* prefill tokens processed in the current batch */
  int64_t kb;   /* admission key: batch of last prefill          */
  int64_t kp;   /* admission key: position within that batch    */
  int64_t id;   /* request id (arrival order)                    */
  int32_t cap_in; /* WAIT, Nested: the cap of the cohort it was admitted with */
} req_t;

typedef struct {
  const or_config *cfg;
  uint64_t seed;
  uint32_t rid;
  /* requests */
  req_t *R;
  int64_t nR, capR;
  vec_t freelist;
  /* queues: WAIT one per type, otherwise one */
  dq_t *q;
  int32_t nq;
  dq_t *bnd; /* Nested boundary queues, index k = 2..nseg (0,1 unused) */
  vec_t res; /* LOC_INT residents */
  vec_t sel; /* selected requests in canonical order */
  /* arrivals */
  double *t_next;
  int32_t *L_next;
  uint32_t *k_next;
  int64_t tr_idx;
  /* clock and aggregates */
  double t;
  int64_t b;
  int64_t N, U, Mres;
  int64_t reserve_tok;
  or_result *out;
  uint32_t *hist;
  or_req_log *rlog;
  int64_t next_id;
  int64_t tmp_cap;
  int64_t *tmp;
  int pre_launch;  /* evictions now are the pre-launch (Q+) repair's */
  int64_t mplus;   /* Nested: M_res(Q+) after the pre-launch repair   */
  int64_t *nsvc;   /* Nested: services of segment k so far, k = 1..nseg */
} sim_t;

static int key_less(const req_t *x, const req_t *y) {
  if (x->kb != y->kb) return x->kb < y->kb;
  return x->kp < y->kp;
}

static __thread const req_t *t_sort_R; /* qsort context */

static int cmp_stage_key(const void *pa, const void *pb) {
  const req_t *x = &t_sort_R[*(const int64_t *)pa];
  const req_t *y = &t_sort_R[*(const int64_t *)pb];
  if (x->j != y->j) return x->j < y->j ? -1 : 1;
  if (x->s != y->s) return x->s < y->s ? -1 : 1;
  if (key_less(x, y)) return -1;
  if (key_less(y, x)) return 1;
  return 0;
}

static int cmp_seg_stage_key(const void *pa, const void *pb) {
  const req_t *x = &t_sort_R[*(const int64_t *)pa];
  const req_t *y = &t_sort_R[*(const int64_t *)pb];
  if (x->seg != y->seg) return x->seg < y->seg ? -1 : 1;
  if (x->s != y->s) return x->s < y->s ? -1 : 1;
  if (key_less(x, y)) return -1;
  if (key_less(y, x)) return 1;
  return 0;
}

/* Sort n request indices (nothing to sort below two: the array may not
 * exist yet). */
static void sort_ids(int64_t *v, int64_t n, int (*cmp)(const void *, const void *)) {
  if (n > 1) qsort(v, (size_t)n, sizeof(int64_t), cmp);
}

static int64_t new_req(sim_t *S) {
  if (S->freelist.len > 0) return S->freelist.v[--S->freelist.len];
  if (S->nR == S->capR) {
    S->capR = S->capR ? S->capR * 2 : 256;
    S->R = (req_t *)realloc(S->R, (size_t)S->capR * sizeof(req_t));
  }
  return S->nR++;
}

/* Memory charge of a resident request (readings: l+s at interior stage s,
 * l+r_{k-1} in the boundary queue of segment k). */
static int64_t charge(const sim_t *S, const req_t *r) {
  const or_config *c = S->cfg;
  int64_t l = c->l[r->j];
  if (r->loc == LOC_INT) return l + r->s;
  if (r->loc == LOC_BND) return l + c->seg_end[r->seg - 2];
  if (r->loc == LOC_PRE) return r->pp;
  return 0;
}

/* -------------------------------------------------------- arrivals ---- */

/* Rate profile of type j (time-varying rates): factors f_j at the points
 * rate_t[0..P-1], row j of rate_f.  seg_of gives -1 before the first point,
 * P-1 from the last point on, else the i with rate_t[i] <= t < rate_t[i+1]. */
static int32_t seg_of(const or_config *c, double t) {
  const int32_t P = c->n_rate_pts;
  if (t < c->rate_t[0]) return -1;
  if (!(t < c->rate_t[P - 1])) return P - 1;
  int32_t i = 0;
  while (!(t < c->rate_t[i + 1])) i++;
  return i;
}

/* f_j(t): constant outside the points, linear between them. */
static double rate_factor(const or_config *c, int32_t j, int32_t i, double t) {
  const int32_t P = c->n_rate_pts;
  const double *f = c->rate_f + (size_t)j * (size_t)P;
  if (i < 0) return f[0];
  if (i == P - 1) return f[P - 1];
  const double frac = (t - c->rate_t[i]) / (c->rate_t[i + 1] - c->rate_t[i]);
  return f[i] + (f[i + 1] - f[i]) * frac;
}

static void draw_next(sim_t *S, int32_t j) {
  const or_config *c = S->cfg;
  double gap = 0.0;
  int32_t L = 0;
  const uint32_t *row =
      (c->lp == NULL) ? c->cdf + (size_t)j * (size_t)(c->out_cap - 1) : NULL;
  if (c->n_rate_pts == 0) {
    oracle_draw(S->seed, S->rid, j, S->k_next[j], c->lambda[j], row, c->out_cap,
                &gap, &L);
    S->t_next[j] = S->t_next[j] + gap;
    S->L_next[j] = (c->lp != NULL) ? c->lp[j] : L;
    return;
  }
  /* Thinning: candidates of a Poisson process at the bound lambda_j f_max,
   * candidate k kept with probability f_j(t_k) / f_max.  A candidate inside a
   * stretch where f_j is zero moves the clock to the end of that stretch. */
  const int32_t P = c->n_rate_pts;
  const double *f = c->rate_f + (size_t)j * (size_t)P;
  double fmax = f[0];
  for (int32_t i = 1; i < P; i++)
    if (f[i] > fmax) fmax = f[i];
  if (!(fmax > 0.0)) {
    S->t_next[j] = INFINITY;
    return;
  }
  const double lam_c = c->lambda[j] * fmax;
  for (uint32_t tries = 0;; tries++) {
    uint32_t w3 = 0;
    oracle_draw_w3(S->seed, S->rid, j, S->k_next[j], lam_c, row, c->out_cap, &gap,
                   &L, &w3);
    const double tc = S->t_next[j] + gap;
    const int32_t i = seg_of(c, tc);
    if ((double)w3 * fmax < rate_factor(c, j, i, tc) * 4294967296.0) {
      S->t_next[j] = tc; /* accepted */
      break;
    }
    if (tries + 1 >= OR_THIN_MAX) {
      S->out->flags |= OR_FLAG_THIN_LIMIT;
      S->t_next[j] = INFINITY;
      return;
    }
    if (i == P - 1 && f[P - 1] == 0.0) {
      S->t_next[j] = INFINITY; /* zero intensity from here on */
      return;
    }
    if (i < 0 && f[0] == 0.0)
      S->t_next[j] = c->rate_t[0];
    else if (i >= 0 && f[i] == 0.0 && f[i + 1] == 0.0)
      S->t_next[j] = c->rate_t[i + 1];
    else
      S->t_next[j] = tc;
    S->k_next[j]++;
  }
  S->L_next[j] = (c->lp != NULL) ? c->lp[j] : L;
}

int oracle_arrival_times(const or_config *cfg, uint64_t seed, uint32_t replica_id,
                         int32_t type, int64_t n, double *t, int32_t *L,
                         uint32_t *k) {
  sim_t S;
  or_result out;
  memset(&S, 0, sizeof(S));
  memset(&out, 0, sizeof(out));
  S.cfg = cfg;
  S.seed = seed;
  S.rid = replica_id;
  S.out = &out;
  S.t_next = (double *)calloc((size_t)cfg->m, sizeof(double));
  S.L_next = (int32_t *)calloc((size_t)cfg->m, sizeof(int32_t));
  S.k_next = (uint32_t *)calloc((size_t)cfg->m, sizeof(uint32_t));
  draw_next(&S, type);
  for (int64_t a = 0; a < n; a++) {
    t[a] = S.t_next[type];
    if (L) L[a] = S.L_next[type];
    if (k) k[a] = S.k_next[type];
    if (!(S.t_next[type] < INFINITY)) continue;
    S.k_next[type]++;
    draw_next(&S, type);
  }
  free(S.t_next);
  free(S.L_next);
  free(S.k_next);
  return (int)out.flags;
}

/* Time and type of the next exogenous arrival (ties: lowest type). */
static double peek_arrival(const sim_t *S, int32_t *jout) {
  const or_config *c = S->cfg;
  if (c->n_trace > 0) {
    if (S->tr_idx >= c->n_trace) {
      *jout = -1;
      return INFINITY;
    }
    *jout = c->tr_type[S->tr_idx];
    return c->tr_time[S->tr_idx];
  }
  int32_t best = 0;
  for (int32_t j = 1; j < c->m; j++)
    if (S->t_next[j] < S->t_next[best]) best = j;
  *jout = best;
  return S->t_next[best];
}

static void push_queue(sim_t *S, int64_t r) {
  const or_config *c = S->cfg;
  int32_t qi = is_wait(c) ? S->R[r].j : 0;
  if (S->q[qi].len >= c->record_capacity) S->out->flags |= OR_FLAG_CAPACITY;
  S->R[r].loc = LOC_QUEUE;
  dq_push(&S->q[qi], r);
}

/* Take the pending arrival (its time is already known to be S->t or within
 * the current batch) and put the new request at the tail of its queue. */
static double take_arrival(sim_t *S) {
  const or_config *c = S->cfg;
  int32_t j;
  double a = peek_arrival(S, &j);
  int32_t L;
  if (c->n_trace > 0) {
    L = (c->lp != NULL) ? c->lp[j] : c->tr_L[S->tr_idx];
    S->tr_idx++;
  } else {
    L = S->L_next[j];
    S->k_next[j]++;
    draw_next(S, j);
  }
  int64_t r = new_req(S);
  req_t *q = &S->R[r];
  memset(q, 0, sizeof(*q));
  q->a = a;
  q->j = j;
  q->L = L;
  q->ft = 0;
  q->id = S->next_id++;
  if (S->rlog && q->id < S->rlog->cap) {
    S->rlog->arr[q->id] = a;
    S->rlog->done[q->id] = -1.0;
    S->rlog->first[q->id] = -1.0;
  }
  S->out->arrivals++;
  S->N++;
  S->U++;
  push_queue(S, r);
  return a;
}

/* ------------------------------------------------------------ decide ---- */

static void ensure_tmp(sim_t *S, int64_t n) {
  if (n > S->tmp_cap) {
    S->tmp_cap = n * 2;
    S->tmp = (int64_t *)realloc(S->tmp, (size_t)S->tmp_cap * sizeof(int64_t));
  }
}

static void select_req(sim_t *S, int64_t r, int32_t sp, int64_t *tokens) {
  req_t *q = &S->R[r];
  q->sel = 1;
  q->sp = sp;
  vec_push(&S->sel, r);
  *tokens += (int64_t)S->cfg->l[q->j] + sp;
}

/* Select min(cap, count) requests from each stage group of a sorted list
 * tmp[lo..hi) (grouped by stage), in key order inside each stage. */
static void select_by_stage(sim_t *S, int64_t lo, int64_t hi, int32_t cap,
                            int64_t *tokens) {
  int64_t i = lo;
  while (i < hi) {
    int32_t s = S->R[S->tmp[i]].s;
    int64_t g = i;
    while (g < hi && S->R[S->tmp[g]].s == s) g++;
    /* cap < 0 (Nested WAIT): a cell holds the cohort that entered the
     * segment together, selected up to the size it entered with */
    const int64_t lim = cap >= 0 ? cap : S->R[S->tmp[i]].cap_in;
    int64_t take = g - i < lim ? g - i : lim;
    for (int64_t k = 0; k < take; k++) select_req(S, S->tmp[i + k], s, tokens);
    i = g;
  }
}

/* Algorithm 1: eligible types J = {j : n_j0 >= n_j}; for every j in J and
 * every stage s select min(n_j, n_js).  Returns 1 if a batch was formed. */
/* Threshold of type j at its next service under WAIT: n_j, or with per-stage
 * caps (Section 6: tl spread over the type's l'_j + 1 prefill and decode
 * stages) the caps of its stages taken in turn, the x-th service (x = 1, 2,
 * ...) taking the cap of stage (x-1) mod (l'_j + 1).  The admitted cohort has
 * that size. */
static int32_t wait_cap(const sim_t *S, int32_t j) {
  const or_config *c = S->cfg;
  if (!c->stage_caps) return c->n[j];
  int64_t lo = 0;
  for (int32_t i = 0; i < j; i++) lo += c->lp[i] + 1;
  return c->stage_caps[lo + S->nsvc[j] % (c->lp[j] + 1)];
}

static int decide_wait(sim_t *S, int64_t *tokens, int64_t *prefill_l) {
  const or_config *c = S->cfg;
  const int nowait = c->policy == OR_WAIT_NOWAIT;
  /* residents per type (WAIT-no-wait also serves a type that has residents
   * and nothing waiting) */
  int64_t nres[c->m];
  int elig[c->m];
  for (int32_t j = 0; j < c->m; j++) nres[j] = 0;
  for (int64_t i = 0; i < S->res.len; i++) nres[S->R[S->res.v[i]].j]++;
  int any = 0;
  for (int32_t j = 0; j < c->m; j++) {
    elig[j] = nowait ? (S->q[j].len > 0 || nres[j] > 0) : (S->q[j].len >= wait_cap(S, j));
    if (elig[j]) any = 1;
  }
  if (!any) return 0;
  int64_t p = 0;
  for (int32_t j = 0; j < c->m; j++) {
    if (!elig[j]) continue;
    const int32_t cap = nowait ? c->n[j] : wait_cap(S, j);
    const int64_t admit = nowait ? (S->q[j].len < c->n[j] ? S->q[j].len : c->n[j]) : cap;
    for (int64_t i = 0; i < admit; i++) {
      int64_t r = dq_pop_front(&S->q[j]);
      S->R[r].kb = S->b;
      S->R[r].kp = p++;
      S->R[r].s = 0;
      S->R[r].cap_in = cap;
      select_req(S, r, 0, tokens);
      *prefill_l += c->l[j];
    }
    /* resident prompts of type j, grouped by stage, FIFO by admission key */
    int64_t cnt = 0;
    ensure_tmp(S, S->res.len);
    for (int64_t i = 0; i < S->res.len; i++)
      if (S->R[S->res.v[i]].j == j) S->tmp[cnt++] = S->res.v[i];
    t_sort_R = S->R;
    sort_ids(S->tmp, cnt, cmp_stage_key);
    select_by_stage(S, 0, cnt, -1, tokens);
    S->nsvc[j]++;
  }
  return 1;
}

/* FCFS: batch every resident prompt, then admit from the head of the
 * external FIFO while the launch memory stays within C minus the reserve;
 * stop at the first prompt that does not fit. */
/* Select a prefill chunk of cq tokens for request r (cached before: pp). */
static void select_chunk(sim_t *S, int64_t r, int32_t cq, int64_t *tokens) {
  req_t *q = &S->R[r];
  q->sel = 1;
  q->sp = 0;
  q->cq = cq;
  vec_push(&S->sel, r);
  *tokens += (int64_t)q->pp + cq;
}

static int decide_fcfs(sim_t *S, int64_t *tokens, int64_t *prefill_l) {
  const or_config *c = S->cfg;
  if (S->res.len == 0 && S->q[0].len == 0) return 0;
  ensure_tmp(S, S->res.len);
  int64_t cnt = 0, part = -1;
  for (int64_t i = 0; i < S->res.len; i++) {
    if (S->R[S->res.v[i]].loc == LOC_PRE)
      part = S->res.v[i];
    else
      S->tmp[cnt++] = S->res.v[i];
  }
  t_sort_R = S->R;
  sort_ids(S->tmp, cnt, cmp_stage_key);
  for (int64_t i = 0; i < cnt; i++) select_req(S, S->tmp[i], S->R[S->tmp[i]].s, tokens);
  /* prefill budget of this iteration */
  int64_t budget = c->chunk > 0 ? c->chunk : INT64_MAX;
  if (part >= 0) {
    const int64_t rest = c->l[S->R[part].j] - S->R[part].pp;
    const int32_t cq = (int32_t)(rest < budget ? rest : budget);
    budget -= cq;
    select_chunk(S, part, cq, tokens);
    *prefill_l += cq;
  }
  int64_t p = 0;
  while (S->q[0].len > 0 && budget > 0) {
    int64_t r = dq_at(&S->q[0], 0);
    int64_t l = c->l[S->R[r].j];
    if (S->Mres + *prefill_l + l > c->C - S->reserve_tok) break;
    dq_pop_front(&S->q[0]);
    S->R[r].kb = S->b;
    S->R[r].kp = p++;
    S->R[r].s = 0;
    S->R[r].pp = 0;
    const int32_t cq = (int32_t)(l < budget ? l : budget);
    budget -= cq;
    select_chunk(S, r, cq, tokens);
    *prefill_l += cq;
  }
  return S->sel.len > 0;
}

static int32_t seg_start(const or_config *c, int32_t k) {
  return k == 1 ? 0 : c->seg_end[k - 2];
}

/* Projected charge after processing at stage sp in segment k, without any
 * early completion (the conservative state Q+). */
static int64_t projected_charge(const or_config *c, int64_t l, int32_t k,
                                int32_t sp) {
  if (sp == c->seg_end[k - 1]) return k < c->nseg ? l + c->seg_end[k - 1] : 0;
  return l + sp + 1;
}

static void evict(sim_t *S, int64_t r, int fallback);

/* Test builds only (-DOR_CHECK_POSITION_ORDER): under Nested WAIT the most
 * recently admitted prompt also stands first in position order (segment 1,
 * boundary queue 2, segment 2, ...): cohorts enter a segment from the front
 * of its FIFO queue, leave it after the same number of services, and their
 * survivors join the next queue in admission order.  The GPU kernels choose
 * the LIFO victim by that position alone; these counters confirm, at every
 * eviction the repairs make, that the victim found by key comparison lies in
 * the lowest non-empty boundary queue (boundary victims) or in the lowest
 * segment holding a candidate (interior victims).  Not part of the model. */
#ifdef OR_CHECK_POSITION_ORDER
static long g_order_checks[2], g_order_misses[2];
long oracle_order_checks(int interior) { return __atomic_load_n(&g_order_checks[interior], __ATOMIC_RELAXED); }
long oracle_order_misses(int interior) { return __atomic_load_n(&g_order_misses[interior], __ATOMIC_RELAXED); }
static void order_check(const sim_t *S, int64_t best, int interior, int only_unselected) {
  const or_config *c = S->cfg;
  int32_t low = 1 << 30;
  if (interior) {
    for (int64_t x = 0; x < S->res.len; x++) {
      const req_t *r = &S->R[S->res.v[x]];
      if (!(only_unselected && r->sel) && r->seg < low) low = r->seg;
    }
  } else {
    for (int32_t k = 2; k <= c->nseg && low > k; k++)
      for (int64_t x = 0; x < S->bnd[k].len; x++)
        if (!(only_unselected && S->R[dq_at(&S->bnd[k], x)].sel)) {
          low = k;
          break;
        }
  }
  __atomic_fetch_add(&g_order_checks[interior], 1, __ATOMIC_RELAXED);
  if (S->R[best].seg != low) __atomic_fetch_add(&g_order_misses[interior], 1, __ATOMIC_RELAXED);
}
#define ORDER_CHECK(S, best, interior, unsel) order_check(S, best, interior, unsel)
#else
#define ORDER_CHECK(S, best, interior, unsel) ((void)0)
#endif

/* Threshold of segment k (1-based) at its next service: n_k, or with
 * per-stage caps (Section 6: the segment cap B_k spread over the segment's
 * decode stages) the cap of the segment's stages taken in turn, the x-th
 * service (x = 1, 2, ...) taking the cap of stage r_{k-1} + 1 + (x-1) mod
 * (r_k - r_{k-1}).  The entering cohort has that size. */
static int32_t entry_cap(const sim_t *S, int32_t k) {
  const or_config *c = S->cfg;
  if (!c->stage_caps) return c->n[k - 1];
  const int32_t lo = seg_start(c, k);
  const int32_t width = c->seg_end[k - 1] - lo;
  return c->stage_caps[lo + (int32_t)(S->nsvc[k] % width)];
}

/* Algorithm 2 / Algorithm 4: largest prefix of segments whose entry queues
 * meet their thresholds; select up to n_k per cell of every prefix segment;
 * then evict unselected boundary prompts (LIFO) until the projected state
 * fits in C, falling back to unselected interior prompts. */
static int decide_nested(sim_t *S, int64_t *tokens, int64_t *prefill_l) {
  const or_config *c = S->cfg;
  if (S->q[0].len < entry_cap(S, 1)) return 0;
  int32_t kmax = 1;
  while (kmax < c->nseg && S->bnd[kmax + 1].len >= entry_cap(S, kmax + 1)) kmax++;

  /* interior residents sorted by (segment, stage, key) */
  ensure_tmp(S, S->res.len);
  for (int64_t i = 0; i < S->res.len; i++) S->tmp[i] = S->res.v[i];
  t_sort_R = S->R;
  sort_ids(S->tmp, S->res.len, cmp_seg_stage_key);

  int64_t p = 0;
  int64_t i = 0;
  for (int32_t k = 1; k <= kmax; k++) {
    int32_t nk = entry_cap(S, k);
    if (k == 1) {
      for (int32_t x = 0; x < nk; x++) {
        int64_t r = dq_pop_front(&S->q[0]);
        S->R[r].kb = S->b;
        S->R[r].kp = p++;
        S->R[r].s = 0;
        S->R[r].seg = 1;
        S->R[r].cap_in = nk;
        select_req(S, r, 0, tokens);
        *prefill_l += c->l[S->R[r].j];
      }
    } else {
      for (int32_t x = 0; x < nk; x++) {
        int64_t r = dq_at(&S->bnd[k], x);
        S->R[r].cap_in = nk;
        select_req(S, r, seg_start(c, k) + 1, tokens);
      }
    }
    while (i < S->res.len && S->R[S->tmp[i]].seg < k) i++;
    int64_t lo = i;
    while (i < S->res.len && S->R[S->tmp[i]].seg == k) i++;
    select_by_stage(S, lo, i, -1, tokens);
    S->nsvc[k]++;
  }

  /* M_res(Q+) */
  int64_t mplus = 0;
  for (int64_t x = 0; x < S->res.len; x++) {
    const req_t *r = &S->R[S->res.v[x]];
    mplus += r->sel ? projected_charge(c, c->l[r->j], r->seg, r->sp)
                    : charge(S, r);
  }
  for (int32_t k = 2; k <= c->nseg; k++)
    for (int64_t x = 0; x < S->bnd[k].len; x++) {
      const req_t *r = &S->R[dq_at(&S->bnd[k], x)];
      mplus += r->sel ? projected_charge(c, c->l[r->j], k, r->sp)
                      : charge(S, r);
    }
  for (int64_t x = 0; x < S->sel.len; x++) {
    const req_t *r = &S->R[S->sel.v[x]];
    if (r->sp == 0) mplus += projected_charge(c, c->l[r->j], 1, 0);
  }

  /* pre-launch repair: unselected boundary prompts, most recent first */
  S->pre_launch = 1;
  while (mplus > c->C) {
    int64_t best = -1;
    for (int32_t k = 2; k <= c->nseg; k++)
      for (int64_t x = 0; x < S->bnd[k].len; x++) {
        int64_t r = dq_at(&S->bnd[k], x);
        if (S->R[r].sel) continue;
        if (best < 0 || key_less(&S->R[best], &S->R[r])) best = r;
      }
    if (best < 0) break;
    ORDER_CHECK(S, best, 0, 1);
    mplus -= charge(S, &S->R[best]);
    evict(S, best, 0);
  }
  /* fallback: unselected interior prompts, most recent first */
  while (mplus > c->C) {
    int64_t best = -1;
    for (int64_t x = 0; x < S->res.len; x++) {
      int64_t r = S->res.v[x];
      if (S->R[r].sel) continue;
      if (best < 0 || key_less(&S->R[best], &S->R[r])) best = r;
    }
    if (best < 0) break;
    ORDER_CHECK(S, best, 1, 1);
    mplus -= charge(S, &S->R[best]);
    evict(S, best, 1);
  }
  S->pre_launch = 0;
  S->mplus = mplus;
  if (mplus > c->C) S->out->flags |= OR_FLAG_OVERFLOW;
  return 1;
}

/* ------------------------------------------------------ transitions ---- */

static void remove_resident(sim_t *S, int64_t r) {
  for (int64_t i = 0; i < S->res.len; i++)
    if (S->res.v[i] == r) {
      S->res.v[i] = S->res.v[S->res.len - 1];
      S->res.len--;
      return;
    }
}

static void remove_boundary(sim_t *S, int64_t r) {
  dq_t *d = &S->bnd[S->R[r].seg];
  for (int64_t i = 0; i < d->len; i++)
    if (dq_at(d, i) == r) {
      dq_remove_at(d, i);
      return;
    }
}

/* Discard the KV cache of a resident prompt and return it to the tail of its
 * external queue as a restart (arrival time, type, length, first-token flag
 * are kept). */
static void evict(sim_t *S, int64_t r, int fallback) {
  req_t *q = &S->R[r];
  int64_t gen; /* decode tokens already produced, lost with the cache */
  if (q->loc == LOC_BND) {
    gen = S->cfg->seg_end[q->seg - 2];
    remove_boundary(S, r);
  } else if (q->loc == LOC_PRE) {
    gen = 0;
    remove_resident(S, r);
  } else {
    gen = q->s - 1;
    remove_resident(S, r);
  }
  S->Mres -= charge(S, q);
  S->out->evictions++;
  S->out->evicted_tokens += gen;
  if (fallback) S->out->fallback_evictions++;
  if (S->rlog && S->rlog->ev_cap > 0 && S->rlog->n_ev < S->rlog->ev_cap) {
    const int64_t e = S->rlog->n_ev++;
    S->rlog->ev_id[e] = q->id;
    S->rlog->ev_batch[e] = S->b;
    S->rlog->ev_kind[e] = (S->pre_launch ? OR_EV_PRE : OR_EV_POST) + (fallback ? 1 : 0);
  }
  q->s = 0;
  q->seg = 0;
  q->sel = 0;
  q->pp = 0;
  push_queue(S, r);
}

static int64_t hist_bin(const or_config *c, double lat) {
  int64_t b = 0;
  while (b < c->n_edges && c->edges[b] <= lat) b++;
  return b;
}

static void complete(sim_t *S, int64_t r, double t_end) {
  req_t *q = &S->R[r];
  const or_config *c = S->cfg;
  S->out->completions++;
  S->out->completed_tokens += q->L;
  double lat = t_end - q->a;
  S->out->lat_completed_sum += lat;
  if (S->hist && c->n_edges >= 0) S->hist[hist_bin(c, lat)]++;
  if (S->rlog && q->id < S->rlog->cap) S->rlog->done[q->id] = t_end;
  S->N--;
  q->loc = LOC_FREE;
  vec_push(&S->freelist, r);
}

/* Apply the completion of the batch to every selected prompt, in the order
 * of the selection list. */
static void transition(sim_t *S, double t_end) {
  const or_config *c = S->cfg;
  for (int64_t x = 0; x < S->sel.len; x++) {
    int64_t r = S->sel.v[x];
    req_t *q = &S->R[r];
    int64_t l = c->l[q->j];
    int32_t sp = q->sp;
    q->sel = 0;
    if (sp == 0 && c->policy == OR_FCFS) { /* a prefill chunk (or a whole prefill) */
      const int64_t old = charge(S, q);
      const int32_t after = q->pp + q->cq;
      if (q->loc != LOC_PRE) vec_push(&S->res, r);
      if (after == l) { /* prefill done: resident at stage 1 */
        q->loc = LOC_INT;
        q->s = 1;
        q->pp = 0;
      } else {
        q->loc = LOC_PRE;
        q->pp = after;
      }
      S->Mres += charge(S, q) - old;
      continue;
    }
    if (sp == 0) { /* prefill done: resident at stage 1 */
      q->loc = LOC_INT;
      q->s = 1;
      if (c->policy == OR_NESTED) q->seg = 1;
      vec_push(&S->res, r);
      S->Mres += l + 1;
      continue;
    }
    /* the processing of stage sp produced output token sp */
    if (sp == 1 && !q->ft) {
      q->ft = 1;
      S->U--;
      if (S->rlog && q->id < S->rlog->cap) S->rlog->first[q->id] = t_end;
    }
    int was_bnd = (q->loc == LOC_BND);
    int64_t old = charge(S, q);
    if (sp == q->L) {
      S->Mres -= old;
      if (was_bnd)
        remove_boundary(S, r);
      else
        remove_resident(S, r);
      complete(S, r, t_end);
      continue;
    }
    if (c->policy == OR_NESTED) {
      int32_t k = q->seg;
      if (sp == c->seg_end[k - 1]) { /* survivor joins boundary queue k+1 */
        S->Mres -= old;
        if (was_bnd)
          remove_boundary(S, r);
        else
          remove_resident(S, r);
        q->loc = LOC_BND;
        q->seg = k + 1;
        dq_push(&S->bnd[k + 1], r);
        S->Mres += charge(S, q);
        continue;
      }
      if (was_bnd) {
        remove_boundary(S, r);
        vec_push(&S->res, r);
      }
      q->loc = LOC_INT;
      q->s = sp + 1;
      S->Mres += charge(S, q) - old;
      continue;
    }
    q->s = sp + 1;
    S->Mres += 1;
  }
  S->sel.len = 0;
}

/* Post-completion repair.  WAIT and FCFS: global LIFO over all resident
 * prompts.  Nested WAIT: boundary prompts first (LIFO), then interior
 * prompts (LIFO, counted as fallback evictions). */
static void repair(sim_t *S) {
  const or_config *c = S->cfg;
  while (S->Mres > c->C) {
    int64_t best = -1;
    if (c->policy == OR_NESTED) {
      for (int32_t k = 2; k <= c->nseg; k++)
        for (int64_t x = 0; x < S->bnd[k].len; x++) {
          int64_t r = dq_at(&S->bnd[k], x);
          if (best < 0 || key_less(&S->R[best], &S->R[r])) best = r;
        }
      if (best >= 0) {
        ORDER_CHECK(S, best, 0, 0);
        evict(S, best, 0);
        continue;
      }
    }
    for (int64_t x = 0; x < S->res.len; x++) {
      int64_t r = S->res.v[x];
      if (best < 0 || key_less(&S->R[best], &S->R[r])) best = r;
    }
    if (best < 0) break;
    if (c->policy == OR_NESTED) ORDER_CHECK(S, best, 1, 0);
    evict(S, best, c->policy == OR_NESTED);
  }
}

/* ------------------------------------------------------------- main ---- */

int oracle_run(const or_config *cfg, uint64_t seed, uint32_t replica_id,
               int64_t horizon, or_result *out, uint32_t *hist,
               or_batch_rec *btrace, int64_t btrace_cap, or_req_log *rlog) {
  const or_config *c = cfg;
  sim_t S;
  memset(&S, 0, sizeof(S));
  memset(out, 0, sizeof(*out));
  if (hist && c->n_edges >= 0)
    memset(hist, 0, sizeof(uint32_t) * (size_t)(c->n_edges + 1));
  S.cfg = c;
  S.seed = seed;
  S.rid = replica_id;
  S.out = out;
  S.hist = hist;
  S.rlog = rlog;
  S.nq = is_wait(c) ? c->m : 1;
  S.q = (dq_t *)calloc((size_t)S.nq, sizeof(dq_t));
  S.bnd = (dq_t *)calloc((size_t)(c->policy == OR_NESTED ? c->nseg + 2 : 1),
                         sizeof(dq_t));
  S.nsvc = (int64_t *)calloc((size_t)(c->policy == OR_NESTED ? c->nseg + 2 : c->m + 1),
                             sizeof(int64_t));
  S.t_next = (double *)calloc((size_t)c->m, sizeof(double));
  S.L_next = (int32_t *)calloc((size_t)c->m, sizeof(int32_t));
  S.k_next = (uint32_t *)calloc((size_t)c->m, sizeof(uint32_t));
  S.reserve_tok =
      (c->policy == OR_FCFS) ? (int64_t)ceil(c->reserve * (double)c->C) : 0;
  S.t = 0.0;
  if (c->n_trace == 0)
    for (int32_t j = 0; j < c->m; j++) {
      S.t_next[j] = 0.0;
      draw_next(&S, j);
    }

  for (S.b = 0; S.b < horizon; S.b++) {
    int64_t tokens = 0, prefill_l = 0;
    int64_t ev0 = out->evictions;
    int stop = 0;
    for (;;) {
      if (out->flags & OR_FLAG_CAPACITY) {
        stop = 1;
        break;
      }
      tokens = 0;
      prefill_l = 0;
      S.mplus = 0;
      int got;
      if (is_wait(c))
        got = decide_wait(&S, &tokens, &prefill_l);
      else if (c->policy == OR_FCFS)
        got = decide_fcfs(&S, &tokens, &prefill_l);
      else
        got = decide_nested(&S, &tokens, &prefill_l);
      if (got) break;
      /* nothing eligible: wait for the next arrival */
      int32_t j;
      double ta = peek_arrival(&S, &j);
      if (!(ta < INFINITY)) {
        out->flags |= OR_FLAG_STALL;
        stop = 1;
        break;
      }
      double dt = ta - S.t;
      out->lat_area += (double)S.N * dt;
      out->ttft_area += (double)S.U * dt;
      out->mem_area += (double)S.Mres * dt;
      S.t = ta;
      /* every arrival at this instant joins before the next decision */
      while (!(out->flags & OR_FLAG_CAPACITY) && peek_arrival(&S, &j) == ta)
        take_arrival(&S);
      out->idle_waits++;
    }
    if (stop) break;
    int64_t evict_pre = out->evictions - ev0;
    int64_t nsel = S.sel.len;
    int64_t nprefill = 0;
    for (int64_t x = 0; x < S.sel.len; x++)
      if (S.R[S.sel.v[x]].sp == 0) nprefill++;

    int64_t m_launch = S.Mres + prefill_l;
    if (m_launch > out->peak_mem) out->peak_mem = m_launch;
    double tau = c->d0 + c->d1 * (double)tokens;
    double t_end = S.t + tau;
    int64_t N0 = S.N, U0 = S.U;
    for (;;) {
      int32_t j;
      if (out->flags & OR_FLAG_CAPACITY) break; /* the replica stops anyway */
      double ta = peek_arrival(&S, &j);
      if (!(ta <= t_end)) break;
      take_arrival(&S);
      out->lat_area += t_end - ta;
      out->ttft_area += t_end - ta;
    }
    out->lat_area += (double)N0 * tau;
    out->ttft_area += (double)U0 * tau;
    out->mem_area += (double)m_launch * tau;
    out->busy_time += tau;
    S.t = t_end;
    int64_t comp0 = out->completions;
    transition(&S, t_end);
    if (S.Mres > out->peak_mem) out->peak_mem = S.Mres;
    int64_t ev1 = out->evictions;
    repair(&S);
    out->batches++;
    out->batch_tokens_sum += tokens;
    if (btrace && S.b < btrace_cap) {
      or_batch_rec *br = &btrace[S.b];
      br->t_launch = t_end - tau;
      br->tau = tau;
      br->tokens = tokens;
      br->prefills = nprefill;
      br->selected = nsel;
      br->completions = out->completions - comp0;
      br->evict_pre = evict_pre;
      br->evict_post = out->evictions - ev1;
      br->mem_after = S.Mres;
      int64_t w = 0;
      for (int32_t qi = 0; qi < S.nq; qi++) w += S.q[qi].len;
      br->waiting_after = w;
      int64_t rr = S.res.len;
      if (c->policy == OR_NESTED)
        for (int32_t k = 2; k <= c->nseg; k++) rr += S.bnd[k].len;
      br->resident_after = rr;
      br->mplus = S.mplus;
    }
  }

  out->t_end = S.t;
  int64_t w = 0;
  for (int32_t qi = 0; qi < S.nq; qi++) w += S.q[qi].len;
  out->waiting_end = w;
  int64_t rr = S.res.len;
  if (c->policy == OR_NESTED)
    for (int32_t k = 2; k <= c->nseg; k++) rr += S.bnd[k].len;
  out->resident_end = rr;

  for (int32_t qi = 0; qi < S.nq; qi++) dq_free(&S.q[qi]);
  if (c->policy == OR_NESTED)
    for (int32_t k = 0; k < c->nseg + 2; k++) dq_free(&S.bnd[k]);
  free(S.q);
  free(S.bnd);
  free(S.nsvc);
  free(S.res.v);
  free(S.sel.v);
  free(S.freelist.v);
  free(S.R);
  free(S.tmp);
  free(S.t_next);
  free(S.L_next);
  free(S.k_next);
  return 0;
}

/* ------------------------------------------------- replica threads ---- */

typedef struct {
  const or_config *cfg;
  uint64_t seed;
  const uint32_t *ids;
  int32_t n;
  int64_t horizon;
  or_result *out;
  uint32_t *hist;
  int32_t next;
  pthread_mutex_t mu;
} pool_t;

static void *worker(void *arg) {
  pool_t *P = (pool_t *)arg;
  int32_t nb = P->cfg->n_edges + 1;
  for (;;) {
    pthread_mutex_lock(&P->mu);
    int32_t i = P->next++;
    pthread_mutex_unlock(&P->mu);
    if (i >= P->n) break;
    oracle_run(P->cfg, P->seed, P->ids[i], P->horizon, &P->out[i],
               P->hist ? P->hist + (size_t)i * (size_t)nb : NULL, NULL, 0,
               NULL);
  }
  return NULL;
}

int oracle_run_many(const or_config *cfg, uint64_t seed,
                    const uint32_t *replica_ids, int32_t n_replicas,
                    int64_t horizon, or_result *out, uint32_t *hist,
                    int32_t n_threads) {
  pool_t P;
  P.cfg = cfg;
  P.seed = seed;
  P.ids = replica_ids;
  P.n = n_replicas;
  P.horizon = horizon;
  P.out = out;
  P.hist = hist;
  P.next = 0;
  pthread_mutex_init(&P.mu, NULL);
  if (n_threads < 1) n_threads = 1;
  pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)n_threads);
  for (int32_t i = 0; i < n_threads; i++)
    pthread_create(&th[i], NULL, worker, &P);
  for (int32_t i = 0; i < n_threads; i++) pthread_join(th[i], NULL);
  free(th);
  pthread_mutex_destroy(&P.mu);
  return 0;
}
