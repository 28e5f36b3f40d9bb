/*
 * wait_sim.h -- C ABI of the batched Monte Carlo simulator (MI355X / gfx950).
 *
 * The library simulates many independent replicas of the multi-stage
 * LLM-inference queueing model of "Optimizing LLM Inference: Fluid-Guided
 * Online Scheduling with Memory Constraints" (arXiv 2504.11320):
 *
 *   - m request types; type j arrives as a Poisson process of rate lambda_j
 *     (Section 2.1), or of time-varying intensity lambda_j f_j(t) (appendix,
 *     time-varying arrival rates), has prompt length l_j and output length
 *     l'_j (known), or an output length drawn per request from a CDF table
 *     (unknown lengths, Section 5.1);
 *   - a batch B takes tau(B) = d0 + d1 * sum_{i in B} (l_i + s_i) where s_i is
 *     the stage being processed, 0 for prefill (eq. time_consump, Section 2.2);
 *   - GPU-resident prompts hold KV cache l_i + s_i and the sum must stay
 *     <= C (eq. memory_constraint, Section 2.3); overflow evicts the most
 *     recently admitted prompt, which restarts from prefill;
 *   - policies: WAIT (Algorithm 1, Section 4.2), Nested WAIT (Algorithm 2,
 *     Section 5.1; event-driven form Algorithm 4, Appendix B.1) and the greedy
 *     FCFS evict-on-overflow baseline (Section 4.1), optionally with chunked
 *     prefill (Section 6);
 *   - metrics: effective throughput, latency and time to first token
 *     censored at the horizon T (Section 2.4).
 *
 * Units: lengths in tokens, times in milliseconds, rates per millisecond.
 * One "batch" is one iteration: launch, then completion.  The horizon of a
 * call counts batches per replica; waiting for arrivals while nothing is
 * eligible is not a batch.
 *
 * Randomness: Philox4x32-10 keyed by the 64-bit stream seed with counter
 * (k, j, replica_id, 0) for the k-th arrival of type j; uniform
 * u = (2x+1) 2^-53 from x = (w0 << 20) | (w1 >> 12); inter-arrival gap
 * -ln(u)/lambda_j; unknown output length = smallest s in 1..cap-1 with
 * w2 < T_j[s], else cap.  A replica's arrival path therefore depends only on
 * (seed, replica_id, lambda, rate profile), identical across policies and
 * thresholds.
 *
 * Time-varying intensities (ws_config.n_rate_pts > 0) are sampled by thinning
 * (Lewis and Shedler, 1979): the draws above at the bound rate
 * lambda_j * max f_j give candidate times; candidate k (counter k) is kept
 * when w3 * max f_j < f_j(t_k) * 2^32 (w3 its fourth Philox word, the product
 * in double), and its w2 gives the output length.  A candidate inside a
 * stretch where f_j is zero moves the clock to the end of that stretch; a
 * type whose f_j is zero from the last point on has no further arrivals.
 *
 * Memory ownership: every pointer in the config structs is HOST memory read
 * during the call only.  d_workspace and d_results are DEVICE memory owned by
 * the caller and sized by wait_sim_workspace_bytes / wait_sim_results_bytes.
 * The library allocates no device memory, keeps no pointer after a call
 * returns, and launches its kernels on the caller's stream.  Calls on one
 * workspace must be serialised by the caller (same stream).
 *
 * Errors: functions return a ws_status.  Validation failures return
 * WS_EINVAL before anything is launched; wait_sim_last_error() then holds a
 * message (thread-local, valid until the next call on the same thread).
 * No C++ exception crosses this interface: a failed host allocation returns
 * WS_ENOMEM, any other exception WS_EINTERNAL.  A call that fails after
 * launching work on the library's side streams still orders that work
 * before the caller's stream (or waits for it) before returning.
 * Conditions met by individual replicas at run time are reported in that
 * replica's flags word, never by aborting the launch.
 */
#ifndef WAIT_SIM_H
#define WAIT_SIM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define WS_ABI_VERSION 4

typedef enum {
  WS_OK = 0,
  WS_EINVAL = -1,      /* invalid configuration or arguments              */
  WS_ENOMEM = -2,      /* host allocation failed                          */
  WS_EDEVICE = -3,     /* HIP runtime error                               */
  WS_EWORKSPACE = -4,  /* workspace or result buffer too small            */
  WS_EUNSUPPORTED = -5, /* valid model, but outside the library's limits */
  WS_EINTERNAL = -6     /* unexpected internal failure (a C++ exception
                           caught at the ABI boundary)                   */
} ws_status;

typedef enum {
  WS_WAIT = 0,         /* Algorithm 1                                          */
  WS_NESTED_WAIT = 1,  /* Algorithm 2 / Algorithm 4                            */
  WS_FCFS = 2,         /* greedy FCFS, LIFO eviction on overflow (Section 4.1) */
  WS_WAIT_NOWAIT = 3   /* WAIT's thresholds without waiting (appendix): a type
                          is served whenever it has a waiting or resident
                          prompt, admitting at most n_j waiting prompts      */
} ws_policy_kind;

/* Per-replica flags (result field "flags"). */
#define WS_FLAG_CAPACITY 1u /* an external queue exceeded record_capacity
                               (FCFS with drawn lengths: also its resident
                               ring, which holds record_capacity entries,
                               or 2^31 - 2^24 batches reached); the replica
                               stopped at its next decision                 */
#define WS_FLAG_STALL 2u    /* nothing eligible and no further arrival       */
#define WS_FLAG_OVERFLOW 4u /* Nested WAIT launched with a projected state
                               above C after every allowed eviction          */
#define WS_FLAG_THIN_LIMIT 8u /* a time-varying type rejected 2^20 candidates
                                 in a row; it has no further arrivals       */

/* Limits of the library. */
#define WS_MAX_TYPES 64
#define WS_MAX_TYPES_KNOWN 16 /* the known-length kernels hold this many types
                                 in registers; WAIT jobs with more run in a
                                 kernel with per-type state in LDS, FCFS jobs
                                 in the kernel for per-request lengths (both
                                 with constant rates only; FCFS without
                                 chunked prefill)                           */
#define WS_MAX_SEGMENTS 16
#define WS_MAX_HIST_EDGES 255
#define WS_MAX_RATE_PTS 32
/* Workspace of wait_sim_run_static: a device array of this many bytes that
   every GPU the library runs on holds until the process ends. */
#define WS_STATIC_WORKSPACE_BYTES (64u << 20)

/* The model (Section 2). */
typedef struct {
  int32_t m;                    /* request types, 1..WS_MAX_TYPES            */
  const int32_t *prompt_len;    /* l_j >= 1                         [m]      */
  const double *lambda;         /* lambda_j >= 0, per ms            [m]      */
  const int32_t *out_len;       /* known output length l'_j >= 1    [m], or
                                   NULL for the distribution mode below (the
                                   unknown-length model of Section 5.1: each
                                   request's length drawn at arrival, never
                                   read by the scheduler; Nested WAIT, and
                                   FCFS without chunked prefill and with
                                   constant rates)                           */
  int32_t out_cap;              /* distribution mode: largest output length  */
  const uint32_t *out_cdf_u32;  /* distribution mode: [m][out_cap-1] row j,
                                   entry s-1 = T_j[s], nondecreasing in s    */
  double d0;                    /* fixed time per iteration, > 0             */
  double d1;                    /* time per cached token, >= 0               */
  int64_t C;                    /* KV-cache budget in tokens, <= 2^30        */
  const double *hist_edges;     /* latency histogram edges (ms), strictly
                                   increasing, or NULL                       */
  int32_t n_hist;               /* number of edges, 0..WS_MAX_HIST_EDGES     */
  int32_t record_capacity;      /* capacity of each external queue, a power
                                   of two >= 16                              */
  /* Trace mode (test hook): if n_trace > 0 these arrivals, in this order,
     replace the random arrivals of every replica.                          */
  const double *trace_time;     /* nondecreasing arrival times     [n_trace] */
  const int32_t *trace_type;    /* type of each arrival            [n_trace] */
  const int32_t *trace_out_len; /* output length (distribution mode)        */
  int64_t n_trace;
  /* Time-varying arrival rates (appendix, time-varying arrival rates): type
     j arrives at intensity lambda_j * f_j(t), f_j linear between the points
     (rate_t[i], rate_f[j * n_rate_pts + i]) and constant outside them.
     n_rate_pts = 0: constant rates (rate_t, rate_f unused); otherwise
     1..WS_MAX_RATE_PTS, no trace, lambda_j * max f_j finite.               */
  int32_t n_rate_pts;
  const double *rate_t;         /* strictly increasing, finite  [n_rate_pts] */
  const double *rate_f;         /* finite, >= 0            [m][n_rate_pts]   */
} ws_config;

/* The scheduling policy. */
typedef struct {
  int32_t kind;          /* ws_policy_kind                                   */
  const int32_t *n;      /* WAIT: n_j >= 1 [m]; NESTED: n_k >= 1 [L]         */
  int32_t L;             /* NESTED: number of segments, 1..WS_MAX_SEGMENTS   */
  const int32_t *seg_end;/* NESTED: r_1 < ... < r_L, r_L = largest output    */
  double fcfs_reserve;   /* FCFS: fraction of C kept free at admission, [0,1)*/
  int32_t fcfs_chunk;    /* FCFS: chunked prefill (the Sarathi-style baseline
                            of Section 6): at most this many prefill tokens
                            per iteration, the partially prefilled prompt
                            first, then admissions from the queue head, each
                            taking min(its remaining prompt, the budget
                            left); a chunk charges the prompt's cache after
                            it; a partial prompt holds its cached tokens, is
                            evicted first and restarts.  0: whole prefills.
                            Must be 0 for the other policies.             */
  const int32_t *stage_caps; /* optional per-stage caps (Section 6, the
                            batch-size cap tl spread over the stages).
                            NESTED: stage_caps[s-1] >= 0 is the cap of
                            decode stage s = 1..r_L; segment k takes the
                            caps of its stages r_{k-1}+1..r_k in turn, one
                            per service, as its threshold and the size of
                            the cohort it admits; n[k] must be the largest
                            cap of segment k and segment 1's caps must be
                            >= 1.  WAIT: for each type j in turn, l'_j + 1
                            caps >= 1 (its prefill and decode stages), taken
                            in turn, one per service of the type, as its
                            threshold and cohort size; n[j] must be the
                            largest.  NULL: every service admits n_k (n_j).
                            Must be NULL for the other policies.          */
} ws_policy;

/* One replica's random stream. */
typedef struct {
  uint64_t seed;
  uint32_t replica_id;
  uint32_t reserved;
} ws_stream;

/* A group of replicas sharing a model and a policy. */
typedef struct {
  const ws_config *cfg;
  const ws_policy *pol;
  const ws_stream *streams; /* [n] */
  int32_t n;
} ws_job;

/* Result layout (device buffer, structure of arrays over the R replicas of
 * all jobs, in job order):
 *   int64  [WS_NI64][R] : batches, arrivals, completions, completed_tokens,
 *                         evictions, evicted_tokens, fallback_evictions,
 *                         batch_tokens_sum, peak_mem, waiting_end,
 *                         resident_end, idle_waits
 *   double [WS_NF64][R] : t_end (T), busy_time, lat_area (sum of censored
 *                         latencies = integral of N dt), ttft_area (sum of
 *                         censored times to first token), lat_completed_sum,
 *                         mem_area (integral of launch memory over batches
 *                         and resident memory while idle)
 *   uint32 [R]          : flags
 *   uint32 [R][H]       : latency histogram of completed requests, bin b =
 *                         number of edges <= latency; H = hist stride
 *                         returned by wait_sim_results_bytes.
 * Byte offsets: i64 at 0, f64 at 8*WS_NI64*R, flags at 8*(WS_NI64+WS_NF64)*R,
 * histogram at that plus 4*R rounded up to a multiple of 8.
 * Results are cumulative over the calls that advanced the same workspace. */
#define WS_NI64 12
#define WS_NF64 6

/* Bytes of device workspace needed for these jobs. */
int wait_sim_workspace_bytes(const ws_job *jobs, int32_t n_jobs,
                             size_t *bytes);

/* Bytes of the result buffer and the histogram stride H (>= 1). */
int wait_sim_results_bytes(const ws_job *jobs, int32_t n_jobs, size_t *bytes,
                           int32_t *hist_stride);

/* Validate the jobs and copy their tables into the workspace.  Blocks the
 * host until the copy on hip_stream (hipStream_t, or NULL for the default
 * stream) has finished. */
int wait_sim_prepare(const ws_job *jobs, int32_t n_jobs, void *d_workspace,
                     size_t ws_bytes, void *hip_stream);

/* Advance every replica of a prepared workspace by `horizon` batches.
 * resume = 0 starts every replica from the empty system at t = 0;
 * resume = 1 continues from the state the previous call left.
 * Checkpoints: the workspace holds each replica's complete state (clock,
 * counters, sums, queues and resident records, histogram); a byte copy of it
 * taken between calls (device to device, or to host and back into a workspace
 * of the same jobs) is a checkpoint, and resume = 1 on the restored copy
 * continues exactly as the original would.  Asynchronous
 * on hip_stream; `jobs` must be the ones given to wait_sim_prepare.  When the
 * jobs use more than one policy kind, the kinds' kernels run concurrently:
 * the second and third on two side streams that the library creates once per
 * device and keeps, forked from hip_stream after its earlier work and joined
 * back into it before the call's later work, so hip_stream still orders
 * everything.  Calls from several host threads share those side streams
 * (their work serialises there). */
int wait_sim_advance(const ws_job *jobs, int32_t n_jobs, int64_t horizon,
                     int32_t resume, void *d_workspace, size_t ws_bytes,
                     void *d_results, size_t results_bytes, void *hip_stream);

/* Test hook: per-batch trace.  One record per replica and batch: the
 * batch's launch time, duration, tokens,
 * prefill processings (FCFS chunks included), selected prompts, completions,
 * evictions before the launch (Nested WAIT's projected-state repair) and
 * after the completion, the resident memory, waiting and resident prompts
 * after the repair, and (Nested WAIT; 0 for the other policies) the
 * projected resident memory M_res(Q+) after the pre-launch repair
 * (Algorithm 4, Appendix B.1). */
typedef struct {
  double t_launch, tau;
  int64_t tokens, prefills, selected, completions, evict_pre, evict_post,
      mem_after, waiting_after, resident_after, mplus;
} ws_batch_rec;

/* wait_sim_advance, also writing ws_batch_rec records to d_btrace (DEVICE
 * memory owned by the caller, btrace_cap records per replica, replica r's
 * batch b at index r * btrace_cap + b, b counted from the replica's start
 * across resumed calls; batches b >= btrace_cap are not recorded, records of
 * batches not run are left as they are).  btrace_cap = 0: no trace.  Runs
 * the kernels' general instantiations (slower than wait_sim_advance). */
int wait_sim_advance_traced(const ws_job *jobs, int32_t n_jobs, int64_t horizon,
                            int32_t resume, void *d_workspace, size_t ws_bytes,
                            void *d_results, size_t results_bytes, void *d_btrace,
                            int64_t btrace_cap, void *hip_stream);

/* Checkpoints of the live state (the simulation state carried from one
 * batch to the next, Section 2; Nested WAIT's segments, cohorts and boundary
 * queues, Algorithm 2).  A checkpoint is a device buffer holding a header,
 * every replica's state slots and latency histogram (structure of arrays over
 * the replicas), and per replica only the live records of its rings: the
 * queued prompts between head and tail, the resident records, and for Nested
 * WAIT every segment's cohort slots and calendar buckets and the boundary
 * queues.  Its size therefore follows the current queue lengths, not the
 * worst-case ring capacities of the workspace.  It is position-independent
 * (it may be copied to the host and back, or to another device) and belongs
 * to the jobs it was taken for: restoring checks a fingerprint of the jobs'
 * tables, seeds, replica ids and layout and of this library's layout rules.
 *
 * wait_sim_save_state: write the checkpoint of the workspace's current state
 * to d_state_out (DEVICE memory owned by the caller, state_out_bytes long).
 * Blocks the host until the checkpoint's size is known (a few small kernels
 * on hip_stream after its earlier work); the copies then run asynchronously
 * on hip_stream.  *state_used (if non-NULL) receives the size in bytes.
 * d_state_out = NULL only sizes the checkpoint.  A buffer smaller than the
 * size returns WS_EWORKSPACE (with *state_used set) and writes nothing.  The
 * workspace must not be advanced on another stream meanwhile. */
int wait_sim_save_state(const ws_job *jobs, int32_t n_jobs, void *d_workspace,
                        size_t ws_bytes, void *d_state_out,
                        size_t state_out_bytes, size_t *state_used,
                        void *hip_stream);

/* wait_sim_load_state: prepare the workspace for the jobs (as
 * wait_sim_prepare) and restore the checkpoint d_state_in (DEVICE memory,
 * state_in_bytes long, written by wait_sim_save_state or
 * wait_sim_run_batch_ex for the same jobs) into it; wait_sim_advance with
 * resume = 1 then continues exactly as the saved workspace would have.
 * Blocks the host until the restore has been checked.  Returns WS_EINVAL for
 * a buffer that is not a checkpoint of these jobs or whose records do not
 * match its state (nothing outside the checkpoint's used bytes is read). */
int wait_sim_load_state(const ws_job *jobs, int32_t n_jobs, void *d_workspace,
                        size_t ws_bytes, const void *d_state_in,
                        size_t state_in_bytes, void *hip_stream);

/* prepare (or, with d_state_in, load_state) + advance + (with d_state_out or
 * state_used) save_state, in one call: advance every replica by `horizon`
 * batches from the empty system, or from the checkpoint d_state_in, and write
 * the checkpoint of the state it leaves to d_state_out.  The results are
 * cumulative from t = 0 as for wait_sim_advance.  When d_state_out is too
 * small the call returns WS_EWORKSPACE after the advance (results written,
 * *state_used = the size needed): wait_sim_save_state with a larger buffer
 * then takes the same checkpoint.  A checkpoint buffer must not overlap the
 * workspace. */
int wait_sim_run_batch_ex(const ws_job *jobs, int32_t n_jobs, int64_t horizon,
                          void *d_workspace, size_t ws_bytes, void *d_results,
                          size_t results_bytes, void *hip_stream,
                          const void *d_state_in, size_t state_in_bytes,
                          void *d_state_out, size_t state_out_bytes,
                          size_t *state_used);

/* prepare + advance(resume = 0) for one job. */
int wait_sim_run(const ws_config *cfg, const ws_policy *pol,
                 const ws_stream *streams, int32_t n_replicas, int64_t horizon,
                 void *d_workspace, size_t ws_bytes, void *d_results,
                 size_t results_bytes, void *hip_stream);

/* prepare + advance(resume = 0) for several jobs in one launch per policy. */
int wait_sim_run_batch(const ws_job *jobs, int32_t n_jobs, int64_t horizon,
                       void *d_workspace, size_t ws_bytes, void *d_results,
                       size_t results_bytes, void *hip_stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * as wait_sim_run, with the workspace taken from a static device array of
 * WS_STATIC_WORKSPACE_BYTES (64 MiB) instead of the caller.  The caller
 * still passes the host structs and the device result buffer (sized by
 * wait_sim_results_bytes).  The call allocates no device memory and creates
 * no stream or event; it blocks the host until the job tables have been
 * copied (as wait_sim_prepare does), then launches asynchronously on
 * hip_stream.  Jobs whose workspace (wait_sim_workspace_bytes) exceeds
 * WS_STATIC_WORKSPACE_BYTES return WS_EWORKSPACE.  Every call on one GPU
 * uses that GPU's one array: calls that overlap on the same GPU (other host
 * threads, or a new call issued before an earlier call's kernels have
 * finished on another stream) race and give undefined results; serialise
 * them, e.g. on one stream.  The array is not cleared between calls (each
 * call rebuilds what it reads). */
int wait_sim_run_static(const ws_config *cfg, const ws_policy *pol,
                        const ws_stream *streams, int32_t n_replicas,
                        int64_t horizon, void *d_results, size_t results_bytes,
                        void *hip_stream);

/* Message of the last failure on this thread ("" if none). */
const char *wait_sim_last_error(void);

/* ABI version compiled into the library (WS_ABI_VERSION). */
int wait_sim_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif
