// sim_common.h -- definitions shared by the simulation kernels and the host
// library: the device job descriptor, the per-replica state slots, the
// launch arguments, the random-number pieces and the request records.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "wait_sim.h"

namespace wsim {

constexpr int kMaxTypes = WS_MAX_TYPES;
constexpr int kMaxSeg = WS_MAX_SEGMENTS;
constexpr uint32_t kFlagCap = WS_FLAG_CAPACITY;
constexpr uint32_t kFlagStall = WS_FLAG_STALL;
constexpr uint32_t kFlagOverflow = WS_FLAG_OVERFLOW;
constexpr uint32_t kFlagThin = WS_FLAG_THIN_LIMIT;
constexpr int kMaxRatePts = WS_MAX_RATE_PTS;
constexpr uint32_t kThinMax = 1u << 20;  // thinning rejections in a row
constexpr uint32_t kNil = 0xFFFFFFFFu;

// One job (a model + policy shared by a group of replicas), in device memory.
struct JobDev {
  int32_t m, policy, n_hist, out_cap;
  int32_t nseg, known, qcap_log2, rec_cap;
  int32_t nowait;  // WAIT: serve without waiting for a full cohort
  int32_t n_rate;  // rate-profile points (0: constant rates)
  int32_t chunk;   // FCFS: prefill tokens per iteration (0: whole prefills)
  int32_t pad_;
  double d0, d1;
  int64_t C, reserve_tok;
  int64_t n_trace;
  int64_t replica_begin;
  int32_t l[kMaxTypes], lp[kMaxTypes], n[kMaxTypes];
  int32_t dcap_log2[kMaxTypes];
  double lambda[kMaxTypes];     // draw rate (the thinning bound with a profile)
  double rate_fmax[kMaxTypes];  // max f_j of the rate profile
  // Nested WAIT segments (index k = 0..nseg-1 is the paper's segment k+1)
  int32_t seg_end[kMaxSeg];    // r_k
  int32_t seg_n[kMaxSeg];      // n_k
  int32_t seg_entry[kMaxSeg];  // processing stage of an entering prompt
  int32_t seg_delta[kMaxSeg];  // number of processing stages (cohort slots)
  int32_t vcap_log2[kMaxSeg];  // boundary-queue ring size (k >= 1)
  uint64_t off_edges, off_cdf, off_tr_time, off_tr_type, off_tr_len;
  uint64_t off_rate;  // rate profile: t [n_rate], then f [m][n_rate]
  uint64_t off_ring, ring_stride;
  uint64_t off_q[kMaxTypes];    // queue rings inside a replica block
  uint64_t off_d[kMaxTypes];    // resident deques inside a replica block
  uint64_t off_rec[kMaxSeg];    // Nested: interior records [delta][n]
  uint64_t off_bkt[kMaxSeg];    // Nested: calendar bucket heads [delta]
  uint64_t off_v[kMaxSeg];      // Nested: boundary-queue rings (k >= 1)
  uint64_t off_caps;            // Nested per-stage caps: int32 [r_L]
  int32_t has_caps, pad2_;
  // FCFS with drawn output lengths: resident ring (32-byte records), its exit
  // batches (u32), calendar of 2^cal_log2 buckets (u32 heads)
  uint64_t off_res, off_exit, off_cal;
  int32_t cal_log2;
  int32_t fdist;  // FCFS job run by the kernel for per-request lengths
};

// Per-replica state slots (8 bytes each), stored [slot][R].
enum Slot : int {
  S_T = 0, S_LAT, S_TTFT, S_LATSUM, S_MEM, S_BUSY,          // f64
  S_BATCHES, S_ARR, S_COMP, S_CTOK, S_EVICT, S_ETOK, S_FALLBACK, S_BTOK,
  S_PEAK, S_IDLE, S_N, S_U, S_MRES, S_TRIDX, S_FLAGS, S_PENDFT,
  S_PARTA, S_PARTJ, S_PARTPP,        // FCFS chunked prefill: the partial prompt
  S_TNEXT,                           // + kMaxTypes f64: next arrival time
  S_K = S_TNEXT + kMaxTypes,         // arrival index of the pending arrival
  S_LNEXT = S_K + kMaxTypes,         // output length of the pending arrival
  S_QH = S_LNEXT + kMaxTypes,        // queue heads
  S_QT = S_QH + kMaxTypes,           // queue tails
  S_DH = S_QT + kMaxTypes,           // deque heads
  S_DT = S_DH + kMaxTypes,           // deque tails
  S_SVC = S_DT + kMaxTypes,          // services per type (WAIT)
  S_MJ = S_SVC + kMaxTypes,          // resident memory per type
  S_KSVC = S_MJ + kMaxTypes,         // Nested: services per segment
  S_KI = S_KSVC + kMaxSeg,           // Nested: interior residents per segment
  S_KM = S_KI + kMaxSeg,             // Nested: interior memory per segment
  S_KB = S_KM + kMaxSeg,             // Nested: boundary-queue memory
  S_KVH = S_KB + kMaxSeg,            // Nested: boundary-queue heads
  S_KVT = S_KVH + kMaxSeg,           // Nested: boundary-queue tails
  S_COUNT = S_KVT + kMaxSeg
};

struct KArgs {
  uint8_t *ws;
  uint64_t off_jobs, off_seed, off_rid, off_job_of, off_list, off_state,
      off_hist;
  int64_t R;           // total replicas
  int32_t n_list;      // replicas in this launch
  int32_t hist_stride;
  int64_t horizon;
  int32_t resume;
  int32_t any_trace;   // some job of this launch replays a fixed arrival list
  int32_t any_tv;      // some job of this launch has time-varying rates
  int32_t lanes;       // replicas per wavefront (lanes >= this are padding)
  int32_t unit_n;      // WAIT launch whose jobs all have thresholds n_j = 1
  int32_t any_caps;    // some Nested WAIT job of this launch has per-stage caps
  uint8_t *btrace;     // per-batch trace [R][btrace_cap] records, or null
  int64_t btrace_cap;
};

// One record of the per-batch trace (layout of ws_batch_rec).
struct BatchRec {
  double t_launch, tau;
  int64_t tokens, prefills, selected, completions, evict_pre, evict_post, mem_after,
      waiting_after, resident_after, mplus;
};
static_assert(sizeof(BatchRec) == 96, "ws_batch_rec layout");

__device__ __forceinline__ int64_t slot_i(const KArgs &A, int s, int64_t r) {
  return ((const int64_t *)(A.ws + A.off_state))[s * A.R + r];
}
__device__ __forceinline__ double slot_f(const KArgs &A, int s, int64_t r) {
  return ((const double *)(A.ws + A.off_state))[s * A.R + r];
}
__device__ __forceinline__ void put_i(const KArgs &A, int s, int64_t r, int64_t v) {
  ((int64_t *)(A.ws + A.off_state))[s * A.R + r] = v;
}
__device__ __forceinline__ void put_f(const KArgs &A, int s, int64_t r, double v) {
  ((double *)(A.ws + A.off_state))[s * A.R + r] = v;
}

// ------------------------------------------------------------------ RNG --

__device__ __forceinline__ void philox10(uint32_t c0, uint32_t c1, uint32_t c2,
                                         uint32_t c3, uint32_t k0, uint32_t k1,
                                         uint32_t w[4]) {
  // Philox4x32-10 (Salmon et al., SC'11).
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
    const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
    c1 = (uint32_t)p1;
    c3 = (uint32_t)p0;
    c0 = n0;
    c2 = n2;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  w[0] = c0;
  w[1] = c1;
  w[2] = c2;
  w[3] = c3;
}

// Natural logarithm of u in (0,1) from IEEE basic operations only:
// u = f 2^e, f in [sqrt(1/2), sqrt(2)), ln f = 2 atanh(z), z = (f-1)/(f+1),
// atanh(z) = z sum_{i=0}^{11} z^{2i}/(2i+1) in Horner form, plus e ln 2 with
// ln 2 split into a head with zero low bits and a tail.
__device__ __forceinline__ double ln_unit(double u) {
  const uint64_t bits = (uint64_t)__double_as_longlong(u);
  int e = (int)((bits >> 52) & 0x7ff) - 1022;
  double f = __longlong_as_double(
      (long long)((bits & 0x000fffffffffffffull) | 0x3fe0000000000000ull));
  if (f < 0x1.6a09e667f3bcdp-1) {
    f = f + f;
    e = e - 1;
  }
  const double z = (f - 1.0) / (f + 1.0);
  const double w = z * z;
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
  const double lnf = (z + z) * p;
  const double de = (double)e;
  return de * 0x1.62e42fefa3800p-1 + (de * 0x1.ef35793c7673p-45 + lnf);
}

// Gap to the k-th arrival of type j, and its output length when a CDF row is
// given (smallest s in 1..cap-1 with w2 < T[s], else cap).
// Remainder by a divisor that is fixed per job (Lemire, Kaser and Kurz,
// "Faster remainder by direct computation", 2019): with M = floor((2^64 - 1)
// / d) + 1 (0 for d = 1), n mod d is the high 64 bits of (M n mod 2^64) d,
// exact for every 32-bit n and d >= 1; three 32-bit multiply steps instead of
// a reciprocal-based division.
__host__ __device__ __forceinline__ uint64_t fastmod_magic(uint32_t d) { return ~0ull / d + 1ull; }
__host__ __device__ __forceinline__ uint32_t fastmod(uint32_t n, uint64_t M, uint32_t d) {
  const uint64_t low = M * (uint64_t)n;
  const uint64_t lo_part = (uint64_t)(uint32_t)low * d;
  const uint64_t hi_part = (low >> 32) * d + (lo_part >> 32);  // < 2^64
  return (uint32_t)(hi_part >> 32);
}

// Output length from a CDF row: the smallest s in 1..cap-1 with w2 < T[s]
// (T[s] at row[s - 1], nondecreasing), else cap.  The table sits in global
// memory, so each probe is a dependent load: an 8-way search probes 7 points
// of the interval at once (independent loads, one round trip) and keeps the
// part between the last probe with T <= w2 and the first with T > w2, so a
// 2048-entry row takes 4 round trips instead of the 11 of a binary search.
__host__ __device__ __forceinline__ int32_t cdf_search_in(const uint32_t *row, int32_t lo,
                                                        int32_t hi, uint32_t w2) {
  constexpr int K = 8;
  // the answer lies in [lo, hi] (1 <= lo <= hi <= cap)
  while (lo < hi) {
    const int32_t span = hi - lo;
    int32_t pos[K - 1];
    uint32_t tv[K - 1];
#pragma unroll
    for (int i = 0; i < K - 1; ++i) {
      pos[i] = lo + (int32_t)(((int64_t)span * (i + 1)) / K);  // in [lo, hi - 1], nondecreasing
      tv[i] = row[pos[i] - 1];
    }
    int32_t nlo = lo, nhi = hi;
#pragma unroll
    for (int i = 0; i < K - 1; ++i) {
      if (tv[i] <= w2)
        nlo = pos[i] + 1;  // T[pos] <= w2: the answer lies above pos
      else if (nhi == hi)
        nhi = pos[i];      // first probe with w2 < T[pos]: the answer is at most pos
    }
    lo = nlo;
    hi = nhi;
  }
  return lo;
}
__host__ __device__ __forceinline__ int32_t cdf_search(const uint32_t *row, int32_t cap,
                                                     uint32_t w2) {
  return cdf_search_in(row, 1, cap, w2);
}

// A guide narrows the search before the first round trip: G[b] (b = 0..64)
// is the length drawn for w2 = b * 2^26, the smallest s with T[s] > b * 2^26
// (G[64] = cap).  Every w2 in [b * 2^26, (b + 1) * 2^26) then draws a
// length in [G[b], G[b + 1]]: T[s] <= w2 below G[b], and T[G[b + 1]] > w2.
constexpr int kCdfGuide = 64;
__host__ __device__ __forceinline__ int32_t cdf_guide_entry(const uint32_t *row, int32_t cap,
                                                          int b) {
  return b >= kCdfGuide ? cap : cdf_search(row, cap, (uint32_t)b << 26);
}

__device__ __forceinline__ double draw_gap(uint64_t seed, uint32_t rid,
                                           uint32_t j, uint32_t k, double lam,
                                           const uint32_t *row, int32_t cap,
                                           int32_t *L, uint32_t *w3 = nullptr,
                                           const uint16_t *guide = nullptr) {
  uint32_t w[4];
  philox10(k, j, rid, 0u, (uint32_t)seed, (uint32_t)(seed >> 32), w);
  if (w3 != nullptr) *w3 = w[3];
  const uint64_t x = ((uint64_t)w[0] << 20) | (uint64_t)(w[1] >> 12);
  const double u = (double)(2 * x + 1) * 0x1p-53;
  if (row != nullptr)
    *L = guide != nullptr ? cdf_search_in(row, guide[w[2] >> 26], guide[(w[2] >> 26) + 1], w[2])
                          : cdf_search(row, cap, w[2]);
  return -ln_unit(u) / lam;
}

// ------------------------------------------------ time-varying rates --
// A type with a rate profile arrives at intensity lambda_j f_j(t), f_j linear
// between the points rt[0..P-1] and constant outside them.

// The profile of one job as the kernels stage it in LDS: points, f_j at the
// points (rows past m are zero) and max f_j.
template <int MT, int NP>
struct RateProfLds {
  double t[NP];
  double f[MT][NP];
  double fmax[MT];
};

// Piece of the profile that holds t: -1 before the first point, P-1 from the
// last point on, else the i with rt[i] <= t < rt[i+1] (rt strictly
// increasing).  A type's candidate times never decrease, so each type keeps a
// cursor at its current piece and moves it forward: cur (-1 at the start of a
// call) is the piece of an earlier time, and on return the piece of t.
__device__ __forceinline__ int rate_seg_from(const double *rt, int P, double t, int &cur) {
  while (cur < P - 1 && !(t < rt[cur + 1])) ++cur;
  return cur;
}

// f(t) for t in piece i.
__device__ __forceinline__ double rate_fac(const double *rt, const double *f, int P, int i,
                                           double t) {
  if (i < 0) return f[0];
  if (i == P - 1) return f[P - 1];
  const double frac = (t - rt[i]) / (rt[i + 1] - rt[i]);
  return f[i] + (f[i + 1] - f[i]) * frac;
}

// Thinning decision for a candidate at time tc with fourth Philox word w3:
// 0 = kept (t = tc); 1 = rejected with zero intensity from the last point on
// (the type stops); 2 = rejected, t = the clock the next candidate starts
// from (the end of a zero stretch that holds tc, else tc).
__device__ __forceinline__ int thin_decide(double tc, uint32_t w3, double fmax,
                                           const double *rt, const double *f, int P,
                                           double &t, int &cur) {
  const int i = rate_seg_from(rt, P, tc, cur);
  if ((double)w3 * fmax < rate_fac(rt, f, P, i, tc) * 4294967296.0) {
    t = tc;
    return 0;
  }
  if (i == P - 1 && f[P - 1] == 0.0) return 1;
  if (i < 0 && f[0] == 0.0)
    t = rt[0];
  else if (i >= 0 && i < P - 1 && f[i] == 0.0 && f[i + 1] == 0.0)
    t = rt[i + 1];
  else
    t = tc;
  return 2;
}

// Next arrival of a type with a rate profile, by thinning: from candidate k
// on (the clock at the previous arrival is t), take candidates of the Poisson
// process at the bound lambda_j fmax from cand(k, &gap, &w3) and keep the first
// that thin_decide keeps.  Returns its time and leaves k at its counter (cur
// at its piece).  A zero intensity from the last point on, or kThinMax
// rejections in a row (flagged), end the type's arrivals (time +inf).
template <typename Cand>
__device__ __forceinline__ double next_thinned(uint32_t &k, double t, double fmax,
                                               const double *rt, const double *f, int P,
                                               int &cur, uint32_t &flags, Cand cand) {
  if (!(fmax > 0.0)) return INFINITY;
  for (uint32_t tries = 0;; ++tries) {
    double g;
    uint32_t w3;
    cand(k, g, w3);
    const int d = thin_decide(t + g, w3, fmax, rt, f, P, t, cur);
    if (d == 0) return t;
    if (tries + 1u >= kThinMax) {
      flags |= kFlagThin;
      return INFINITY;
    }
    if (d == 1) return INFINITY;
    ++k;
  }
}

// next_thinned with every candidate drawn here (output length into *L when a
// CDF row is given).
__device__ __forceinline__ double draw_thinned(uint64_t seed, uint32_t rid, uint32_t j,
                                               uint32_t &k, double t, double lam_c,
                                               double fmax, const double *rt,
                                               const double *f, int P,
                                               const uint32_t *row, int32_t cap,
                                               int32_t *L, int &cur, uint32_t &flags) {
  return next_thinned(k, t, fmax, rt, f, P, cur, flags,
                      [&](uint32_t kc, double &g, uint32_t &w3) {
                        g = draw_gap(seed, rid, j, kc, lam_c, row, cap, L, &w3);
                      });
}

// Histogram bin through a bucket index: the non-negative edges are bucketed
// by the top bits of their IEEE patterns (which order non-negative doubles
// like their values), so a latency (always >= 0) finds its bin with one table
// read and a few comparisons instead of a chain of dependent searches.  The
// result is the number of edges <= lat (edges strictly increasing, at most
// 255 of them).
constexpr int kHistTab = 512;  // bucket-table entries

struct HistIdx {
  int32_t shift;  // bucket = (bits >> shift) - kmin, clamped to [0, K)
  int32_t kmin;
  int32_t K;
  int32_t steps;  // most edges in one bucket
};

__device__ __forceinline__ uint64_t dbits(double x) {
  return (uint64_t)__double_as_longlong(x);
}

// Block-cooperative (every thread of the block calls it): E[0..n-1] are the
// edges staged in LDS with E[n] = +infinity; fills the table T (kHistTab
// bytes of LDS) and returns the block-uniform index parameters.
__device__ __forceinline__ HistIdx hist_index_build(const double *E, int n, uint8_t *T,
                                                    int *s_steps) {
  int p0 = 0;  // negative edges (a prefix) are below every latency
  while (p0 < n && __builtin_signbit(E[p0])) ++p0;
  HistIdx H;
  if (p0 == n) {
    H.shift = 63;
    H.kmin = 0;
    H.K = 1;
  } else {
    const uint64_t b0 = dbits(E[p0]), b1 = dbits(E[n - 1]);
    int s = 44;
    while ((b1 >> s) - (b0 >> s) >= (uint64_t)kHistTab) ++s;
    H.shift = s;
    H.kmin = (int32_t)(b0 >> s);
    H.K = (int32_t)((b1 >> s) - (b0 >> s)) + 1;
  }
  for (int k = threadIdx.x; k < H.K; k += blockDim.x) {
    // edges whose bucket is below k: the first edge at or above the
    // smallest pattern of bucket k
    const uint64_t lower = (uint64_t)(H.kmin + k) << H.shift;
    int lo = p0, hi = n;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (dbits(E[mid]) < lower)
        lo = mid + 1;
      else
        hi = mid;
    }
    T[k] = (uint8_t)(p0 == n ? n : lo);
  }
  if (threadIdx.x == 0) *s_steps = 0;
  __syncthreads();
  int mx = 0;
  for (int k = threadIdx.x; k < H.K; k += blockDim.x) {
    const int next = k + 1 < H.K ? (int)T[k + 1] : n;
    mx = max(mx, next - (int)T[k]);
  }
  atomicMax(s_steps, mx);
  __syncthreads();
  H.steps = *s_steps;
  H.shift = __builtin_amdgcn_readfirstlane(H.shift);
  H.kmin = __builtin_amdgcn_readfirstlane(H.kmin);
  H.K = __builtin_amdgcn_readfirstlane(H.K);
  H.steps = __builtin_amdgcn_readfirstlane(H.steps);
  return H;
}

__device__ __forceinline__ int hist_bin_idx(const double *E, const uint8_t *T, const HistIdx &H,
                                            double lat) {
  const int64_t key = (int64_t)(dbits(lat) >> H.shift) - H.kmin;
  const int kc = key < 0 ? 0 : (key >= H.K ? H.K - 1 : (int)key);
  int pos = T[kc];
  // a few steps at most (the table lands within H.steps edges): a copy of
  // the loop unrolled for run-time trip counts only adds branches and code
#pragma unroll 1
  for (int s = 0; s < H.steps; ++s) pos += E[pos] <= lat ? 1 : 0;
  return pos;
}

// ------------------------------------------------------------- records --

// The first-token flag travels in the sign bit of the arrival time.
__device__ __forceinline__ double with_ft(double a) { return -fabs(a); }
__device__ __forceinline__ bool has_ft(double a_ft) { return __builtin_signbit(a_ft); }
__device__ __forceinline__ double arrival_of(double a_ft) { return fabs(a_ft); }

struct DRec {   // known-length resident record, 16 bytes
  double a_ft;  // arrival time, sign = first token produced
  uint32_t kb;  // admission batch
  uint32_t kc;  // WAIT: admission service of its type; FCFS: position p
};

struct QRec {   // shared FIFO record, 16 bytes
  double a_ft;
  int32_t j;
  int32_t L;
};

struct NRec {   // Nested WAIT boundary / interior record, 32 bytes
  double a_ft;  // arrival time, sign = first token produced
  uint32_t kb;  // admission batch of the last prefill (FCFS with drawn
                // lengths; Nested WAIT leaves it unset: its record positions
                // already give the admission order)
  uint32_t kp;  // position within that batch (likewise)
  int32_t j;    // type
  int32_t L;    // output length; 0 marks an evicted interior slot
  uint32_t c;   // service of its segment at which it entered
  uint32_t next;// calendar-bucket link
};

// Orders LDS accesses between the lanes of one wavefront.  The simulation
// kernels run one wavefront per workgroup, and a wavefront's LDS operations
// complete in issue order, so a compiler barrier with wavefront-scope fences
// suffices; a workgroup barrier would also wait for every outstanding global
// store of the wavefront.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Opaque copy: stops the compiler from turning a chain of selects over the
// elements of a register array back into a dynamically indexed access (which
// would move the array to scratch memory).
template <typename T>
__device__ __forceinline__ T opaque(T x) {
  asm volatile("" : "+v"(x));
  return x;
}

// a[j] for a lane-dependent j, as selects over the elements.
template <typename T, int MT>
__device__ __forceinline__ T pick(const T (&a)[MT], int j) {
  // the barriers run unconditionally so the choice stays a select
  T e[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) e[i] = opaque(a[i]);
  T v = e[0];
#pragma unroll
  for (int i = 1; i < MT; ++i) v = (i == j) ? e[i] : v;
  return v;
}

// a[j] = v for a lane-dependent j, as selects over the elements.
template <typename T, int MT>
__device__ __forceinline__ void place(T (&a)[MT], int j, T v) {
#pragma unroll
  for (int i = 0; i < MT; ++i) a[i] = opaque((i == j) ? v : a[i]);
}

// if (c) a[j] = v, without a branch.
template <typename T, int MT>
__device__ __forceinline__ void place_if(T (&a)[MT], int j, bool c, T v) {
#pragma unroll
  for (int i = 0; i < MT; ++i) a[i] = opaque((c && i == j) ? v : a[i]);
}

// Widest wavefront (replicas per wavefront) of the known-length kernel with
// MT type slots: 64 replicas, 32 with 16 slots (see the note on 16 types in
// the design notes).
__host__ __device__ constexpr int known_max_lanes(int mt) { return mt > 8 ? 32 : 64; }

// Launch a simulation kernel on g workgroups of one 64-lane wavefront, after
// checking that its static LDS fits a workgroup on the current device (a
// kernel declaring more would otherwise run with the excess unaddressable).
template <typename Kernel>
hipError_t launch_checked(Kernel kernel, dim3 g, hipStream_t s, const KArgs &A) {
  hipFuncAttributes fa;
  hipError_t e = hipFuncGetAttributes(&fa, reinterpret_cast<const void *>(kernel));
  if (e != hipSuccess) return e;
  int dev = 0, lim = 0;
  e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&lim, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
  if (e != hipSuccess) return e;
  if (fa.sharedSizeBytes > (size_t)lim) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(kernel, g, dim3(64), 0, s, A);
  return hipGetLastError();
}

// Lanes per replica of the Nested WAIT kernel: the smallest of 4, 8, 16 that
// covers the types and the segments (one type and one segment per lane).
__host__ __device__ constexpr int nested_group_width(int max_m, int max_seg) {
  return (max_m > max_seg ? max_m : max_seg) <= 4    ? 4
         : (max_m > max_seg ? max_m : max_seg) <= 8  ? 8
         : (max_m > max_seg ? max_m : max_seg) <= 16 ? 16
         : (max_m > max_seg ? max_m : max_seg) <= 32 ? 32
                                                     : 64;
}

// Launchers, one per kernel family (defined next to their kernels).
hipError_t launch_known_wait(int max_m, const KArgs &A, hipStream_t s);
hipError_t launch_known_fcfs(int max_m, const KArgs &A, hipStream_t s);
hipError_t launch_nested(int max_m, int max_seg, const KArgs &A, hipStream_t s);
hipError_t launch_fcfs_dist(int max_m, const KArgs &A, hipStream_t s);
hipError_t launch_wait_many(int max_m, const KArgs &A, hipStream_t s);
// the kernels for launches with time-varying rates or an arrival list
hipError_t launch_known_wait_tv(int max_m, const KArgs &A, hipStream_t s);
hipError_t launch_known_fcfs_tv(int max_m, const KArgs &A, hipStream_t s);
hipError_t launch_nested_tv(int max_m, int max_seg, const KArgs &A, hipStream_t s);

}  // namespace wsim
