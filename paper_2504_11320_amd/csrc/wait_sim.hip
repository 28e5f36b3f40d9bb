// wait_sim.hip -- batched Monte Carlo simulation of the multi-stage
// LLM-inference queueing model (arXiv 2504.11320) on MI355X (gfx950).
//
// Layout: one lane per replica.  A replica's state is a handful of scalars
// (clock, per-type next arrival, counters, areas) held in registers for the
// whole run, plus ring buffers of request records in HBM:
//   - external queues (WAIT: one per type, FCFS: one shared FIFO);
//   - one resident deque per type, in admission order.
// Under WAIT a served type advances every resident prompt of that type
// (each stage holds at most n_j prompts, so min(n_j, n_js) = n_js: the
// resident-memory lemma of the Theorem 1 proof), and under FCFS every
// resident is batched every iteration; in both cases a prompt's stage is
// (services of its type since admission) and residents of one type complete
// in admission order.  A per-type deque therefore replaces the
// (type, stage) count matrix: admissions push at the back, completions pop at
// the front, LIFO evictions pop at the back, and every step costs O(events)
// instead of O(stages).
//
// Arithmetic follows the model contract exactly (same operations, same
// order, no FMA contraction) so that integer state is bit-identical to the
// oracle and floating sums match to rounding.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <string>
#include <vector>

#include "wait_sim.h"

namespace {

constexpr int kMaxTypes = WS_MAX_TYPES;
constexpr int kMaxSeg = WS_MAX_SEGMENTS;
constexpr uint32_t kFlagCap = WS_FLAG_CAPACITY;
constexpr uint32_t kFlagStall = WS_FLAG_STALL;

// ------------------------------------------------------------ device job --

struct JobDev {
  int32_t m, policy, n_hist, out_cap;
  int32_t nseg, known, qcap_log2, rec_cap;
  double d0, d1;
  int64_t C, reserve_tok;
  int64_t n_trace;
  int64_t replica_begin;
  int32_t l[kMaxTypes], lp[kMaxTypes], n[kMaxTypes];
  int32_t dcap_log2[kMaxTypes];
  double lambda[kMaxTypes];
  int32_t seg_end[kMaxSeg];
  uint64_t off_edges, off_cdf, off_tr_time, off_tr_type, off_tr_len;
  uint64_t off_ring, ring_stride;
  uint64_t off_q[kMaxTypes];  // queue ring offset inside a replica block
  uint64_t off_d[kMaxTypes];  // deque ring offset inside a replica block
};

// Per-replica state slots (8 bytes each), stored [slot][R].
enum Slot : int {
  S_T = 0, S_LAT, S_TTFT, S_LATSUM, S_MEM, S_BUSY,          // f64
  S_BATCHES, S_ARR, S_COMP, S_CTOK, S_EVICT, S_ETOK, S_FALLBACK, S_BTOK,
  S_PEAK, S_IDLE, S_N, S_U, S_MRES, S_TRIDX, S_FLAGS,       // i64
  S_TNEXT,                                                  // + kMaxTypes f64
  S_K = S_TNEXT + kMaxTypes,
  S_QH = S_K + kMaxTypes,
  S_QT = S_QH + kMaxTypes,
  S_DH = S_QT + kMaxTypes,
  S_DT = S_DH + kMaxTypes,
  S_SVC = S_DT + kMaxTypes,
  S_MJ = S_SVC + kMaxTypes,
  S_COUNT = S_MJ + kMaxTypes
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
};

// --------------------------------------------------------------- RNG -----

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

// Gap to the k-th arrival of type j (and its output length when the table
// row is given).
__device__ __forceinline__ double draw_gap(uint64_t seed, uint32_t rid,
                                           uint32_t j, uint32_t k, double lam,
                                           const uint32_t *row, int32_t cap,
                                           int32_t *L) {
  uint32_t w[4];
  philox10(k, j, rid, 0u, (uint32_t)seed, (uint32_t)(seed >> 32), w);
  const uint64_t x = ((uint64_t)w[0] << 20) | (uint64_t)(w[1] >> 12);
  const double u = (double)(2 * x + 1) * 0x1p-53;
  if (row != nullptr) {
    // smallest s in 1..cap-1 with w2 < T[s], else cap
    int32_t lo = 1, hi = cap;
    while (lo < hi) {
      const int32_t mid = (lo + hi) >> 1;
      if (w[2] < row[mid - 1])
        hi = mid;
      else
        lo = mid + 1;
    }
    *L = lo;
  }
  return -ln_unit(u) / lam;
}

// ------------------------------------------------------------ records ----

// First-token flag travels in the sign bit of the arrival time.
__device__ __forceinline__ double with_ft(double a) { return -a; }
__device__ __forceinline__ bool has_ft(double a_ft) { return __builtin_signbit(a_ft); }
__device__ __forceinline__ double arrival_of(double a_ft) { return fabs(a_ft); }

struct DRec {   // resident record, 16 bytes
  double a_ft;  // arrival time, sign = first token produced
  uint32_t kb;  // admission batch
  uint32_t kc;  // WAIT: admission service of its type; FCFS: position p
};

struct QRec {   // FCFS queue record, 16 bytes
  double a_ft;
  int32_t j;
  int32_t L;
};

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

template <typename T, int MT>
__device__ __forceinline__ T pick(const T (&a)[MT], int j) {
  T v = a[0];
#pragma unroll
  for (int i = 1; i < MT; ++i)
    if (i == j) v = a[i];
  return v;
}

template <typename T, int MT>
__device__ __forceinline__ void place(T (&a)[MT], int j, T v) {
#pragma unroll
  for (int i = 0; i < MT; ++i)
    if (i == j) a[i] = v;
}

// ------------------------------------------------------- the kernel ------
//
// POL = WS_WAIT or WS_FCFS, known output lengths.  MT = compile-time bound on
// the number of types (loops over types are unrolled so per-type state
// stays in registers).

template <int MT, int POL>
__global__ void __launch_bounds__(64) sim_known_kernel(KArgs A) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= A.n_list) return;
  const int64_t r = ((const int32_t *)(A.ws + A.off_list))[gid];
  const uint32_t jix = ((const uint32_t *)(A.ws + A.off_job_of))[r];
  const JobDev &J = ((const JobDev *)(A.ws + A.off_jobs))[jix];
  const uint64_t seed = ((const uint64_t *)(A.ws + A.off_seed))[r];
  const uint32_t rid = ((const uint32_t *)(A.ws + A.off_rid))[r];

  const int m = J.m;
  const double d0 = J.d0, d1 = J.d1;
  const int64_t C = J.C;
  const int64_t cap_adm = J.C - J.reserve_tok;
  const int n_hist = J.n_hist;
  const double *edges = (const double *)(A.ws + J.off_edges);
  const bool trace = J.n_trace > 0;
  const double *tr_time = (const double *)(A.ws + J.off_tr_time);
  const int32_t *tr_type = (const int32_t *)(A.ws + J.off_tr_type);
  const uint32_t qmask = (1u << J.qcap_log2) - 1u;
  const uint32_t rec_cap = (uint32_t)J.rec_cap;
  uint8_t *blk = A.ws + J.off_ring + (uint64_t)(r - J.replica_begin) * J.ring_stride;
  uint32_t *hist = (uint32_t *)(A.ws + A.off_hist) + r * (int64_t)A.hist_stride;

  int32_t l[MT], lp[MT], nth[MT];
  double lam[MT];
  uint32_t dmask[MT];
  uint32_t qoff[MT], doff[MT];  // ring offsets inside the replica block
  double tnext[MT];
  uint32_t kk[MT], qh[MT], qt[MT], dh[MT], dt[MT], svc[MT];
  int64_t Mj[MT];
#pragma unroll
  for (int j = 0; j < MT; ++j) {
    const bool on = j < m;
    l[j] = on ? J.l[j] : 0;
    lp[j] = on ? J.lp[j] : 1;
    nth[j] = on ? J.n[j] : 0;
    lam[j] = on ? J.lambda[j] : 0.0;
    dmask[j] = on ? (1u << J.dcap_log2[j]) - 1u : 0u;
    qoff[j] = (uint32_t)J.off_q[on ? j : 0];
    doff[j] = (uint32_t)J.off_d[on ? j : 0];
  }

  double t, lat_area, ttft_area, lat_sum, mem_area, busy;
  int64_t batches, arrivals, comps, ctok, evicts, etok, btok, peak, idle, N, U, Mres, tridx;
  uint32_t flags;

  if (!A.resume) {
    t = lat_area = ttft_area = lat_sum = mem_area = busy = 0.0;
    batches = arrivals = comps = ctok = evicts = etok = btok = peak = idle = 0;
    N = U = Mres = tridx = 0;
    flags = 0;
#pragma unroll
    for (int j = 0; j < MT; ++j) {
      kk[j] = qh[j] = qt[j] = dh[j] = dt[j] = svc[j] = 0;
      Mj[j] = 0;
      tnext[j] = INFINITY;
      if (j < m && !trace) {
        int32_t dummy;
        tnext[j] = 0.0 + draw_gap(seed, rid, (uint32_t)j, 0u, lam[j], nullptr, 0, &dummy);
      }
    }
    for (int b = 0; b <= n_hist; ++b) hist[b] = 0;
  } else {
    t = slot_f(A, S_T, r);
    lat_area = slot_f(A, S_LAT, r);
    ttft_area = slot_f(A, S_TTFT, r);
    lat_sum = slot_f(A, S_LATSUM, r);
    mem_area = slot_f(A, S_MEM, r);
    busy = slot_f(A, S_BUSY, r);
    batches = slot_i(A, S_BATCHES, r);
    arrivals = slot_i(A, S_ARR, r);
    comps = slot_i(A, S_COMP, r);
    ctok = slot_i(A, S_CTOK, r);
    evicts = slot_i(A, S_EVICT, r);
    etok = slot_i(A, S_ETOK, r);
    btok = slot_i(A, S_BTOK, r);
    peak = slot_i(A, S_PEAK, r);
    idle = slot_i(A, S_IDLE, r);
    N = slot_i(A, S_N, r);
    U = slot_i(A, S_U, r);
    Mres = slot_i(A, S_MRES, r);
    tridx = slot_i(A, S_TRIDX, r);
    flags = (uint32_t)slot_i(A, S_FLAGS, r);
#pragma unroll
    for (int j = 0; j < MT; ++j) {
      tnext[j] = slot_f(A, S_TNEXT + j, r);
      kk[j] = (uint32_t)slot_i(A, S_K + j, r);
      qh[j] = (uint32_t)slot_i(A, S_QH + j, r);
      qt[j] = (uint32_t)slot_i(A, S_QT + j, r);
      dh[j] = (uint32_t)slot_i(A, S_DH + j, r);
      dt[j] = (uint32_t)slot_i(A, S_DT + j, r);
      svc[j] = (uint32_t)slot_i(A, S_SVC + j, r);
      Mj[j] = slot_i(A, S_MJ + j, r);
    }
  }

  // Next exogenous arrival (ties: lowest type); trace mode reads the list.
  auto peek = [&](int &jn) -> double {
    if (trace) {
      if (tridx >= J.n_trace) {
        jn = 0;
        return INFINITY;
      }
      jn = tr_type[tridx];
      return tr_time[tridx];
    }
    double best = tnext[0];
    jn = 0;
#pragma unroll
    for (int j = 1; j < MT; ++j)
      if (j < m && tnext[j] < best) {
        best = tnext[j];
        jn = j;
      }
    return best;
  };

  // Append the pending arrival of type jn (time a) to its external queue
  // and draw that type's next arrival.
  auto take = [&](int jn, double a) {
    if (trace) {
      tridx++;
    } else {
      uint32_t k = pick(kk, jn) + 1u;
      place(kk, jn, k);
      int32_t dummy;
      const double g = draw_gap(seed, rid, (uint32_t)jn, k, pick(lam, jn), nullptr, 0, &dummy);
      place(tnext, jn, pick(tnext, jn) + g);
    }
    arrivals++;
    N++;
    U++;
    if (POL == WS_WAIT) {
      const uint32_t h = pick(qh, jn), tt = pick(qt, jn);
      if (tt - h >= rec_cap)
        flags |= kFlagCap;
      else
        ((double *)(blk + pick(qoff, jn)))[tt & qmask] = a;
      place(qt, jn, tt + 1u);
    } else {
      const uint32_t h = qh[0], tt = qt[0];
      if (tt - h >= rec_cap) {
        flags |= kFlagCap;
      } else {
        QRec rec;
        rec.a_ft = a;
        rec.j = jn;
        rec.L = pick(lp, jn);
        ((QRec *)(blk + qoff[0]))[tt & qmask] = rec;
      }
      qt[0] = tt + 1u;
    }
  };

  bool stopped = (flags & (kFlagCap | kFlagStall)) != 0;
  uint32_t newcnt[MT];

  for (int64_t it = 0; it < A.horizon && !stopped; ++it) {
    // ---- decision: form a batch or wait for the next arrival ------------
    uint32_t elig = 0;
    int64_t tokens = 0, prefill_l = 0;
    for (;;) {
      if (flags & kFlagCap) {
        stopped = true;
        break;
      }
      elig = 0;
      if (POL == WS_WAIT) {
#pragma unroll
        for (int j = 0; j < MT; ++j)
          if (j < m && (qt[j] - qh[j]) >= (uint32_t)nth[j]) elig |= 1u << j;
      } else {
        int64_t resident = 0;
#pragma unroll
        for (int j = 0; j < MT; ++j) resident += (int64_t)(dt[j] - dh[j]);
        if (resident > 0 || qt[0] != qh[0]) elig = 1;
      }
      if (elig) break;
      int jn;
      const double ta = peek(jn);
      if (!(ta < INFINITY)) {
        flags |= kFlagStall;
        stopped = true;
        break;
      }
      const double dtm = ta - t;
      lat_area += (double)N * dtm;
      ttft_area += (double)U * dtm;
      mem_area += (double)Mres * dtm;
      t = ta;
      // every arrival at this instant joins before the next decision; a full
      // queue ends the replica, which also bounds this loop
      for (;;) {
        if (flags & kFlagCap) break;
        int j2;
        const double a2 = peek(j2);
        if (a2 != ta) break;
        take(j2, a2);
      }
      idle++;
    }
    if (stopped) break;

    // ---- launch: admissions and batch tokens --------------------------
#pragma unroll
    for (int j = 0; j < MT; ++j) newcnt[j] = 0;
    const uint32_t bidx = (uint32_t)batches;
    if (POL == WS_WAIT) {
#pragma unroll
      for (int j = 0; j < MT; ++j) {
        if (!(elig & (1u << j))) continue;
        const double *q = (const double *)(blk + qoff[j]);
        DRec *d = (DRec *)(blk + doff[j]);
        const uint32_t c = svc[j] + 1u;
        for (int x = 0; x < nth[j]; ++x) {
          DRec rec;
          rec.a_ft = q[qh[j] & qmask];
          rec.kb = bidx;
          rec.kc = c;
          d[dt[j] & dmask[j]] = rec;
          qh[j]++;
          dt[j]++;
        }
        newcnt[j] = (uint32_t)nth[j];
        tokens += (int64_t)nth[j] * l[j] + Mj[j];
        prefill_l += (int64_t)nth[j] * l[j];
      }
    } else {
      tokens = Mres;
      const QRec *q = (const QRec *)(blk + qoff[0]);
      uint32_t p = 0;
      while (qt[0] != qh[0]) {
        const QRec head = q[qh[0] & qmask];
        const int hj = head.j;
        const int64_t hl = pick(l, hj);
        if (Mres + prefill_l + hl > cap_adm) break;
        qh[0]++;
        DRec rec;
        rec.a_ft = head.a_ft;
        rec.kb = bidx;
        rec.kc = p++;
#pragma unroll
        for (int j = 0; j < MT; ++j)
          if (j == hj) {
            DRec *d = (DRec *)(blk + doff[j]);
            d[dt[j] & dmask[j]] = rec;
            dt[j]++;
            newcnt[j]++;
          }
        prefill_l += hl;
      }
      tokens += prefill_l;
    }

    const int64_t m_launch = Mres + prefill_l;
    if (m_launch > peak) peak = m_launch;
    const double tau = d0 + d1 * (double)tokens;
    const double t_end = t + tau;
    const int64_t N0 = N, U0 = U;

    // ---- arrivals during the batch ------------------------------------
    for (;;) {
      if (flags & kFlagCap) break;  // the replica stops at its next decision
      int jn;
      const double ta = peek(jn);
      if (!(ta <= t_end)) break;
      take(jn, ta);
      lat_area += t_end - ta;
      ttft_area += t_end - ta;
    }
    lat_area += (double)N0 * tau;
    ttft_area += (double)U0 * tau;
    mem_area += (double)m_launch * tau;
    busy += tau;
    t = t_end;

    // ---- completion transition ------------------------------------------
#pragma unroll
    for (int j = 0; j < MT; ++j) {
      const bool served = (POL == WS_WAIT) ? ((elig >> j) & 1u) != 0
                                           : (j < m && (dt[j] - dh[j]) > 0);
      if (!served) continue;
      DRec *d = (DRec *)(blk + doff[j]);
      // stage reached by a record: WAIT counts services of its type, FCFS
      // counts batches
      const uint32_t now = (POL == WS_WAIT) ? svc[j] + 1u : bidx;
      if (POL == WS_WAIT) svc[j] = now;
      const uint32_t fresh = newcnt[j];
      const uint32_t before = (dt[j] - dh[j]) - fresh;  // residents at launch
      // completions: processed at stage l'_j
      uint32_t done = 0;
      while (done < before) {
        const DRec rec = d[dh[j] & dmask[j]];
        const uint32_t adm = rec.kc;
        const uint32_t admb = (POL == WS_WAIT) ? adm : rec.kb;
        if (admb + (uint32_t)lp[j] != now) break;
        if (!has_ft(rec.a_ft)) U--;  // l'_j = 1: first token at completion
        const double lat = t_end - arrival_of(rec.a_ft);
        lat_sum += lat;
        int lo = 0, hi = n_hist;
        while (lo < hi) {
          const int mid = (lo + hi) >> 1;
          if (edges[mid] <= lat)
            lo = mid + 1;
          else
            hi = mid;
        }
        hist[lo] += 1u;
        comps++;
        ctok += lp[j];
        N--;
        Mj[j] -= (int64_t)l[j] + lp[j];
        dh[j]++;
        done++;
      }
      // first tokens: residents processed at stage 1 (admitted one service
      // earlier), located just before this launch's admissions
      if (lp[j] > 1) {
        uint32_t idx = dt[j] - fresh;
        uint32_t left = before - done;
        while (left > 0) {
          DRec *pr = &d[(idx - 1u) & dmask[j]];
          const uint32_t admb = (POL == WS_WAIT) ? pr->kc : pr->kb;
          if (admb + 1u != now) break;
          if (!has_ft(pr->a_ft)) {
            pr->a_ft = with_ft(pr->a_ft);
            U--;
          }
          idx--;
          left--;
        }
      }
      Mj[j] += (int64_t)(before - done) + (int64_t)fresh * (l[j] + 1);
    }
    Mres = 0;
#pragma unroll
    for (int j = 0; j < MT; ++j) Mres += Mj[j];
    if (Mres > peak) peak = Mres;

    // ---- repair: evict the most recently admitted resident ------------
    while (Mres > C) {
      int jb = -1;
      uint32_t bb = 0, bp = 0;
#pragma unroll
      for (int j = 0; j < MT; ++j) {
        if (j >= m || dt[j] == dh[j]) continue;
        const DRec *d = (const DRec *)(blk + doff[j]);
        const DRec rec = d[(dt[j] - 1u) & dmask[j]];
        const uint32_t pb = (POL == WS_WAIT) ? (uint32_t)j : rec.kc;
        if (jb < 0 || rec.kb > bb || (rec.kb == bb && pb > bp)) {
          jb = j;
          bb = rec.kb;
          bp = pb;
        }
      }
      if (jb < 0) break;
#pragma unroll
      for (int j = 0; j < MT; ++j) {
        if (j != jb) continue;
        DRec *d = (DRec *)(blk + doff[j]);
        const DRec rec = d[(dt[j] - 1u) & dmask[j]];
        dt[j]--;
        const uint32_t admb = (POL == WS_WAIT) ? rec.kc : rec.kb;
        const uint32_t now = (POL == WS_WAIT) ? svc[j] : bidx;
        const int64_t stage = (int64_t)(now - admb) + 1;
        Mj[j] -= (int64_t)l[j] + stage;
        Mres -= (int64_t)l[j] + stage;
        evicts++;
        etok += stage - 1;
        // back to the tail of the external queue
        if (POL == WS_WAIT) {
          double *q = (double *)(blk + qoff[j]);
          if (qt[j] - qh[j] >= rec_cap)
            flags |= kFlagCap;
          else
            q[qt[j] & qmask] = rec.a_ft;
          qt[j]++;
        } else {
          QRec *q = (QRec *)(blk + qoff[0]);
          if (qt[0] - qh[0] >= rec_cap) {
            flags |= kFlagCap;
          } else {
            QRec qr;
            qr.a_ft = rec.a_ft;
            qr.j = j;
            qr.L = lp[j];
            q[qt[0] & qmask] = qr;
          }
          qt[0]++;
        }
      }
    }
    batches++;
    btok += tokens;
  }

  // ---- save state --------------------------------------------------------
  put_f(A, S_T, r, t);
  put_f(A, S_LAT, r, lat_area);
  put_f(A, S_TTFT, r, ttft_area);
  put_f(A, S_LATSUM, r, lat_sum);
  put_f(A, S_MEM, r, mem_area);
  put_f(A, S_BUSY, r, busy);
  put_i(A, S_BATCHES, r, batches);
  put_i(A, S_ARR, r, arrivals);
  put_i(A, S_COMP, r, comps);
  put_i(A, S_CTOK, r, ctok);
  put_i(A, S_EVICT, r, evicts);
  put_i(A, S_ETOK, r, etok);
  put_i(A, S_FALLBACK, r, 0);
  put_i(A, S_BTOK, r, btok);
  put_i(A, S_PEAK, r, peak);
  put_i(A, S_IDLE, r, idle);
  put_i(A, S_N, r, N);
  put_i(A, S_U, r, U);
  put_i(A, S_MRES, r, Mres);
  put_i(A, S_TRIDX, r, tridx);
  put_i(A, S_FLAGS, r, (int64_t)flags);
#pragma unroll
  for (int j = 0; j < MT; ++j) {
    put_f(A, S_TNEXT + j, r, tnext[j]);
    put_i(A, S_K + j, r, kk[j]);
    put_i(A, S_QH + j, r, qh[j]);
    put_i(A, S_QT + j, r, qt[j]);
    put_i(A, S_DH + j, r, dh[j]);
    put_i(A, S_DT + j, r, dt[j]);
    put_i(A, S_SVC + j, r, svc[j]);
    put_i(A, S_MJ + j, r, Mj[j]);
  }
}

// Copy the per-replica state of a workspace into the result layout.
__global__ void __launch_bounds__(256) export_kernel(KArgs A, uint8_t *out) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= A.R) return;
  const int64_t R = A.R;
  int64_t *oi = (int64_t *)out;
  double *of = (double *)(out + 8 * WS_NI64 * R);
  uint32_t *ofl = (uint32_t *)(out + 8 * (WS_NI64 + WS_NF64) * R);
  const uint32_t jix = ((const uint32_t *)(A.ws + A.off_job_of))[r];
  const JobDev &J = ((const JobDev *)(A.ws + A.off_jobs))[jix];
  const int fi[WS_NI64] = {S_BATCHES, S_ARR, S_COMP, S_CTOK, S_EVICT, S_ETOK,
                           S_FALLBACK, S_BTOK, S_PEAK, -1, -1, S_IDLE};
  for (int f = 0; f < WS_NI64; ++f)
    if (fi[f] >= 0) oi[f * R + r] = slot_i(A, fi[f], r);
  // waiting and resident counts at T
  int64_t waiting = 0, resident = 0;
  const int nq = (J.policy == WS_WAIT) ? J.m : 1;
  for (int j = 0; j < nq; ++j) waiting += slot_i(A, S_QT + j, r) - slot_i(A, S_QH + j, r);
  for (int j = 0; j < J.m; ++j) resident += slot_i(A, S_DT + j, r) - slot_i(A, S_DH + j, r);
  oi[9 * R + r] = waiting;
  oi[10 * R + r] = resident;
  const int ff[WS_NF64] = {S_T, S_BUSY, S_LAT, S_TTFT, S_LATSUM, S_MEM};
  for (int f = 0; f < WS_NF64; ++f) of[f * R + r] = slot_f(A, ff[f], r);
  ofl[r] = (uint32_t)slot_i(A, S_FLAGS, r);
}

// ------------------------------------------------------------- host -----

thread_local std::string g_err;

int fail(int code, const std::string &msg) {
  g_err = msg;
  return code;
}

int ceil_log2(uint64_t x) {
  int k = 0;
  while ((1ull << k) < x) ++k;
  return k;
}

uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

struct JobHost {
  JobDev d;
  int64_t reserve_tok;
  uint64_t edges_bytes, cdf_bytes, trace_bytes;
};

struct Layout {
  int64_t R = 0;
  int32_t hist_stride = 1;
  uint64_t off_jobs = 0, off_seed = 0, off_rid = 0, off_job_of = 0,
           off_list = 0, off_tables = 0, off_state = 0, off_hist = 0,
           off_rings = 0, total = 0;
  std::vector<JobHost> jobs;
  int32_t list_count[3] = {0, 0, 0};
  uint64_t list_off[3] = {0, 0, 0};
  int32_t max_m[3] = {0, 0, 0};
};

int validate_job(const ws_job &jb, int idx, JobHost &H) {
  const std::string at = "job " + std::to_string(idx) + ": ";
  if (!jb.cfg || !jb.pol) return fail(WS_EINVAL, at + "cfg and pol must be non-NULL");
  if (jb.n < 0) return fail(WS_EINVAL, at + "negative replica count");
  if (jb.n > 0 && !jb.streams) return fail(WS_EINVAL, at + "streams must be non-NULL");
  const ws_config &c = *jb.cfg;
  const ws_policy &p = *jb.pol;
  if (c.m < 1 || c.m > WS_MAX_TYPES)
    return fail(WS_EINVAL, at + "m must be in 1.." + std::to_string(WS_MAX_TYPES));
  if (!c.prompt_len || !c.lambda) return fail(WS_EINVAL, at + "prompt_len and lambda required");
  for (int j = 0; j < c.m; ++j) {
    if (c.prompt_len[j] < 1) return fail(WS_EINVAL, at + "prompt lengths must be >= 1");
    if (!(c.lambda[j] >= 0.0) || !std::isfinite(c.lambda[j]))
      return fail(WS_EINVAL, at + "rates must be finite and >= 0");
  }
  if (!(c.d0 > 0.0) || !std::isfinite(c.d0)) return fail(WS_EINVAL, at + "d0 must be > 0");
  if (!(c.d1 >= 0.0) || !std::isfinite(c.d1)) return fail(WS_EINVAL, at + "d1 must be >= 0");
  if (c.C < 1 || c.C > (int64_t(1) << 30)) return fail(WS_EINVAL, at + "C must be in 1..2^30");
  const bool known = c.out_len != nullptr;
  int64_t maxL = 0;
  if (known) {
    for (int j = 0; j < c.m; ++j) {
      if (c.out_len[j] < 1) return fail(WS_EINVAL, at + "output lengths must be >= 1");
      maxL = std::max<int64_t>(maxL, c.out_len[j]);
    }
  } else {
    if (c.out_cap < 1) return fail(WS_EINVAL, at + "out_cap must be >= 1 without out_len");
    maxL = c.out_cap;
    if (c.n_trace == 0) {
      if (c.out_cap > 1 && !c.out_cdf_u32) return fail(WS_EINVAL, at + "out_cdf_u32 required");
      for (int j = 0; j < c.m; ++j)
        for (int s = 1; s + 1 < c.out_cap; ++s)
          if (c.out_cdf_u32[(size_t)j * (c.out_cap - 1) + s] <
              c.out_cdf_u32[(size_t)j * (c.out_cap - 1) + s - 1])
            return fail(WS_EINVAL, at + "CDF table rows must be nondecreasing");
    }
  }
  if (c.n_hist < 0 || c.n_hist > WS_MAX_HIST_EDGES)
    return fail(WS_EINVAL, at + "n_hist out of range");
  if (c.n_hist > 0) {
    if (!c.hist_edges) return fail(WS_EINVAL, at + "hist_edges required");
    for (int b = 0; b < c.n_hist; ++b) {
      if (!std::isfinite(c.hist_edges[b])) return fail(WS_EINVAL, at + "edges must be finite");
      if (b > 0 && !(c.hist_edges[b] > c.hist_edges[b - 1]))
        return fail(WS_EINVAL, at + "edges must be strictly increasing");
    }
  }
  if (c.record_capacity < 16 || c.record_capacity > (1 << 26) ||
      (c.record_capacity & (c.record_capacity - 1)) != 0)
    return fail(WS_EINVAL, at + "record_capacity must be a power of two in 16..2^26");
  if (c.n_trace < 0) return fail(WS_EINVAL, at + "n_trace must be >= 0");
  if (c.n_trace > 0) {
    if (!c.trace_time || !c.trace_type) return fail(WS_EINVAL, at + "trace arrays required");
    if (!known && !c.trace_out_len) return fail(WS_EINVAL, at + "trace_out_len required");
    for (int64_t i = 0; i < c.n_trace; ++i) {
      if (!(c.trace_time[i] >= 0.0) || !std::isfinite(c.trace_time[i]))
        return fail(WS_EINVAL, at + "trace times must be finite and >= 0");
      if (i > 0 && c.trace_time[i] < c.trace_time[i - 1])
        return fail(WS_EINVAL, at + "trace times must be nondecreasing");
      if (c.trace_type[i] < 0 || c.trace_type[i] >= c.m)
        return fail(WS_EINVAL, at + "trace type out of range");
      if (!known && (c.trace_out_len[i] < 1 || c.trace_out_len[i] > c.out_cap))
        return fail(WS_EINVAL, at + "trace output length out of range");
    }
  }
  int64_t reserve_tok = 0;
  if (p.kind == WS_WAIT) {
    if (!known) return fail(WS_EINVAL, at + "WAIT needs known output lengths");
    if (!p.n) return fail(WS_EINVAL, at + "thresholds required");
    for (int j = 0; j < c.m; ++j)
      if (p.n[j] < 1) return fail(WS_EINVAL, at + "thresholds must be >= 1");
  } else if (p.kind == WS_FCFS) {
    if (!(p.fcfs_reserve >= 0.0 && p.fcfs_reserve < 1.0))
      return fail(WS_EINVAL, at + "fcfs_reserve must be in [0,1)");
    reserve_tok = (int64_t)std::ceil(p.fcfs_reserve * (double)c.C);
    for (int j = 0; j < c.m; ++j)
      if (c.prompt_len[j] > c.C - reserve_tok)
        return fail(WS_EINVAL, at + "a prompt does not fit below the FCFS reserve");
    if (!known) return fail(WS_EUNSUPPORTED, at + "FCFS with unknown lengths is not in this build");
  } else if (p.kind == WS_NESTED_WAIT) {
    if (p.L < 1 || p.L > WS_MAX_SEGMENTS) return fail(WS_EINVAL, at + "L out of range");
    if (!p.n || !p.seg_end) return fail(WS_EINVAL, at + "thresholds and seg_end required");
    for (int k = 0; k < p.L; ++k) {
      if (p.n[k] < 1) return fail(WS_EINVAL, at + "thresholds must be >= 1");
      if (p.seg_end[k] < 1 || (k > 0 && p.seg_end[k] <= p.seg_end[k - 1]))
        return fail(WS_EINVAL, at + "seg_end must be strictly increasing and >= 1");
    }
    if (p.seg_end[p.L - 1] != maxL)
      return fail(WS_EINVAL, at + "last segment must end at the largest output length");
    return fail(WS_EUNSUPPORTED, at + "Nested WAIT kernel is not in this build");
  } else {
    return fail(WS_EINVAL, at + "unknown policy kind");
  }
  for (int j = 0; j < c.m; ++j) {
    const int64_t Lj = known ? c.out_len[j] : c.out_cap;
    if (c.prompt_len[j] + Lj > c.C)
      return fail(WS_EINVAL, at + "a single prompt does not fit in C (atomic feasibility)");
  }

  JobDev &d = H.d;
  std::memset(&d, 0, sizeof(d));
  d.m = c.m;
  d.policy = p.kind;
  d.n_hist = c.n_hist;
  d.out_cap = c.out_cap;
  d.nseg = p.kind == WS_NESTED_WAIT ? p.L : 0;
  d.known = known ? 1 : 0;
  d.qcap_log2 = ceil_log2((uint64_t)c.record_capacity);
  d.rec_cap = c.record_capacity;
  d.d0 = c.d0;
  d.d1 = c.d1;
  d.C = c.C;
  d.reserve_tok = reserve_tok;
  d.n_trace = c.n_trace;
  for (int j = 0; j < c.m; ++j) {
    d.l[j] = c.prompt_len[j];
    d.lp[j] = known ? c.out_len[j] : c.out_cap;
    d.lambda[j] = c.lambda[j];
    d.n[j] = (p.kind == WS_WAIT) ? p.n[j] : 0;
    uint64_t dcap;
    if (p.kind == WS_WAIT)  // launch holds <= (l'_j + 1) n_j records
      dcap = (uint64_t)(c.out_len[j] + 1) * (uint64_t)p.n[j];
    else                    // residents of type j charge >= l_j each
      dcap = (uint64_t)(c.C / c.prompt_len[j]) + 2;
    d.dcap_log2[j] = ceil_log2(std::max<uint64_t>(dcap, 2));
  }
  H.reserve_tok = reserve_tok;
  H.edges_bytes = align_up(8ull * (uint64_t)std::max(c.n_hist, 1), 256);
  H.cdf_bytes = (!known && c.n_trace == 0 && c.out_cap > 1)
                    ? align_up(4ull * (uint64_t)c.m * (uint64_t)(c.out_cap - 1), 256)
                    : 0;
  H.trace_bytes = c.n_trace > 0 ? align_up(16ull * (uint64_t)c.n_trace, 256) : 0;
  // ring block of one replica
  uint64_t off = 0;
  const uint64_t qrec = (p.kind == WS_WAIT) ? 8 : 16;
  const int nq = (p.kind == WS_WAIT) ? c.m : 1;
  for (int j = 0; j < nq; ++j) {
    d.off_q[j] = off;
    off += align_up(qrec << d.qcap_log2, 256);
  }
  for (int j = 0; j < c.m; ++j) {
    d.off_d[j] = off;
    off += align_up(16ull << d.dcap_log2[j], 256);
  }
  d.ring_stride = off;
  return WS_OK;
}

int make_layout(const ws_job *jobs, int32_t n_jobs, Layout &Lo) {
  if (n_jobs < 1 || !jobs) return fail(WS_EINVAL, "need at least one job");
  Lo = Layout();
  Lo.jobs.resize(n_jobs);
  int64_t R = 0;
  int32_t hmax = 0;
  for (int i = 0; i < n_jobs; ++i) {
    int rc = validate_job(jobs[i], i, Lo.jobs[i]);
    if (rc != WS_OK) return rc;
    Lo.jobs[i].d.replica_begin = R;
    R += jobs[i].n;
    hmax = std::max(hmax, jobs[i].cfg->n_hist + 1);
    const int pk = jobs[i].pol->kind;
    Lo.list_count[pk] += jobs[i].n;
    Lo.max_m[pk] = std::max(Lo.max_m[pk], jobs[i].cfg->m);
  }
  if (R < 1) return fail(WS_EINVAL, "no replicas");
  if (R > (int64_t(1) << 30)) return fail(WS_EINVAL, "too many replicas");
  Lo.R = R;
  Lo.hist_stride = hmax;
  uint64_t off = 256;
  Lo.off_jobs = off;
  off = align_up(off + sizeof(JobDev) * (uint64_t)n_jobs, 256);
  Lo.off_seed = off;
  off = align_up(off + 8ull * R, 256);
  Lo.off_rid = off;
  off = align_up(off + 4ull * R, 256);
  Lo.off_job_of = off;
  off = align_up(off + 4ull * R, 256);
  Lo.off_list = off;
  for (int pk = 0; pk < 3; ++pk) {
    Lo.list_off[pk] = off;
    off = align_up(off + 4ull * (uint64_t)Lo.list_count[pk], 256);
  }
  Lo.off_tables = off;
  for (int i = 0; i < n_jobs; ++i) {
    JobHost &H = Lo.jobs[i];
    H.d.off_edges = off;
    off += H.edges_bytes;
    H.d.off_cdf = off;
    off += H.cdf_bytes;
    H.d.off_tr_time = off;
    H.d.off_tr_type = off + 8ull * (uint64_t)jobs[i].cfg->n_trace;
    H.d.off_tr_len = off + 12ull * (uint64_t)jobs[i].cfg->n_trace;
    off += H.trace_bytes;
  }
  off = align_up(off, 256);
  Lo.off_state = off;
  off = align_up(off + 8ull * S_COUNT * (uint64_t)R, 256);
  Lo.off_hist = off;
  off = align_up(off + 4ull * (uint64_t)hmax * (uint64_t)R, 256);
  Lo.off_rings = off;
  for (int i = 0; i < n_jobs; ++i) {
    JobHost &H = Lo.jobs[i];
    H.d.off_ring = off;
    off += H.d.ring_stride * (uint64_t)jobs[i].n;
    off = align_up(off, 256);
  }
  Lo.total = off;
  return WS_OK;
}

uint64_t results_size(const Layout &Lo) {
  const uint64_t R = (uint64_t)Lo.R;
  uint64_t off = 8ull * (WS_NI64 + WS_NF64) * R + 4ull * R;
  off = align_up(off, 8);
  return off + 4ull * (uint64_t)Lo.hist_stride * R;
}

uint64_t results_hist_offset(const Layout &Lo) {
  const uint64_t R = (uint64_t)Lo.R;
  return align_up(8ull * (WS_NI64 + WS_NF64) * R + 4ull * R, 8);
}

#define HIP_TRY(expr)                                                       \
  do {                                                                      \
    hipError_t e_ = (expr);                                                 \
    if (e_ != hipSuccess)                                                   \
      return fail(WS_EDEVICE, std::string(#expr) + ": " + hipGetErrorString(e_)); \
  } while (0)

KArgs base_args(const Layout &Lo, void *d_ws) {
  KArgs A;
  std::memset(&A, 0, sizeof(A));
  A.ws = (uint8_t *)d_ws;
  A.off_jobs = Lo.off_jobs;
  A.off_seed = Lo.off_seed;
  A.off_rid = Lo.off_rid;
  A.off_job_of = Lo.off_job_of;
  A.off_state = Lo.off_state;
  A.off_hist = Lo.off_hist;
  A.R = Lo.R;
  A.hist_stride = Lo.hist_stride;
  return A;
}

template <int MT, int POL>
hipError_t launch_known(KArgs A, hipStream_t s) {
  const int threads = 64;
  const int blocks = (A.n_list + threads - 1) / threads;
  hipLaunchKernelGGL((sim_known_kernel<MT, POL>), dim3(blocks), dim3(threads), 0, s, A);
  return hipGetLastError();
}

template <int POL>
hipError_t launch_by_m(int max_m, KArgs A, hipStream_t s) {
  if (max_m <= 2) return launch_known<2, POL>(A, s);
  if (max_m <= 4) return launch_known<4, POL>(A, s);
  if (max_m <= 8) return launch_known<8, POL>(A, s);
  return launch_known<16, POL>(A, s);
}

}  // namespace

// ---------------------------------------------------------------- C ABI --

extern "C" {

const char *wait_sim_last_error(void) { return g_err.c_str(); }

int wait_sim_abi_version(void) { return WS_ABI_VERSION; }

int wait_sim_workspace_bytes(const ws_job *jobs, int32_t n_jobs, size_t *bytes) {
  g_err.clear();
  if (!bytes) return fail(WS_EINVAL, "bytes must be non-NULL");
  Layout Lo;
  int rc = make_layout(jobs, n_jobs, Lo);
  if (rc != WS_OK) return rc;
  *bytes = (size_t)Lo.total;
  return WS_OK;
}

int wait_sim_results_bytes(const ws_job *jobs, int32_t n_jobs, size_t *bytes,
                           int32_t *hist_stride) {
  g_err.clear();
  if (!bytes) return fail(WS_EINVAL, "bytes must be non-NULL");
  Layout Lo;
  int rc = make_layout(jobs, n_jobs, Lo);
  if (rc != WS_OK) return rc;
  *bytes = (size_t)results_size(Lo);
  if (hist_stride) *hist_stride = Lo.hist_stride;
  return WS_OK;
}

int wait_sim_prepare(const ws_job *jobs, int32_t n_jobs, void *d_workspace,
                     size_t ws_bytes, void *hip_stream) {
  g_err.clear();
  Layout Lo;
  int rc = make_layout(jobs, n_jobs, Lo);
  if (rc != WS_OK) return rc;
  if (!d_workspace) return fail(WS_EINVAL, "workspace must be non-NULL");
  if (ws_bytes < Lo.total) return fail(WS_EWORKSPACE, "workspace too small");
  hipStream_t s = (hipStream_t)hip_stream;
  // host image of everything up to the state region
  std::vector<uint8_t> img(Lo.off_state, 0);
  for (int i = 0; i < n_jobs; ++i)
    std::memcpy(img.data() + Lo.off_jobs + sizeof(JobDev) * i, &Lo.jobs[i].d, sizeof(JobDev));
  int64_t r = 0;
  std::vector<int32_t> lists[3];
  for (int i = 0; i < n_jobs; ++i) {
    const ws_job &jb = jobs[i];
    for (int x = 0; x < jb.n; ++x, ++r) {
      std::memcpy(img.data() + Lo.off_seed + 8 * r, &jb.streams[x].seed, 8);
      std::memcpy(img.data() + Lo.off_rid + 4 * r, &jb.streams[x].replica_id, 4);
      const uint32_t ji = (uint32_t)i;
      std::memcpy(img.data() + Lo.off_job_of + 4 * r, &ji, 4);
      lists[jb.pol->kind].push_back((int32_t)r);
    }
    const ws_config &c = *jb.cfg;
    const JobDev &d = Lo.jobs[i].d;
    if (c.n_hist > 0) std::memcpy(img.data() + d.off_edges, c.hist_edges, 8ull * c.n_hist);
    if (Lo.jobs[i].cdf_bytes)
      std::memcpy(img.data() + d.off_cdf, c.out_cdf_u32, 4ull * c.m * (c.out_cap - 1));
    if (c.n_trace > 0) {
      std::memcpy(img.data() + d.off_tr_time, c.trace_time, 8ull * c.n_trace);
      std::memcpy(img.data() + d.off_tr_type, c.trace_type, 4ull * c.n_trace);
      if (c.trace_out_len)
        std::memcpy(img.data() + d.off_tr_len, c.trace_out_len, 4ull * c.n_trace);
    }
  }
  for (int pk = 0; pk < 3; ++pk)
    if (!lists[pk].empty())
      std::memcpy(img.data() + Lo.list_off[pk], lists[pk].data(), 4 * lists[pk].size());
  HIP_TRY(hipMemcpyAsync(d_workspace, img.data(), img.size(), hipMemcpyHostToDevice, s));
  HIP_TRY(hipStreamSynchronize(s));
  return WS_OK;
}

int wait_sim_advance(const ws_job *jobs, int32_t n_jobs, int64_t horizon,
                     int32_t resume, void *d_workspace, size_t ws_bytes,
                     void *d_results, size_t results_bytes, void *hip_stream) {
  g_err.clear();
  Layout Lo;
  int rc = make_layout(jobs, n_jobs, Lo);
  if (rc != WS_OK) return rc;
  if (horizon < 0) return fail(WS_EINVAL, "horizon must be >= 0");
  if (!d_workspace || !d_results) return fail(WS_EINVAL, "device buffers must be non-NULL");
  if (ws_bytes < Lo.total) return fail(WS_EWORKSPACE, "workspace too small");
  if (results_bytes < results_size(Lo)) return fail(WS_EWORKSPACE, "result buffer too small");
  hipStream_t s = (hipStream_t)hip_stream;
  KArgs A = base_args(Lo, d_workspace);
  A.horizon = horizon;
  A.resume = resume ? 1 : 0;
  for (int pk = 0; pk < 3; ++pk) {
    if (Lo.list_count[pk] == 0) continue;
    KArgs B = A;
    B.off_list = Lo.list_off[pk];
    B.n_list = Lo.list_count[pk];
    hipError_t e = hipSuccess;
    if (pk == WS_WAIT)
      e = launch_by_m<WS_WAIT>(Lo.max_m[pk], B, s);
    else if (pk == WS_FCFS)
      e = launch_by_m<WS_FCFS>(Lo.max_m[pk], B, s);
    if (e != hipSuccess) return fail(WS_EDEVICE, std::string("launch: ") + hipGetErrorString(e));
  }
  const int tb = 256;
  hipLaunchKernelGGL(export_kernel, dim3((unsigned)((Lo.R + tb - 1) / tb)), dim3(tb), 0, s, A,
                     (uint8_t *)d_results);
  HIP_TRY(hipGetLastError());
  HIP_TRY(hipMemcpyAsync((uint8_t *)d_results + results_hist_offset(Lo),
                         (uint8_t *)d_workspace + Lo.off_hist,
                         4ull * (uint64_t)Lo.hist_stride * (uint64_t)Lo.R,
                         hipMemcpyDeviceToDevice, s));
  return WS_OK;
}

int wait_sim_run_batch(const ws_job *jobs, int32_t n_jobs, int64_t horizon,
                       void *d_workspace, size_t ws_bytes, void *d_results,
                       size_t results_bytes, void *hip_stream) {
  int rc = wait_sim_prepare(jobs, n_jobs, d_workspace, ws_bytes, hip_stream);
  if (rc != WS_OK) return rc;
  return wait_sim_advance(jobs, n_jobs, horizon, 0, d_workspace, ws_bytes, d_results,
                          results_bytes, hip_stream);
}

int wait_sim_run(const ws_config *cfg, const ws_policy *pol, const ws_stream *streams,
                 int32_t n_replicas, int64_t horizon, void *d_workspace, size_t ws_bytes,
                 void *d_results, size_t results_bytes, void *hip_stream) {
  ws_job jb;
  jb.cfg = cfg;
  jb.pol = pol;
  jb.streams = streams;
  jb.n = n_replicas;
  return wait_sim_run_batch(&jb, 1, horizon, d_workspace, ws_bytes, d_results, results_bytes,
                            hip_stream);
}

}  // extern "C"
