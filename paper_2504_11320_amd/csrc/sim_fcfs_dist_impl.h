// sim_fcfs_dist_impl.h -- simulation kernel for FCFS when output lengths are
// unknown to the scheduler (arXiv 2504.11320: Section 4.1's FCFS with LIFO
// eviction on overflow; the unknown-length model of Section 5.1, each
// request's length drawn once at arrival from its type's distribution).  It
// also runs FCFS with known lengths l'_j for more types than the
// known-length kernels hold: the structure below takes any per-request
// length.
//
// One lane per replica.  FCFS batches every resident every iteration, so a
// prompt admitted (prefilled) at batch kb with output length L completes at
// batch kb + L: the exit is known at admission, although the policy never
// reads it.  Residents of one type no longer complete in admission order, so
// instead of per-type deques each replica keeps, in its block of the
// workspace:
//   - the external FIFO queue (16-byte records: arrival time with the
//     first-token flag in the sign bit, type word, length);
//   - a ring of resident records in admission order (32 bytes), with a
//     parallel array of exit batches (bit 31: evicted);
//   - a calendar of W >= out_cap + 1 buckets (exit batch mod W), each the head
//     of a list of the records that exit at that batch, linked through the
//     records.  A batch's admissions are linked in reverse admission order,
//     so a bucket is traversed newest batch first and in admission order
//     within a batch: by (stage, admission key), the order in which the
//     model's transition meets the completing prompts (their stage is their
//     own length).
// LIFO repair evicts the newest live entry of the ring (found from the back,
// skipping entries that completed or were evicted); an evicted record stays
// in its bucket as a hole (length 0) until its exit batch, and the ring's
// front releases an entry only after its exit batch, so no slot a calendar
// list still reaches is reused.
#pragma once

#include "sim_common.h"

namespace wsim {
namespace {

constexpr uint32_t kEvicted = 0x80000000u;  // exit-array flag

__device__ __forceinline__ NRec load_rec32(const NRec *p) {
  const uint4 lo = ((const uint4 *)p)[0], hi = ((const uint4 *)p)[1];
  NRec r;
  r.a_ft = __longlong_as_double((long long)(((uint64_t)lo.y << 32) | lo.x));
  r.kb = lo.z;
  r.kp = lo.w;
  r.j = (int32_t)hi.x;
  r.L = (int32_t)hi.y;
  r.c = hi.z;
  r.next = hi.w;
  return r;
}

// MT: type slots (>= m); TV: general instantiation (per-batch trace).
template <int MT, bool TV>
__global__ void __launch_bounds__(64) sim_fcfs_dist_kernel(KArgs A) {
  __shared__ double s_edges[WS_MAX_HIST_EDGES + 1];
  __shared__ uint8_t s_htab[kHistTab];
  __shared__ int s_hsteps;
  __shared__ uint16_t s_cdfg[MT][kCdfGuide + 1];
  // per type and lane: the pending arrival's time, index and length
  __shared__ double s_tn[MT][64];
  __shared__ uint32_t s_k[MT][64];
  __shared__ int32_t s_len[MT][64];
  __shared__ int32_t s_l[MT], s_lp[MT];
  __shared__ double s_lam[MT];

  const int tx = threadIdx.x;
  const int32_t r32 =
      tx < A.lanes ? ((const int32_t *)(A.ws + A.off_list))[(int64_t)blockIdx.x * 64 + tx] : -1;
  const int64_t r = r32 < 0 ? 0 : r32;
  // every replica of a wavefront belongs to the same job
  const uint32_t jix =
      __builtin_amdgcn_readfirstlane(((const uint32_t *)(A.ws + A.off_job_of))[r]);
  const JobDev &J = ((const JobDev *)(A.ws + A.off_jobs))[jix];
  const int m = J.m;
  const int n_hist = J.n_hist;
  const int32_t cap = J.out_cap;
  const bool known = J.known != 0;  // lengths l'_j of the type
  const uint32_t *cdf = (const uint32_t *)(A.ws + J.off_cdf);
  const bool use_guide = !known && J.n_trace == 0 && cap > 1 && cap <= 65535;
  {
    const double *edges_g = (const double *)(A.ws + J.off_edges);
    for (int b = tx; b <= n_hist; b += 64) s_edges[b] = b < n_hist ? edges_g[b] : INFINITY;
    for (int j = tx; j < MT; j += 64) {
      s_l[j] = j < m ? J.l[j] : 0;
      s_lp[j] = j < m ? J.lp[j] : 1;
      s_lam[j] = j < m ? J.lambda[j] : 0.0;
    }
    if (use_guide) {
      for (int x = tx; x < MT * (kCdfGuide + 1); x += 64) {
        const int j = x / (kCdfGuide + 1), b = x % (kCdfGuide + 1);
        s_cdfg[j][b] = j < m ? (uint16_t)cdf_guide_entry(cdf + (size_t)j * (size_t)(cap - 1), cap, b)
                             : (uint16_t)0;
      }
    }
    __syncthreads();
  }
  const HistIdx hidx = hist_index_build(s_edges, n_hist, s_htab, &s_hsteps);
  if (r32 < 0) return;  // padding lane
  const uint64_t seed = ((const uint64_t *)(A.ws + A.off_seed))[r];
  const uint32_t rid = ((const uint32_t *)(A.ws + A.off_rid))[r];

  const double d0 = J.d0, d1 = J.d1;
  const int64_t C = J.C;
  const int64_t cap_adm = J.C - J.reserve_tok;
  const bool trace = J.n_trace > 0;
  const double *tr_time = (const double *)(A.ws + J.off_tr_time);
  const int32_t *tr_type = (const int32_t *)(A.ws + J.off_tr_type);
  const int32_t *tr_len = (const int32_t *)(A.ws + J.off_tr_len);
  const uint32_t qmask = (1u << J.qcap_log2) - 1u;
  const uint32_t rec_cap = (uint32_t)J.rec_cap;
  const uint32_t wmask = (1u << J.cal_log2) - 1u;
  uint8_t *blk = A.ws + J.off_ring + (uint64_t)(r - J.replica_begin) * J.ring_stride;
  QRec *q10 = (QRec *)(blk + J.off_q[0]);
  NRec *res = (NRec *)(blk + J.off_res);
  uint32_t *ex = (uint32_t *)(blk + J.off_exit);
  uint32_t *cal = (uint32_t *)(blk + J.off_cal);
  uint32_t *hist = (uint32_t *)(A.ws + A.off_hist) + r * (int64_t)A.hist_stride;
  auto row_of = [&](int j) __attribute__((always_inline)) -> const uint32_t * {
    return known || cap <= 1 ? nullptr : cdf + (size_t)j * (size_t)(cap - 1);
  };
  auto guide_of = [&](int j) __attribute__((always_inline)) -> const uint16_t * {
    return use_guide ? s_cdfg[j] : nullptr;
  };

  double t, lat_area, ttft_area, lat_sum, mem_area, busy;
  int64_t batches, arrivals, comps, ctok, evicts, etok, btok, peak, idle, tridx, Mres;
  int32_t N, U, pendft;  // in the system; without a first token; stage-1 cohort
  uint32_t flags, qh, qt, rh, rt, I;  // queue and resident-ring ends; live residents
  if (!A.resume) {
    t = lat_area = ttft_area = lat_sum = mem_area = busy = 0.0;
    batches = arrivals = comps = ctok = evicts = etok = btok = peak = idle = tridx = Mres = 0;
    N = U = pendft = 0;
    flags = qh = qt = rh = rt = I = 0;
    for (int j = 0; j < MT; ++j) {
      double tn = INFINITY;
      int32_t Lj = 1;
      if (j < m && !trace) tn = 0.0 + draw_gap(seed, rid, (uint32_t)j, 0u, s_lam[j], row_of(j), cap,
                                               &Lj, nullptr, guide_of(j));
      s_tn[j][tx] = tn;
      s_k[j][tx] = 0;
      s_len[j][tx] = known ? s_lp[j] : (cap <= 1 ? 1 : Lj);
    }
    for (uint32_t b = 0; b <= wmask; ++b) cal[b] = kNil;
    for (int b = 0; b < A.hist_stride; ++b) hist[b] = 0;  // whole row, padding included
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
    tridx = slot_i(A, S_TRIDX, r);
    Mres = slot_i(A, S_MRES, r);
    N = (int32_t)slot_i(A, S_N, r);
    U = (int32_t)slot_i(A, S_U, r);
    pendft = (int32_t)slot_i(A, S_PENDFT, r);
    flags = (uint32_t)slot_i(A, S_FLAGS, r);
    qh = (uint32_t)slot_i(A, S_QH, r);
    qt = (uint32_t)slot_i(A, S_QT, r);
    rh = (uint32_t)slot_i(A, S_DH, r);
    rt = (uint32_t)slot_i(A, S_DT, r);
    I = (uint32_t)slot_i(A, S_KI, r);
    for (int j = 0; j < MT; ++j) {
      s_tn[j][tx] = slot_f(A, S_TNEXT + j, r);
      s_k[j][tx] = (uint32_t)slot_i(A, S_K + j, r);
      s_len[j][tx] = (int32_t)slot_i(A, S_LNEXT + j, r);
    }
  }

  // ---- arrivals ---------------------------------------------------------------
  // The next arrival (ties: the lowest type), kept up to date by take().
  double tmin = INFINITY;
  int jmin = 0;
  auto next_arrival = [&]() __attribute__((always_inline)) {
    tmin = INFINITY;
    jmin = 0;
    for (int j = 0; j < m; ++j) {
      const double v = s_tn[j][tx];
      if (v < tmin) {
        tmin = v;
        jmin = j;
      }
    }
  };
  auto peek = [&](int &jn) __attribute__((always_inline)) -> double {
    if (trace) {
      if (tridx >= J.n_trace) {
        jn = 0;
        return INFINITY;
      }
      jn = tr_type[tridx];
      return tr_time[tridx];
    }
    jn = jmin;
    return tmin;
  };
  // Append to the external queue (a full queue ends the replica at its next
  // decision; the record is then not written).
  auto push_q = [&](double a_ft, int32_t jw, int32_t L) __attribute__((always_inline)) {
    if (qt - qh >= rec_cap) {
      flags |= kFlagCap;
    } else {
      QRec rec;
      rec.a_ft = a_ft;
      rec.j = jw;
      rec.L = L;
      q10[qt & qmask] = rec;
    }
    qt++;
  };
  auto take = [&](int jn, double a) __attribute__((always_inline)) {
    int32_t Lr;
    if (trace) {
      Lr = known ? s_lp[jn] : tr_len[tridx];
      tridx++;
    } else {
      Lr = s_len[jn][tx];
      const uint32_t k = s_k[jn][tx] + 1u;
      int32_t Lj = 1;
      const double g = draw_gap(seed, rid, (uint32_t)jn, k, s_lam[jn], row_of(jn), cap, &Lj,
                                nullptr, guide_of(jn));
      s_k[jn][tx] = k;
      s_tn[jn][tx] = s_tn[jn][tx] + g;
      s_len[jn][tx] = known ? s_lp[jn] : (cap <= 1 ? 1 : Lj);
      next_arrival();
    }
    arrivals++;
    N++;
    U++;
    push_q(a, (s_l[jn] << 8) | jn, Lr);
  };

  bool stopped = (flags & (kFlagCap | kFlagStall)) != 0;
  if (!trace) next_arrival();

  for (int64_t it = 0; it < A.horizon && !stopped; ++it) {
    // ---- decision: batch every resident, admit from the queue head ---------
    for (;;) {
      // exit batches are kept below 2^31 (bit 31 of the exit array marks
      // evicted entries)
      if (batches >= (int64_t(1) << 31) - (int64_t(1) << 24)) flags |= kFlagCap;
      if (flags & kFlagCap) {
        stopped = true;
        break;
      }
      if (I > 0 || qt != qh) break;
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
      for (;;) {  // every arrival at this instant joins before the next decision
        if (flags & kFlagCap) break;
        int j2;
        const double a2 = peek(j2);
        if (a2 != ta) break;
        take(j2, a2);
      }
      idle++;
    }
    if (stopped) break;

    // ---- launch: head-of-line admissions while the launch memory fits -------
    const uint32_t bidx = (uint32_t)batches;
    int64_t prefill_l = 0;
    uint32_t nadm = 0;
    while (qh + nadm != qt) {
      if (rt - rh + nadm >= rec_cap) {  // the resident ring is full: the replica
        flags |= kFlagCap;              // stops at its next decision
        break;
      }
      const QRec head = q10[(qh + nadm) & qmask];
      const int64_t hl = head.j >> 8;
      if (Mres + prefill_l + hl > cap_adm) break;
      prefill_l += hl;
      nadm++;
    }
    const int64_t tokens = Mres + prefill_l;  // residents at stage s cost l + s
    const int64_t m_launch = Mres + prefill_l;
    if (m_launch > peak) peak = m_launch;
    const double tau = d0 + d1 * (double)tokens;
    const double t_end = t + tau;
    const int32_t N0 = N, U0 = U;
    const uint32_t I0 = I;

    // ---- admissions into the resident ring and the calendar -----------------
    // linked in reverse admission order (traversal: admission order)
    int32_t pend_new = 0;
    for (int32_t i = (int32_t)nadm - 1; i >= 0; --i) {
      const QRec qr = q10[(qh + (uint32_t)i) & qmask];
      const uint32_t idx = rt + (uint32_t)i;
      const uint32_t exit = bidx + (uint32_t)qr.L;
      NRec e;
      e.a_ft = qr.a_ft;
      e.kb = bidx;
      e.kp = (uint32_t)i;
      e.j = qr.j;
      e.L = qr.L;
      e.c = 0u;
      e.next = cal[exit & wmask];
      res[idx & qmask] = e;
      ex[idx & qmask] = exit;
      cal[exit & wmask] = idx;
      pend_new += has_ft(qr.a_ft) ? 0 : 1;
    }
    qh += nadm;
    rt += nadm;

    // ---- arrivals during the batch -------------------------------------------
    for (;;) {
      if (flags & kFlagCap) break;
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

    // ---- completion transition ------------------------------------------------
    // the stage-1 cohort produces its first tokens
    U -= pendft;
    pendft = pend_new;
    const int64_t bt_comps0 = comps;
    uint32_t node = cal[bidx & wmask];
    cal[bidx & wmask] = kNil;
    uint32_t nc = 0, steps = 0;
    int64_t freed = 0;
    while (node != kNil) {
      if (++steps > rec_cap) {  // a list longer than the ring: a corrupted link
        flags |= kFlagCap;
        break;
      }
      const NRec rec = load_rec32(res + (node & qmask));
      if (rec.L != 0) {  // holes left by evictions are skipped
        const double lat = t_end - arrival_of(rec.a_ft);
        lat_sum += lat;
        __hip_atomic_fetch_add(&hist[hist_bin_idx(s_edges, s_htab, hidx, lat)], 1u,
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        comps++;
        ctok += rec.L;
        N--;
        nc++;
        freed += (int64_t)(rec.j >> 8) + rec.L;
      }
      node = rec.next;
    }
    // residents advance one stage, completions leave, admissions hold l + 1
    Mres += (int64_t)(I0 - nc) - freed + prefill_l + (int64_t)nadm;
    I = I0 - nc + nadm;
    if (Mres > peak) peak = Mres;
    // release ring entries whose calendar entry has been consumed
    while (rh != rt && (int32_t)((ex[rh & qmask] & ~kEvicted) - bidx) <= 0) rh++;

    // ---- repair: evict the most recently admitted resident ------------------
    const int64_t bt_ev0 = evicts;
    uint32_t scan = rt;  // entries at or above scan hold no live resident
    while (Mres > C && I > 0) {
      uint32_t v = scan;
      while (v != rh) {
        const uint32_t e = ex[(v - 1u) & qmask];
        if ((e & kEvicted) == 0 && (int32_t)(e - bidx) > 0) break;  // live
        v--;
      }
      if (v == rh) break;  // none live (I counts them: cannot happen)
      const uint32_t idx = v - 1u;
      scan = idx;
      NRec rec = load_rec32(res + (idx & qmask));
      const int32_t stage = (int32_t)(bidx - rec.kb) + 1;
      const int64_t ch = (int64_t)(rec.j >> 8) + stage;
      Mres -= ch;
      I--;
      evicts++;
      etok += stage - 1;
      const bool ft = has_ft(rec.a_ft);
      pendft -= (stage == 1 && !ft) ? 1 : 0;
      ex[idx & qmask] = ex[idx & qmask] | kEvicted;
      res[idx & qmask].L = 0;  // a hole in its calendar list
      push_q((ft || stage >= 2) ? with_ft(rec.a_ft) : rec.a_ft, rec.j, rec.L);
    }
    if constexpr (TV) {
      if (A.btrace != nullptr && batches < A.btrace_cap) {
        BatchRec br;
        br.t_launch = t_end - tau;
        br.tau = tau;
        br.tokens = tokens;
        br.prefills = nadm;
        br.selected = (int64_t)I0 + nadm;
        br.completions = comps - bt_comps0;
        br.evict_pre = 0;
        br.evict_post = evicts - bt_ev0;
        br.mem_after = Mres;
        br.waiting_after = qt - qh;
        br.resident_after = I;
        br.mplus = 0;
        ((BatchRec *)A.btrace)[r * A.btrace_cap + batches] = br;
      }
    }
    batches++;
    btok += tokens;
  }

  // ---- save state ------------------------------------------------------------
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
  put_i(A, S_PENDFT, r, pendft);
  put_i(A, S_FLAGS, r, (int64_t)flags);
  put_i(A, S_QH, r, qh);
  put_i(A, S_QT, r, qt);
  put_i(A, S_DH, r, rh);
  put_i(A, S_DT, r, rt);
  put_i(A, S_KI, r, I);
  put_i(A, S_PARTJ, r, -1);
  for (int j = 0; j < MT; ++j) {
    put_f(A, S_TNEXT + j, r, s_tn[j][tx]);
    put_i(A, S_K + j, r, s_k[j][tx]);
    put_i(A, S_LNEXT + j, r, s_len[j][tx]);
  }
}

template <int MT, bool TV>
hipError_t launch_fd(const KArgs &A, hipStream_t s) {
  return launch_checked(sim_fcfs_dist_kernel<MT, TV>, dim3(A.n_list / 64), s, A);
}

template <bool TV>
hipError_t launch_fcfs_dist_k(int max_m, const KArgs &A, hipStream_t s) {
  if (A.n_list % 64 != 0) return hipErrorInvalidValue;
  if (max_m <= 4) return launch_fd<4, TV>(A, s);
  if (max_m <= 16) return launch_fd<16, TV>(A, s);
  if (max_m <= 64) return launch_fd<64, TV>(A, s);
  return hipErrorInvalidValue;  // the host admits at most WS_MAX_TYPES types
}

}  // namespace
}  // namespace wsim
