// sim_wait_many_impl.h -- simulation kernel for WAIT with more request types
// than the known-length kernel holds in registers (arXiv 2504.11320:
// Algorithm 1; the threshold-without-waiting form of the appendix; per-stage
// caps of Section 6).
//
// One lane per replica, the same model and ring layout as the known-length
// kernel (per type: an external queue ring of 8-byte records, the arrival
// time with the first-token flag in the sign bit, and a resident deque of
// 16-byte records in admission order), but every per-type scalar -- next
// arrival, queue and deque ends, services, resident memory, the first-token
// cohort count, the admission batch of the deque's back -- sits in an LDS
// column per lane, so up to 64 types cost no registers.  A batch visits the
// types in order: eligibility (the queue holds the type's threshold, or under
// no-wait any waiting or resident prompt), admissions, then the completion of
// every served type (its residents complete in admission order, at service
// admission + l'_j), and the LIFO repair picks the largest (admission batch,
// type) over the deque backs.
#pragma once

#include "sim_common.h"

namespace wsim {
namespace {

// MT: type slots; LN: replicas per wavefront (the LDS columns); TV: general
// instantiation (per-batch trace, arrival lists).
template <int MT, int LN, bool TV>
__global__ void __launch_bounds__(64) sim_wait_many_kernel(KArgs A) {
  __shared__ double s_edges[WS_MAX_HIST_EDGES + 1];
  __shared__ uint8_t s_htab[kHistTab];
  __shared__ int s_hsteps;
  __shared__ int32_t s_l[MT], s_lp[MT], s_n[MT], s_coff[MT];
  __shared__ double s_lam[MT];
  // per type and lane
  __shared__ double s_tn[MT][LN];
  __shared__ uint32_t s_k[MT][LN], s_qh[MT][LN], s_qt[MT][LN], s_dh[MT][LN], s_dt[MT][LN],
      s_svc[MT][LN], s_bkb[MT][LN];
  __shared__ int32_t s_pend[MT][LN], s_Mj[MT][LN];
  __shared__ uint8_t s_elig[MT][LN];
  __shared__ uint16_t s_fresh[MT][LN], s_pnew[MT][LN];

  const int tx = threadIdx.x;
  const int32_t r32 =
      tx < A.lanes && tx < LN ? ((const int32_t *)(A.ws + A.off_list))[(int64_t)blockIdx.x * 64 + tx]
                              : -1;
  const int64_t r = r32 < 0 ? 0 : r32;
  const uint32_t jix =
      __builtin_amdgcn_readfirstlane(((const uint32_t *)(A.ws + A.off_job_of))[r]);
  const JobDev &J = ((const JobDev *)(A.ws + A.off_jobs))[jix];
  const int m = J.m;
  const int n_hist = J.n_hist;
  {
    const double *edges_g = (const double *)(A.ws + J.off_edges);
    for (int b = tx; b <= n_hist; b += 64) s_edges[b] = b < n_hist ? edges_g[b] : INFINITY;
    if (tx == 0) {
      int32_t off = 0;
      for (int j = 0; j < MT; ++j) {
        const bool on = j < m;
        s_l[j] = on ? J.l[j] : 0;
        s_lp[j] = on ? J.lp[j] : 1;
        s_n[j] = on ? J.n[j] : 0;
        s_lam[j] = on ? J.lambda[j] : 0.0;
        s_coff[j] = off;  // first cap of type j in the per-stage cap table
        off += s_lp[j] + 1;
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
  const bool nowait = J.nowait != 0;
  const bool capped = J.has_caps != 0;
  const int32_t *capt = (const int32_t *)(A.ws + J.off_caps);
  const bool trace = J.n_trace > 0;
  const double *tr_time = (const double *)(A.ws + J.off_tr_time);
  const int32_t *tr_type = (const int32_t *)(A.ws + J.off_tr_type);
  const uint32_t qmask = (1u << J.qcap_log2) - 1u;
  const uint32_t rec_cap = (uint32_t)J.rec_cap;
  uint8_t *blk = A.ws + J.off_ring + (uint64_t)(r - J.replica_begin) * J.ring_stride;
  uint32_t *hist = (uint32_t *)(A.ws + A.off_hist) + r * (int64_t)A.hist_stride;
  auto qring = [&](int j) __attribute__((always_inline)) { return (double *)(blk + J.off_q[j]); };
  auto dring = [&](int j) __attribute__((always_inline)) { return (DRec *)(blk + J.off_d[j]); };
  auto dmask = [&](int j) __attribute__((always_inline)) { return (1u << J.dcap_log2[j]) - 1u; };
  // threshold of type j at its next service (per-stage caps: in turn)
  auto thr = [&](int j) __attribute__((always_inline)) -> int32_t {
    return capped ? capt[s_coff[j] + (int32_t)(s_svc[j][tx] % (uint32_t)(s_lp[j] + 1))]
                  : s_n[j];
  };

  double t, lat_area, ttft_area, lat_sum, mem_area, busy;
  int64_t batches, arrivals, comps, ctok, evicts, etok, btok, peak, idle, tridx, Mres;
  int32_t N, U;
  uint32_t flags;
  if (!A.resume) {
    t = lat_area = ttft_area = lat_sum = mem_area = busy = 0.0;
    batches = arrivals = comps = ctok = evicts = etok = btok = peak = idle = tridx = Mres = 0;
    N = U = 0;
    flags = 0;
    for (int j = 0; j < MT; ++j) {
      s_tn[j][tx] = j < m && !trace
                        ? 0.0 + draw_gap(seed, rid, (uint32_t)j, 0u, s_lam[j], nullptr, 0, nullptr)
                        : INFINITY;
      s_k[j][tx] = s_qh[j][tx] = s_qt[j][tx] = s_dh[j][tx] = s_dt[j][tx] = s_svc[j][tx] = 0;
      s_pend[j][tx] = s_Mj[j][tx] = 0;
      s_bkb[j][tx] = 0;
    }
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
    flags = (uint32_t)slot_i(A, S_FLAGS, r);
    for (int j = 0; j < MT; ++j) {
      s_tn[j][tx] = slot_f(A, S_TNEXT + j, r);
      s_k[j][tx] = (uint32_t)slot_i(A, S_K + j, r);
      s_qh[j][tx] = (uint32_t)slot_i(A, S_QH + j, r);
      s_qt[j][tx] = (uint32_t)slot_i(A, S_QT + j, r);
      s_dh[j][tx] = (uint32_t)slot_i(A, S_DH + j, r);
      s_dt[j][tx] = (uint32_t)slot_i(A, S_DT + j, r);
      s_svc[j][tx] = (uint32_t)slot_i(A, S_SVC + j, r);
      s_Mj[j][tx] = (int32_t)slot_i(A, S_MJ + j, r);
      s_pend[j][tx] = (int32_t)slot_i(A, S_LNEXT + j, r);
      const uint32_t dt = s_dt[j][tx];
      s_bkb[j][tx] = j < m && dt != s_dh[j][tx] ? dring(j)[(dt - 1u) & dmask(j)].kb : 0u;
    }
  }

  // ---- arrivals ---------------------------------------------------------------
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
  // Append to queue j (a full queue ends the replica at its next decision).
  auto push_q = [&](int j, double a_ft) __attribute__((always_inline)) {
    const uint32_t h = s_qh[j][tx], tq = s_qt[j][tx];
    if (tq - h >= rec_cap)
      flags |= kFlagCap;
    else
      qring(j)[tq & qmask] = a_ft;
    s_qt[j][tx] = tq + 1u;
  };
  auto take = [&](int jn, double a) __attribute__((always_inline)) {
    if (trace) {
      tridx++;
    } else {
      const uint32_t k = s_k[jn][tx] + 1u;
      const double g = draw_gap(seed, rid, (uint32_t)jn, k, s_lam[jn], nullptr, 0, nullptr);
      s_k[jn][tx] = k;
      s_tn[jn][tx] = s_tn[jn][tx] + g;
      next_arrival();
    }
    arrivals++;
    N++;
    U++;
    push_q(jn, a);
  };

  bool stopped = (flags & (kFlagCap | kFlagStall)) != 0;
  if (!trace) next_arrival();

  for (int64_t it = 0; it < A.horizon && !stopped; ++it) {
    // ---- decision: the eligible types, or wait for the next arrival --------
    bool any = false;
    for (;;) {
      if (flags & kFlagCap) {
        stopped = true;
        break;
      }
      any = false;
      for (int j = 0; j < m; ++j) {
        const uint32_t waiting = s_qt[j][tx] - s_qh[j][tx];
        const bool e = nowait ? (waiting != 0u || s_dt[j][tx] != s_dh[j][tx])
                              : waiting >= (uint32_t)thr(j);
        s_elig[j][tx] = e ? 1 : 0;
        any = any || e;
      }
      if (any) break;
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

    // ---- launch: admissions of the eligible types, in type order ------------
    const uint32_t bidx = (uint32_t)batches;
    int64_t tokens = 0, prefill_l = 0, bt_pre = 0, bt_sel = 0;
    for (int j = 0; j < m; ++j) {
      s_fresh[j][tx] = 0;
      s_pnew[j][tx] = 0;
      if (!s_elig[j][tx]) continue;
      const uint32_t c = s_svc[j][tx] + 1u;
      const uint32_t waiting = s_qt[j][tx] - s_qh[j][tx];
      const int32_t na = nowait ? (waiting < (uint32_t)s_n[j] ? (int32_t)waiting : s_n[j]) : thr(j);
      uint32_t qh = s_qh[j][tx], dt = s_dt[j][tx];
      const uint32_t dm = dmask(j);
      int32_t pn = 0;
      for (int32_t x = 0; x < na; ++x) {
        const double a_ft = qring(j)[qh & qmask];
        qh++;
        DRec rec;
        rec.a_ft = a_ft;
        rec.kb = bidx;
        rec.kc = c;
        dring(j)[dt & dm] = rec;
        dt++;
        pn += has_ft(a_ft) ? 0 : 1;
      }
      s_qh[j][tx] = qh;
      s_dt[j][tx] = dt;
      if (na > 0) s_bkb[j][tx] = bidx;
      s_fresh[j][tx] = (uint16_t)na;
      s_pnew[j][tx] = (uint16_t)pn;
      bt_pre += na;
      bt_sel += (int64_t)(dt - s_dh[j][tx]);
      tokens += (int64_t)na * s_l[j] + s_Mj[j][tx];
      prefill_l += (int64_t)na * s_l[j];
    }
    const int64_t m_launch = Mres + prefill_l;
    if (m_launch > peak) peak = m_launch;
    const double tau = d0 + d1 * (double)tokens;
    const double t_end = t + tau;
    const int32_t N0 = N, U0 = U;

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

    // ---- completion transition, type by type -----------------------------------
    const int64_t bt_comps0 = comps;
    Mres = 0;
    for (int j = 0; j < m; ++j) {
      if (s_elig[j][tx]) {
        // the stage-1 cohort produces its first tokens
        U -= s_pend[j][tx];
        s_pend[j][tx] = s_pnew[j][tx];
        const uint32_t now = s_svc[j][tx] + 1u;
        s_svc[j][tx] = now;
        const uint32_t fresh = s_fresh[j][tx];
        uint32_t dh = s_dh[j][tx];
        const uint32_t before = (s_dt[j][tx] - dh) - fresh;
        const uint32_t dm = dmask(j);
        const int32_t lpj = s_lp[j];
        uint32_t done = 0;
        while (done < before) {
          const DRec f = dring(j)[dh & dm];
          if (f.kc + (uint32_t)lpj != now) break;
          const double lat = t_end - arrival_of(f.a_ft);
          lat_sum += lat;
          __hip_atomic_fetch_add(&hist[hist_bin_idx(s_edges, s_htab, hidx, lat)], 1u,
                                 __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          comps++;
          ctok += lpj;
          N--;
          dh++;
          done++;
        }
        s_dh[j][tx] = dh;
        s_Mj[j][tx] += (int32_t)(before - done) + (int32_t)fresh * (s_l[j] + 1) -
                       (int32_t)done * (s_l[j] + lpj);
      }
      Mres += s_Mj[j][tx];
    }
    if (Mres > peak) peak = Mres;

    // ---- repair: evict the most recently admitted resident -------------------
    const int64_t bt_ev0 = evicts;
    while (Mres > C) {
      int jb = -1;
      uint32_t bb = 0;
      for (int j = 0; j < m; ++j) {  // largest (admission batch, type)
        if (s_dt[j][tx] == s_dh[j][tx]) continue;
        const uint32_t kb = s_bkb[j][tx];
        if (jb < 0 || kb >= bb) {
          jb = j;
          bb = kb;
        }
      }
      if (jb < 0) break;
      const uint32_t dm = dmask(jb);
      const uint32_t tq = s_dt[jb][tx] - 1u;
      const DRec rec = dring(jb)[tq & dm];
      s_dt[jb][tx] = tq;
      if (tq != s_dh[jb][tx]) s_bkb[jb][tx] = dring(jb)[(tq - 1u) & dm].kb;
      const int32_t stage = (int32_t)(s_svc[jb][tx] - rec.kc) + 1;
      const int32_t ch = s_l[jb] + stage;
      s_Mj[jb][tx] -= ch;
      Mres -= ch;
      evicts++;
      etok += stage - 1;
      const bool ft = has_ft(rec.a_ft);
      s_pend[jb][tx] -= (stage == 1 && !ft) ? 1 : 0;
      push_q(jb, (ft || stage >= 2) ? with_ft(rec.a_ft) : rec.a_ft);
    }
    if constexpr (TV) {
      if (A.btrace != nullptr && batches < A.btrace_cap) {
        BatchRec br;
        br.t_launch = t_end - tau;
        br.tau = tau;
        br.tokens = tokens;
        br.prefills = bt_pre;
        br.selected = bt_sel;
        br.completions = comps - bt_comps0;
        br.evict_pre = 0;
        br.evict_post = evicts - bt_ev0;
        br.mem_after = Mres;
        int64_t w = 0, res = 0;
        for (int j = 0; j < m; ++j) {
          w += s_qt[j][tx] - s_qh[j][tx];
          res += s_dt[j][tx] - s_dh[j][tx];
        }
        br.waiting_after = w;
        br.resident_after = res;
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
  put_i(A, S_FLAGS, r, (int64_t)flags);
  put_i(A, S_PARTJ, r, -1);
  for (int j = 0; j < MT; ++j) {
    put_f(A, S_TNEXT + j, r, s_tn[j][tx]);
    put_i(A, S_K + j, r, s_k[j][tx]);
    put_i(A, S_QH + j, r, s_qh[j][tx]);
    put_i(A, S_QT + j, r, s_qt[j][tx]);
    put_i(A, S_DH + j, r, s_dh[j][tx]);
    put_i(A, S_DT + j, r, s_dt[j][tx]);
    put_i(A, S_SVC + j, r, s_svc[j][tx]);
    put_i(A, S_MJ + j, r, s_Mj[j][tx]);
    put_i(A, S_LNEXT + j, r, s_pend[j][tx]);
  }
}

// Replicas per wavefront of this kernel (its LDS columns).
constexpr int kWaitManyLanes = 16;

template <bool TV>
hipError_t launch_wait_many_k(int max_m, const KArgs &A, hipStream_t s) {
  if (A.n_list % 64 != 0 || A.lanes > kWaitManyLanes) return hipErrorInvalidValue;
  if (max_m <= 32)
    return launch_checked(sim_wait_many_kernel<32, kWaitManyLanes, TV>, dim3(A.n_list / 64), s, A);
  if (max_m <= 64)
    return launch_checked(sim_wait_many_kernel<64, kWaitManyLanes, TV>, dim3(A.n_list / 64), s, A);
  return hipErrorInvalidValue;  // the host admits at most WS_MAX_TYPES types
}

}  // namespace
}  // namespace wsim
