// sim_known.hip -- simulation kernel for WAIT and FCFS with known output
// lengths (arXiv 2504.11320: Algorithm 1, Section 4.1).
//
// One lane per replica.  A replica's state is a handful of scalars (clock,
// per-type next arrival, counters, areas) held in registers, plus ring
// buffers of request records in HBM: external queues (WAIT: one per type,
// FCFS: one shared FIFO) and one resident deque per type in admission order.
// Under WAIT a served type advances every resident prompt of that type (each
// stage holds at most n_j prompts, so min(n_j, n_js) = n_js, as in the
// resident-memory lemma of the Theorem 1 proof); under FCFS every resident is
// batched every iteration.  In both cases a prompt's stage is the number of
// services of its type since admission and the residents of one type complete
// in admission order, so a per-type deque replaces the (type, stage) count
// matrix: admissions push at the back, completions pop at the front, LIFO
// evictions pop at the back, and each step costs O(events), not O(stages).
//
// Arithmetic follows the model contract exactly (same IEEE operations in the
// same order, no FMA contraction), so integer state is bit-identical to the
// oracle's and floating sums agree to rounding.
#include "sim_common.h"

namespace wsim {
namespace {

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

template <int MT, int POL>
hipError_t launch_mt(const KArgs &A, hipStream_t s) {
  const int threads = 64;
  const int blocks = (A.n_list + threads - 1) / threads;
  hipLaunchKernelGGL((sim_known_kernel<MT, POL>), dim3(blocks), dim3(threads), 0, s, A);
  return hipGetLastError();
}

template <int POL>
hipError_t launch_pol(int max_m, const KArgs &A, hipStream_t s) {
  if (max_m <= 2) return launch_mt<2, POL>(A, s);
  if (max_m <= 3) return launch_mt<3, POL>(A, s);
  if (max_m <= 4) return launch_mt<4, POL>(A, s);
  if (max_m <= 8) return launch_mt<8, POL>(A, s);
  return launch_mt<16, POL>(A, s);
}

}  // namespace

hipError_t launch_known(int policy, int max_m, const KArgs &A, hipStream_t s) {
  if (policy == WS_WAIT) return launch_pol<WS_WAIT>(max_m, A, s);
  return launch_pol<WS_FCFS>(max_m, A, s);
}

}  // namespace wsim
