// sim_nested_impl.h -- simulation kernel for Nested WAIT (arXiv 2504.11320:
// Algorithm 2, Section 5.1; event-driven form Algorithm 4, Appendix B.1;
// coarse segments with heterogeneous prompts, Appendix A).
//
// One lane per replica.  Per-type arrival state and per-segment counters
// live in the lane's own column of LDS; request records live in HBM:
//   - the external queue Q_{1,0} (FIFO ring);
//   - for segment k >= 2 the resident boundary queue (a ring kept in
//     admission-key order, so FIFO selection pops the front and LIFO eviction
//     pops the back);
//   - for every segment a ring of cohort slots indexed by the segment's
//     service number modulo delta_k (its number of processing stages).  All
//     prompts that entered the segment at one service form one cohort of at
//     most n_k prompts and share a stage, so each stage holds one cohort (the
//     stage-cap invariant of the Nested WAIT analysis) and every interior
//     prompt of a served segment is selected.
// A prompt's exit from its segment (completion at its own output length, or
// survival to the next boundary queue at r_k) happens at a known service, so
// each segment keeps a calendar: bucket (service mod delta_k) heads a linked
// list of the prompts that exit at that service.  Cohorts are linked in
// reverse admission order, so a bucket is traversed youngest cohort first and
// in admission order within a cohort: the same (stage, key) order as the
// oracle's selection list, which fixes the order of floating-point sums and
// of survivors joining the next boundary queue.
//
// The projected state Q+ of the pre-launch repair (apply the selected moves
// with no early completion) is computed from per-segment counts and the
// prompts still live in the terminal cohort slot (a record with L = 0 has left
// its segment).
#pragma once

#include "sim_common.h"

namespace wsim {
namespace {

// Per-segment constants, staged in LDS: a segment index is often
// lane-dependent (it starts at a lane's own prefix length), and LDS serves
// such reads without a round trip to the job table in memory.
struct SegConst {
  uint64_t dmagic;  // fastmod multiplier for delta
  int32_t end;      // r_k
  int32_t n;        // n_k
  int32_t delta;    // processing stages (cohort slots)
  int32_t entry;    // processing stage of an entering prompt
  uint32_t vmask;   // boundary-queue ring mask (k >= 1)
  uint32_t off_rec; // ring offsets inside a replica block
  uint32_t off_bkt;
  uint32_t off_v;
};

__device__ __forceinline__ NRec nrec_of(uint4 a, uint4 b) {
  NRec r;
  r.a_ft = __longlong_as_double((long long)(((uint64_t)a.y << 32) | a.x));
  r.kb = a.z;
  r.kp = a.w;
  r.j = (int32_t)b.x;
  r.L = (int32_t)b.y;
  r.c = b.z;
  r.next = b.w;
  return r;
}
__device__ __forceinline__ uint4 nrec_lo(const NRec &r) {
  const uint64_t u = (uint64_t)__double_as_longlong(r.a_ft);
  return make_uint4((uint32_t)u, (uint32_t)(u >> 32), r.kb, r.kp);
}
__device__ __forceinline__ uint4 nrec_hi(const NRec &r) {
  return make_uint4((uint32_t)r.j, (uint32_t)r.L, r.c, r.next);
}
__device__ __forceinline__ QRec qrec_of(uint4 a) {
  QRec q;
  q.a_ft = __longlong_as_double((long long)(((uint64_t)a.y << 32) | a.x));
  q.j = (int32_t)a.z;
  q.L = (int32_t)a.w;
  return q;
}
__device__ __forceinline__ uint4 qrec_u4(const QRec &q) {
  const uint64_t u = (uint64_t)__double_as_longlong(q.a_ft);
  return make_uint4((uint32_t)u, (uint32_t)(u >> 32), (uint32_t)q.j, (uint32_t)q.L);
}
// Asynchronous copy of 4 or 16 bytes per lane from HBM into LDS: lane t
// writes lds_base + t * size, so lds_base is the start of a per-lane array
// (and must be the same for all lanes).
__device__ __forceinline__ void copy4_to_lds(const void *src, void *lds_base) {
  __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void *)lds_base, 4, 0,
                                   0);
}
__device__ __forceinline__ void copy16_to_lds(const void *src, void *lds_base) {
  __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void *)lds_base, 16, 0,
                                   0);
}
__device__ __forceinline__ uint4 opaque4(uint4 v) {
  v.x = opaque(v.x);
  v.y = opaque(v.y);
  v.z = opaque(v.z);
  v.w = opaque(v.w);
  return v;
}
// Wait for every outstanding memory operation of the wavefront (including the
// asynchronous copies); also a compiler barrier for memory accesses.
__device__ __forceinline__ void wait_memory() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// MT: type slots (>= m); LT: segment slots (>= L); LN: replicas per
// wavefront (lanes LN..63 are padding), which sizes the per-lane LDS columns;
// TV: jobs with time-varying rates are supported (compiled out of the common
// kernels).
template <int MT, int LT, int LN, bool TV>
__global__ void __launch_bounds__(64) sim_nested_kernel(KArgs A) {
  // Inter-arrival gaps and output lengths are drawn ahead of use by the
  // whole wavefront at once into a ring of GR draws per type and lane; a
  // lane whose ring runs dry draws for itself.
  constexpr int GR = 4;
  constexpr int GU = GR / 2;         // draws added per refill
  constexpr uint32_t kLow = GU / 2;  // a lane below this triggers a refill
  __shared__ double s_tnext[MT][LN];
  __shared__ uint32_t s_k[MT][LN], s_gend[MT][LN];
  __shared__ int32_t s_Ln[MT][LN];
  // With time-varying rates the rings hold candidates of the thinning bound
  // process with their fourth Philox words (the acceptance draws), and the
  // rate profile sits in LDS beside them.
  __shared__ double s_gap[MT][GR][LN];
  __shared__ int32_t s_glen[MT][GR][LN];
  constexpr int NP = TV ? kMaxRatePts : 1;
  __shared__ uint32_t s_w3[TV ? MT : 1][TV ? GR : 1][TV ? LN : 1];
  __shared__ RateProfLds<MT, NP> s_prof;
  __shared__ int8_t s_cur[TV ? MT : 1][TV ? LN : 1];  // profile piece per type
  double(&s_rt)[NP] = s_prof.t;
  double(&s_rf)[MT][NP] = s_prof.f;
  double(&s_fmax)[MT] = s_prof.fmax;
  __shared__ uint64_t s_seed[LN];
  __shared__ uint32_t s_rid[LN];
  // refill requests of one pass, all types together: lane, type, first draw
  __shared__ uint8_t s_req_lane[MT * LN], s_req_j[MT * LN];
  __shared__ uint32_t s_req_k[MT * LN];
  __shared__ double s_lam[MT];
  __shared__ uint32_t s_svc[LT][LN], s_I[LT][LN], s_vh[LT][LN], s_vt[LT][LN];
  __shared__ int64_t s_M[LT][LN], s_B[LT][LN];
  __shared__ int32_t s_l[MT], s_lp[MT];
  __shared__ SegConst s_seg[LT];
  // Per lane: the back record of each boundary queue, and the youngest live
  // interior record of each segment with its index (kNil: not known; found by
  // a scan when next needed).  LIFO selections then read no HBM.
  __shared__ NRec s_vb[LT][LN], s_yi[LT][LN];
  __shared__ uint32_t s_yidx[LT][LN];
  // Per lane and segment: the index of the last youngest interior record that
  // left the segment (kNil: none known).  Every record entered after it has
  // left too, so the scan for the next youngest starts just below it; s_yi
  // still holds it while s_yidx is kNil.
  __shared__ uint32_t s_ydead[LT][LN];
  // per type: the guide of its output-length CDF row (kCdfGuide + 1 entries)
  __shared__ uint16_t s_cdfg[MT][kCdfGuide + 1];
  // Prefetch landing slots, one per lane, filled by asynchronous copies from
  // HBM (global_load_lds) issued at the end of an iteration and waited for at
  // the start of the next: the head of Q_{1,0}; per segment that can launch
  // next, the front of its boundary queue, the first record of the next
  // launch's terminal cohort slot and the head of the calendar bucket served
  // next.  32-byte records land as two 16-byte halves.
  __shared__ uint4 s_q0[LN];
  __shared__ uint4 s_vfa[LT][LN], s_vfb[LT][LN];
  __shared__ uint4 s_tra[LT][LN], s_trb[LT][LN];
  __shared__ uint32_t s_bh[LT][LN];
  // per lane and segment: the entering cohort's accounting, formed at launch
  __shared__ int32_t s_eB[LT][LN], s_eM[LT][LN];
  __shared__ uint32_t s_eI[LT][LN];
  __shared__ double s_edges[WS_MAX_HIST_EDGES + 1];
  __shared__ uint8_t s_htab[kHistTab];
  __shared__ int s_hsteps;

  const int tx = threadIdx.x;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + tx;
  // replica of this lane, or -1 for padding (padding only ends a job's
  // wavefront, so lane 0 of every wavefront holds a replica)
  const int32_t r32 = gid < A.n_list ? ((const int32_t *)(A.ws + A.off_list))[gid] : -1;
  const int64_t r = r32 < 0 ? 0 : r32;
  // every lane of a wavefront belongs to the same job: its constants are
  // wavefront-uniform
  const uint32_t jix =
      __builtin_amdgcn_readfirstlane(((const uint32_t *)(A.ws + A.off_job_of))[r]);
  const JobDev &J = ((const JobDev *)(A.ws + A.off_jobs))[jix];
  const int m = J.m;
  const int n_hist = J.n_hist;
  const int P = TV ? J.n_rate : 0;  // rate-profile points, 0 for constant rates
  const bool tv = TV && P > 0;
  // per-type prompt lengths (indexed by a lane's request type) and the
  // histogram edges with their bucket index, staged in LDS by the block
  {
    const double *edges_g = (const double *)(A.ws + J.off_edges);
    for (int b = tx; b <= n_hist; b += 64) s_edges[b] = b < n_hist ? edges_g[b] : INFINITY;
    for (int j = tx; j < MT; j += 64) {
      s_l[j] = j < m ? J.l[j] : 0;
      s_lp[j] = j < m ? J.lp[j] : 1;
      s_lam[j] = j < m ? J.lambda[j] : 0.0;
    }
    for (int k = tx; k < LT; k += 64) {
      SegConst c;
      const bool on = k < J.nseg;
      c.end = on ? J.seg_end[k] : 0;
      c.n = on ? J.seg_n[k] : 0;
      c.delta = on ? J.seg_delta[k] : 1;
      c.dmagic = fastmod_magic((uint32_t)c.delta);
      c.entry = on ? J.seg_entry[k] : 0;
      c.vmask = on && k >= 1 ? (1u << J.vcap_log2[k]) - 1u : 0u;
      c.off_rec = on ? (uint32_t)J.off_rec[k] : 0u;
      c.off_bkt = on ? (uint32_t)J.off_bkt[k] : 0u;
      c.off_v = on && k >= 1 ? (uint32_t)J.off_v[k] : 0u;
      s_seg[k] = c;
    }
    if (J.known == 0 && J.n_trace == 0 && J.out_cap > 1 && J.out_cap <= 65535) {
      const uint32_t *cdf_g = (const uint32_t *)(A.ws + J.off_cdf);
      for (int x = tx; x < MT * (kCdfGuide + 1); x += 64) {
        const int j = x / (kCdfGuide + 1), b = x % (kCdfGuide + 1);
        s_cdfg[j][b] = j < m ? (uint16_t)cdf_guide_entry(cdf_g + (size_t)j * (size_t)(J.out_cap - 1),
                                                         J.out_cap, b)
                             : (uint16_t)0;
      }
    }
    if (tv) {
      const double *rg = (const double *)(A.ws + J.off_rate);
      for (int i = tx; i < P; i += 64) s_rt[i] = rg[i];
      for (int x = tx; x < MT * NP; x += 64) {
        const int j = x / NP, i = x % NP;
        s_rf[j][i] = j < m && i < P ? rg[P + j * P + i] : 0.0;
      }
      for (int j = tx; j < MT; j += 64) s_fmax[j] = j < m ? J.rate_fmax[j] : 0.0;
    }
    __syncthreads();
  }
  const HistIdx hidx = hist_index_build(s_edges, n_hist, s_htab, &s_hsteps);
  const double *edges = s_edges;
  if (r32 < 0 || tx >= LN) return;  // padding lane: uses only its own LDS columns
  const uint64_t seed = ((const uint64_t *)(A.ws + A.off_seed))[r];
  const uint32_t rid = ((const uint32_t *)(A.ws + A.off_rid))[r];
  s_seed[tx] = seed;
  s_rid[tx] = rid;

  const int L = J.nseg;
  const double d0 = J.d0, d1 = J.d1;
  const int64_t C = J.C;
  const bool trace = J.n_trace > 0;
  const bool known = J.known != 0;
  const int32_t cap = J.out_cap;
  const uint32_t *cdf = (const uint32_t *)(A.ws + J.off_cdf);
  const double *tr_time = (const double *)(A.ws + J.off_tr_time);
  const int32_t *tr_type = (const int32_t *)(A.ws + J.off_tr_type);
  const int32_t *tr_len = (const int32_t *)(A.ws + J.off_tr_len);
  const uint32_t qmask = (1u << J.qcap_log2) - 1u;
  const uint32_t rec_cap = (uint32_t)J.rec_cap;
  uint8_t *blk = A.ws + J.off_ring + (uint64_t)(r - J.replica_begin) * J.ring_stride;
  QRec *q10 = (QRec *)(blk + J.off_q[0]);
  uint32_t *hist = (uint32_t *)(A.ws + A.off_hist) + r * (int64_t)A.hist_stride;

  auto recs = [&](int k) __attribute__((always_inline)) { return (NRec *)(blk + s_seg[k].off_rec); };
  auto bkts = [&](int k) __attribute__((always_inline)) { return (uint32_t *)(blk + s_seg[k].off_bkt); };
  auto vring = [&](int k) __attribute__((always_inline)) { return (NRec *)(blk + s_seg[k].off_v); };
  auto vmask = [&](int k) __attribute__((always_inline)) { return s_seg[k].vmask; };
  auto row_of = [&](int j) __attribute__((always_inline)) -> const uint32_t * {
    return (known || cap <= 1) ? nullptr : cdf + (size_t)j * (size_t)(cap - 1);
  };
  const bool use_guide = !known && !trace && cap > 1 && cap <= 65535;
  auto guide_of = [&](int j) __attribute__((always_inline)) -> const uint16_t * {
    return use_guide ? s_cdfg[j] : nullptr;
  };

  double t, lat_area, ttft_area, lat_sum, mem_area, busy;
  int64_t batches, arrivals, comps, ctok, evicts, etok, fallback, btok, peak, idle, N, U,
      Mres, tridx, pendft;
  uint32_t flags, qh, qt;

  if (!A.resume) {
    t = lat_area = ttft_area = lat_sum = mem_area = busy = 0.0;
    batches = arrivals = comps = ctok = evicts = etok = fallback = btok = peak = idle = 0;
    N = U = Mres = tridx = pendft = 0;
    flags = 0;
    qh = qt = 0;
    for (int j = 0; j < MT; ++j) {
      s_k[j][tx] = 0;
      s_tnext[j][tx] = INFINITY;
      s_Ln[j][tx] = 1;
      if (j < m && !trace) {
        int32_t Lj = 1;
        if (tv) {
          uint32_t k0 = 0;
          int cur = -1;
          s_tnext[j][tx] = draw_thinned(seed, rid, (uint32_t)j, k0, 0.0, J.lambda[j], s_fmax[j],
                                        s_rt, s_rf[j], P, row_of(j), cap, &Lj, cur, flags);
          s_k[j][tx] = k0;
        } else {
          const double g = draw_gap(seed, rid, (uint32_t)j, 0u, J.lambda[j], row_of(j), cap, &Lj,
                                    nullptr, guide_of(j));
          s_tnext[j][tx] = 0.0 + g;
        }
        s_Ln[j][tx] = known ? J.lp[j] : (cap <= 1 ? 1 : Lj);
      }
    }
    for (int k = 0; k < LT; ++k) {
      s_svc[k][tx] = s_I[k][tx] = s_vh[k][tx] = s_vt[k][tx] = 0;
      s_M[k][tx] = s_B[k][tx] = 0;
      if (k < L) {
        uint32_t *bk = bkts(k);
        for (int x = 0; x < s_seg[k].delta; ++x) bk[x] = kNil;
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
    fallback = slot_i(A, S_FALLBACK, r);
    btok = slot_i(A, S_BTOK, r);
    peak = slot_i(A, S_PEAK, r);
    idle = slot_i(A, S_IDLE, r);
    N = slot_i(A, S_N, r);
    U = slot_i(A, S_U, r);
    Mres = slot_i(A, S_MRES, r);
    tridx = slot_i(A, S_TRIDX, r);
    pendft = slot_i(A, S_PENDFT, r);
    flags = (uint32_t)slot_i(A, S_FLAGS, r);
    qh = (uint32_t)slot_i(A, S_QH, r);
    qt = (uint32_t)slot_i(A, S_QT, r);
    for (int j = 0; j < MT; ++j) {
      s_tnext[j][tx] = slot_f(A, S_TNEXT + j, r);
      s_k[j][tx] = (uint32_t)slot_i(A, S_K + j, r);
      s_Ln[j][tx] = (int32_t)slot_i(A, S_LNEXT + j, r);
    }
    for (int k = 0; k < LT; ++k) {
      s_svc[k][tx] = (uint32_t)slot_i(A, S_KSVC + k, r);
      s_I[k][tx] = (uint32_t)slot_i(A, S_KI + k, r);
      s_M[k][tx] = slot_i(A, S_KM + k, r);
      s_B[k][tx] = slot_i(A, S_KB + k, r);
      s_vh[k][tx] = (uint32_t)slot_i(A, S_KVH + k, r);
      s_vt[k][tx] = (uint32_t)slot_i(A, S_KVT + k, r);
    }
  }

  for (int j = 0; j < MT; ++j) {
    s_gend[j][tx] = s_k[j][tx] + 1u;  // gap rings start empty
    if constexpr (TV) s_cur[j][tx] = -1;  // profile cursors before the first piece
  }
  for (int k = 0; k < LT; ++k) {
    s_yidx[k][tx] = kNil;
    s_ydead[k][tx] = kNil;
    if (k >= 1 && k < L && s_vt[k][tx] != s_vh[k][tx])
      s_vb[k][tx] = vring(k)[(s_vt[k][tx] - 1u) & vmask(k)];
  }

  // ---- arrivals ------------------------------------------------------------
  auto peek = [&](int &jn) __attribute__((always_inline)) -> double {
    if (trace) {
      if (tridx >= J.n_trace) {
        jn = 0;
        return INFINITY;
      }
      jn = tr_type[tridx];
      return tr_time[tridx];
    }
    double best = s_tnext[0][tx];
    jn = 0;
    for (int j = 1; j < m; ++j) {
      const double v = s_tnext[j][tx];
      if (v < best) {
        best = v;
        jn = j;
      }
    }
    return best;
  };

  auto push_q10 = [&](double a_ft, int32_t j, int32_t Lr) __attribute__((always_inline)) {
    if (qt - qh >= rec_cap) {
      flags |= kFlagCap;
    } else {
      QRec rec;
      rec.a_ft = a_ft;
      rec.j = j;
      rec.L = Lr;
      q10[qt & qmask] = rec;
      if (qt == qh) s_q0[tx] = qrec_u4(rec);  // the new head
    }
    qt++;
  };

  auto take = [&](int jn, double a) __attribute__((always_inline)) {
    int32_t Lr;
    if (trace) {
      Lr = known ? s_lp[jn] : tr_len[tridx];
      tridx++;
    } else if (tv) {
      if constexpr (TV) {  // thinning over the candidates in the ring
        Lr = s_Ln[jn][tx];
        uint32_t k = s_k[jn][tx] + 1u;
        uint32_t ge = s_gend[jn][tx];
        int32_t Lj = 1;
        int cur = s_cur[jn][tx];
        const double tn = next_thinned(k, s_tnext[jn][tx], s_fmax[jn], s_rt, s_rf[jn], P, cur, flags,
                                       [&](uint32_t kc, double &g, uint32_t &w3) {
                                         if (kc < ge) {
                                           g = s_gap[jn][kc % GR][tx];
                                           w3 = s_w3[jn][kc % GR][tx];
                                           Lj = s_glen[jn][kc % GR][tx];
                                         } else {
                                           g = draw_gap(seed, rid, (uint32_t)jn, kc, J.lambda[jn],
                                                        row_of(jn), cap, &Lj, &w3);
                                           ge = kc + 1u;
                                         }
                                       });
        s_cur[jn][tx] = (int8_t)cur;
        s_gend[jn][tx] = ge;
        s_k[jn][tx] = k;
        s_tnext[jn][tx] = tn;
        s_Ln[jn][tx] = known ? s_lp[jn] : (cap <= 1 ? 1 : Lj);
      }
    } else {
      Lr = s_Ln[jn][tx];
      const uint32_t k = s_k[jn][tx] + 1u;
      s_k[jn][tx] = k;
      int32_t Lj = 1;
      double g;
      if (k < s_gend[jn][tx]) {
        g = s_gap[jn][k % GR][tx];
        Lj = s_glen[jn][k % GR][tx];
      } else {
        g = draw_gap(seed, rid, (uint32_t)jn, k, J.lambda[jn], row_of(jn), cap, &Lj, nullptr,
                     guide_of(jn));
        s_gend[jn][tx] = k + 1u;
      }
      s_tnext[jn][tx] = s_tnext[jn][tx] + g;
      s_Ln[jn][tx] = known ? s_lp[jn] : (cap <= 1 ? 1 : Lj);
    }
    arrivals++;
    N++;
    U++;
    push_q10(a, jn, Lr);
  };

  // ---- evictions -------------------------------------------------------------
  // Evict the back (most recently admitted) prompt of boundary queue h >= 1.
  auto evict_boundary = [&](int h) __attribute__((always_inline)) -> int64_t {
    const uint32_t vt = s_vt[h][tx] - 1u;
    const NRec rec = s_vb[h][tx];
    s_vt[h][tx] = vt;
    if (vt != s_vh[h][tx]) s_vb[h][tx] = vring(h)[(vt - 1u) & vmask(h)];  // the new back
    const int32_t rprev = s_seg[h - 1].end;
    const int64_t ch = (int64_t)s_l[rec.j] + rprev;
    s_B[h][tx] -= ch;
    Mres -= ch;
    evicts++;
    etok += rprev;
    push_q10(with_ft(rec.a_ft), rec.j, rec.L);  // it has produced r_{h-1} >= 1 tokens
    return ch;
  };

  // Most recently admitted live interior prompt of segment k: the newest
  // non-empty cohort slot, its highest live index.  Returns the record index
  // or kNil.
  auto youngest_interior = [&](int k, uint32_t &kb, uint32_t &kp) __attribute__((always_inline)) -> uint32_t {
    if (s_I[k][tx] == 0) return kNil;
    const uint32_t y = s_yidx[k][tx];
    if (y != kNil) {
      kb = s_yi[k][tx].kb;
      kp = s_yi[k][tx].kp;
      return y;
    }
    const int32_t delta = s_seg[k].delta;
    const int32_t nk = s_seg[k].n;
    const uint64_t dmg = s_seg[k].dmagic;
    const uint32_t svc = s_svc[k][tx];
    const NRec *rc = recs(k);
    // start just below the youngest that left last (its cohort entered at
    // service c, no later cohort has entered since: an entering cohort sets
    // the cache), else at the newest cohort slot
    int32_t back = 0, ifrom = nk - 1;
    const uint32_t dead = s_ydead[k][tx];
    if (dead != kNil) {
      const uint32_t c0 = s_yi[k][tx].c;
      back = (int32_t)(svc - c0);
      ifrom = (int32_t)(dead - fastmod(c0, dmg, (uint32_t)delta) * (uint32_t)nk) - 1;
      ifrom = ifrom < nk - 1 ? ifrom : nk - 1;  // indices stay inside the cohort slot
    }
    for (; back < delta && (int64_t)svc - back >= 1; ++back, ifrom = nk - 1) {
      const uint32_t slot = fastmod(svc - (uint32_t)back, dmg, (uint32_t)delta);
      // a record with L = 0 has left the segment (exit or eviction)
      for (int32_t i = ifrom; i >= 0; --i) {
        const uint32_t idx = slot * (uint32_t)nk + (uint32_t)i;
        // the whole record in one round trip (both halves issued together)
        uint4 lo = ((const uint4 *)(rc + idx))[0], hi = ((const uint4 *)(rc + idx))[1];
        lo = opaque4(lo);
        hi = opaque4(hi);
        const NRec rec = nrec_of(lo, hi);
        if (rec.L != 0) {
          kb = rec.kb;
          kp = rec.kp;
          s_yi[k][tx] = rec;
          s_yidx[k][tx] = idx;
          return idx;
        }
      }
    }
    return kNil;
  };

  auto evict_interior = [&](int k, uint32_t idx) __attribute__((always_inline)) -> int64_t {
    NRec *rc = recs(k);
    NRec rec = s_yi[k][tx];  // idx is the segment's youngest live interior record
    s_yidx[k][tx] = kNil;
    s_ydead[k][tx] = idx;
    const int32_t delta = s_seg[k].delta;
    const int32_t nk = s_seg[k].n;
    const int64_t stage = (int64_t)s_seg[k].entry + (int64_t)(s_svc[k][tx] - rec.c) + 1;
    const int64_t ch = (int64_t)s_l[rec.j] + stage;
    (void)delta;
    (void)nk;
    const int32_t Lr = rec.L;
    rec.L = 0;  // leaves a hole; the calendar skips it
    rc[idx] = rec;
    s_I[k][tx] -= 1u;
    s_M[k][tx] -= ch;
    Mres -= ch;
    evicts++;
    fallback++;
    etok += stage - 1;
    const bool ft = has_ft(rec.a_ft) || stage >= 2;
    if (stage == 1 && !ft) pendft--;
    push_q10(ft ? with_ft(rec.a_ft) : arrival_of(rec.a_ft), rec.j, Lr);
    return ch;
  };

  // Evict the most recently admitted prompt among the boundary queues and,
  // if allow_interior is set and none holds a prompt, among the interior of
  // segments [klo, L).  Returns the memory freed, 0 if nothing was left.
  // `boundary` is cleared once the boundary queues are found empty: within
  // one repair they stay empty (evicted prompts go back to the entry queue),
  // so later calls skip that scan.
  auto evict_lifo = [&](int klo, bool allow_interior, bool &boundary)
                        __attribute__((always_inline)) -> int64_t {
    int hb = -1;
    uint32_t bkb = 0, bkp = 0;
    for (int h = 1; boundary && h < L; ++h) {
      if (s_vt[h][tx] == s_vh[h][tx]) continue;
      const uint32_t rkb = s_vb[h][tx].kb, rkp = s_vb[h][tx].kp;
      if (hb < 0 || rkb > bkb || (rkb == bkb && rkp > bkp)) {
        hb = h;
        bkb = rkb;
        bkp = rkp;
      }
    }
    if (hb >= 0) return evict_boundary(hb);
    boundary = false;
    if (!allow_interior) return 0;
    int kbest = -1;
    uint32_t ibest = kNil;
    for (int k = klo; k < L; ++k) {
      uint32_t kb = 0, kp = 0;
      const uint32_t idx = youngest_interior(k, kb, kp);
      if (idx == kNil) continue;
      if (kbest < 0 || kb > bkb || (kb == bkb && kp > bkp)) {
        kbest = k;
        ibest = idx;
        bkb = kb;
        bkp = kp;
      }
    }
    if (kbest < 0) return 0;
    return evict_interior(kbest, ibest);
  };

  // Stage A of the prefetch (end of an iteration): everything the next
  // launch and completion read first.  Slot indices are masked into their
  // rings, so a slot past a queue's tail reads a stale record that is never
  // used (a push into the empty queue writes the landing slot instead).
  // A segment k >= 1 can be in the next launch only if its boundary queue
  // already holds n_k prompts (boundary queues change only in the completion
  // step); only those segments are prefetched.
  auto may_launch = [&](int k) __attribute__((always_inline)) {
    return k == 0 || (int32_t)(s_vt[k][tx] - s_vh[k][tx]) >= s_seg[k].n;
  };
  auto prefetch_a = [&]() __attribute__((always_inline)) {
    copy16_to_lds(q10 + (qh & qmask), &s_q0[0]);
    for (int k = 0; k < L; ++k) {
      if (!may_launch(k)) continue;
      const int32_t delta = s_seg[k].delta;
      const uint32_t x = s_svc[k][tx] + 1u;  // the segment's next service
      copy4_to_lds(bkts(k) + fastmod(x, s_seg[k].dmagic, (uint32_t)delta), &s_bh[k][0]);
      if (k >= 1) {
        const NRec *f = vring(k) + (s_vh[k][tx] & vmask(k));
        copy16_to_lds(f, &s_vfa[k][0]);
        copy16_to_lds((const uint8_t *)f + 16, &s_vfb[k][0]);
      }
      if (s_seg[k].n == 1) {
        const NRec *tr = recs(k) + fastmod(x - (uint32_t)(delta - 1), s_seg[k].dmagic, (uint32_t)delta);
        copy16_to_lds(tr, &s_tra[k][0]);
        copy16_to_lds((const uint8_t *)tr + 16, &s_trb[k][0]);
      }
    }
  };
  bool stopped = (flags & (kFlagCap | kFlagStall)) != 0;
  if (!stopped) prefetch_a();

  for (int64_t it = 0; it < A.horizon && !stopped; ++it) {
    // ---- refill the draw rings, all active lanes together -----------------
    if (!trace) {
      const uint64_t act = __ballot(1);
      const int nact = __popcll(act);
      const int wrank = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(act >> 32),
                                                      __builtin_amdgcn_mbcnt_lo((uint32_t)act, 0u));
      // the requests of every type are gathered first and drawn in one pass,
      // so the types' memory round trips (CDF searches) overlap
      int nreq = 0;  // wavefront-uniform
      for (int j = 0; j < m; ++j) {
        const uint32_t ge = s_gend[j][tx];
        const uint32_t avail = ge - s_k[j][tx] - 1u;
        if (__ballot(avail < kLow) == 0) continue;
        const bool room = avail <= (uint32_t)(GR - GU);
        const uint64_t need = __ballot(room);
        if (room) {
          const int rk = nreq + (int)__builtin_amdgcn_mbcnt_hi(
                                    (uint32_t)(need >> 32),
                                    __builtin_amdgcn_mbcnt_lo((uint32_t)need, 0u));
          s_req_lane[rk] = (uint8_t)tx;
          s_req_j[rk] = (uint8_t)j;
          s_req_k[rk] = ge;
          s_gend[j][tx] = ge + GU;  // read again only after the pass
        }
        nreq += __popcll(need);
      }
      if (nreq > 0) {
        wave_lds_sync();
        const int total = nreq * GU;
        for (int base = 0; base < total; base += nact) {
          const int w = base + wrank;
          if (w < total) {
            const int ln = (int)s_req_lane[w / GU];
            const int j = (int)s_req_j[w / GU];
            const uint32_t k = s_req_k[w / GU] + (uint32_t)(w % GU);
            int32_t Lj = 1;
            uint32_t w3;
            s_gap[j][k % GR][ln] = draw_gap(s_seed[ln], s_rid[ln], (uint32_t)j, k, s_lam[j],
                                            row_of(j), cap, &Lj, TV ? &w3 : nullptr,
                                            guide_of(j));
            s_glen[j][k % GR][ln] = Lj;
            if constexpr (TV) s_w3[j][k % GR][ln] = w3;
          }
        }
        wave_lds_sync();
      }
    }

    wait_memory();  // stage A has landed

    // ---- decision: largest prefix of segments meeting their thresholds -----
    int kmax = 0;
    for (;;) {
      if (flags & kFlagCap) {
        stopped = true;
        break;
      }
      if ((int64_t)(qt - qh) >= s_seg[0].n) {
        kmax = 1;
        while (kmax < L && (int64_t)(s_vt[kmax][tx] - s_vh[kmax][tx]) >= s_seg[kmax].n) kmax++;
        break;
      }
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


    // ---- launch: entering cohorts, calendar links, batch tokens -----------
    const uint32_t bidx = (uint32_t)batches;
    int64_t tokens = 0, prefill_l = 0, mplus = Mres;
    int64_t pend_new = 0;
    // per-batch trace: every interior prompt of a served segment and the
    // entering cohorts are processed
    int64_t bt_sel = 0;
    const int64_t bt_ev0 = evicts;
    if constexpr (TV)
      for (int k = 0; k < kmax; ++k) bt_sel += (int64_t)s_I[k][tx] + s_seg[k].n;
    for (int k = 0; k < kmax; ++k) {
      const int32_t delta = s_seg[k].delta;
      const int32_t nk = s_seg[k].n;
      const int32_t rk = s_seg[k].end;
      const int32_t ent = s_seg[k].entry;
      const uint32_t x = s_svc[k][tx] + 1u;
      const uint64_t dmg = s_seg[k].dmagic;
      const uint32_t slot = fastmod(x, dmg, (uint32_t)delta);
      NRec *rc = recs(k);
      uint32_t *bk = bkts(k);
      tokens += s_M[k][tx];
      uint32_t suml = 0;
      int32_t eB = 0, eM = 0;
      uint32_t eI = 0;
      // link in reverse selection order: traversal is then in key order
      for (int32_t i = nk - 1; i >= 0; --i) {
        NRec e;
        if (k == 0) {
          QRec qr;
          if (i == 0) {
            qr = qrec_of(s_q0[tx]);  // the head, prefetched
          } else {
            qr = q10[(qh + (uint32_t)i) & qmask];
            qr.a_ft = opaque(qr.a_ft);  // waited for inside this branch
            qr.j = opaque(qr.j);
            qr.L = opaque(qr.L);
          }
          e.a_ft = qr.a_ft;
          e.j = qr.j;
          e.L = qr.L;
          e.kb = bidx;
          e.kp = (uint32_t)i;
          tokens += s_l[qr.j];
          prefill_l += s_l[qr.j];
          if (!has_ft(qr.a_ft)) pend_new++;
        } else {
          if (i == 0) {
            e = nrec_of(s_vfa[k][tx], s_vfb[k][tx]);  // the front, prefetched
          } else {
            const NRec *src = vring(k) + ((s_vh[k][tx] + (uint32_t)i) & vmask(k));
            uint4 lo = ((const uint4 *)src)[0], hi = ((const uint4 *)src)[1];
            lo = opaque4(lo);  // both halves in flight before the wait
            hi = opaque4(hi);
            e = nrec_of(lo, hi);
          }
          tokens += (int64_t)s_l[e.j] + s_seg[k - 1].end + 1;
        }
        e.c = x;
        const int32_t pexit = e.L < rk ? e.L : rk;
        const uint32_t b = fastmod(x + (uint32_t)(pexit - ent), dmg, (uint32_t)delta);
        const uint32_t idx = slot * (uint32_t)nk + (uint32_t)i;
        if (b == slot) {  // exits at this very service: heads the bucket served now
          e.next = s_bh[k][tx];
          s_bh[k][tx] = idx;
        } else {
          e.next = bk[b];
        }
        bk[b] = idx;
        rc[idx] = e;
        if (i == nk - 1) {  // the cohort's last record is the segment's youngest
          s_yi[k][tx] = e;
          s_yidx[k][tx] = idx;
        }
        suml += (uint32_t)s_l[e.j];
        // what the completion step does with the entering prompts
        const int32_t le = s_l[e.j];
        if (k > 0) eB += le + s_seg[k - 1].end;
        if (pexit > ent) {
          eI += 1u;
          eM += le + ent + 1;
        }
      }
      s_eB[k][tx] = eB;
      s_eI[k][tx] = eI;
      s_eM[k][tx] = eM;
      if (k == 0)
        qh += (uint32_t)nk;
      else
        s_vh[k][tx] += (uint32_t)nk;  // still charged in s_B until the completion
      // projected change of the segment's memory (no early completion)
      if (delta >= 2) {
        uint32_t T = 0, Tl = 0;
        if ((int64_t)x - (delta - 1) >= 1) {
          // the terminal cohort slot: its prompts still in the segment
          const uint32_t ts = fastmod(x - (uint32_t)(delta - 1), dmg, (uint32_t)delta);
          if (nk == 1) {  // prefetched
            const int32_t trL = (int32_t)s_trb[k][tx].y, trj = (int32_t)s_trb[k][tx].x;
            T = trL != 0 ? 1u : 0u;
            Tl = trL != 0 ? (uint32_t)s_l[trj] : 0u;
          } else {
            for (int32_t i = 0; i < nk; ++i) {
              // j and L (the second half's first two words) in one load
              const uint2 jl = opaque(*(const uint2 *)((const uint8_t *)(rc + ts * (uint32_t)nk +
                                                                          (uint32_t)i) + 16));
              const bool live = (int32_t)jl.y != 0;
              T += live ? 1u : 0u;
              Tl += live ? (uint32_t)s_l[(int32_t)jl.x] : 0u;
            }
          }
        }
        mplus += (int64_t)s_I[k][tx] - T;
        if (k == L - 1) mplus -= (int64_t)Tl + (int64_t)T * rk;
        if (k == 0)
          mplus += (int64_t)suml + nk;  // prefills land at stage 1
        else
          mplus += 2ll * nk;            // l + r_{k-1} -> l + r_{k-1} + 2
      } else {                          // entering prompts are processed at r_k
        if (k < L - 1)
          mplus += nk;                  // l + r_{k-1} -> l + r_k
        else
          mplus -= (int64_t)suml + (int64_t)nk * s_seg[k - 1].end;
      }
    }

    // ---- pre-launch repair on the projected state ----------------------------
    bool bnd_pre = true;
    while (mplus > C) {
      const int64_t freed = evict_lifo(kmax, false, bnd_pre);
      if (freed == 0) break;
      mplus -= freed;
    }
    while (mplus > C) {  // unselected interior prompts (segments after the prefix)
      const int64_t freed = evict_lifo(kmax, true, bnd_pre);
      if (freed == 0) break;
      mplus -= freed;
    }
    if (mplus > C) flags |= kFlagOverflow;
    const int64_t bt_ev1 = evicts;
    const int64_t bt_comps0 = comps;

    const int64_t m_launch = Mres + prefill_l;
    if (m_launch > peak) peak = m_launch;
    const double tau = d0 + d1 * (double)tokens;
    const double t_end = t + tau;
    const int64_t N0 = N, U0 = U;

    // ---- arrivals during the batch -----------------------------------------
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

    // ---- completion transition, segment by segment ---------------------------
    for (int k = 0; k < kmax; ++k) {
      const int32_t delta = s_seg[k].delta;
      const int32_t rk = s_seg[k].end;
      const uint32_t x = s_svc[k][tx] + 1u;
      s_svc[k][tx] = x;
      NRec *rc = recs(k);
      if (k == 0) {  // the stage-1 cohort produces its first tokens
        U -= pendft;
        pendft = pend_new;
      }
      int64_t Mk = s_M[k][tx] + (int64_t)s_I[k][tx];  // every interior prompt advances
      uint32_t Ik = s_I[k][tx];
      // entering prompts: leave the entry queue, stay unless they exit now
      // (their sums were formed at launch)
      if (k > 0) {
        s_B[k][tx] -= s_eB[k][tx];
        Mres -= s_eB[k][tx];
      }
      Ik += s_eI[k][tx];
      Mk += s_eM[k][tx];
      // prompts whose exit is at this service: the bucket's head was
      // prefetched, the list's records are read on demand
      uint32_t *bk = bkts(k);
      const uint32_t b = fastmod(x, s_seg[k].dmagic, (uint32_t)delta);
      uint32_t idx = s_bh[k][tx];
      bk[b] = kNil;
      // Each record is loaded whole (both 16-byte halves at once) one node
      // ahead: the next record's load is issued before this node's stores,
      // so waiting for it does not wait for them.
      uint4 clo = make_uint4(0u, 0u, 0u, 0u), chi = make_uint4(0u, 0u, 0u, kNil);
      if (idx != kNil) {
        clo = ((const uint4 *)(rc + idx))[0];
        chi = ((const uint4 *)(rc + idx))[1];
      }
      while (idx != kNil) {
        const NRec rec = nrec_of(opaque4(clo), opaque4(chi));
        const uint32_t nxt = rec.next;
        if (nxt != kNil) {
          clo = ((const uint4 *)(rc + nxt))[0];
          chi = ((const uint4 *)(rc + nxt))[1];
        }
        if (rec.L != 0) {  // holes left by evictions are skipped
          if (idx == s_yidx[k][tx]) {  // the youngest leaves
            s_ydead[k][tx] = idx;
            s_yidx[k][tx] = kNil;
          }
          const int64_t le = s_l[rec.j];
          const int32_t p = rec.L < rk ? rec.L : rk;
          if (rec.c != x) {  // an interior prompt: it had advanced to p + 1
            Mk -= le + p + 1;
            Ik -= 1u;
          }
          if (rec.L == p) {  // completion at its own output length
            const double lat = t_end - arrival_of(rec.a_ft);
            lat_sum += lat;
            __hip_atomic_fetch_add(&hist[hist_bin_idx(edges, s_htab, hidx, lat)], 1u,
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            comps++;
            ctok += rec.L;
            N--;
          } else {  // survivor joins the boundary queue of segment k+1
            const int h = k + 1;
            NRec v = rec;
            v.a_ft = with_ft(rec.a_ft);
            const uint32_t vt = s_vt[h][tx];
            if (vt - s_vh[h][tx] <= vmask(h)) {
              vring(h)[vt & vmask(h)] = v;
              if (vt == s_vh[h][tx]) {  // pushed into an empty queue: its front
                s_vfa[h][tx] = nrec_lo(v);
                s_vfb[h][tx] = nrec_hi(v);
              }
              s_vt[h][tx] = vt + 1u;
              s_vb[h][tx] = v;
            } else {
              flags |= kFlagCap;  // bounded by construction; guards the ring
            }
            s_B[h][tx] += le + rk;
            Mres += le + rk;
          }
          rc[idx].L = 0;  // no longer in the segment
        }
        idx = nxt;
      }
      Mres += Mk - s_M[k][tx];
      s_M[k][tx] = Mk;
      s_I[k][tx] = Ik;
    }
    if (Mres > peak) peak = Mres;

    // ---- repair: boundary prompts first, then interior prompts -------------
    bool bnd_post = true;
    while (Mres > C) {
      if (evict_lifo(0, true, bnd_post) == 0) break;
    }
    if constexpr (TV) {
      if (A.btrace != nullptr && batches < A.btrace_cap) {
        BatchRec br;
        br.t_launch = t_end - tau;
        br.tau = tau;
        br.tokens = tokens;
        br.prefills = s_seg[0].n;
        br.selected = bt_sel;
        br.completions = comps - bt_comps0;
        br.evict_pre = bt_ev1 - bt_ev0;
        br.evict_post = evicts - bt_ev1;
        br.mem_after = Mres;
        br.waiting_after = qt - qh;
        int64_t res = 0;
        for (int k = 0; k < L; ++k) {
          res += s_I[k][tx];
          if (k > 0) res += s_vt[k][tx] - s_vh[k][tx];
        }
        br.resident_after = res;
        br.mplus = mplus;
        ((BatchRec *)A.btrace)[r * A.btrace_cap + batches] = br;
      }
    }
    batches++;
    btok += tokens;
    prefetch_a();
  }
  // no asynchronous copy may still target this workgroup's LDS when it ends
  wait_memory();

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
  put_i(A, S_FALLBACK, r, fallback);
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
  for (int j = 0; j < MT; ++j) {
    put_f(A, S_TNEXT + j, r, s_tnext[j][tx]);
    put_i(A, S_K + j, r, s_k[j][tx]);
    put_i(A, S_LNEXT + j, r, s_Ln[j][tx]);
  }
  for (int k = 0; k < LT; ++k) {
    put_i(A, S_KSVC + k, r, s_svc[k][tx]);
    put_i(A, S_KI + k, r, s_I[k][tx]);
    put_i(A, S_KM + k, r, s_M[k][tx]);
    put_i(A, S_KB + k, r, s_B[k][tx]);
    put_i(A, S_KVH + k, r, s_vh[k][tx]);
    put_i(A, S_KVT + k, r, s_vt[k][tx]);
  }
}

template <int MT, int LT, bool TV>
hipError_t launch_ml(const KArgs &A, hipStream_t s) {
  const dim3 g((A.n_list + 63) / 64), b(64);
  if (A.lanes == 32)
    hipLaunchKernelGGL((sim_nested_kernel<MT, LT, 32, TV>), g, b, 0, s, A);
  else if (A.lanes == 16)
    hipLaunchKernelGGL((sim_nested_kernel<MT, LT, 16, TV>), g, b, 0, s, A);
  else if (A.lanes == 8)
    hipLaunchKernelGGL((sim_nested_kernel<MT, LT, 8, TV>), g, b, 0, s, A);
  else if (A.lanes == 4)
    hipLaunchKernelGGL((sim_nested_kernel<MT, LT, 4, TV>), g, b, 0, s, A);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

template <bool TV>
hipError_t launch_nested_k(int max_m, int max_seg, const KArgs &A, hipStream_t s) {
  if (max_m <= 4) {
    if (max_seg <= 4) return launch_ml<4, 4, TV>(A, s);
    if (max_seg <= 8) return launch_ml<4, 8, TV>(A, s);
    return launch_ml<4, 16, TV>(A, s);
  }
  if (max_seg <= 8) return launch_ml<16, 8, TV>(A, s);
  return launch_ml<16, 16, TV>(A, s);
}

}  // namespace
}  // namespace wsim
