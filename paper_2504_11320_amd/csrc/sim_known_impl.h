// sim_known_impl.h -- simulation kernel for WAIT and FCFS with known output
// lengths (arXiv 2504.11320: Algorithm 1, Section 4.1).  Included by one
// translation unit per policy (sim_known_wait.hip, sim_known_fcfs.hip).
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
// Latency: the hot ends of every ring are cached in registers.  The queue
// head and the first two deque records are prefetched one pop ahead with
// unconditional loads (a slot past the tail reads a stale value that a later
// push replaces through a separate register and a bit mask), and the loads
// of one iteration are waited for once, at the start of the next, so a pop
// consumes a value loaded long before; the deque back is served from a
// window of the most recent pushes kept in LDS.  First tokens are counted per
// cohort (how many prompts of the newest cohort have not produced one yet),
// so resident records are never rewritten.  All lanes of a wavefront belong to
// one job (the replica lists are padded per job), so the job's constants are
// wavefront-uniform and live in scalar registers.
//
// Arithmetic follows the model contract exactly (same IEEE operations in the
// same order, no FMA contraction), so integer state is bit-identical to the
// oracle's and floating sums agree to rounding.
#pragma once

#include "sim_common.h"

namespace wsim {
namespace {

// MT: type slots (>= m, at most 16); POL: WS_WAIT or WS_FCFS; TRACE: some job of the
// launch replays an arrival list; LN: replicas per wavefront (lanes LN..63
// are padding), which sizes the per-lane LDS arrays; TV: jobs with
// time-varying rates are supported (compiled out of the common kernels);
// ONE: WAIT with every threshold n_j = 1 (at most one admission and one
// completion per type and batch), which defers ring reloads to the ends of
// the admission and completion phases.
// Wavefronts of at most 16 replicas with up to 3 types run two per SIMD
// (their LDS allows it), so their register budget is stated to the compiler:
// one register past it would halve their occupancy.
template <int MT, int LN>
constexpr int kKnownMinWaves = MT <= 3 && LN <= 16 ? 2 : 1;

template <int MT, int POL, bool TRACE, int LN, bool TV, bool ONE>
__global__ void __launch_bounds__(64)
    __attribute__((amdgpu_waves_per_eu(kKnownMinWaves<MT, LN>, 2))) sim_known_kernel(KArgs A) {
  constexpr bool WAIT = POL == WS_WAIT;
  // Inter-arrival gaps are drawn ahead of use by the whole wavefront at once
  // (64 draws per pass, no divergence) into a ring of GR gaps per type and
  // lane; a lane whose ring runs dry draws the gap itself.
  // With time-varying rates the rings hold candidates of the thinning bound
  // process with their fourth Philox words (the acceptance draws), and the
  // rate profile sits in LDS beside them.
  constexpr int GR = MT <= 4 ? (TV ? 8 : 16) : 4;  // ring size per (type, lane)
  constexpr int GU = GR / 2;            // gaps added per refill
  constexpr uint32_t kLow = GU / 2;     // a lane below this triggers a refill
  __shared__ double s_edges[WS_MAX_HIST_EDGES + 1];
  __shared__ uint8_t s_htab[kHistTab];
  __shared__ int s_hsteps;
  __shared__ double s_gap[MT][GR][LN];
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
  __shared__ double s_lamj[MT];
  // The last WB records pushed on each resident deque are also kept in LDS,
  // so LIFO evictions (which pop the back) rarely read HBM.  Launches with
  // time-varying rates run two wavefronts per SIMD at 16 replicas each; a
  // window of 8 lets eight workgroups share a CU's LDS.  Constant-rate
  // launches at 16 replicas per wavefront (jobs of 16 replicas, as in
  // threshold sweeps) also run two per SIMD: a window of 14 keeps the
  // 3-type kernel within a CU's LDS for eight workgroups.
  constexpr int WB = MT <= 4 ? (TV && LN <= 16 ? 8 : (LN == 16 ? 14 : 16)) : 2;
  __shared__ DRec s_win[MT][WB][LN];
  const int tx = threadIdx.x;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  // replica of this lane, or -1 for padding (padding only ends a job's last
  // wavefront, so lane 0 of every wavefront holds a replica)
  const int32_t r32 = gid < A.n_list ? ((const int32_t *)(A.ws + A.off_list))[gid] : -1;
  const int64_t r = r32 < 0 ? 0 : r32;
  // every lane of a wavefront belongs to the same job
  const uint32_t jix =
      __builtin_amdgcn_readfirstlane(((const uint32_t *)(A.ws + A.off_job_of))[r]);
  const JobDev *J = ((const JobDev *)(A.ws + A.off_jobs)) + jix;

  const int m = J->m;
  const double d0 = J->d0, d1 = J->d1;
  const int32_t C = (int32_t)J->C;  // <= 2^30
  const int32_t cap_adm = (int32_t)(J->C - J->reserve_tok);
  // FCFS with chunked prefill: prefill tokens per iteration (0: whole)
  const int32_t chunk = WAIT ? 0 : J->chunk;
  const int n_hist = J->n_hist;
  const int P = TV ? J->n_rate : 0;  // rate-profile points, 0 for constant rates
  const bool tv = TV && P > 0;
  // the latency histogram's edges, searched at every completion, and the
  // rate profile, staged in LDS (the edges with their bucket index) by all
  // lanes of the block (one wavefront, one job)
  {
    const double *edges_g = (const double *)(A.ws + J->off_edges);
    for (int b = threadIdx.x; b <= n_hist; b += 64)
      s_edges[b] = b < n_hist ? edges_g[b] : INFINITY;
    for (int j = threadIdx.x; j < MT; j += 64) s_lamj[j] = j < m ? J->lambda[j] : 0.0;
    if (tv) {
      const double *rg = (const double *)(A.ws + J->off_rate);
      for (int i = threadIdx.x; i < P; i += 64) s_rt[i] = rg[i];
      for (int x = threadIdx.x; x < MT * NP; x += 64) {
        const int j = x / NP, i = x % NP;
        s_rf[j][i] = j < m && i < P ? rg[P + j * P + i] : 0.0;
      }
      for (int j = threadIdx.x; j < MT; j += 64) s_fmax[j] = j < m ? J->rate_fmax[j] : 0.0;
    }
    __syncthreads();
  }
  const HistIdx hidx = hist_index_build(s_edges, n_hist, s_htab, &s_hsteps);
  const double *edges = s_edges;
  if (r32 < 0 || tx >= LN) return;  // padding lane
  const uint64_t seed = ((const uint64_t *)(A.ws + A.off_seed))[r];
  const uint32_t rid = ((const uint32_t *)(A.ws + A.off_rid))[r];
  s_seed[tx] = seed;
  s_rid[tx] = rid;
  const bool trace = TRACE && J->n_trace > 0;  // compiled out of the common kernel
  // WAIT-no-wait: a type is served whenever it has a waiting or resident
  // prompt and admits at most n_j waiting ones (job-uniform)
  const bool nowait = WAIT && J->nowait != 0;
  const int64_t n_trace = J->n_trace;
  const double *tr_time = (const double *)(A.ws + J->off_tr_time);
  const int32_t *tr_type = (const int32_t *)(A.ws + J->off_tr_type);
  const uint32_t qmask = (1u << J->qcap_log2) - 1u;
  const uint32_t rec_cap = (uint32_t)J->rec_cap;
  uint8_t *blk = A.ws + J->off_ring + (uint64_t)(r - J->replica_begin) * J->ring_stride;
  uint32_t *hist = (uint32_t *)(A.ws + A.off_hist) + r * (int64_t)A.hist_stride;

  int32_t l[MT], lp[MT], nth[MT];
  // WAIT per-stage caps (Section 6; general instantiation only): type j takes
  // the caps of its l'_j + 1 stages in turn, one per service, as its
  // threshold and cohort size; ncap[j] is the cap of its next service
  const bool capped = TV && WAIT && J->has_caps != 0;
  const int32_t *capt = (const int32_t *)(A.ws + J->off_caps);
  int32_t coff[MT], ncap[MT];
  double lam[MT];
  uint32_t dmask[MT];
  uint32_t qoff[MT], doff[MT];  // ring offsets inside the replica block
#pragma unroll
  for (int j = 0; j < MT; ++j) {
    const bool on = j < m;
    l[j] = on ? J->l[j] : 0;
    lp[j] = on ? J->lp[j] : 1;
    nth[j] = on ? J->n[j] : 0;
    coff[j] = j == 0 ? 0 : coff[j - 1] + lp[j - 1] + 1;
    lam[j] = on ? J->lambda[j] : 0.0;
    dmask[j] = on ? (1u << J->dcap_log2[j]) - 1u : 0u;
    qoff[j] = (uint32_t)J->off_q[on && WAIT ? j : 0];
    doff[j] = (uint32_t)J->off_d[on ? j : 0];
  }

  // per-type state
  double tnext[MT];
  uint32_t kk[MT], qh[MT], qt[MT], dh[MT], dt[MT], svc[MT], pend[MT];
  uint32_t gend[MT];  // gaps of arrivals kk+1 .. gend-1 are in the ring
  uint32_t wv[MT];    // deque records dt-wv .. dt-1 are also in the LDS window
  // WAIT with general thresholds, constant rates: the records of deque j
  // admitted in the current batch and still resident (the last fr[j] ones)
  constexpr bool BULK = WAIT && !ONE && !TV;
  uint32_t fr[MT];
  int32_t Mj[MT];  // resident memory per type (< 2C <= 2^31)
  // Queue heads.  WAIT: the head of queue j is qpu[j] if bit j of qsrc is
  // set (pushed into an empty queue), else qld[j] (loaded when the previous
  // head left).  FCFS: the same for the shared queue with q0pu / q0ld.
  double qld[MT], qpu[MT];
  uint32_t qsrc = 0;
  QRec q0ld, q0pu;
  bool q0src = false;
  // Deque fronts: the first record (fa = arrival, fadm = admission service
  // under WAIT, admission batch under FCFS) and the second, which is s1pa /
  // s1padm if bit j of s1src is set, else s1a / s1adm (prefetched).  The
  // back record (ba, bkb, bkc) is kept for the LIFO repair.  One array per
  // field: arrays of structs would be indexed as memory by the compiler.
  double fa[MT], s1a[MT], s1pa[MT], ba[MT];
  uint32_t fadm[MT], s1adm[MT], s1padm[MT], bkb[MT], bkc[MT];
  uint32_t s1src = 0;

  double t, lat_area, ttft_area, lat_sum, mem_area, busy;
  int64_t batches, arrivals, comps, ctok, evicts, etok, btok, peak, idle, tridx;
  // resident memory: at most C after a repair, plus one batch's growth (at
  // most C/2: every resident holds >= 2 tokens) and admissions (FCFS: within
  // C; WAIT: sum_j n_j (l_j + 1) < 2^29, checked on the host), so < 2^31
  int32_t Mres;
  int32_t N, U;  // requests in system, and those without a first token
  uint32_t flags;
  // FCFS chunked prefill: the partially prefilled prompt (at most one, the
  // last admitted), outside the deques until its last chunk: arrival time
  // with first-token flag, type (-1: none) and prompt tokens cached so far
  double part_a;
  int32_t part_j, part_pp;

  uint32_t bidx_cur = 0;  // index of the batch being formed

  auto qring = [&](int j) __attribute__((always_inline)) { return (double *)(blk + qoff[j]); };
  auto qring0 = [&]() __attribute__((always_inline)) { return (QRec *)(blk + qoff[0]); };
  auto dring = [&](int j) __attribute__((always_inline)) { return (DRec *)(blk + doff[j]); };

  if (!A.resume) {
    t = lat_area = ttft_area = lat_sum = mem_area = busy = 0.0;
    batches = arrivals = comps = ctok = evicts = etok = btok = peak = idle = 0;
    N = U = Mres = 0;
    tridx = 0;
    flags = 0;
    part_a = 0.0;
    part_j = -1;
    part_pp = 0;
#pragma unroll
    for (int j = 0; j < MT; ++j) {
      kk[j] = qh[j] = qt[j] = dh[j] = dt[j] = svc[j] = pend[j] = 0;
      Mj[j] = 0;
      tnext[j] = INFINITY;
      if (j < m && !trace && tv) {
        uint32_t k0 = 0;
        int cur = -1;
        tnext[j] = draw_thinned(seed, rid, (uint32_t)j, k0, 0.0, lam[j], s_fmax[j], s_rt, s_rf[j],
                                P, nullptr, 0, nullptr, cur, flags);
        kk[j] = k0;
      } else if (j < m && !trace) {
        tnext[j] = 0.0 + draw_gap(seed, rid, (uint32_t)j, 0u, lam[j], nullptr, 0, nullptr);
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
    N = (int32_t)slot_i(A, S_N, r);
    U = (int32_t)slot_i(A, S_U, r);
    Mres = (int32_t)slot_i(A, S_MRES, r);
    tridx = slot_i(A, S_TRIDX, r);
    flags = (uint32_t)slot_i(A, S_FLAGS, r);
    part_a = slot_f(A, S_PARTA, r);
    part_j = (int32_t)slot_i(A, S_PARTJ, r);
    part_pp = (int32_t)slot_i(A, S_PARTPP, r);
#pragma unroll
    for (int j = 0; j < MT; ++j) {
      tnext[j] = slot_f(A, S_TNEXT + j, r);
      kk[j] = (uint32_t)slot_i(A, S_K + j, r);
      qh[j] = (uint32_t)slot_i(A, S_QH + j, r);
      qt[j] = (uint32_t)slot_i(A, S_QT + j, r);
      dh[j] = (uint32_t)slot_i(A, S_DH + j, r);
      dt[j] = (uint32_t)slot_i(A, S_DT + j, r);
      svc[j] = (uint32_t)slot_i(A, S_SVC + j, r);
      Mj[j] = (int32_t)slot_i(A, S_MJ + j, r);
      pend[j] = (uint32_t)slot_i(A, S_LNEXT + j, r);
    }
  }
#pragma unroll
  for (int j = 0; j < MT; ++j)
    ncap[j] = capped && j < m ? capt[coff[j] + (int32_t)(svc[j] % (uint32_t)(lp[j] + 1))] : nth[j];
  // caches of the ring ends; the gap rings start empty; profile cursors start
  // before the first piece
#pragma unroll
  for (int j = 0; j < MT; ++j) {
    if constexpr (TV) s_cur[j][tx] = -1;
    gend[j] = kk[j] + 1u;
    wv[j] = 0;
    fr[j] = 0;
    // unconditional loads: a slot past the tail holds a stale record that is
    // never used (the masks keep every index inside its ring)
    if (WAIT) qld[j] = qring(j)[qh[j] & qmask];
    const DRec f = dring(j)[dh[j] & dmask[j]];
    const DRec f2 = dring(j)[(dh[j] + 1u) & dmask[j]];
    const DRec b = dring(j)[(dt[j] - 1u) & dmask[j]];
    fa[j] = f.a_ft;
    fadm[j] = WAIT ? f.kc : f.kb;
    s1a[j] = f2.a_ft;
    s1adm[j] = WAIT ? f2.kc : f2.kb;
    ba[j] = b.a_ft;
    bkb[j] = b.kb;
    bkc[j] = b.kc;
  }
  if (!WAIT) q0ld = qring0()[qh[0] & qmask];
  // wait for these loads here: otherwise the first use inside the loop would
  // carry a wait that runs on every iteration
#pragma unroll
  for (int j = 0; j < MT; ++j) {
    fa[j] = opaque(fa[j]);
    fadm[j] = opaque(fadm[j]);
    ba[j] = opaque(ba[j]);
    bkb[j] = opaque(bkb[j]);
    bkc[j] = opaque(bkc[j]);
  }

  // ---- ring operations ------------------------------------------------------
  // Operations with a compile-time type index j (inside unrolled loops).
  auto dpush = [&](int j, double a_ft, uint32_t kb, uint32_t kc) __attribute__((always_inline)) {
    DRec rec;
    rec.a_ft = a_ft;
    rec.kb = kb;
    rec.kc = kc;
    dring(j)[dt[j] & dmask[j]] = rec;
    s_win[j][dt[j] % WB][tx] = rec;
    wv[j] = wv[j] < (uint32_t)WB ? wv[j] + 1u : wv[j];
    const uint32_t adm = WAIT ? kc : kb;
    const bool empty = dt[j] == dh[j], second = dt[j] == dh[j] + 1u;
    fa[j] = empty ? a_ft : fa[j];
    fadm[j] = empty ? adm : fadm[j];
    s1pa[j] = second ? a_ft : s1pa[j];
    s1padm[j] = second ? adm : s1padm[j];
    s1src |= (second ? 1u : 0u) << j;
    ba[j] = a_ft;
    bkb[j] = kb;
    bkc[j] = kc;
    dt[j]++;
  };
  // Front pop: the new front is the cached second record.  dpop_front loads
  // the next second record at once (used by a further pop in the same batch
  // or at the next iteration).  With unit thresholds (ONE) a type completes
  // at most one prompt per batch, and dpop_front_cached leaves the reload to
  // the end of the completion phase: no load is then issued inside the
  // phase, where the compiler's waits for a pending load (one in-order
  // counter per wavefront) would also wait for every earlier memory
  // operation.
  auto dpop_front_cached = [&](int j) __attribute__((always_inline)) {
    dh[j]++;
    const bool pushed = (s1src >> j) & 1u;
    fa[j] = pushed ? s1pa[j] : s1a[j];
    fadm[j] = pushed ? s1padm[j] : s1adm[j];
    s1src &= ~(1u << j);
  };
  auto dpop_front = [&](int j) __attribute__((always_inline)) {
    dpop_front_cached(j);
    const DRec n = dring(j)[(dh[j] + 1u) & dmask[j]];  // next second record
    s1a[j] = n.a_ft;
    s1adm[j] = WAIT ? n.kc : n.kb;
  };
  // Operations with a lane-dependent type index: every per-type array is
  // read and written through selects (pick / place).
  auto push_wait_dyn = [&](int j, double a_ft) __attribute__((always_inline)) {
    // (flag and head updates are branch-free: stores to different variables
    // in the two arms of a branch get merged into one store through a
    // selected address, which would move both variables to scratch memory)
    const uint32_t h = pick(qh, j), tq = pick(qt, j);
    const bool full = tq - h >= rec_cap;  // the replica stops at its next decision
    flags |= full ? kFlagCap : 0u;
    const bool first = !full && tq == h;
    place_if(qpu, j, first, a_ft);
    qsrc |= (first ? 1u : 0u) << j;
    ((double *)(blk + pick(qoff, j)))[tq & qmask] = a_ft;  // see evict
    place(qt, j, tq + 1u);
  };
  auto push_fcfs = [&](double a_ft, int32_t j, int32_t L) __attribute__((always_inline)) {
    const bool full = qt[0] - qh[0] >= rec_cap;
    flags |= full ? kFlagCap : 0u;
    const bool first = !full && qt[0] == qh[0];
    QRec rec;
    rec.a_ft = a_ft;
    rec.j = j;
    rec.L = L;
    q0pu.a_ft = first ? a_ft : q0pu.a_ft;
    q0pu.j = first ? j : q0pu.j;
    q0pu.L = first ? L : q0pu.L;
    q0src = q0src || first;
    if (!full) qring0()[qt[0] & qmask] = rec;
    qt[0]++;
  };
  auto dpush_dyn = [&](int j, double a_ft, uint32_t kb, uint32_t kc) __attribute__((always_inline)) {
    const uint32_t tq = pick(dt, j);
    DRec rec;
    rec.a_ft = a_ft;
    rec.kb = kb;
    rec.kc = kc;
    ((DRec *)(blk + pick(doff, j)))[tq & pick(dmask, j)] = rec;
    s_win[j][tq % WB][tx] = rec;
    const uint32_t wvj = pick(wv, j);
    place(wv, j, wvj < (uint32_t)WB ? wvj + 1u : wvj);
    const uint32_t h = pick(dh, j);
    const uint32_t adm = WAIT ? kc : kb;
    const bool empty = tq == h, second = tq == h + 1u;
    place_if(fa, j, empty, a_ft);
    place_if(fadm, j, empty, adm);
    place_if(s1pa, j, second, a_ft);
    place_if(s1padm, j, second, adm);
    s1src |= (second ? 1u : 0u) << j;
    place(ba, j, a_ft);
    place(bkb, j, kb);
    place(bkc, j, kc);
    place(dt, j, tq + 1u);
  };
  // LIFO eviction of the back record of deque j (static j): it returns to
  // the tail of its external queue with its first-token flag.
  auto evict = [&](int j) __attribute__((always_inline)) {
    const double ra = ba[j];
    const uint32_t rkb = bkb[j], rkc = bkc[j];
    const uint32_t tq = dt[j] - 1u;
    dt[j] = tq;
    if (tq != dh[j]) {  // the new back record, read from the window
      if (wv[j] < 2u) {
        // rare: not in the window; copy it in from HBM.  The load is consumed
        // inside this branch, so no wait for memory operations (such as the
        // prefetches of this iteration) follows the branch.
        s_win[j][(tq - 1u) % WB][tx] = dring(j)[(tq - 1u) & dmask[j]];
        wv[j] = 2u;  // after the pop below: the new back is valid
      }
      const DRec b = s_win[j][(tq - 1u) % WB][tx];
      ba[j] = b.a_ft;
      bkb[j] = b.kb;
      bkc[j] = b.kc;
    }
    wv[j] = wv[j] > 0u ? wv[j] - 1u : 0u;
    const uint32_t admb = WAIT ? rkc : rkb;
    const uint32_t now = WAIT ? svc[j] : bidx_cur;
    const int32_t stage = (int32_t)(now - admb) + 1;
    const int32_t ch = l[j] + stage;
    Mj[j] -= ch;
    Mres -= ch;
    evicts++;
    etok += stage - 1;
    const bool ft = has_ft(ra);
    pend[j] -= (stage == 1 && !ft) ? 1u : 0u;
    const double a_ft = (ft || stage >= 2) ? with_ft(ra) : ra;
    if (WAIT) {
      const uint32_t h = qh[j], tq2 = qt[j];
      const bool full = tq2 - h >= rec_cap;
      flags |= full ? kFlagCap : 0u;
      const bool first = !full && tq2 == h;
      qpu[j] = first ? a_ft : qpu[j];
      qsrc |= (first ? 1u : 0u) << j;
      // unconditional (no branch): a full queue ends the replica at its next
      // decision and its ring is not read again
      qring(j)[tq2 & qmask] = a_ft;
      qt[j] = tq2 + 1u;
    } else {
      push_fcfs(a_ft, j, lp[j]);
    }
    if constexpr (BULK) fr[j] -= fr[j] > 0u ? 1u : 0u;  // the back was admitted now
  };
  // LIFO eviction of the last k records of deque j (static j, WAIT), all
  // admitted in the current batch: they share the key (batch, type), are at
  // stage 1 with the charge l_j + 1 and lose no decode token, so they leave
  // back first, one after another as single evictions would, and join the
  // tail of queue j in that order with their own first-token flags.
  auto evict_fresh = [&](int j, uint32_t k) __attribute__((always_inline)) {
    const int32_t ch = l[j] + 1;
    const uint32_t h = qh[j], tq2 = qt[j], t0 = dt[j];
    double* qr = qring(j);
    uint32_t nopend = 0;
    double a0 = 0.0;
    for (uint32_t i = 0; i < k; ++i) {
      const uint32_t p = t0 - 1u - i;
      const double a = i < wv[j] ? s_win[j][p % WB][tx].a_ft : dring(j)[p & dmask[j]].a_ft;
      nopend += has_ft(a) ? 0u : 1u;
      a0 = i == 0 ? a : a0;
      // unconditional, as in evict: a full queue ends the replica
      qr[(tq2 + i) & qmask] = a;
    }
    flags |= tq2 + k - h > rec_cap ? kFlagCap : 0u;
    const bool first = tq2 == h;  // the queue was empty: the first one is its head
    qpu[j] = first ? a0 : qpu[j];
    qsrc |= (first ? 1u : 0u) << j;
    qt[j] = tq2 + k;
    const uint32_t tq = t0 - k;
    dt[j] = tq;
    fr[j] -= k;
    wv[j] = wv[j] > k ? wv[j] - k : 0u;
    if (tq != dh[j]) {  // the new back record
      if (wv[j] < 1u) {  // not in the window: copy it in from HBM
        s_win[j][(tq - 1u) % WB][tx] = dring(j)[(tq - 1u) & dmask[j]];
        wv[j] = 1u;
      }
      const DRec b = s_win[j][(tq - 1u) % WB][tx];
      ba[j] = b.a_ft;
      bkb[j] = b.kb;
      bkc[j] = b.kc;
    }
    pend[j] -= nopend;
    Mj[j] -= (int32_t)k * ch;
    Mres -= (int32_t)k * ch;
    evicts += k;
  };

  // ---- arrivals ---------------------------------------------------------------
  // Next exogenous arrival (ties: lowest type); trace mode reads the list.
  auto peek = [&](int &jn) __attribute__((always_inline)) -> double {
    if (trace) {
      if (tridx >= n_trace) {
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

  // Append the pending arrival of type jn (time a) to its external queue and
  // draw that type's next arrival.
  auto take = [&](int jn, double a) __attribute__((always_inline)) {
    if (trace) {
      tridx++;
    } else if (tv) {
      if constexpr (TV) {  // thinning over the candidates in the ring
        uint32_t k = pick(kk, jn) + 1u;
        uint32_t ge = pick(gend, jn);
        const double lamc = pick(lam, jn);
        int cur = s_cur[jn][tx];
        const double tn = next_thinned(k, pick(tnext, jn), s_fmax[jn], s_rt, s_rf[jn], P, cur, flags,
                                       [&](uint32_t kc, double &g, uint32_t &w3) {
                                         if (kc < ge) {
                                           g = s_gap[jn][kc % GR][tx];
                                           w3 = s_w3[jn][kc % GR][tx];
                                         } else {
                                           g = draw_gap(seed, rid, (uint32_t)jn, kc, lamc,
                                                        nullptr, 0, nullptr, &w3);
                                           ge = kc + 1u;
                                         }
                                       });
        s_cur[jn][tx] = (int8_t)cur;
        place(gend, jn, ge);
        place(kk, jn, k);
        place(tnext, jn, tn);
      }
    } else {
      const uint32_t k = pick(kk, jn) + 1u;
      place(kk, jn, k);
      double g;
      if (k < pick(gend, jn)) {
        g = s_gap[jn][k % GR][tx];
      } else {
        g = draw_gap(seed, rid, (uint32_t)jn, k, pick(lam, jn), nullptr, 0, nullptr);
        place(gend, jn, k + 1u);
      }
      place(tnext, jn, pick(tnext, jn) + g);
    }
    arrivals++;
    N++;
    U++;
    if (WAIT)
      push_wait_dyn(jn, a);
    else
      push_fcfs(a, jn, pick(lp, jn));
  };

  bool stopped = (flags & (kFlagCap | kFlagStall)) != 0;
  uint32_t fresh[MT], pendnew[MT], popped[MT];

  for (int64_t it = 0; it < A.horizon && !stopped; ++it) {
    // ---- refill the gap rings, all active lanes together ----------------
    if (!TRACE) {
      const uint64_t act = __ballot(1);
      const int nact = __popcll(act);
      const int wrank = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(act >> 32),
                                                      __builtin_amdgcn_mbcnt_lo((uint32_t)act, 0u));
      // the requests of every type are gathered first and drawn in one pass
      // (fewer passes when several types run low in the same batch)
      int nreq = 0;  // wavefront-uniform
#pragma unroll
      for (int j = 0; j < MT; ++j) {
        if (j >= m) continue;
        const uint32_t avail = gend[j] - kk[j] - 1u;
        if (__ballot(avail < kLow) == 0) continue;
        const bool room = avail <= (uint32_t)(GR - GU);
        const uint64_t need = __ballot(room);
        if (room) {
          const int rk = nreq + (int)__builtin_amdgcn_mbcnt_hi(
                                    (uint32_t)(need >> 32),
                                    __builtin_amdgcn_mbcnt_lo((uint32_t)need, 0u));
          s_req_lane[rk] = (uint8_t)tx;
          s_req_j[rk] = (uint8_t)j;
          s_req_k[rk] = gend[j];
          gend[j] += GU;  // the draws land before the next use
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
            uint32_t w3;
            s_gap[j][k % GR][ln] = draw_gap(s_seed[ln], s_rid[ln], (uint32_t)j, k, s_lamj[j],
                                            nullptr, 0, nullptr, TV ? &w3 : nullptr);
            if constexpr (TV) s_w3[j][k % GR][ln] = w3;
          }
        }
        wave_lds_sync();
      }
    }

    // The prefetched ring records become usable here, with one wait for the
    // loads issued during the previous iteration (their uses below need no
    // further wait).
#pragma unroll
    for (int j = 0; j < MT; ++j) {
      if (WAIT) qld[j] = opaque(qld[j]);
      s1a[j] = opaque(s1a[j]);
      s1adm[j] = opaque(s1adm[j]);
    }
    if (!WAIT) {
      q0ld.a_ft = opaque(q0ld.a_ft);
      q0ld.j = opaque(q0ld.j);
      q0ld.L = opaque(q0ld.L);
    }

    // ---- decision: form a batch or wait for the next arrival ------------
    uint32_t elig = 0;
    for (;;) {
      if (flags & kFlagCap) {
        stopped = true;
        break;
      }
      elig = 0;
      if (WAIT) {
#pragma unroll
        for (int j = 0; j < MT; ++j)
          if (j < m && (nowait ? (qt[j] != qh[j] || dt[j] != dh[j])
                               : (qt[j] - qh[j]) >= (uint32_t)ncap[j]))
            elig |= 1u << j;
      } else {
        uint32_t resident = 0;
#pragma unroll
        for (int j = 0; j < MT; ++j) resident += dt[j] - dh[j];
        if (resident > 0 || qt[0] != qh[0] || part_j >= 0) elig = 1;
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
    const uint32_t bidx = (uint32_t)batches;
    bidx_cur = bidx;
    int64_t tokens = 0, prefill_l = 0;
    int64_t bt_pre = 0;  // per-batch trace: prefill processings
#pragma unroll
    for (int j = 0; j < MT; ++j) fresh[j] = pendnew[j] = 0;
    if (WAIT) {
#pragma unroll
      for (int j = 0; j < MT; ++j) {
        if (!(elig & (1u << j))) continue;
        const uint32_t c = svc[j] + 1u;
        // admissions: n_j (WAIT), at most n_j of those waiting (no-wait)
        const uint32_t waiting = qt[j] - qh[j];
        const int32_t na = nowait ? (waiting < (uint32_t)nth[j] ? (int32_t)waiting : nth[j]) : ncap[j];
        if constexpr (BULK) {
          // a cohort of na records (same batch and service): copied from the
          // queue ring (the cached head, then the records behind it, read KA
          // at a time) into the deque ring and the LDS window; the cached
          // ends of the deque are set once
          const double head = ((qsrc >> j) & 1u) ? qpu[j] : qld[j];
          const double *qr = qring(j);
          DRec *dr = dring(j);
          const uint32_t d0 = dt[j], h0 = qh[j];
          uint32_t nopend = 0;
          double a1 = 0.0, alast = head;
          for (int x = 0; x < na; x += 4) {
            double nx[4];
#pragma unroll
            for (int u = 0; u < 4; ++u)
              nx[u] = (x + u) == 0 ? head : qr[(h0 + (uint32_t)(x + u)) & qmask];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              if (x + u < na) {
                DRec rec;
                rec.a_ft = nx[u];
                rec.kb = bidx;
                rec.kc = c;
                dr[(d0 + (uint32_t)(x + u)) & dmask[j]] = rec;
                s_win[j][(d0 + (uint32_t)(x + u)) % WB][tx] = rec;
                nopend += has_ft(nx[u]) ? 0u : 1u;
                a1 = x + u == 1 ? nx[u] : a1;
                alast = nx[u];
              }
            }
          }
          if (na > 0) {
            qsrc &= ~(1u << j);
            const bool was_empty = d0 == dh[j], was_one = d0 == dh[j] + 1u;
            fa[j] = was_empty ? head : fa[j];
            fadm[j] = was_empty ? c : fadm[j];
            const bool sec = (was_empty && na >= 2) || was_one;
            const double sa = was_one ? head : a1;
            s1pa[j] = sec ? sa : s1pa[j];
            s1padm[j] = sec ? c : s1padm[j];
            s1src |= (sec ? 1u : 0u) << j;
            ba[j] = alast;
            bkb[j] = bidx;
            bkc[j] = c;
            dt[j] = d0 + (uint32_t)na;
            wv[j] = wv[j] + (uint32_t)na < (uint32_t)WB ? wv[j] + (uint32_t)na : (uint32_t)WB;
            qh[j] = h0 + (uint32_t)na;
            qld[j] = qr[qh[j] & qmask];  // the next head
            pendnew[j] += nopend;
          }
        } else {
          // each admission takes the cached head and loads the next one (ONE:
          // at most one admission, and the reload follows all admissions)
          for (int x = 0; x < (ONE ? min(na, 1) : na); ++x) {
            const double a_ft = ((qsrc >> j) & 1u) ? qpu[j] : qld[j];
            qsrc &= ~(1u << j);
            qh[j]++;
            if (!ONE) qld[j] = qring(j)[qh[j] & qmask];  // the next head
            dpush(j, a_ft, bidx, c);
            pendnew[j] += has_ft(a_ft) ? 0u : 1u;
          }
        }
        fresh[j] = (uint32_t)na;
        bt_pre += na;
        tokens += (int64_t)na * l[j] + Mj[j];
        prefill_l += (int64_t)na * l[j];
      }
      if (ONE) {  // reload the heads of the queues that admitted
#pragma unroll
        for (int j = 0; j < MT; ++j)
          if (fresh[j] > 0u) qld[j] = qring(j)[qh[j] & qmask];
      }
    } else if (chunk > 0) {
      // chunked prefill: the partial prompt first, then admissions from the
      // head of the queue, within `chunk` prefill tokens; a chunk charges the
      // prompt's cache after it
      tokens = Mres - part_pp;  // decode residents
      uint32_t p = 0;
      int32_t budget = chunk;
      if (part_j >= 0) {
        bt_pre++;
        const int32_t pl = pick(l, part_j);
        const int32_t cq = min(pl - part_pp, budget);
        budget -= cq;
        const int32_t after = part_pp + cq;
        tokens += after;
        prefill_l += cq;
        if (after == pl) {  // last chunk: a fresh resident of its type
          dpush_dyn(part_j, part_a, bidx, p++);
          place(fresh, part_j, pick(fresh, part_j) + 1u);
          place(pendnew, part_j, pick(pendnew, part_j) + (has_ft(part_a) ? 0u : 1u));
          part_j = -1;
          part_pp = 0;
        } else {
          part_pp = after;
        }
      }
      while (qt[0] != qh[0] && budget > 0) {
        const QRec head = q0src ? q0pu : q0ld;
        const int hj = head.j;
        const int32_t hl = pick(l, hj);
        if (Mres + prefill_l + hl > cap_adm) break;
        qh[0]++;
        q0src = false;
        q0ld = qring0()[qh[0] & qmask];
        const int32_t cq = min(hl, budget);
        budget -= cq;
        tokens += cq;
        prefill_l += cq;
        bt_pre++;
        if (cq == hl) {
          dpush_dyn(hj, head.a_ft, bidx, p++);
          place(fresh, hj, pick(fresh, hj) + 1u);
          place(pendnew, hj, pick(pendnew, hj) + (has_ft(head.a_ft) ? 0u : 1u));
        } else {  // the budget ends inside this prompt
          part_a = head.a_ft;
          part_j = hj;
          part_pp = cq;
        }
      }
    } else {
      tokens = Mres;
      uint32_t p = 0;
      while (qt[0] != qh[0]) {
        const QRec head = q0src ? q0pu : q0ld;
        const int hj = head.j;
        const int64_t hl = pick(l, hj);
        if (Mres + prefill_l + hl > cap_adm) break;
        qh[0]++;
        q0src = false;
        q0ld = qring0()[qh[0] & qmask];
        dpush_dyn(hj, head.a_ft, bidx, p++);
        place(fresh, hj, pick(fresh, hj) + 1u);
        place(pendnew, hj, pick(pendnew, hj) + (has_ft(head.a_ft) ? 0u : 1u));
        prefill_l += hl;
        bt_pre++;
      }
      tokens += prefill_l;
    }

    const int64_t m_launch = (int64_t)Mres + prefill_l;
    if (m_launch > peak) peak = m_launch;
    const double tau = d0 + d1 * (double)tokens;
    const double t_end = t + tau;
    const int64_t N0 = N, U0 = U;

    // ---- arrivals during the batch ------------------------------------
    // This loop and the repair chase dependent LDS reads one event at a time:
    // at raised priority the wavefront issues ahead of the other one on its
    // SIMD (launches of 16 replicas per wavefront run two per SIMD).
    __builtin_amdgcn_s_setprio(2);
    for (;;) {
      if (flags & kFlagCap) break;  // the replica stops at its next decision
      int jn;
      const double ta = peek(jn);
      if (!(ta <= t_end)) break;
      take(jn, ta);
      lat_area += t_end - ta;
      ttft_area += t_end - ta;
    }
    __builtin_amdgcn_s_setprio(0);
    lat_area += (double)N0 * tau;
    ttft_area += (double)U0 * tau;
    mem_area += (double)m_launch * tau;
    busy += tau;
    t = t_end;

    // ---- completion transition ------------------------------------------
    // (per-batch trace: selected prompts and completions of this batch)
    int64_t bt_sel = 0;
    const int64_t bt_comps0 = comps;
    if constexpr (TV) bt_sel = !WAIT && part_j >= 0 ? 1 : 0;
#pragma unroll
    for (int j = 0; j < MT; ++j) popped[j] = 0;
#pragma unroll
    for (int j = 0; j < MT; ++j) {
      const bool served = WAIT ? ((elig >> j) & 1u) != 0 : j < m;
      if (!served) continue;
      if constexpr (TV) bt_sel += dt[j] - dh[j];  // every resident of a served type
      // the stage-1 cohort produces its first tokens
      U -= pend[j];
      pend[j] = pendnew[j];
      // stage reached: WAIT counts services of the type, FCFS counts batches
      const uint32_t now = WAIT ? svc[j] + 1u : bidx;
      if (WAIT) svc[j] = now;
      if (capped) ncap[j] = capt[coff[j] + (int32_t)(now % (uint32_t)(lp[j] + 1))];
      const uint32_t before = (dt[j] - dh[j]) - fresh[j];  // residents at launch
      uint32_t done = 0;
      // completions: processed at stage l'_j (fresh records never qualify)
      auto complete_front = [&]() __attribute__((always_inline)) {
        const double lat = t_end - arrival_of(fa[j]);
        lat_sum += lat;
        __hip_atomic_fetch_add(&hist[hist_bin_idx(edges, s_htab, hidx, lat)], 1u, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        comps++;
        ctok += lp[j];
        N--;
      };
      if constexpr (ONE) {
        // unit thresholds: one admission per service, so at most one resident
        // of the type reaches its last stage in a batch
        if (before > 0u && fadm[j] + (uint32_t)lp[j] == now) {
          complete_front();
          dpop_front_cached(j);
          done = 1;
        }
      } else {
        while (done < before) {
          if (fadm[j] + (uint32_t)lp[j] != now) break;
          complete_front();
          dpop_front(j);
          done++;
        }
      }
      popped[j] = done;
      Mj[j] += (int32_t)(before - done) + (int32_t)fresh[j] * (l[j] + 1) -
               (int32_t)done * (l[j] + lp[j]);
    }
    // ONE: reload the second records of the deques that popped
#pragma unroll
    for (int j = 0; j < MT; ++j) {
      if (ONE && popped[j] > 0u) {
        const DRec n = dring(j)[(dh[j] + 1u) & dmask[j]];
        s1a[j] = n.a_ft;
        s1adm[j] = WAIT ? n.kc : n.kb;
      }
    }
    Mres = WAIT ? 0 : part_pp;
#pragma unroll
    for (int j = 0; j < MT; ++j) Mres += Mj[j];
    if (Mres > peak) peak = Mres;

    // ---- repair: evict the most recently admitted resident ------------
    // (FCFS: a partially prefilled prompt first; it restarts from scratch)
    const int64_t bt_ev0 = evicts;
    if constexpr (BULK) {
#pragma unroll
      for (int j = 0; j < MT; ++j) fr[j] = fresh[j];
    }
    if (!WAIT && part_j >= 0 && Mres > C) {
      Mres -= part_pp;
      evicts++;
      push_fcfs(part_a, part_j, pick(lp, part_j));
      part_j = -1;
      part_pp = 0;
    }
    __builtin_amdgcn_s_setprio(2);
    if constexpr (ONE) {
      // this batch's admissions (at most one per type) hold the largest keys,
      // the type breaking the tie: they go first, highest type first
#pragma unroll
      for (int j = MT - 1; j >= 0; --j)
        if (fresh[j] != 0u && Mres > C) evict(j);
    }
    if constexpr (WAIT && TV) {
      // this batch's cohorts hold the largest keys, the type breaking the
      // tie: they go first, highest type first
#pragma unroll
      for (int j = MT - 1; j >= 0; --j)
        for (uint32_t x = 0; x < fresh[j] && Mres > C; ++x) evict(j);
    }
    if constexpr (BULK) {
      // this batch's cohorts hold the largest keys, the type breaking the
      // tie: they go first, highest type first, each as many at a time as
      // the memory in excess needs
#pragma unroll
      for (int j = MT - 1; j >= 0; --j) {
        if (fr[j] != 0u && Mres > C) {
          const int32_t ch = l[j] + 1;
          const uint32_t need = (uint32_t)((Mres - C + ch - 1) / ch);
          const uint32_t k = need < fr[j] ? need : fr[j];
          if (k == 1u)
            evict(j);
          else
            evict_fresh(j, k);
        }
      }
    }
    while (Mres > C) {
      int jb = -1;
      uint32_t bb = 0, bp = 0;
#pragma unroll
      for (int j = 0; j < MT; ++j) {
        if (j >= m || dt[j] == dh[j]) continue;
        const uint32_t pb = WAIT ? (uint32_t)j : bkc[j];
        if (jb < 0 || bkb[j] > bb || (bkb[j] == bb && pb > bp)) {
          jb = j;
          bb = bkb[j];
          bp = pb;
        }
      }
      if (jb < 0) break;
      // one unrolled body per type, each with static register indices; the
      // lanes of a wavefront mostly evict the same type, so usually one body
      // runs.  Records admitted in this batch leave as many at a time as the
      // memory in excess needs.
#pragma unroll
      for (int j = 0; j < MT; ++j) {
        if (jb != j) continue;
        if constexpr (BULK) {
          if (fr[j] >= 2u) {
            const int32_t ch = l[j] + 1;
            const uint32_t need = (uint32_t)((Mres - C + ch - 1) / ch);
            evict_fresh(j, need < fr[j] ? need : fr[j]);
            continue;
          }
        }
        evict(j);
      }
    }
    __builtin_amdgcn_s_setprio(0);
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
        int64_t w = 0, res = !WAIT && part_j >= 0 ? 1 : 0;
#pragma unroll
        for (int j = 0; j < MT; ++j) {
          if (WAIT || j == 0) w += qt[j] - qh[j];
          res += dt[j] - dh[j];
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
  put_f(A, S_PARTA, r, part_a);
  put_i(A, S_PARTJ, r, part_j);
  put_i(A, S_PARTPP, r, part_pp);
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
    put_i(A, S_LNEXT + j, r, pend[j]);
  }
}

template <int MT, int POL, bool TV, bool ONE>
hipError_t launch_lanes(const KArgs &A, hipStream_t s) {
  // the widest wavefront for this many type slots (known_max_lanes)
  constexpr int kMax = known_max_lanes(MT);
  const dim3 g((A.n_list + 63) / 64);
  if (A.lanes > kMax) return hipErrorInvalidValue;
  if (A.any_trace) {  // arrival-list replay (tests, small jobs): the widest wavefront
    if constexpr (TV) {
      if (A.lanes != kMax) return hipErrorInvalidValue;
      return launch_checked(sim_known_kernel<MT, POL, true, kMax, TV, ONE>, g, s, A);
    } else {
      return hipErrorInvalidValue;  // replays run on the TV kernels
    }
  }
  if constexpr (kMax == 64) {
    if (A.lanes == 64) return launch_checked(sim_known_kernel<MT, POL, false, 64, TV, ONE>, g, s, A);
  }
  if (A.lanes == 32) return launch_checked(sim_known_kernel<MT, POL, false, 32, TV, ONE>, g, s, A);
  if (A.lanes == 16) return launch_checked(sim_known_kernel<MT, POL, false, 16, TV, ONE>, g, s, A);
  if (A.lanes == 8) return launch_checked(sim_known_kernel<MT, POL, false, 8, TV, ONE>, g, s, A);
  return hipErrorInvalidValue;
}

// The unit-threshold kernels exist for constant-rate WAIT only.
template <int MT, int POL, bool TV>
hipError_t launch_mt(const KArgs &A, hipStream_t s) {
  if constexpr (POL == WS_WAIT && !TV) {
    if (A.unit_n) return launch_lanes<MT, POL, TV, true>(A, s);
  }
  return launch_lanes<MT, POL, TV, false>(A, s);
}

template <int POL, bool TV>
hipError_t launch_pol(int max_m, const KArgs &A, hipStream_t s) {
  if (max_m <= 2) return launch_mt<2, POL, TV>(A, s);
  if (max_m <= 3) return launch_mt<3, POL, TV>(A, s);
  if (max_m <= 4) return launch_mt<4, POL, TV>(A, s);
  if (max_m <= 8) return launch_mt<8, POL, TV>(A, s);
  if (max_m <= 16) return launch_mt<16, POL, TV>(A, s);
  return hipErrorInvalidValue;  // the host admits at most WS_MAX_TYPES types
}

}  // namespace
}  // namespace wsim
