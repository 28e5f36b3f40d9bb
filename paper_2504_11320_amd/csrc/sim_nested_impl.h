// sim_nested_impl.h -- simulation kernel for Nested WAIT (arXiv 2504.11320:
// Algorithm 2, Section 5.1; event-driven form Algorithm 4, Appendix B.1;
// coarse segments with heterogeneous prompts, Appendix A).
//
// A group of G lanes (G = 4, 8, 16, 32 or 64, a power of two >= the job's
// types and segments) runs one replica; a 64-lane wavefront holds 64/G
// replicas.  Lane
// g of a group owns request type g (its arrival clock, draw counter and the
// length of its pending arrival) and segment g (its service count, interior
// count and memory, calendar, cohort slots, the cache of its two youngest
// interior prompts, and its boundary queue's ends, memory and back two
// records, in registers: the survivors lane g-1 pushes are handed over by a
// lane shift after the walk).  What a batch does segment by segment -- the
// entering cohorts, the calendar links, the projected state Q+ of the
// pre-launch repair, the completion walk -- runs on the segment lanes at
// once; the sums over segments and types (batch tokens, Q+, the earliest
// arrival, the prefix of segments meeting their thresholds) are group
// reductions with DPP lane permutations inside the 16-lane rows, on the ALU;
// the most recently admitted eviction candidate is found from its position
// alone (a ballot).  Replica-wide scalars (clock, counters, censored areas,
// resident memory) are kept identical in every lane of the group.
//
// Request records live in HBM, in the replica's block of the workspace:
//   - the external queue Q_{1,0} (FIFO ring of 16-byte records);
//   - for segment k >= 2 the resident boundary queue (a ring in admission
//     order: FIFO selection pops the front, LIFO eviction pops the back);
//   - for every segment a ring of cohort slots indexed by the segment's
//     service number modulo delta_k (its number of processing stages).  The
//     prompts that entered the segment at one service form a cohort of at
//     most n_k prompts and share a stage (the stage-cap invariant), so every
//     interior prompt of a served segment is selected.
// A prompt's exit from its segment (completion at its own output length, or
// survival to the next boundary queue at r_k) happens at a known service, so
// each segment keeps a calendar: bucket (service mod delta_k) heads a linked
// list of the prompts that exit at that service.  Cohorts are linked in
// reverse admission order, so a bucket is traversed youngest cohort first and
// in admission order within a cohort: the same (stage, key) order as the
// oracle's selection list.  The completion latencies a segment lane meets are
// buffered in LDS and added to the replica's latency sum in segment order, so
// the floating-point sum takes the oracle's order exactly.
//
// The projected state Q+ of the pre-launch repair (apply the selected moves
// with no early completion) is computed from per-segment counts and the
// prompts still live in the terminal cohort slot (a record with L = 0 has left
// its segment).
//
// Memory handoffs between lanes of one wavefront (a survivor pushed by lane k
// into the boundary queue of segment k+1, a record appended to Q_{1,0} by a
// type lane and read by lane 0) need no hardware fence: the memory operations
// of a wavefront are performed in order.  wave_lds_sync() keeps the compiler
// from reordering them.
#pragma once

#include "sim_common.h"

namespace wsim {
namespace {

// Per-segment constants, staged in LDS.
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
__device__ __forceinline__ QRec qrec_of(uint4 a) {
  QRec q;
  q.a_ft = __longlong_as_double((long long)(((uint64_t)a.y << 32) | a.x));
  q.j = (int32_t)a.z;
  q.L = (int32_t)a.w;
  return q;
}
// A 32-byte record in one round trip: both 16-byte halves issued together.
__device__ __forceinline__ NRec load_nrec(const NRec *p) {
  const uint4 lo = ((const uint4 *)p)[0], hi = ((const uint4 *)p)[1];
  return nrec_of(lo, hi);
}
// A record's type word carries the prompt length with the type, so the
// charges a record implies need no table lookup: (l << 8) | type.
__device__ __forceinline__ int32_t type_word(int32_t l, int32_t j) { return (l << 8) | j; }
__device__ __forceinline__ int32_t plen(int32_t jw) { return jw >> 8; }

// ---------------------------------------------------------- group lanes --
// DPP lane permutations inside 16-lane rows (gfx9 encodings): swap neighbours
// (quad_perm [1,0,3,2]), swap pairs (quad_perm [2,3,0,1]), mirror each half
// row (lane i <-> 7-i), mirror the row (i <-> 15-i).  After the first two a
// lane holds its quad's reduction; the half-row mirror pairs each lane with
// one of the other quad of its 8, the row mirror with one of the other 8 of
// its 16: an all-reduce over groups of 4, 8 or 16 aligned lanes that reads
// no lane outside the group.
constexpr int kDppSwap1 = 0xB1;
constexpr int kDppSwap2 = 0x4E;
constexpr int kDppHalfMirror = 0x141;
constexpr int kDppMirror = 0x140;

template <int CTRL>
__device__ __forceinline__ uint32_t dpp32(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ uint64_t dpp64(uint64_t v) {
  return ((uint64_t)dpp32<CTRL>((uint32_t)(v >> 32)) << 32) | dpp32<CTRL>((uint32_t)v);
}

// Shift by one lane inside the 16-lane rows: row_shl:1 (lane i takes lane
// i+1) and row_shr:1 (lane i takes lane i-1); a row's end lane keeps 0.
constexpr int kDppShl1 = 0x101;
constexpr int kDppShr1 = 0x111;

// Groups of 32 or 64 lanes combine the 16-lane rows with lane-index XOR
// exchanges (16, then 32).
template <int MASK>
__device__ __forceinline__ uint32_t xor32(uint32_t v) {
  return (uint32_t)__shfl_xor((int)v, MASK, 64);
}
template <int MASK>
__device__ __forceinline__ uint64_t xor64(uint64_t v) {
  return ((uint64_t)xor32<MASK>((uint32_t)(v >> 32)) << 32) | xor32<MASK>((uint32_t)v);
}

template <int G, typename Op>
__device__ __forceinline__ uint64_t group_reduce64(uint64_t v, Op op) {
  v = op(v, dpp64<kDppSwap1>(v));
  v = op(v, dpp64<kDppSwap2>(v));
  if constexpr (G >= 8) v = op(v, dpp64<kDppHalfMirror>(v));
  if constexpr (G >= 16) v = op(v, dpp64<kDppMirror>(v));
  if constexpr (G >= 32) v = op(v, xor64<16>(v));
  if constexpr (G >= 64) v = op(v, xor64<32>(v));
  return v;
}
template <int G>
__device__ __forceinline__ int64_t group_sum(int64_t v) {
  return (int64_t)group_reduce64<G>((uint64_t)v, [](uint64_t a, uint64_t b) { return a + b; });
}
template <int G, typename Op>
__device__ __forceinline__ uint32_t group_reduce32(uint32_t v, Op op) {
  v = op(v, dpp32<kDppSwap1>(v));
  v = op(v, dpp32<kDppSwap2>(v));
  if constexpr (G >= 8) v = op(v, dpp32<kDppHalfMirror>(v));
  if constexpr (G >= 16) v = op(v, dpp32<kDppMirror>(v));
  if constexpr (G >= 32) v = op(v, xor32<16>(v));
  if constexpr (G >= 64) v = op(v, xor32<32>(v));
  return v;
}
// Sum of values whose group total fits in 32 bits (per-batch memory changes
// and counts).
template <int G>
__device__ __forceinline__ int32_t group_sum32(int32_t v) {
  return (int32_t)group_reduce32<G>((uint32_t)v, [](uint32_t a, uint32_t b) { return a + b; });
}
template <int G>
__device__ __forceinline__ uint32_t group_or(uint32_t v) {
  return group_reduce32<G>(v, [](uint32_t a, uint32_t b) { return a | b; });
}
template <int G>
__device__ __forceinline__ double group_min(double v) {
  const uint64_t r = group_reduce64<G>((uint64_t)__double_as_longlong(v), [](uint64_t a, uint64_t b) {
    const double x = __longlong_as_double((long long)a), y = __longlong_as_double((long long)b);
    return y < x ? b : a;
  });
  return __longlong_as_double((long long)r);
}
// The value of segment lane k+1 (seg_next) or k-1 (seg_prev) of the group;
// the group's end lanes get values they do not use.
template <int G>
__device__ __forceinline__ uint32_t seg_next(uint32_t v) {
  if constexpr (G <= 16)
    return dpp32<kDppShl1>(v);
  else
    return (uint32_t)__shfl_down((int)v, 1u, G);
}
template <int G>
__device__ __forceinline__ uint32_t seg_prev(uint32_t v) {
  if constexpr (G <= 16)
    return dpp32<kDppShr1>(v);
  else
    return (uint32_t)__shfl_up((int)v, 1u, G);
}
template <int G>
__device__ __forceinline__ uint64_t seg_prev64(uint64_t v) {
  return ((uint64_t)seg_prev<G>((uint32_t)(v >> 32)) << 32) | seg_prev<G>((uint32_t)v);
}

// The group's G bits of a wavefront ballot (bit g = group lane g).
template <int G>
__device__ __forceinline__ uint64_t group_bits(bool pred) {
  const uint64_t b = __ballot(pred);
  if constexpr (G == 64) {
    return b;
  } else {
    return (b >> (threadIdx.x & (64 - G))) & ((1ull << G) - 1ull);
  }
}

// Wait for every outstanding memory operation of the wavefront; also a
// compiler barrier for memory accesses.
__device__ __forceinline__ void wait_memory() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// G: lanes per replica (types and segments per group); TV: jobs with
// time-varying rates are supported (compiled out of the common kernels).
template <int G, bool TV>
__global__ void __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(2))) sim_nested_kernel(KArgs A) {
  constexpr int NR = 64 / G;  // replicas per wavefront
  constexpr int MT = G;       // type slots
  constexpr int LT = G;       // segment slots
  // Inter-arrival gaps and output lengths are drawn ahead of use by the
  // whole wavefront at once into a ring of GR draws per type and replica; a
  // type lane whose ring runs dry draws for itself.  Eight draws keep refill
  // passes (whose table lookups wait for every outstanding memory operation)
  // rare and still leave LDS for two wavefronts per SIMD; the general
  // instantiation (more LDS per draw) and 64-lane groups keep four.
  constexpr int GR = TV || G > 32 ? 4 : 8;
  constexpr int GU = GR / 2;         // draws added per refill
  constexpr uint32_t kLow = GU / 2;  // a ring below this triggers a refill
  // completion latencies buffered per segment lane before they are summed
  constexpr int KL = 8;
  __shared__ double s_gap[MT][GR][NR];
  __shared__ int32_t s_glen[MT][GR][NR];
  constexpr int NP = TV ? kMaxRatePts : 1;
  __shared__ uint32_t s_w3[TV ? MT : 1][TV ? GR : 1][TV ? NR : 1];
  __shared__ RateProfLds<MT, NP> s_prof;
  double(&s_rt)[NP] = s_prof.t;
  double(&s_rf)[MT][NP] = s_prof.f;
  double(&s_fmax)[MT] = s_prof.fmax;
  __shared__ uint64_t s_seed[NR];
  __shared__ uint32_t s_rid[NR];
  // refill requests of one pass: requesting lane, first draw
  __shared__ uint8_t s_req_ln[64];
  __shared__ uint32_t s_req_k[64];
  __shared__ double s_lam[MT];
  __shared__ int32_t s_l[MT], s_lp[MT];
  __shared__ SegConst s_seg[LT];
  // completion latencies of one batch, per segment, in traversal order
  __shared__ double s_lat[LT][KL][NR];
  __shared__ int32_t s_latn[LT][NR];
  __shared__ int32_t s_latdone[LT][NR];
  __shared__ uint16_t s_cdfg[MT][kCdfGuide + 1];
  __shared__ double s_edges[WS_MAX_HIST_EDGES + 1];
  __shared__ uint8_t s_htab[kHistTab];
  __shared__ int s_hsteps;

  const int tx = threadIdx.x;
  const int gl = tx & (G - 1);  // lane in the group: type gl, segment gl
  const int q = tx / G;         // replica slot of the wavefront
  // replica of this group, or -1 for padding (padding only ends a job's
  // wavefront, so group 0 of every wavefront holds a replica)
  const int32_t r32 =
      q < A.lanes ? ((const int32_t *)(A.ws + A.off_list))[(int64_t)blockIdx.x * 64 + q] : -1;
  const int64_t r = r32 < 0 ? 0 : r32;
  // every replica of a wavefront belongs to the same job: its constants are
  // wavefront-uniform
  const uint32_t jix =
      __builtin_amdgcn_readfirstlane(((const uint32_t *)(A.ws + A.off_job_of))[r]);
  const JobDev &J = ((const JobDev *)(A.ws + A.off_jobs))[jix];
  const int m = J.m;
  const int L = J.nseg;
  const int n_hist = J.n_hist;
  const int P = TV ? J.n_rate : 0;  // rate-profile points, 0 for constant rates
  const bool tv = TV && P > 0;
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
      const bool on = k < L;
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
  if (r32 < 0) return;  // padding group: uses nothing of the others
  const uint64_t seed = ((const uint64_t *)(A.ws + A.off_seed))[r];
  const uint32_t rid = ((const uint32_t *)(A.ws + A.off_rid))[r];
  if (gl == 0) {
    s_seed[q] = seed;
    s_rid[q] = rid;
  }

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
  const uint32_t o_q10 = (uint32_t)J.off_q[0];
#define q10 ((QRec *)(blk + opaque(o_q10)))
  uint32_t *hist = (uint32_t *)(A.ws + A.off_hist) + r * (int64_t)A.hist_stride;

  // this lane's type and segment
  const bool is_t = gl < m;
  const int32_t tword = is_t ? type_word(J.l[gl], gl) : 0;  // this lane's type
  const bool is_s = gl < L;
  const int k = gl;
  const SegConst sc = s_seg[gl];
  const int32_t rk = sc.end, nk = sc.n, delta = sc.delta, ent = sc.entry;
  // per-stage caps (Section 6; general instantiation only): the segment's
  // services take the caps of its decode stages r_{k-1}+1..r_k in turn as
  // the size of the entering cohort; n_k, the largest, is the row width of
  // the cohort slots
  const bool capped = TV && J.has_caps != 0;
  const int32_t nrow = nk;
  const int32_t clo = k >= 1 ? ent - 1 : 0;  // r_{k-1}
  const int32_t *capt = (const int32_t *)(A.ws + J.off_caps);
  auto cap_at = [&](uint32_t services) __attribute__((always_inline)) -> int32_t {
    return capped && is_s ? capt[clo + (int32_t)(services % (uint32_t)(rk - clo))] : nk;
  };
  const int32_t rprev = k >= 1 ? ent - 1 : 0;  // r_{k-1}
  const uint64_t dmg = sc.dmagic;
  const uint32_t o_rc = sc.off_rec, o_bk = sc.off_bkt, o_vr = sc.off_v;
#define rc ((NRec *)(blk + opaque(o_rc)))
#define bk ((uint32_t *)(blk + opaque(o_bk)))
#define vr ((NRec *)(blk + opaque(o_vr)))
  const uint32_t vmask = sc.vmask;
  const int32_t n0 = s_seg[0].n;
  // the next segment (survivors of this one join its boundary queue)
  const bool has_next = is_s && k + 1 < L;
  const int kn = has_next ? k + 1 : gl;
  const SegConst scn = s_seg[kn];
  const uint32_t o_vrn = scn.off_v;
#define vrn ((NRec *)(blk + opaque(o_vrn)))
  const uint32_t vmaskn = scn.vmask;

  auto row_of = [&](int j) __attribute__((always_inline)) -> const uint32_t * {
    return (known || cap <= 1) ? nullptr : cdf + (size_t)j * (size_t)(cap - 1);
  };
  const bool use_guide = !known && !trace && cap > 1 && cap <= 65535;
  auto guide_of = [&](int j) __attribute__((always_inline)) -> const uint16_t * {
    return use_guide ? s_cdfg[j] : nullptr;
  };

  // replica-wide scalars, identical in every lane of the group (lat_sum:
  // group lane 0 only)
  double t, lat_area, ttft_area, lat_sum, mem_area, busy;
  int64_t batches, arrivals, comps, ctok, evicts, etok, fallback, btok, peak, idle, Mres, tridx;
  // requests in the system and without a first token (bounded by the rings)
  int32_t N, U, pendft;
  uint32_t flags, qh, qt;
  // type lane: next arrival time, its counter and output length, ring end
  double tn = INFINITY;
  uint32_t kj = 0, gend = 0;
  int32_t Lnj = 1;
  int cur = -1;  // time-varying rates: profile piece of the type's clock
  // segment lane: services, interior prompts and their memory
  uint32_t svc = 0, I = 0;
  int64_t M = 0;
  // segment lane k >= 2 (1-based): its boundary queue's ring ends and memory,
  // and what LIFO eviction needs of its back record and of the record before
  // it (arrival with first-token mark, type word, length): an eviction takes
  // the back and promotes the second at once, and the next second is loaded
  // while the repair goes on
  uint32_t vh = 0, vt = 0;
  int64_t Bk = 0;
  double vba = 0.0, v2a = 0.0;
  int32_t vbj = 0, vbL = 0, v2j = 0, v2L = 0;
  auto set_back = [&](const NRec &b) __attribute__((always_inline)) {
    vba = b.a_ft;
    vbj = b.j;
    vbL = b.L;
  };
  // the record before the back (valid while the queue holds two)
  auto load_second = [&]() __attribute__((always_inline)) {
    const NRec b = load_nrec(vr + ((vt - 2u) & vmask));
    v2a = b.a_ft;
    v2j = b.j;
    v2L = b.L;
  };

  if (!A.resume) {
    t = lat_area = ttft_area = lat_sum = mem_area = busy = 0.0;
    batches = arrivals = comps = ctok = evicts = etok = fallback = btok = peak = idle = 0;
    N = U = Mres = tridx = pendft = 0;
    flags = 0;
    qh = qt = 0;
    if (is_t && !trace) {
      int32_t Lj = 1;
      if (tv) {
        uint32_t k0 = 0;
        uint32_t fl = 0;
        tn = draw_thinned(seed, rid, (uint32_t)gl, k0, 0.0, J.lambda[gl], s_fmax[gl], s_rt,
                          s_rf[gl], P, row_of(gl), cap, &Lj, cur, fl);
        kj = k0;
        flags |= fl;
      } else {
        tn = 0.0 + draw_gap(seed, rid, (uint32_t)gl, 0u, J.lambda[gl], row_of(gl), cap, &Lj,
                            nullptr, guide_of(gl));
      }
      Lnj = known ? J.lp[gl] : (cap <= 1 ? 1 : Lj);
    }
    // flags are replica-wide
    flags = group_or<G>(flags);
    // calendar buckets start empty: each segment's buckets by the whole group
    for (int kk = 0; kk < L; ++kk) {
      uint32_t *b = (uint32_t *)(blk + s_seg[kk].off_bkt);
      for (int x = gl; x < s_seg[kk].delta; x += G) b[x] = kNil;
    }
    for (int b = gl; b < A.hist_stride; b += G) hist[b] = 0;  // whole row, padding included
    if (capped) {  // a cohort smaller than the row leaves records unwritten: none is live
      for (int kk = 0; kk < L; ++kk) {
        NRec *rr = (NRec *)(blk + s_seg[kk].off_rec);
        const int cells = s_seg[kk].delta * s_seg[kk].n;
        for (int x = gl; x < cells; x += G) rr[x].L = 0;
      }
    }
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
    N = (int32_t)slot_i(A, S_N, r);
    U = (int32_t)slot_i(A, S_U, r);
    Mres = slot_i(A, S_MRES, r);
    tridx = slot_i(A, S_TRIDX, r);
    pendft = (int32_t)slot_i(A, S_PENDFT, r);
    flags = (uint32_t)slot_i(A, S_FLAGS, r);
    qh = (uint32_t)slot_i(A, S_QH, r);
    qt = (uint32_t)slot_i(A, S_QT, r);
    if (is_t) {
      tn = slot_f(A, S_TNEXT + gl, r);
      kj = (uint32_t)slot_i(A, S_K + gl, r);
      Lnj = (int32_t)slot_i(A, S_LNEXT + gl, r);
    }
    if (is_s) {
      svc = (uint32_t)slot_i(A, S_KSVC + k, r);
      I = (uint32_t)slot_i(A, S_KI + k, r);
      M = slot_i(A, S_KM + k, r);
      Bk = slot_i(A, S_KB + k, r);
      vh = (uint32_t)slot_i(A, S_KVH + k, r);
      vt = (uint32_t)slot_i(A, S_KVT + k, r);
    }
  }
  gend = kj + 1u;  // draw rings start empty
  // cohort slot of the segment's last service (svc mod delta_k), kept step by
  // step: the next service's slot, its exit buckets and the terminal slot
  // follow from it without a division
  uint32_t xs = is_s ? fastmod(svc, dmg, (uint32_t)delta) : 0u;
  auto slot_after = [&](uint32_t v) __attribute__((always_inline)) -> uint32_t {
    return v + 1u == (uint32_t)delta ? 0u : v + 1u;
  };
  // size of the cohort this segment admits at its next service
  int32_t ncap = cap_at(svc);
  // youngest live interior record of this segment and its index (kNil: not
  // known, found by a scan when next needed); ydead: the index of the last
  // youngest that left (every record entered after it has left too, so the
  // scan for the next one starts just below it; yi still holds it while yidx
  // is kNil)
  uint32_t yidx = kNil, ydead = kNil;
  NRec yi;
  yi.a_ft = 0.0;
  yi.kb = yi.kp = 0;
  yi.j = 0;
  yi.L = 0;
  yi.c = 0;
  yi.next = kNil;
  // the segment's second youngest live interior record and its index (kNil:
  // not known): it takes the youngest's place when that one leaves, so a
  // second eviction in a row waits for no load (the specialised
  // instantiation only: the general one, short of registers, would spill it)
  uint32_t y2idx = kNil;
  NRec y2 = yi;
  if (is_s && k >= 1 && vt != vh) set_back(load_nrec(vr + ((vt - 1u) & vmask)));
  if (is_s && k >= 1 && vt - vh >= 2u) load_second();

  // What the next launch reads first, loaded ahead (see prefetch below).
  uint4 pf_q0 = make_uint4(0u, 0u, 0u, 0u);
  bool pf_q0_ok = false;  // the head was prefetched (the queue was not empty)
  uint32_t bh = kNil;     // head of the bucket served next
  NRec pf_vf = yi;        // front of this segment's boundary queue
  uint2 pf_tr = make_uint2(0u, 0u);  // (j, L) of the terminal slot's record (n_k = 1)
  uint32_t pf_ti = kNil;             // its index

  // ---- arrivals --------------------------------------------------------------
  // The group's next arrival: its time, and its type (ties: the lowest type).
  double tmin = INFINITY;
  int jmin = 0;
  auto next_arrival = [&]() __attribute__((always_inline)) {
    const double v = is_t ? tn : INFINITY;
    tmin = group_min<G>(v);
    const uint64_t b = group_bits<G>(is_t && v == tmin);
    jmin = b != 0 ? __builtin_ctzll(b) : 0;
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

  // Append a record to Q_{1,0}: the counters in every lane, the record by the
  // lane given.
  auto push_q10 = [&](bool writer, double a_ft, int32_t j, int32_t Lr)
                      __attribute__((always_inline)) {
    if (qt - qh >= rec_cap) {
      flags |= kFlagCap;
    } else if (writer) {
      QRec rec;
      rec.a_ft = a_ft;
      rec.j = j;
      rec.L = Lr;
      q10[qt & qmask] = rec;
    }
    qt++;
  };

  // Take the group's pending arrival of type jn at time a.
  auto take = [&](int jn, double a) __attribute__((always_inline)) {
    int32_t Lr = 0;
    bool writer;
    if (trace) {
      Lr = known ? s_lp[jn] : tr_len[tridx];
      tridx++;
      writer = gl == 0;
    } else {
      writer = gl == jn;
      if (writer) {
        Lr = Lnj;
        if (tv) {
          if constexpr (TV) {  // thinning over the candidates in the ring
            uint32_t kk = kj + 1u;
            uint32_t ge = gend;
            int32_t Lj = 1;
            uint32_t fl = 0;
            tn = next_thinned(kk, tn, s_fmax[jn], s_rt, s_rf[jn], P, cur, fl,
                              [&](uint32_t kc, double &g, uint32_t &w3) {
                                if (kc < ge) {
                                  g = s_gap[jn][kc % GR][q];
                                  w3 = s_w3[jn][kc % GR][q];
                                  Lj = s_glen[jn][kc % GR][q];
                                } else {
                                  g = draw_gap(seed, rid, (uint32_t)jn, kc, J.lambda[jn],
                                               row_of(jn), cap, &Lj, &w3);
                                  ge = kc + 1u;
                                }
                              });
            gend = ge;
            kj = kk;
            flags |= fl;
            Lnj = known ? s_lp[jn] : (cap <= 1 ? 1 : Lj);
          }
        } else {
          const uint32_t kk = kj + 1u;
          kj = kk;
          int32_t Lj = 1;
          double g;
          if (kk < gend) {
            g = s_gap[jn][kk % GR][q];
            Lj = s_glen[jn][kk % GR][q];
          } else {
            g = draw_gap(seed, rid, (uint32_t)jn, kk, J.lambda[jn], row_of(jn), cap, &Lj,
                         nullptr, guide_of(jn));
            gend = kk + 1u;
          }
          tn = tn + g;
          Lnj = known ? s_lp[jn] : (cap <= 1 ? 1 : Lj);
        }
      }
      if constexpr (TV) flags = group_or<G>(flags);  // thinning limit
      next_arrival();
    }
    arrivals++;
    N++;
    U++;
    // the writer's type word: its own type's (non-trace), or a lookup (trace)
    push_q10(writer, a, trace ? type_word(s_l[jn], jn) : tword, Lr);
  };

  // ---- evictions -------------------------------------------------------------
  // Most recently admitted live interior prompt of this lane's segment: the
  // newest non-empty cohort slot, its highest live index.  Lane-local;
  // returns the record index or kNil (and caches the record in yi).
  auto youngest_interior = [&]() __attribute__((always_inline)) -> uint32_t {
    if (!is_s || I == 0) return kNil;
    if (yidx != kNil) return yidx;
    // start just below the youngest that left last (its cohort entered at
    // service yi.c, no later cohort has entered since: an entering cohort
    // sets the cache), else at the newest cohort slot
    int32_t back = 0, ifrom = nrow - 1;
    if (ydead != kNil) {
      const uint32_t c0 = yi.c;
      back = (int32_t)(svc - c0);
      ifrom = (int32_t)(ydead - fastmod(c0, dmg, (uint32_t)delta) * (uint32_t)nrow) - 1;
      ifrom = ifrom < nrow - 1 ? ifrom : nrow - 1;  // indices stay inside the cohort slot
    }
    for (; back < delta && (int64_t)svc - back >= 1; ++back, ifrom = nrow - 1) {
      const uint32_t slot = fastmod(svc - (uint32_t)back, dmg, (uint32_t)delta);
      // a record with L = 0 has left the segment (exit or eviction)
      for (int32_t i = ifrom; i >= 0; --i) {
        const uint32_t idx = slot * (uint32_t)nrow + (uint32_t)i;
        const NRec rec = load_nrec(rc + idx);
        if (rec.L != 0) {
          yi = rec;
          yidx = idx;
          return idx;
        }
      }
    }
    return kNil;
  };

  // Evict the most recently admitted prompt among the boundary queues and,
  // if allow_interior is set and none holds a prompt, among the interior of
  // segments [klo, L).  Group-uniform: returns the memory freed (0 if
  // nothing was left).  `boundary` is cleared once the boundary queues are
  // found empty: within one repair they stay empty (evicted prompts go back
  // to the entry queue), so later calls skip that step.
  //
  // Admission order is also position order: a prompt admitted later never
  // stands further along than one admitted earlier (segment 1, boundary
  // queue 2, segment 2, ..., in that order).  A cohort enters a segment from
  // the front of its queue, every cohort of a segment leaves it after the
  // same number of services, and the survivors of one exit join the next
  // queue in admission order; a prompt evicted re-enters with a new key.  So
  // the most recent boundary prompt is the back of the lowest non-empty
  // boundary queue, and the most recent interior prompt of segments >= klo
  // is the youngest of the lowest such segment that holds one: no key
  // comparison across lanes.
  auto evict_lifo = [&](int klo, bool allow_interior, bool &boundary)
                        __attribute__((always_inline)) -> int64_t {
    if (boundary) {
      const bool cand = is_s && k >= 1 && vt != vh;
      const uint64_t cb = group_bits<G>(cand);
      if (cb != 0) {
        const int h = __builtin_ctzll(cb);
        const bool me = gl == h;
        // the victim is the back of boundary queue h: its charge l + r_{h-1}
        // and lost tokens r_{h-1}, from lane h
        const uint64_t cg = group_sum<G>(
            me ? ((uint64_t)(uint32_t)rprev << 32) | (uint32_t)(plen(vbj) + rprev) : 0ull);
        const int64_t ch = (int64_t)(uint32_t)cg, gen = (int64_t)(cg >> 32);
        const double va = vba;
        const int32_t vj = vbj, vL = vbL;
        if (me) {
          vt -= 1u;
          if (vt != vh) {  // the second is the new back
            vba = v2a;
            vbj = v2j;
            vbL = v2L;
            if (vt - vh >= 2u) load_second();
          }
          Bk -= ch;
        }
        Mres -= ch;
        evicts++;
        etok += gen;
        push_q10(me, with_ft(va), vj, vL);  // it has produced r_{h-1} >= 1 tokens
        wave_lds_sync();
        return ch;
      }
      boundary = false;
    }
    if (!allow_interior) return 0;
    // every candidate segment refreshes its cache (the scans' loads overlap,
    // and a later repair that starts at a higher segment finds its youngest
    // known); the victim is the lowest one's
    uint32_t idx = kNil;
    if (k >= klo) idx = youngest_interior();
    const uint64_t ib = group_bits<G>(idx != kNil);
    if (ib == 0) return 0;
    const int w = __builtin_ctzll(ib);
    const bool me = gl == w;
    int32_t ch = 0, gen = 0, dpend = 0;
    const NRec rec = yi;
    bool ft = false;
    if (me) {
      // idx is the segment's youngest live interior record
      if (!TV && y2idx != kNil) {  // the second is the new youngest
        yi = y2;
        yidx = y2idx;
        y2idx = kNil;
      } else {
        yidx = kNil;
        ydead = idx;
      }
      const int32_t stage = ent + (int32_t)(svc - rec.c) + 1;
      ch = plen(rec.j) + stage;
      gen = stage - 1;
      rc[idx].L = 0;  // leaves a hole; the calendar skips it
      if (idx == pf_ti) pf_tr.y = 0u;  // the prefetched terminal record has left
      I -= 1u;
      M -= ch;
      ft = has_ft(rec.a_ft) || stage >= 2;
      if (stage == 1 && !ft) dpend = 1;
    }
    // the victim's charge, lost tokens and first-token state, from its lane
    // (the other lanes hold zeros)
    const uint64_t cg =
        group_sum<G>(((uint64_t)(uint32_t)(gen * 2 + dpend) << 32) | (uint32_t)ch);
    ch = (int32_t)(uint32_t)cg;
    gen = (int32_t)(cg >> 33);
    dpend = (int32_t)(cg >> 32) & 1;
    Mres -= ch;
    evicts++;
    fallback++;
    etok += gen;
    pendft -= dpend;
    push_q10(me, ft ? with_ft(rec.a_ft) : arrival_of(rec.a_ft), rec.j, rec.L);
    wave_lds_sync();
    return ch;
  };

  // Prefetch, right after the completion walk, what the next launch reads
  // first: the head of Q_{1,0}; per segment that can launch next, the head of
  // the calendar bucket served next, the front of its boundary queue and the
  // (type, length) words of the next launch's terminal cohort slot.  A
  // segment k >= 2 can be in the next launch only if its boundary queue
  // holds n_k prompts now (the repair that follows can only remove prompts;
  // the front it keeps is the one loaded here, and an interior eviction that
  // empties the terminal slot clears the prefetched length).
  auto prefetch = [&]() __attribute__((always_inline)) {
    pf_q0_ok = qt != qh;
    if (gl == 0 && pf_q0_ok) pf_q0 = ((const uint4 *)q10)[qh & qmask];
    if (is_s && (k == 0 || (int32_t)(vt - vh) >= ncap)) {
      const uint32_t x = svc + 1u;  // the segment's next service
      const uint32_t nx = slot_after(xs);
      bh = bk[nx];
      if (k >= 1) pf_vf = load_nrec(vr + (vh & vmask));
      pf_ti = kNil;
      if (nrow == 1 && delta >= 2 && (int64_t)x - (delta - 1) >= 1) {
        pf_ti = slot_after(nx);  // x - (delta - 1) = x + 1 mod delta
        pf_tr = *(const uint2 *)((const uint8_t *)(rc + pf_ti) + 16);
      }
    }
  };
  bool stopped = (flags & (kFlagCap | kFlagStall)) != 0;
  if (!trace) next_arrival();
  if (!stopped) prefetch();

  for (int64_t it = 0; it < A.horizon && !stopped; ++it) {
    // ---- refill the draw rings, all active lanes together -----------------
    if (!trace) {
      const uint64_t act = __ballot(1);
      const int nact = __popcll(act);
      const int wrank = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(act >> 32),
                                                      __builtin_amdgcn_mbcnt_lo((uint32_t)act, 0u));
      const uint32_t avail = gend - kj - 1u;
      if (__ballot(is_t && avail < kLow) != 0) {
        const bool room = is_t && avail <= (uint32_t)(GR - GU);
        const uint64_t need = __ballot(room);
        if (room) {
          const int rq = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(need >> 32),
                                                        __builtin_amdgcn_mbcnt_lo((uint32_t)need, 0u));
          s_req_ln[rq] = (uint8_t)tx;
          s_req_k[rq] = gend;
          gend += GU;  // read again only after the pass
        }
        const int nreq = __popcll(need);
        wave_lds_sync();
        const int total = nreq * GU;
        for (int base = 0; base < total; base += nact) {
          const int w = base + wrank;
          if (w < total) {
            const int ln = (int)s_req_ln[w / GU];
            const int j = ln & (G - 1), qq = ln / G;
            const uint32_t kk = s_req_k[w / GU] + (uint32_t)(w % GU);
            int32_t Lj = 1;
            uint32_t w3;
            s_gap[j][kk % GR][qq] = draw_gap(s_seed[qq], s_rid[qq], (uint32_t)j, kk, s_lam[j],
                                             row_of(j), cap, &Lj, TV ? &w3 : nullptr, guide_of(j));
            s_glen[j][kk % GR][qq] = Lj;
            if constexpr (TV) s_w3[j][kk % GR][qq] = w3;
          }
        }
        wave_lds_sync();
      }
    }

    // ---- decision: largest prefix of segments meeting their thresholds -----
    int kmax = 0;
    for (;;) {
      if (flags & kFlagCap) {
        stopped = true;
        break;
      }
      const bool ok = gl == 0 ? (int64_t)(qt - qh) >= (capped ? ncap : n0)
                              : (is_s && (int32_t)(vt - vh) >= ncap);
      const uint64_t okb = group_bits<G>(ok);
      if (okb & 1u) {
        kmax = __builtin_ctzll(~okb);  // lanes >= L never meet it
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
      for (;;) {  // every arrival at this instant joins before the next decision
        if (flags & kFlagCap) break;
        int j2;
        const double a2 = peek(j2);
        if (a2 != ta) break;
        take(j2, a2);
      }
      idle++;
      wave_lds_sync();
    }
    if (stopped) break;

    // ---- launch: entering cohorts, calendar links, batch tokens -----------
    const bool served = is_s && k < kmax;
    const uint32_t x = svc + 1u;
    int64_t tok = 0, sel = 0;
    int32_t pre_l = 0, pend_new = 0, dplus = 0;
    int32_t eB = 0, eM = 0;
    uint32_t eI = 0;
    // n_k = 1: the entering record is stored only at the completion step, so
    // the launch never waits for the bucket head it links to; the walk's
    // first record (the head prefetched for this service) is loaded at once
    NRec pend = yi;
    uint32_t pend_idx = kNil;
    const uint32_t bh0 = bh;
    NRec crec0 = yi;
    const bool pre_ok = served && nrow == 1 && bh0 != kNil;
    // the walk's first record, loaded now: the walk waits for it last, and
    // with the boundary queues' back records and each segment's two youngest
    // interior records at hand the repair seldom waits for a load of its own
    // (memory operations complete in issue order); the pre-launch repair
    // leaves the served segments' records alone
    if (pre_ok) crec0 = load_nrec(rc + bh0);
    // prompts entering segment 1 now (the cap of its service)
    const int32_t n0c = capped ? __shfl(ncap, 0, G) : n0;
    if (served) {
      const uint32_t slot = slot_after(xs);
      tok = M;  // every interior prompt is processed at its stage
      sel = (int64_t)I + ncap;
      uint32_t suml = 0;
      // link in reverse selection order: traversal is then in key order
      for (int32_t i = ncap - 1; i >= 0; --i) {
        NRec e;
        if (k == 0) {
          QRec qr;
          if (i == 0 && pf_q0_ok)
            qr = qrec_of(pf_q0);  // the head, prefetched
          else
            qr = q10[(qh + (uint32_t)i) & qmask];
          e.a_ft = qr.a_ft;
          e.j = qr.j;
          e.L = qr.L;
          tok += plen(qr.j);
          pre_l += plen(qr.j);
          if (!has_ft(qr.a_ft)) pend_new++;
        } else {
          e = i == 0 ? pf_vf : load_nrec(vr + ((vh + (uint32_t)i) & vmask));
          tok += (int64_t)plen(e.j) + ent;  // processed at stage r_{k-1} + 1
        }
        e.c = x;
        const int32_t pexit = e.L < rk ? e.L : rk;
        // entry stage <= pexit <= r_k: the exit is 0..delta-1 services ahead
        uint32_t b = slot + (uint32_t)(pexit - ent);
        b = b >= (uint32_t)delta ? b - (uint32_t)delta : b;
        const uint32_t idx = slot * (uint32_t)nrow + (uint32_t)i;
        // (the bucket served now was prefetched as bh: the same head)
        e.next = b == slot ? bh : bk[b];
        bk[b] = idx;
        if (b == slot) bh = idx;  // exits at this very service: heads the bucket served now
        if (nrow == 1) {
          pend = e;
          pend_idx = idx;
        } else {
          rc[idx] = e;
        }
        if (i == ncap - 1) {  // the cohort's last record is the segment's youngest
          if constexpr (!TV) {
            y2 = yi;  // the youngest so far is second (a cohort of one)
            y2idx = yidx;
          }
          yi = e;
          yidx = idx;
        } else if (!TV && i == ncap - 2) {  // the cohort's record before it is second
          y2 = e;
          y2idx = idx;
        }
        const int32_t le = plen(e.j);
        suml += (uint32_t)le;
        // what the completion step does with the entering prompts
        if (k > 0) eB += le + rprev;
        if (pexit > ent) {
          eI += 1u;
          eM += le + ent + 1;
        }
      }
      if (k > 0) vh += (uint32_t)ncap;  // still charged in Bk until the completion
      // projected change of the segment's memory (no early completion)
      if (delta >= 2) {
        uint32_t T = 0, Tl = 0;
        if ((int64_t)x - (delta - 1) >= 1) {
          // the terminal cohort slot: its prompts still in the segment
          if (nrow == 1) {  // prefetched
            const int32_t trL = (int32_t)pf_tr.y, trj = (int32_t)pf_tr.x;
            T = trL != 0 ? 1u : 0u;
            Tl = trL != 0 ? (uint32_t)plen(trj) : 0u;
          } else {
            const uint32_t ts = slot_after(slot);  // x - (delta - 1) = x + 1 mod delta
            for (int32_t i = 0; i < nrow; ++i) {
              // j and L (the second half's first two words) in one load
              const uint2 jl = *(const uint2 *)((const uint8_t *)(rc + ts * (uint32_t)nrow +
                                                                  (uint32_t)i) + 16);
              const bool live = (int32_t)jl.y != 0;
              T += live ? 1u : 0u;
              Tl += live ? (uint32_t)plen((int32_t)jl.x) : 0u;
            }
          }
        }
        dplus = (int32_t)I - (int32_t)T;
        if (k == L - 1) dplus -= (int32_t)Tl + (int32_t)T * rk;
        if (k == 0)
          dplus += (int32_t)suml + ncap;  // prefills land at stage 1
        else
          dplus += 2 * ncap;            // l + r_{k-1} -> l + r_{k-1} + 2
      } else {                          // entering prompts are processed at r_k
        if (k < L - 1)
          dplus = ncap;                 // l + r_{k-1} -> l + r_k
        else
          dplus = -((int32_t)suml + ncap * rprev);
      }
    }
    const int64_t tokens = group_sum<G>(tok);
    const int64_t prefill_l = group_sum32<G>(pre_l);
    pend_new = group_sum32<G>(pend_new);
    int64_t mplus = Mres + group_sum32<G>(dplus);
    int64_t bt_sel = 0;
    if constexpr (TV) bt_sel = group_sum<G>(sel);
    qh += (uint32_t)n0c;
    const int64_t bt_ev0 = evicts;
    wave_lds_sync();

    // ---- pre-launch repair on the projected state ----------------------------
    // The repairs and the walk chase dependent loads: at raised priority the
    // wavefront issues ahead of the other one on its SIMD, so each of its
    // next loads leaves sooner.
    __builtin_amdgcn_s_setprio(2);
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
    __builtin_amdgcn_s_setprio(0);
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
    wave_lds_sync();

    // ---- completion transition, every served segment at once ----------------
    // the stage-1 cohort produces its first tokens
    U -= pendft;
    pendft = pend_new;
    int64_t Mk = M, dctok = 0;
    int32_t dM = 0, dcomp = 0;
    uint32_t Ik = I, lflags = 0;
    uint32_t node = kNil;
    if (pend_idx != kNil) rc[pend_idx] = pend;  // the entering record (n_k = 1)
    if (served) {
      svc = x;
      if (capped) ncap = cap_at(svc);  // the cap of the next service
      Mk = M + (int64_t)I + eM;  // every interior prompt advances
      Ik = I + eI;
      if (k > 0) {  // entering prompts leave the boundary queue's charge
        Bk -= eB;
        dM -= eB;
      }
      node = bh;
      xs = slot_after(xs);  // the slot of service x
      bk[xs] = kNil;
    }
    wave_lds_sync();
    // Walk the buckets served now.  A lane stops after KL completions until
    // the group's latency sum has taken them: the sum runs over segments in
    // order, each segment's latencies in traversal order.
    // survivors join the back of segment k+1's boundary queue: its ring ends,
    // from lane k+1; what was pushed goes to lane k+1 after the walk
    const uint32_t vtn = seg_next<G>(vt), vhn = seg_next<G>(vh);
    uint32_t npush = 0;
    int32_t bpush = 0;
    NRec vlast = yi;
    NRec crec = yi;
    if (node != kNil) {
      if (node == pend_idx)
        crec = pend;
      else if (pre_ok && node == bh0)
        crec = crec0;
      else
        crec = load_nrec(rc + node);
    }
    __builtin_amdgcn_s_setprio(2);  // the walk (see the pre-launch repair)
    int32_t nbuf = 0;
    // a bucket lists at most the segment's delta_k * n_k records: a longer
    // walk could only follow a corrupted link, so it stops the replica
    uint32_t steps = 0;
    const uint32_t max_steps = (uint32_t)delta * (uint32_t)nrow;
    for (;;) {
      while (node != kNil && nbuf < KL) {
        if (++steps > max_steps) {
          lflags |= kFlagCap;
          node = kNil;
          break;
        }
        const NRec rec = crec;
        const uint32_t nxt = rec.next;
        if (nxt != kNil) {  // one node ahead
          if (pre_ok && nxt == bh0)
            crec = crec0;
          else
            crec = load_nrec(rc + nxt);
        }
        if (rec.L != 0) {  // holes left by evictions are skipped
          if (!TV && node == y2idx) y2idx = kNil;  // the second leaves
          if (node == yidx) {  // the youngest leaves
            if (!TV && y2idx != kNil) {  // the second is the new youngest
              yi = y2;
              yidx = y2idx;
              y2idx = kNil;
            } else {
              ydead = node;
              yidx = kNil;
            }
          }
          const int64_t le = plen(rec.j);
          const int32_t p = rec.L < rk ? rec.L : rk;
          if (rec.c != x) {  // an interior prompt: it had advanced to p + 1
            Mk -= le + p + 1;
            Ik -= 1u;
          }
          if (rec.L == p) {  // completion at its own output length
            const double lat = t_end - arrival_of(rec.a_ft);
            s_lat[k][nbuf][q] = lat;
            nbuf++;
            __hip_atomic_fetch_add(&hist[hist_bin_idx(edges, s_htab, hidx, lat)], 1u,
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            dcomp++;
            dctok += rec.L;
          } else {  // survivor joins the boundary queue of segment k+1
            NRec v = rec;
            v.a_ft = with_ft(rec.a_ft);
            const uint32_t vp = vtn + npush;
            if (vp - vhn <= vmaskn) {
              vrn[vp & vmaskn] = v;
              npush++;
              vlast = v;
            } else {
              lflags |= kFlagCap;  // bounded by construction; guards the ring
            }
            bpush += (int32_t)(le + rk);
            dM += (int32_t)(le + rk);
          }
          rc[node].L = 0;  // no longer in the segment
        }
        node = nxt;
      }
      // the group's latency sum takes the buffered latencies in segment order,
      // up to the first segment still walking
      if (group_bits<G>(nbuf != 0) != 0) {
        if (is_s) {
          s_latn[k][q] = nbuf;
          s_latdone[k][q] = node == kNil ? 1 : 0;
        }
        wave_lds_sync();
        if (gl == 0) {
          for (int kk = 0; kk < kmax; ++kk) {
            const int32_t nb = s_latn[kk][q];
            for (int32_t i = 0; i < nb; ++i) lat_sum += s_lat[kk][i][q];
            s_latn[kk][q] = 0;
            if (!s_latdone[kk][q]) break;
          }
        }
        wave_lds_sync();
        if (is_s) nbuf = s_latn[k][q];
      }
      if (group_bits<G>(node != kNil || nbuf != 0) == 0) break;
    }
    {
      const uint32_t np = seg_prev<G>(npush);
      const int32_t bp = (int32_t)seg_prev<G>((uint32_t)bpush);
      const double la = __longlong_as_double((long long)seg_prev64<G>(
          (uint64_t)__double_as_longlong(vlast.a_ft)));
      const int32_t lj = (int32_t)seg_prev<G>((uint32_t)vlast.j);
      const int32_t lL = (int32_t)seg_prev<G>((uint32_t)vlast.L);
      if (is_s && k >= 1) {
        Bk += bp;
        if (np != 0) {
          vt += np;
          if (np == 1) {  // the old back (if any) is the second
            v2a = vba;
            v2j = vbj;
            v2L = vbL;
          } else {
            load_second();
          }
          vba = la;
          vbj = lj;
          vbL = lL;
        }
      }
    }
    __builtin_amdgcn_s_setprio(0);
    Mres += group_sum32<G>((int32_t)(Mk - M) + dM);
    const int32_t nc = group_sum32<G>(dcomp);
    comps += nc;
    N -= nc;
    ctok += group_sum<G>(dctok);
    flags |= group_or<G>(lflags);
    M = Mk;
    I = Ik;
    if (Mres > peak) peak = Mres;
    wave_lds_sync();
    prefetch();

    // ---- repair: boundary prompts first, then interior prompts -------------
    __builtin_amdgcn_s_setprio(2);
    bool bnd_post = true;
    while (Mres > C) {
      if (evict_lifo(0, true, bnd_post) == 0) break;
    }
    __builtin_amdgcn_s_setprio(0);
    if constexpr (TV) {
      if (A.btrace != nullptr && batches < A.btrace_cap) {
        const int64_t res = group_sum<G>(
            is_s ? (int64_t)I + (k > 0 ? (int64_t)(vt - vh) : 0) : 0);
        if (gl == 0) {
          BatchRec br;
          br.t_launch = t_end - tau;
          br.tau = tau;
          br.tokens = tokens;
          br.prefills = n0c;
          br.selected = bt_sel;
          br.completions = comps - bt_comps0;
          br.evict_pre = bt_ev1 - bt_ev0;
          br.evict_post = evicts - bt_ev1;
          br.mem_after = Mres;
          br.waiting_after = qt - qh;
          br.resident_after = res;
          br.mplus = mplus;
          ((BatchRec *)A.btrace)[r * A.btrace_cap + batches] = br;
        }
      }
    }
    batches++;
    btok += tokens;
    wave_lds_sync();
  }
  wait_memory();

  // ---- save state ------------------------------------------------------------
  if (gl == 0) {
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
  }
  put_f(A, S_TNEXT + gl, r, is_t ? tn : INFINITY);
  put_i(A, S_K + gl, r, kj);
  put_i(A, S_LNEXT + gl, r, Lnj);
  if (k < kMaxSeg) {  // groups wider than the segment limit: lanes without one
    put_i(A, S_KSVC + k, r, svc);
    put_i(A, S_KI + k, r, I);
    put_i(A, S_KM + k, r, M);
    put_i(A, S_KB + k, r, is_s ? Bk : 0);
    put_i(A, S_KVH + k, r, is_s ? vh : 0);
    put_i(A, S_KVT + k, r, is_s ? vt : 0);
  }
}

template <int G, bool TV>
hipError_t launch_g(const KArgs &A, hipStream_t s) {
  return launch_checked(sim_nested_kernel<G, TV>, dim3(A.n_list / 64), s, A);
}

template <bool TV>
hipError_t launch_nested_k(int max_m, int max_seg, const KArgs &A, hipStream_t s) {
  const int G = nested_group_width(max_m, max_seg);
  // the host's replica list holds 64 / G replicas per wavefront
  if (A.lanes != 64 / G || A.n_list % 64 != 0) return hipErrorInvalidValue;
  if (G == 4) return launch_g<4, TV>(A, s);
  if (G == 8) return launch_g<8, TV>(A, s);
  if (G == 16) return launch_g<16, TV>(A, s);
  if (G == 32) return launch_g<32, TV>(A, s);
  return launch_g<64, TV>(A, s);
}

}  // namespace
}  // namespace wsim
