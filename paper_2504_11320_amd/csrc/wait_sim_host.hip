// wait_sim_host.hip -- host side of the simulator library: validation of the
// model and policy (arXiv 2504.11320, Sections 2, 4 and 5), workspace layout,
// table upload, kernel launches and the C ABI declared in include/wait_sim.h.
#include <algorithm>
#include <array>
#include <cmath>
#include <cstddef>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "sim_common.h"

namespace {

using namespace wsim;

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
  if (J.policy == WS_NESTED_WAIT) {
    for (int k = 0; k < J.nseg; ++k) {
      resident += slot_i(A, S_KI + k, r);
      if (k > 0) resident += slot_i(A, S_KVT + k, r) - slot_i(A, S_KVH + k, r);
    }
  } else if (J.fdist) {
    resident = slot_i(A, S_KI, r);  // live residents (the ring also holds released ones)
  } else {
    for (int j = 0; j < J.m; ++j) resident += slot_i(A, S_DT + j, r) - slot_i(A, S_DH + j, r);
    if (J.policy == WS_FCFS && slot_i(A, S_PARTJ, r) >= 0) resident += 1;  // partial prefill
  }
  oi[9 * R + r] = waiting;
  oi[10 * R + r] = resident;
  const int ff[WS_NF64] = {S_T, S_BUSY, S_LAT, S_TTFT, S_LATSUM, S_MEM};
  for (int f = 0; f < WS_NF64; ++f) of[f * R + r] = slot_f(A, ff[f], r);
  ofl[r] = (uint32_t)slot_i(A, S_FLAGS, r);
}

// ------------------------------------------------------- checkpoints -----
// A checkpoint holds a workspace's live state: every replica's state slots
// and histogram (copied whole, coalesced) and, per replica, the live part of
// its record rings -- the queued records between head and tail, the resident
// deques, and for Nested WAIT the cohort slots and calendar buckets of every
// segment and the boundary queues -- packed back to back.  Ring positions
// follow from the indices in the state slots, so a restore writes each
// record back to its slot.  Layout (all offsets multiples of 256):
//   [header][state slots S_COUNT x R x 8][histograms H x R x 4]
//   [blob offsets R x 8][blobs]
struct CkptHeader {
  uint64_t magic;        // kCkptMagic
  uint64_t fingerprint;  // of the jobs' workspace layout
  uint64_t used;         // bytes of the checkpoint in use (header included)
  uint64_t R;            // replicas
  uint64_t state_off, hist_off, dir_off, blob_off;
  uint64_t pad[24];
};
static_assert(sizeof(CkptHeader) == 256, "checkpoint header layout");
constexpr uint64_t kCkptMagic = 0x31504B434D495357ull;  // "WSIMCKP1"

// The live ring segments of replica r, in a fixed order: f(ring base, index
// mask, log2 of the 4-byte words per record, first index, records).  A ring
// holds at most its capacity (a full queue counts the pushes it could not
// store and flags the replica).
template <typename F>
__device__ __forceinline__ void for_each_segment(const KArgs &A, int64_t r, F f) {
  const uint32_t jix = ((const uint32_t *)(A.ws + A.off_job_of))[r];
  const JobDev &J = ((const JobDev *)(A.ws + A.off_jobs))[jix];
  uint8_t *blk = A.ws + J.off_ring + (uint64_t)(r - J.replica_begin) * J.ring_stride;
  auto hd = [&](int s) { return (uint32_t)slot_i(A, s, r); };
  auto ring = [&](uint8_t *base, int cap_log2, int wl, int sh, int st) {
    const uint32_t cap = 1u << cap_log2, h = hd(sh), n = hd(st) - h;
    f(base, cap - 1u, wl, h, n < cap ? n : cap);
  };
  if (J.policy == WS_NESTED_WAIT) {
    ring(blk + J.off_q[0], J.qcap_log2, 2, S_QH, S_QT);
    for (int k = 0; k < J.nseg; ++k) {
      const uint32_t cells = (uint32_t)J.seg_delta[k] * (uint32_t)J.seg_n[k];
      f(blk + J.off_rec[k], ~0u, 3, 0u, cells);
      f(blk + J.off_bkt[k], ~0u, 0, 0u, (uint32_t)J.seg_delta[k]);
      if (k >= 1) ring(blk + J.off_v[k], J.vcap_log2[k], 3, S_KVH + k, S_KVT + k);
    }
    return;
  }
  if (J.fdist) {  // FCFS in the kernel for per-request lengths
    ring(blk + J.off_q[0], J.qcap_log2, 2, S_QH, S_QT);
    ring(blk + J.off_res, J.qcap_log2, 3, S_DH, S_DT);
    ring(blk + J.off_exit, J.qcap_log2, 0, S_DH, S_DT);
    f(blk + J.off_cal, ~0u, 0, 0u, 1u << J.cal_log2);
    return;
  }
  const bool wait = J.policy == WS_WAIT;
  for (int j = 0; j < (wait ? J.m : 1); ++j)
    ring(blk + J.off_q[j], J.qcap_log2, wait ? 1 : 2, S_QH + j, S_QT + j);
  for (int j = 0; j < J.m; ++j) ring(blk + J.off_d[j], J.dcap_log2[j], 2, S_DH + j, S_DT + j);
}

__device__ __forceinline__ uint64_t packed_bytes(const KArgs &A, int64_t r) {
  uint64_t words = 0;
  for_each_segment(A, r, [&](uint8_t *, uint32_t, int wl, uint32_t, uint32_t n) {
    words += (uint64_t)n << wl;
  });
  return 4ull * words;
}

// Bytes of each replica's packed rings.
__global__ void __launch_bounds__(256) ckpt_size_kernel(KArgs A, uint64_t *bytes) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r < A.R) bytes[r] = packed_bytes(A, r);
}

// Exclusive prefix sum of the blob sizes in place (one workgroup of 1024
// threads, each over a contiguous chunk); writes the header with the total.
__global__ void __launch_bounds__(1024) ckpt_scan_kernel(uint64_t *dir, int64_t R, CkptHeader hdr,
                                                         CkptHeader *out) {
  __shared__ uint64_t part[1024];
  const int tid = threadIdx.x;
  const int64_t chunk = (R + 1023) / 1024;
  const int64_t lo = tid * chunk < R ? tid * chunk : R;
  const int64_t hi = lo + chunk < R ? lo + chunk : R;
  uint64_t sum = 0;
  for (int64_t i = lo; i < hi; ++i) sum += dir[i];
  part[tid] = sum;
  __syncthreads();
  if (tid == 0) {
    uint64_t run = 0;
    for (int i = 0; i < 1024; ++i) {
      const uint64_t v = part[i];
      part[i] = run;
      run += v;
    }
    hdr.used = hdr.blob_off + run;
    *out = hdr;
  }
  __syncthreads();
  uint64_t run = part[tid];
  for (int64_t i = lo; i < hi; ++i) {
    const uint64_t v = dir[i];
    dir[i] = run;
    run += v;
  }
}

// Copy every replica's live ring segments into its blob (to_ckpt) or back
// into the workspace: one wavefront per replica, lanes over 4-byte words.  A
// blob that would end beyond `limit` bytes of blob space is not copied and
// sets *bad (a checkpoint whose blobs do not match its state slots).
__global__ void __launch_bounds__(64) ckpt_copy_kernel(KArgs A, uint8_t *ckpt, const uint64_t *dir,
                                                       uint64_t blob_off, uint64_t limit,
                                                       int to_ckpt, uint32_t *bad) {
  const int64_t r = blockIdx.x;
  if (r >= A.R) return;
  const uint64_t start = dir[r], bytes = packed_bytes(A, r);
  if (start > limit || bytes > limit - start) {
    if (threadIdx.x == 0) atomicOr(bad, 1u);
    return;
  }
  uint32_t *blob = (uint32_t *)(ckpt + blob_off + start);
  uint64_t pos = 0;
  for_each_segment(A, r, [&](uint8_t *base, uint32_t mask, int wl, uint32_t lo, uint32_t n) {
    uint32_t *ring = (uint32_t *)base;
    const uint64_t total = (uint64_t)n << wl;
    const uint32_t wmask = (1u << wl) - 1u;
    for (uint64_t x = threadIdx.x; x < total; x += 64) {
      const uint32_t rec = (uint32_t)(x >> wl), word = (uint32_t)x & wmask;
      uint32_t *cell = ring + ((uint64_t)((lo + rec) & mask) << wl) + word;
      if (to_ckpt)
        blob[pos + x] = *cell;
      else
        *cell = blob[pos + x];
    }
    pos += total;
  });
}

// Write the finished header (after every copy on the stream).
__global__ void ckpt_seal_kernel(CkptHeader hdr, CkptHeader *out) {
  if (threadIdx.x == 0) *out = hdr;
}

// ------------------------------------------------------------- host -----

thread_local std::string g_err;

// Record the message of a failure and return its code.  Never throws: if the
// message cannot be stored the previous one is cleared instead.
int fail(int code, const char *msg) noexcept {
  try {
    g_err = msg;
  } catch (...) {
    g_err.clear();
  }
  return code;
}
int fail(int code, const std::string &msg) noexcept { return fail(code, msg.c_str()); }

// A failure of job `idx`; the message is only built on this (failure) path.
int fail_job(int code, int idx, const char *what) noexcept {
  try {
    g_err = "job " + std::to_string(idx) + ": " + what;
  } catch (...) {
    g_err.clear();
  }
  return code;
}
int fail_job(int code, int idx, const std::string &what) noexcept {
  return fail_job(code, idx, what.c_str());
}

// Body of an extern "C" entry point: no C++ exception crosses the C ABI.
template <class F>
int guarded(F &&body) noexcept {
  try {
    return body();
  } catch (const std::bad_alloc &) {
    return fail(WS_ENOMEM, "host memory allocation failed");
  } catch (...) {
    return fail(WS_EINTERNAL, "internal error (unexpected C++ exception)");
  }
}

// Replicas per 64-lane wavefront.  A replica is a serial chain of events, so
// a wavefront's time per batch is set by latency, not by how many of its lanes
// are busy: when a launch has few replicas they are spread over more
// wavefronts (64, 32, 16 or 8 per wavefront; Nested WAIT 32 down to 4) until
// the launch has at least the target number of wavefronts or reaches the
// smallest width.  The WAIT/FCFS kernel targets one wavefront per SIMD (1024):
// a second one per SIMD gains nothing there; with time-varying rates (longer
// chains of dependent LDS reads per arrival) it targets two per SIMD.  The
// Nested WAIT kernel, which waits on dependent loads of records, targets two
// per SIMD (2048).  A wavefront never has more lanes than the largest job has replicas
// (fewer lanes, less LDS).
#ifndef WS_TARGET_WAVES
#define WS_TARGET_WAVES 1024
#endif
constexpr int64_t kTargetWaves = WS_TARGET_WAVES;
constexpr int64_t kTargetWavesNested = 2 * WS_TARGET_WAVES;

int ceil_log2(uint64_t x) {
  int k = 0;
  while ((1ull << k) < x) ++k;
  return k;
}

uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

// Launch kinds: the policy kinds, and FCFS with drawn lengths.
constexpr int kKinds = 4;
constexpr int kFcfsDist = 3;

struct JobHost {
  JobDev d;
  int64_t reserve_tok;
  uint64_t edges_bytes, cdf_bytes, trace_bytes, rate_bytes, caps_bytes;
  int64_t caps_count;  // per-stage caps in the job's table
};

struct Layout {
  Layout() = default;
  Layout(Layout &&) = default;
  Layout &operator=(Layout &&) = default;
  Layout(const Layout &) = delete;
  Layout &operator=(const Layout &) = delete;
  int64_t R = 0;
  int32_t hist_stride = 1;
  uint64_t off_jobs = 0, off_seed = 0, off_rid = 0, off_job_of = 0,
           off_list = 0, off_tables = 0, off_state = 0, off_hist = 0,
           off_dir = 0, off_rings = 0, total = 0;
  JobHost *jobs = nullptr;     // [n_jobs]: `own`, or storage of the caller
  std::vector<JobHost> own;
  int32_t list_count[kKinds] = {0, 0, 0, 0};
  int32_t lanes[kKinds] = {64, 64, 64, 64};  // replicas per wavefront, per launch
  uint64_t list_off[kKinds] = {0, 0, 0, 0};
  int32_t max_m[kKinds] = {0, 0, 0, 0};
  int32_t max_seg = 0;
};

// The launch (kernel family and replica list) a job runs in: WAIT (and
// WAIT-no-wait), Nested WAIT, FCFS with known output lengths, FCFS with
// lengths drawn per request.
int launch_kind(const ws_job &jb) {
  const ws_policy *p = jb.pol;
  if (p->kind == WS_FCFS && (jb.cfg->out_len == nullptr || jb.cfg->m > WS_MAX_TYPES_KNOWN))
    return kFcfsDist;
  return p->kind == WS_WAIT_NOWAIT ? (int)WS_WAIT : (int)p->kind;
}

int validate_job(const ws_job &jb, int idx, JobHost &H) {
  if (!jb.cfg || !jb.pol) return fail_job(WS_EINVAL, idx, "cfg and pol must be non-NULL");
  if (jb.n < 0) return fail_job(WS_EINVAL, idx, "negative replica count");
  if (jb.n > 0 && !jb.streams) return fail_job(WS_EINVAL, idx, "streams must be non-NULL");
  const ws_config &c = *jb.cfg;
  const ws_policy &p = *jb.pol;
  // WAIT-no-wait runs on the WAIT kernel with a flag
  const int kind = p.kind == WS_WAIT_NOWAIT ? (int)WS_WAIT : (int)p.kind;
  if (c.m < 1 || c.m > WS_MAX_TYPES)
    return fail_job(WS_EINVAL, idx, std::string("m must be in 1..") + std::to_string(WS_MAX_TYPES));
  if (!c.prompt_len || !c.lambda) return fail_job(WS_EINVAL, idx, "prompt_len and lambda required");
  for (int j = 0; j < c.m; ++j) {
    if (c.prompt_len[j] < 1) return fail_job(WS_EINVAL, idx, "prompt lengths must be >= 1");
    if (!(c.lambda[j] >= 0.0) || !std::isfinite(c.lambda[j]))
      return fail_job(WS_EINVAL, idx, "rates must be finite and >= 0");
  }
  if (!(c.d0 > 0.0) || !std::isfinite(c.d0)) return fail_job(WS_EINVAL, idx, "d0 must be > 0");
  if (!(c.d1 >= 0.0) || !std::isfinite(c.d1)) return fail_job(WS_EINVAL, idx, "d1 must be >= 0");
  if (c.C < 1 || c.C > (int64_t(1) << 30)) return fail_job(WS_EINVAL, idx, "C must be in 1..2^30");
  const bool known = c.out_len != nullptr;
  int64_t maxL = 0;
  if (known) {
    for (int j = 0; j < c.m; ++j) {
      if (c.out_len[j] < 1) return fail_job(WS_EINVAL, idx, "output lengths must be >= 1");
      maxL = std::max<int64_t>(maxL, c.out_len[j]);
    }
  } else {
    if (c.out_cap < 1) return fail_job(WS_EINVAL, idx, "out_cap must be >= 1 without out_len");
    maxL = c.out_cap;
    if (c.n_trace == 0) {
      if (c.out_cap > 1 && !c.out_cdf_u32) return fail_job(WS_EINVAL, idx, "out_cdf_u32 required");
      for (int j = 0; j < c.m; ++j)
        for (int s = 1; s + 1 < c.out_cap; ++s)
          if (c.out_cdf_u32[(size_t)j * (c.out_cap - 1) + s] <
              c.out_cdf_u32[(size_t)j * (c.out_cap - 1) + s - 1])
            return fail_job(WS_EINVAL, idx, "CDF table rows must be nondecreasing");
    }
  }
  if (c.n_hist < 0 || c.n_hist > WS_MAX_HIST_EDGES)
    return fail_job(WS_EINVAL, idx, "n_hist out of range");
  if (c.n_hist > 0) {
    if (!c.hist_edges) return fail_job(WS_EINVAL, idx, "hist_edges required");
    for (int b = 0; b < c.n_hist; ++b) {
      if (!std::isfinite(c.hist_edges[b])) return fail_job(WS_EINVAL, idx, "edges must be finite");
      if (b > 0 && !(c.hist_edges[b] > c.hist_edges[b - 1]))
        return fail_job(WS_EINVAL, idx, "edges must be strictly increasing");
    }
  }
  if (c.record_capacity < 16 || c.record_capacity > (1 << 26) ||
      (c.record_capacity & (c.record_capacity - 1)) != 0)
    return fail_job(WS_EINVAL, idx, "record_capacity must be a power of two in 16..2^26");
  if (c.n_trace < 0) return fail_job(WS_EINVAL, idx, "n_trace must be >= 0");
  if (c.n_trace > 0) {
    if (!c.trace_time || !c.trace_type) return fail_job(WS_EINVAL, idx, "trace arrays required");
    if (!known && !c.trace_out_len) return fail_job(WS_EINVAL, idx, "trace_out_len required");
    for (int64_t i = 0; i < c.n_trace; ++i) {
      if (!(c.trace_time[i] >= 0.0) || !std::isfinite(c.trace_time[i]))
        return fail_job(WS_EINVAL, idx, "trace times must be finite and >= 0");
      if (i > 0 && c.trace_time[i] < c.trace_time[i - 1])
        return fail_job(WS_EINVAL, idx, "trace times must be nondecreasing");
      if (c.trace_type[i] < 0 || c.trace_type[i] >= c.m)
        return fail_job(WS_EINVAL, idx, "trace type out of range");
      if (!known && (c.trace_out_len[i] < 1 || c.trace_out_len[i] > c.out_cap))
        return fail_job(WS_EINVAL, idx, "trace output length out of range");
    }
  }
  double fmax[WS_MAX_TYPES] = {};
  if (c.n_rate_pts != 0) {
    if (c.n_rate_pts < 0 || c.n_rate_pts > WS_MAX_RATE_PTS)
      return fail_job(WS_EINVAL, idx, std::string("n_rate_pts must be in 0..") + std::to_string(WS_MAX_RATE_PTS));
    if (c.n_trace > 0) return fail_job(WS_EINVAL, idx, "a rate profile and a trace are exclusive");
    if (!c.rate_t || !c.rate_f) return fail_job(WS_EINVAL, idx, "rate_t and rate_f required");
    const int P = c.n_rate_pts;
    for (int i = 0; i < P; ++i) {
      if (!std::isfinite(c.rate_t[i])) return fail_job(WS_EINVAL, idx, "rate_t must be finite");
      if (i > 0 && !(c.rate_t[i] > c.rate_t[i - 1]))
        return fail_job(WS_EINVAL, idx, "rate_t must be strictly increasing");
    }
    for (int j = 0; j < c.m; ++j) {
      for (int i = 0; i < P; ++i) {
        const double f = c.rate_f[(size_t)j * P + i];
        if (!(f >= 0.0) || !std::isfinite(f))
          return fail_job(WS_EINVAL, idx, "rate_f must be finite and >= 0");
        fmax[j] = std::max(fmax[j], f);
      }
      if (!std::isfinite(c.lambda[j] * fmax[j]))
        return fail_job(WS_EINVAL, idx, "lambda_j * max f_j must be finite");
    }
  }
  int64_t reserve_tok = 0;
  if (kind != WS_FCFS && p.fcfs_chunk != 0)
    return fail_job(WS_EINVAL, idx, "fcfs_chunk applies to FCFS only");
  if (p.stage_caps && !(kind == WS_NESTED_WAIT || p.kind == WS_WAIT))
    return fail_job(WS_EINVAL, idx, "stage_caps apply to WAIT and Nested WAIT only");
  int64_t caps_count = 0;
  // FCFS jobs the kernel for per-request lengths runs (drawn lengths, or
  // more types than the known-length kernels hold)
  const bool fdist = kind == WS_FCFS && (!known || c.m > WS_MAX_TYPES_KNOWN);
  if (kind == WS_WAIT) {
    if (!known) return fail_job(WS_EINVAL, idx, "WAIT needs known output lengths");
    if (c.m > WS_MAX_TYPES_KNOWN && c.n_rate_pts > 0)
      return fail_job(WS_EUNSUPPORTED, idx,
                      "WAIT with more than 16 types takes constant rates only");
    if (!p.n) return fail_job(WS_EINVAL, idx, "thresholds required");
    int64_t fresh = 0;  // memory one batch can admit
    for (int j = 0; j < c.m; ++j) {
      if (p.n[j] < 1) return fail_job(WS_EINVAL, idx, "thresholds must be >= 1");
      fresh += (int64_t)p.n[j] * (c.prompt_len[j] + 1);
    }
    if (fresh >= (int64_t(1) << 29))
      return fail_job(WS_EUNSUPPORTED, idx, "sum_j n_j (l_j + 1) must stay below 2^29");
    if (p.stage_caps) {  // per type j, l'_j + 1 caps >= 1 whose largest is n_j
      for (int j = 0; j < c.m; ++j) {
        int32_t mx = 0;
        for (int32_t st = 0; st <= c.out_len[j]; ++st) {
          const int32_t cp = p.stage_caps[caps_count + st];
          if (cp < 1) return fail_job(WS_EINVAL, idx, "WAIT stage caps must be >= 1");
          mx = std::max(mx, cp);
        }
        if (mx != p.n[j]) return fail_job(WS_EINVAL, idx, "n[j] must be the largest stage cap of type j");
        caps_count += c.out_len[j] + 1;
      }
    }
  } else if (kind == WS_FCFS) {
    if (!(p.fcfs_reserve >= 0.0 && p.fcfs_reserve < 1.0))
      return fail_job(WS_EINVAL, idx, "fcfs_reserve must be in [0,1)");
    reserve_tok = (int64_t)std::ceil(p.fcfs_reserve * (double)c.C);
    if (p.fcfs_chunk < 0) return fail_job(WS_EINVAL, idx, "fcfs_chunk must be >= 0");
    for (int j = 0; j < c.m; ++j)
      if (c.prompt_len[j] > c.C - reserve_tok)
        return fail_job(WS_EINVAL, idx, "a prompt does not fit below the FCFS reserve");
    if (fdist && p.fcfs_chunk != 0)
      return fail_job(WS_EUNSUPPORTED, idx,
                      "chunked prefill needs known output lengths and at most 16 types");
    if (fdist && c.n_rate_pts > 0)
      return fail_job(WS_EUNSUPPORTED, idx,
                      "FCFS with drawn output lengths or more than 16 types takes constant "
                      "rates only");
  } else if (kind == WS_NESTED_WAIT) {
    if (p.L < 1 || p.L > WS_MAX_SEGMENTS) return fail_job(WS_EINVAL, idx, "L out of range");
    if (!p.n || !p.seg_end) return fail_job(WS_EINVAL, idx, "thresholds and seg_end required");
    for (int k = 0; k < p.L; ++k) {
      if (p.n[k] < 1) return fail_job(WS_EINVAL, idx, "thresholds must be >= 1");
      if (p.seg_end[k] < 1 || (k > 0 && p.seg_end[k] <= p.seg_end[k - 1]))
        return fail_job(WS_EINVAL, idx, "seg_end must be strictly increasing and >= 1");
    }
    if (p.seg_end[p.L - 1] != maxL)
      return fail_job(WS_EINVAL, idx, "last segment must end at the largest output length");
    for (int j = 0; j < c.m; ++j)  // records carry the prompt length in 24 bits
      if (c.prompt_len[j] >= (1 << 23))
        return fail_job(WS_EUNSUPPORTED, idx, "Nested WAIT prompt lengths must stay below 2^23");
    if (p.stage_caps) {  // per-stage caps: n_k is the largest of segment k's
      for (int k = 0; k < p.L; ++k) {
        int32_t mx = 0;
        for (int32_t st = k == 0 ? 0 : p.seg_end[k - 1]; st < p.seg_end[k]; ++st) {
          const int32_t cp = p.stage_caps[st];
          if (cp < 0 || (k == 0 && cp < 1))
            return fail_job(WS_EINVAL, idx, "stage caps must be >= 0, and >= 1 in segment 1");
          mx = std::max(mx, cp);
        }
        if (mx != p.n[k])
          return fail_job(WS_EINVAL, idx, "n[k] must be the largest stage cap of segment k");
      }
      caps_count = maxL;
    }
  } else {
    return fail_job(WS_EINVAL, idx, "unknown policy kind");
  }
  for (int j = 0; j < c.m; ++j) {
    const int64_t Lj = known ? c.out_len[j] : c.out_cap;
    if (c.prompt_len[j] + Lj > c.C)
      return fail_job(WS_EINVAL, idx, "a single prompt does not fit in C (atomic feasibility)");
  }

  JobDev &d = H.d;
  std::memset(&d, 0, sizeof(d));
  d.m = c.m;
  d.policy = kind;
  d.nowait = p.kind == WS_WAIT_NOWAIT ? 1 : 0;
  d.chunk = kind == WS_FCFS ? p.fcfs_chunk : 0;
  d.n_hist = c.n_hist;
  d.out_cap = c.out_cap;
  d.nseg = kind == WS_NESTED_WAIT ? p.L : 0;
  d.known = known ? 1 : 0;
  d.qcap_log2 = ceil_log2((uint64_t)c.record_capacity);
  d.rec_cap = c.record_capacity;
  d.d0 = c.d0;
  d.d1 = c.d1;
  d.C = c.C;
  d.reserve_tok = reserve_tok;
  d.n_trace = c.n_trace;
  d.n_rate = c.n_rate_pts;
  for (int j = 0; j < c.m; ++j) {
    d.l[j] = c.prompt_len[j];
    d.lp[j] = known ? c.out_len[j] : c.out_cap;
    // with a rate profile the draws run at the thinning bound lambda_j max f_j
    d.lambda[j] = c.n_rate_pts > 0 ? c.lambda[j] * fmax[j] : c.lambda[j];
    d.rate_fmax[j] = fmax[j];
    d.n[j] = (kind == WS_WAIT) ? p.n[j] : 0;
    uint64_t dcap;
    if (kind == WS_WAIT)  // launch holds <= (l'_j + 1) n_j records
      dcap = (uint64_t)(c.out_len[j] + 1) * (uint64_t)p.n[j];
    else                    // residents of type j charge >= l_j each
      dcap = (uint64_t)(c.C / c.prompt_len[j]) + 2;
    if (kind == WS_NESTED_WAIT) dcap = 2;
    d.dcap_log2[j] = ceil_log2(std::max<uint64_t>(dcap, 2));
  }
  if (kind == WS_NESTED_WAIT) {
    int32_t lmin = c.prompt_len[0];
    for (int j = 1; j < c.m; ++j) lmin = std::min(lmin, c.prompt_len[j]);
    for (int k = 0; k < p.L; ++k) {
      const int32_t prev = k == 0 ? 0 : p.seg_end[k - 1];
      d.seg_end[k] = p.seg_end[k];
      d.seg_n[k] = p.n[k];
      d.seg_entry[k] = k == 0 ? 0 : prev + 1;
      d.seg_delta[k] = p.seg_end[k] - d.seg_entry[k] + 1;
      if (k > 0) {
        // boundary queue k holds <= C/(l_min + r_{k-1}) prompts after any
        // repair, plus one batch of survivors from segment k-1
        const uint64_t vcap = (uint64_t)(c.C / (lmin + prev)) + 2ull * (uint64_t)p.n[k - 1] + 2;
        d.vcap_log2[k] = ceil_log2(vcap);
      }
    }
  }
  H.reserve_tok = reserve_tok;
  H.edges_bytes = align_up(8ull * (uint64_t)std::max(c.n_hist, 1), 256);
  H.cdf_bytes = (!known && c.n_trace == 0 && c.out_cap > 1)
                    ? align_up(4ull * (uint64_t)c.m * (uint64_t)(c.out_cap - 1), 256)
                    : 0;
  H.trace_bytes = c.n_trace > 0 ? align_up(16ull * (uint64_t)c.n_trace, 256) : 0;
  H.rate_bytes = align_up(8ull * (uint64_t)c.n_rate_pts * (uint64_t)(c.m + 1), 256);
  H.caps_count = caps_count;
  H.caps_bytes = p.stage_caps ? align_up(4ull * (uint64_t)caps_count, 256) : 0;
  d.has_caps = p.stage_caps ? 1 : 0;
  // ring block of one replica
  uint64_t off = 0;
  const uint64_t qrec = (kind == WS_WAIT) ? 8 : 16;
  const int nq = (kind == WS_WAIT) ? c.m : 1;
  for (int j = 0; j < nq; ++j) {
    d.off_q[j] = off;
    off += align_up(qrec << d.qcap_log2, 256);
  }
  if (kind == WS_NESTED_WAIT) {
    for (int k = 0; k < p.L; ++k) {
      const uint64_t slots = (uint64_t)d.seg_delta[k];
      d.off_rec[k] = off;
      off += align_up(sizeof(NRec) * slots * (uint64_t)p.n[k], 256);
      d.off_bkt[k] = off;
      off += align_up(4ull * slots, 256);
      if (k > 0) {
        d.off_v[k] = off;
        off += align_up(sizeof(NRec) << d.vcap_log2[k], 256);
      }
    }
  } else if (fdist) {
    // resident ring in admission order, its exit batches, exit calendar
    d.fdist = 1;
    d.cal_log2 = ceil_log2((uint64_t)maxL + 1);
    d.off_res = off;
    off += align_up(sizeof(NRec) << d.qcap_log2, 256);
    d.off_exit = off;
    off += align_up(4ull << d.qcap_log2, 256);
    d.off_cal = off;
    off += align_up(4ull << d.cal_log2, 256);
  } else {
    for (int j = 0; j < c.m; ++j) {
      d.off_d[j] = off;
      off += align_up(16ull << d.dcap_log2[j], 256);
    }
  }
  d.ring_stride = off;
  // ring offsets inside a replica block are kept as 32-bit values on the device
  if (off >= (1ull << 32)) return fail_job(WS_EUNSUPPORTED, idx, "record rings exceed 4 GiB per replica");
  return WS_OK;
}

// Validate the jobs and lay out the workspace.  `storage`: room for n_jobs
// job descriptors supplied by the caller (no host allocation), or null.
int make_layout(const ws_job *jobs, int32_t n_jobs, Layout &Lo, JobHost *storage = nullptr) {
  if (n_jobs < 1 || !jobs) return fail(WS_EINVAL, "need at least one job");
  Lo = Layout();
  if (storage) {
    Lo.jobs = storage;
  } else {
    Lo.own.resize(n_jobs);
    Lo.jobs = Lo.own.data();
  }
  int64_t R = 0;
  int32_t hmax = 0;
  for (int i = 0; i < n_jobs; ++i) {
    int rc = validate_job(jobs[i], i, Lo.jobs[i]);
    if (rc != WS_OK) return rc;
    Lo.jobs[i].d.replica_begin = R;
    R += jobs[i].n;
    hmax = std::max(hmax, jobs[i].cfg->n_hist + 1);
    const int pk = launch_kind(jobs[i]);
    Lo.max_m[pk] = std::max(Lo.max_m[pk], jobs[i].cfg->m);
    if (pk == WS_NESTED_WAIT) Lo.max_seg = std::max(Lo.max_seg, jobs[i].pol->L);
  }
  for (int pk = 0; pk < kKinds; ++pk) {
    auto waves = [&](int lanes) {
      // each job starts a new wavefront: its constants are wavefront-uniform
      int64_t w = 0;
      for (int i = 0; i < n_jobs; ++i)
        if (launch_kind(jobs[i]) == pk) w += (jobs[i].n + lanes - 1) / lanes;
      return w;
    };
    bool any_trace = false;
    for (int i = 0; i < n_jobs; ++i)
      any_trace |= launch_kind(jobs[i]) == pk && jobs[i].cfg->n_trace > 0;
    int32_t nmax = 0;  // largest job: no wavefront needs more lanes
    for (int i = 0; i < n_jobs; ++i)
      if (launch_kind(jobs[i]) == pk) nmax = std::max(nmax, jobs[i].n);
    // the known-length kernels with up to 4 types stop at 32 replicas per
    // wavefront (their 64-lane LDS footprint would leave half of a CU's SIMDs
    // idle), except replays
    int lanes = Lo.max_m[pk] <= 4 && !any_trace ? 32 : known_max_lanes(Lo.max_m[pk]);
    const int min_lanes = 8;
    bool any_tv = false;
    for (int i = 0; i < n_jobs; ++i)
      any_tv |= launch_kind(jobs[i]) == pk && jobs[i].cfg->n_rate_pts > 0;
    const int64_t target = any_tv ? kTargetWavesNested : kTargetWaves;
    if (pk == kFcfsDist) lanes = 64;  // per-lane state in registers and LDS columns
    if (pk == WS_WAIT && Lo.max_m[pk] > WS_MAX_TYPES_KNOWN) lanes = 16;  // LDS columns
    if (pk == WS_NESTED_WAIT) {
      // a group of lanes per replica: 64 / G replicas per wavefront
      lanes = 64 / nested_group_width(Lo.max_m[pk], Lo.max_seg);
    } else if (!any_trace) {  // known-length replays keep the widest
      while (lanes > min_lanes && lanes / 2 >= nmax) lanes /= 2;
      while (lanes > min_lanes && waves(lanes) < target) lanes /= 2;
    }
    Lo.lanes[pk] = lanes;
    const int64_t count = waves(lanes) * 64;
    if (count > INT32_MAX) return fail(WS_EINVAL, "too many replicas");
    Lo.list_count[pk] = (int32_t)count;
  }
  if (R < 1) return fail(WS_EINVAL, "no replicas");
  if (R > (int64_t(1) << 30)) return fail(WS_EINVAL, "too many replicas");
  Lo.R = R;
  Lo.hist_stride = hmax;
  uint64_t off = 256;  // [0, 256): control block (checkpoint header, status)
  Lo.off_jobs = off;
  off = align_up(off + sizeof(JobDev) * (uint64_t)n_jobs, 256);
  Lo.off_seed = off;
  off = align_up(off + 8ull * R, 256);
  Lo.off_rid = off;
  off = align_up(off + 4ull * R, 256);
  Lo.off_job_of = off;
  off = align_up(off + 4ull * R, 256);
  Lo.off_list = off;
  for (int pk = 0; pk < kKinds; ++pk) {
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
    H.d.off_rate = off;
    off += H.rate_bytes;
    H.d.off_caps = off;
    off += H.caps_bytes;
  }
  off = align_up(off, 256);
  Lo.off_state = off;
  off = align_up(off + 8ull * S_COUNT * (uint64_t)R, 256);
  Lo.off_hist = off;
  off = align_up(off + 4ull * (uint64_t)hmax * (uint64_t)R, 256);
  Lo.off_dir = off;  // checkpoints: per-replica blob offsets
  off = align_up(off + 8ull * (uint64_t)R, 256);
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

// Side streams (default priority) on which the launches of a call's second
// and later launch kinds run beside the first: the kinds touch disjoint
// replicas, so they can share the GPU.  Created once per device and kept for
// the life of the process; each call orders them with events of its own.
constexpr int kSide = kKinds - 1;
hipError_t side_streams(hipStream_t out[kSide]) {
  static std::mutex mu;
  static std::map<int, std::array<hipStream_t, kSide>> streams;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(mu);
  auto it = streams.find(dev);
  if (it == streams.end()) {
    std::array<hipStream_t, kSide> made{};
    for (int i = 0; i < kSide; ++i) {
      e = hipStreamCreateWithFlags(&made[i], hipStreamNonBlocking);
      if (e != hipSuccess) {
        for (int x = 0; x < i; ++x) (void)hipStreamDestroy(made[x]);
        return e;
      }
    }
    it = streams.emplace(dev, made).first;
  }
  for (int i = 0; i < kSide; ++i) out[i] = it->second[i];
  return hipSuccess;
}

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

// Write the table image (everything in front of the state region: the
// control block, job descriptors, streams, replica lists and per-job tables)
// into `img` (Lo.off_state bytes).
void build_image(const ws_job *jobs, int32_t n_jobs, const Layout &Lo, uint8_t *img) {
  std::memset(img, 0, Lo.off_state);
  for (int i = 0; i < n_jobs; ++i)
    std::memcpy(img + Lo.off_jobs + sizeof(JobDev) * i, &Lo.jobs[i].d, sizeof(JobDev));
  // replica lists per launch kind: each job starts a new wavefront, whose
  // lanes beyond the launch's width are padding (-1)
  int64_t pos[kKinds] = {0, 0, 0, 0};
  auto put = [&](int pk, int32_t v) {
    std::memcpy(img + Lo.list_off[pk] + 4 * pos[pk], &v, 4);
    pos[pk]++;
  };
  int64_t r = 0;
  for (int i = 0; i < n_jobs; ++i) {
    const ws_job &jb = jobs[i];
    const int pk = launch_kind(jb);
    for (int x = 0; x < jb.n; ++x, ++r) {
      std::memcpy(img + Lo.off_seed + 8 * r, &jb.streams[x].seed, 8);
      std::memcpy(img + Lo.off_rid + 4 * r, &jb.streams[x].replica_id, 4);
      const uint32_t ji = (uint32_t)i;
      std::memcpy(img + Lo.off_job_of + 4 * r, &ji, 4);
      put(pk, (int32_t)r);
      if (pos[pk] % 64 == Lo.lanes[pk])
        while (pos[pk] % 64 != 0) put(pk, -1);
    }
    while (pos[pk] % 64 != 0) put(pk, -1);
    const ws_config &c = *jb.cfg;
    const JobDev &d = Lo.jobs[i].d;
    if (c.n_hist > 0) std::memcpy(img + d.off_edges, c.hist_edges, 8ull * c.n_hist);
    if (Lo.jobs[i].cdf_bytes)
      std::memcpy(img + d.off_cdf, c.out_cdf_u32, 4ull * c.m * (c.out_cap - 1));
    if (c.n_trace > 0) {
      std::memcpy(img + d.off_tr_time, c.trace_time, 8ull * c.n_trace);
      std::memcpy(img + d.off_tr_type, c.trace_type, 4ull * c.n_trace);
      if (c.trace_out_len) std::memcpy(img + d.off_tr_len, c.trace_out_len, 4ull * c.n_trace);
    }
    if (Lo.jobs[i].caps_bytes)
      std::memcpy(img + d.off_caps, jb.pol->stage_caps, 4ull * (uint64_t)Lo.jobs[i].caps_count);
    if (c.n_rate_pts > 0) {  // rate_t [P], then rate_f [m][P]
      std::memcpy(img + d.off_rate, c.rate_t, 8ull * c.n_rate_pts);
      std::memcpy(img + d.off_rate + 8ull * c.n_rate_pts, c.rate_f, 8ull * c.n_rate_pts * c.m);
    }
  }
}

// build_image, then copy the image to the workspace on stream s and wait for
// the copy.  Allocates nothing.
int prepare_image(const ws_job *jobs, int32_t n_jobs, const Layout &Lo, uint8_t *img,
                  void *d_workspace, hipStream_t s) {
  build_image(jobs, n_jobs, Lo, img);
  HIP_TRY(hipMemcpyAsync(d_workspace, img, Lo.off_state, hipMemcpyHostToDevice, s));
  HIP_TRY(hipStreamSynchronize(s));
  return WS_OK;
}

// Orders the launches a call puts on the library's side streams before the
// caller's stream: every side stream that received work is joined back into
// it (an event recorded there, waited for by the caller's stream), also when
// the call fails part-way; if even that fails the side stream is
// synchronised, so no launch of the call outlives its return unordered.
struct SideJoin {
  hipStream_t main = nullptr;
  hipEvent_t fork = nullptr;
  hipStream_t pending[kSide] = {};
  int n_pending = 0;

  static hipError_t join_one(hipStream_t main, hipStream_t side) {
    hipEvent_t ev = nullptr;
    hipError_t e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventRecord(ev, side);
    if (e == hipSuccess) e = hipStreamWaitEvent(main, ev, 0);
    if (ev != nullptr) (void)hipEventDestroy(ev);  // released once it has completed
    if (e != hipSuccess) (void)hipStreamSynchronize(side);
    return e;
  }
  // Join every pending side stream; returns the first error.
  hipError_t join_all() {
    hipError_t first = hipSuccess;
    for (int i = 0; i < n_pending; ++i) {
      const hipError_t e = join_one(main, pending[i]);
      if (first == hipSuccess) first = e;
    }
    n_pending = 0;
    return first;
  }
  ~SideJoin() {
    (void)join_all();
    if (fork != nullptr) (void)hipEventDestroy(fork);
  }
};

// Launch the simulation kernels of every policy kind, then the export of the
// results.  Allocates no device memory; a call with one policy kind creates
// no stream or event.
int advance_impl(const ws_job *jobs, int32_t n_jobs, const Layout &Lo, int64_t horizon,
                 int32_t resume, void *d_workspace, void *d_results, void *d_btrace,
                 int64_t btrace_cap, hipStream_t s) {
  KArgs A = base_args(Lo, d_workspace);
  A.horizon = horizon;
  A.resume = resume ? 1 : 0;
  A.btrace = btrace_cap > 0 ? (uint8_t *)d_btrace : nullptr;
  A.btrace_cap = btrace_cap;
  // a call with several policy kinds runs the second and third kinds on side
  // streams, forked from and joined back into the caller's stream
  int kinds = 0;
  for (int pk = 0; pk < kKinds; ++pk) kinds += Lo.list_count[pk] > 0 ? 1 : 0;
  hipStream_t side[kSide] = {};
  SideJoin sj;
  sj.main = s;
  if (kinds > 1) {
    HIP_TRY(side_streams(side));
    HIP_TRY(hipEventCreateWithFlags(&sj.fork, hipEventDisableTiming));
    HIP_TRY(hipEventRecord(sj.fork, s));
  }
  int launched = 0;
  for (int pk = 0; pk < kKinds; ++pk) {
    if (Lo.list_count[pk] == 0) continue;
    hipStream_t ls = s;
    if (launched > 0) {
      ls = side[launched - 1];
      HIP_TRY(hipStreamWaitEvent(ls, sj.fork, 0));
    }
    KArgs B = A;
    B.off_list = Lo.list_off[pk];
    B.n_list = Lo.list_count[pk];
    B.lanes = Lo.lanes[pk];
    B.any_trace = B.any_tv = B.any_caps = 0;
    B.unit_n = pk == WS_WAIT ? 1 : 0;
    for (int i = 0; i < n_jobs; ++i) {
      if (launch_kind(jobs[i]) != pk) continue;
      if (jobs[i].cfg->n_trace > 0) B.any_trace = 1;
      if (jobs[i].cfg->n_rate_pts > 0) B.any_tv = 1;
      if (jobs[i].pol->stage_caps) B.any_caps = 1;
      if (pk == WS_WAIT)
        for (int j = 0; j < jobs[i].cfg->m; ++j)
          if (jobs[i].pol->n[j] != 1) B.unit_n = 0;
    }
    if (launched > 0) sj.pending[sj.n_pending++] = ls;  // joined even if the launch fails
    hipError_t e = hipSuccess;
    if (pk == WS_NESTED_WAIT)
      e = launch_nested(Lo.max_m[pk], Lo.max_seg, B, ls);
    else if (pk == kFcfsDist)
      e = launch_fcfs_dist(Lo.max_m[pk], B, ls);
    else
      e = pk == WS_WAIT ? launch_known_wait(Lo.max_m[pk], B, ls)
                        : launch_known_fcfs(Lo.max_m[pk], B, ls);
    if (e != hipSuccess) return fail(WS_EDEVICE, std::string("launch: ") + hipGetErrorString(e));
    launched++;
  }
  HIP_TRY(sj.join_all());  // the caller's stream waits for every kind
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

// Checks shared by the entry points that advance a workspace.
int check_advance(const Layout &Lo, int64_t horizon, const void *d_workspace, size_t ws_bytes,
                  const void *d_results, size_t results_bytes) {
  if (horizon < 0) return fail(WS_EINVAL, "horizon must be >= 0");
  if (!d_workspace || !d_results) return fail(WS_EINVAL, "device buffers must be non-NULL");
  if (ws_bytes < Lo.total) return fail(WS_EWORKSPACE, "workspace too small");
  if (results_bytes < results_size(Lo)) return fail(WS_EWORKSPACE, "result buffer too small");
  return WS_OK;
}

// ---------------------------------------------------- checkpoint host --

// Fingerprint of the jobs a checkpoint belongs to: a 64-bit hash of the
// table image (job descriptors with every workspace offset, seeds, replica
// ids, replica lists, tables) and of the layout's sizes.
uint64_t fingerprint(const Layout &Lo, const uint8_t *img) {
  uint64_t h = 0x9E3779B97F4A7C15ull;
  auto mix = [&](uint64_t w) {
    h ^= w;
    h *= 0xBF58476D1CE4E5B9ull;
    h ^= h >> 31;
  };
  for (uint64_t i = 0; i + 8 <= Lo.off_state; i += 8) {
    uint64_t w;
    std::memcpy(&w, img + i, 8);
    mix(w);
  }
  mix((uint64_t)Lo.R);
  mix((uint64_t)Lo.hist_stride);
  mix(Lo.total);
  return h;
}

// The checkpoint's header as the jobs lay it out (used = 0, magic = 0).
CkptHeader ckpt_geometry(const Layout &Lo, uint64_t fp) {
  CkptHeader h;
  std::memset(&h, 0, sizeof(h));
  const uint64_t R = (uint64_t)Lo.R;
  h.fingerprint = fp;
  h.R = R;
  h.state_off = sizeof(CkptHeader);
  h.hist_off = align_up(h.state_off + 8ull * S_COUNT * R, 256);
  h.dir_off = align_up(h.hist_off + 4ull * (uint64_t)Lo.hist_stride * R, 256);
  h.blob_off = align_up(h.dir_off + 8ull * R, 256);
  return h;
}

// Size the checkpoint of the workspace's current state (blocks until known)
// and, when d_out holds it, write it on stream s.
int save_impl(const ws_job *jobs, int32_t n_jobs, const Layout &Lo, void *d_ws, void *d_out,
              size_t out_bytes, size_t *used, hipStream_t s) {
  std::vector<uint8_t> img(Lo.off_state);
  build_image(jobs, n_jobs, Lo, img.data());
  CkptHeader hdr = ckpt_geometry(Lo, fingerprint(Lo, img.data()));
  KArgs A = base_args(Lo, d_ws);
  uint8_t *ws = (uint8_t *)d_ws;
  uint64_t *dir = (uint64_t *)(ws + Lo.off_dir);
  CkptHeader *ctl = (CkptHeader *)ws;  // control block
  const int tb = 256;
  hipLaunchKernelGGL(ckpt_size_kernel, dim3((unsigned)((Lo.R + tb - 1) / tb)), dim3(tb), 0, s, A,
                     dir);
  HIP_TRY(hipGetLastError());
  hipLaunchKernelGGL(ckpt_scan_kernel, dim3(1), dim3(1024), 0, s, dir, (int64_t)Lo.R, hdr, ctl);
  HIP_TRY(hipGetLastError());
  CkptHeader got;
  HIP_TRY(hipMemcpyAsync(&got, ctl, sizeof(got), hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  if (used) *used = (size_t)got.used;
  if (!d_out) return WS_OK;
  if (out_bytes < got.used)
    return fail(WS_EWORKSPACE, "checkpoint buffer too small: the state needs " +
                                   std::to_string(got.used) + " bytes");
  uint8_t *out = (uint8_t *)d_out;
  const uint64_t R = (uint64_t)Lo.R;
  HIP_TRY(hipMemcpyAsync(out + hdr.state_off, ws + Lo.off_state, 8ull * S_COUNT * R,
                         hipMemcpyDeviceToDevice, s));
  HIP_TRY(hipMemcpyAsync(out + hdr.hist_off, ws + Lo.off_hist,
                         4ull * (uint64_t)Lo.hist_stride * R, hipMemcpyDeviceToDevice, s));
  HIP_TRY(hipMemcpyAsync(out + hdr.dir_off, dir, 8ull * R, hipMemcpyDeviceToDevice, s));
  uint32_t *bad = (uint32_t *)(ws + offsetof(CkptHeader, pad));
  hipLaunchKernelGGL(ckpt_copy_kernel, dim3((unsigned)R), dim3(64), 0, s, A, out,
                     (const uint64_t *)dir, hdr.blob_off, got.used - hdr.blob_off, 1, bad);
  HIP_TRY(hipGetLastError());
  got.magic = kCkptMagic;
  hipLaunchKernelGGL(ckpt_seal_kernel, dim3(1), dim3(64), 0, s, got, (CkptHeader *)out);
  HIP_TRY(hipGetLastError());
  return WS_OK;
}

// Prepare the workspace for the jobs and restore the checkpoint d_in into it
// on stream s (blocks until the checks are done).
int load_impl(const ws_job *jobs, int32_t n_jobs, const Layout &Lo, void *d_ws, const void *d_in,
              size_t in_bytes, hipStream_t s) {
  if (in_bytes < sizeof(CkptHeader)) return fail(WS_EINVAL, "checkpoint smaller than its header");
  std::vector<uint8_t> img(Lo.off_state);
  int rc = prepare_image(jobs, n_jobs, Lo, img.data(), d_ws, s);
  if (rc != WS_OK) return rc;
  const CkptHeader want = ckpt_geometry(Lo, fingerprint(Lo, img.data()));
  CkptHeader got;
  HIP_TRY(hipMemcpyAsync(&got, d_in, sizeof(got), hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  if (got.magic != kCkptMagic) return fail(WS_EINVAL, "not a checkpoint (bad magic)");
  if (got.fingerprint != want.fingerprint || got.R != want.R || got.state_off != want.state_off ||
      got.hist_off != want.hist_off || got.dir_off != want.dir_off ||
      got.blob_off != want.blob_off)
    return fail(WS_EINVAL, "checkpoint taken for other jobs (fingerprint or layout differs)");
  if (got.used < got.blob_off || got.used > in_bytes)
    return fail(WS_EINVAL, "checkpoint size does not match its header");
  const uint8_t *in = (const uint8_t *)d_in;
  uint8_t *ws = (uint8_t *)d_ws;
  const uint64_t R = (uint64_t)Lo.R;
  HIP_TRY(hipMemcpyAsync(ws + Lo.off_state, in + got.state_off, 8ull * S_COUNT * R,
                         hipMemcpyDeviceToDevice, s));
  HIP_TRY(hipMemcpyAsync(ws + Lo.off_hist, in + got.hist_off,
                         4ull * (uint64_t)Lo.hist_stride * R, hipMemcpyDeviceToDevice, s));
  KArgs A = base_args(Lo, d_ws);
  uint32_t *bad = (uint32_t *)(ws + offsetof(CkptHeader, pad));  // zeroed by the image
  hipLaunchKernelGGL(ckpt_copy_kernel, dim3((unsigned)R), dim3(64), 0, s, A,
                     const_cast<uint8_t *>(in), (const uint64_t *)(in + got.dir_off),
                     got.blob_off, got.used - got.blob_off, 0, bad);
  HIP_TRY(hipGetLastError());
  uint32_t status = 0;
  HIP_TRY(hipMemcpyAsync(&status, bad, 4, hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  if (status != 0) return fail(WS_EINVAL, "checkpoint blobs do not match its state slots");
  return WS_OK;
}

// ----------------------------------------------- workspace of run_static --

// The workspace of wait_sim_run_static.  Every device the library runs on
// holds its own copy until the process ends.  In host code this name is only
// a stand-in for the symbol: its device address comes from
// hipGetSymbolAddress, once per device (static_workspace()).
__device__ __align__(256) uint8_t scratch[WS_STATIC_WORKSPACE_BYTES];

constexpr int kMaxDevices = 64;

// Device address of `scratch` on the current device, looked up on the first
// call there.
int static_workspace(void **out) {
  static std::mutex mu;
  static void *addr[kMaxDevices] = {};
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(WS_EDEVICE, "device index out of range");
  std::lock_guard<std::mutex> lock(mu);
  if (addr[dev] == nullptr) {
    void *p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (p == nullptr) return fail(WS_EDEVICE, "no device address for the static workspace");
    addr[dev] = p;
  }
  *out = addr[dev];
  return WS_OK;
}

// Host staging of the table image for wait_sim_run_static (its image is at
// most the static workspace's size); used under static_mu.
std::mutex static_mu;
uint8_t static_img[WS_STATIC_WORKSPACE_BYTES];

}  // namespace

// ---------------------------------------------------------------- C ABI --

extern "C" {

const char *wait_sim_last_error(void) { return g_err.c_str(); }

int wait_sim_abi_version(void) { return WS_ABI_VERSION; }

int wait_sim_workspace_bytes(const ws_job *jobs, int32_t n_jobs, size_t *bytes) {
  return guarded([&]() -> int {
    g_err.clear();
    if (!bytes) return fail(WS_EINVAL, "bytes must be non-NULL");
    Layout Lo;
    int rc = make_layout(jobs, n_jobs, Lo);
    if (rc != WS_OK) return rc;
    *bytes = (size_t)Lo.total;
    return WS_OK;
  });
}

int wait_sim_results_bytes(const ws_job *jobs, int32_t n_jobs, size_t *bytes,
                           int32_t *hist_stride) {
  return guarded([&]() -> int {
    g_err.clear();
    if (!bytes) return fail(WS_EINVAL, "bytes must be non-NULL");
    Layout Lo;
    int rc = make_layout(jobs, n_jobs, Lo);
    if (rc != WS_OK) return rc;
    *bytes = (size_t)results_size(Lo);
    if (hist_stride) *hist_stride = Lo.hist_stride;
    return WS_OK;
  });
}

int wait_sim_prepare(const ws_job *jobs, int32_t n_jobs, void *d_workspace,
                     size_t ws_bytes, void *hip_stream) {
  return guarded([&]() -> int {
    g_err.clear();
    Layout Lo;
    int rc = make_layout(jobs, n_jobs, Lo);
    if (rc != WS_OK) return rc;
    if (!d_workspace) return fail(WS_EINVAL, "workspace must be non-NULL");
    if (ws_bytes < Lo.total) return fail(WS_EWORKSPACE, "workspace too small");
    std::vector<uint8_t> img(Lo.off_state);
    return prepare_image(jobs, n_jobs, Lo, img.data(), d_workspace, (hipStream_t)hip_stream);
  });
}

int wait_sim_advance(const ws_job *jobs, int32_t n_jobs, int64_t horizon,
                     int32_t resume, void *d_workspace, size_t ws_bytes,
                     void *d_results, size_t results_bytes, void *hip_stream) {
  return wait_sim_advance_traced(jobs, n_jobs, horizon, resume, d_workspace, ws_bytes,
                                 d_results, results_bytes, nullptr, 0, hip_stream);
}

int wait_sim_advance_traced(const ws_job *jobs, int32_t n_jobs, int64_t horizon,
                            int32_t resume, void *d_workspace, size_t ws_bytes,
                            void *d_results, size_t results_bytes, void *d_btrace,
                            int64_t btrace_cap, void *hip_stream) {
  return guarded([&]() -> int {
    g_err.clear();
    Layout Lo;
    int rc = make_layout(jobs, n_jobs, Lo);
    if (rc != WS_OK) return rc;
    rc = check_advance(Lo, horizon, d_workspace, ws_bytes, d_results, results_bytes);
    if (rc != WS_OK) return rc;
    if (btrace_cap < 0) return fail(WS_EINVAL, "btrace_cap must be >= 0");
    if (btrace_cap > 0 && !d_btrace) return fail(WS_EINVAL, "d_btrace must be non-NULL");
    return advance_impl(jobs, n_jobs, Lo, horizon, resume, d_workspace, d_results, d_btrace,
                        btrace_cap, (hipStream_t)hip_stream);
  });
}

int wait_sim_run_batch(const ws_job *jobs, int32_t n_jobs, int64_t horizon,
                       void *d_workspace, size_t ws_bytes, void *d_results,
                       size_t results_bytes, void *hip_stream) {
  int rc = wait_sim_prepare(jobs, n_jobs, d_workspace, ws_bytes, hip_stream);
  if (rc != WS_OK) return rc;
  return wait_sim_advance(jobs, n_jobs, horizon, 0, d_workspace, ws_bytes, d_results,
                          results_bytes, hip_stream);
}

int wait_sim_save_state(const ws_job *jobs, int32_t n_jobs, void *d_workspace, size_t ws_bytes,
                        void *d_state_out, size_t state_out_bytes, size_t *state_used,
                        void *hip_stream) {
  return guarded([&]() -> int {
    g_err.clear();
    Layout Lo;
    int rc = make_layout(jobs, n_jobs, Lo);
    if (rc != WS_OK) return rc;
    if (!d_workspace) return fail(WS_EINVAL, "workspace must be non-NULL");
    if (ws_bytes < Lo.total) return fail(WS_EWORKSPACE, "workspace too small");
    if (!d_state_out && !state_used)
      return fail(WS_EINVAL, "need a checkpoint buffer or state_used");
    return save_impl(jobs, n_jobs, Lo, d_workspace, d_state_out, state_out_bytes, state_used,
                     (hipStream_t)hip_stream);
  });
}

int wait_sim_load_state(const ws_job *jobs, int32_t n_jobs, void *d_workspace, size_t ws_bytes,
                        const void *d_state_in, size_t state_in_bytes, void *hip_stream) {
  return guarded([&]() -> int {
    g_err.clear();
    Layout Lo;
    int rc = make_layout(jobs, n_jobs, Lo);
    if (rc != WS_OK) return rc;
    if (!d_workspace || !d_state_in) return fail(WS_EINVAL, "device buffers must be non-NULL");
    if (ws_bytes < Lo.total) return fail(WS_EWORKSPACE, "workspace too small");
    return load_impl(jobs, n_jobs, Lo, d_workspace, d_state_in, state_in_bytes,
                     (hipStream_t)hip_stream);
  });
}

int wait_sim_run_batch_ex(const ws_job *jobs, int32_t n_jobs, int64_t horizon,
                          void *d_workspace, size_t ws_bytes, void *d_results,
                          size_t results_bytes, void *hip_stream, const void *d_state_in,
                          size_t state_in_bytes, void *d_state_out, size_t state_out_bytes,
                          size_t *state_used) {
  return guarded([&]() -> int {
    g_err.clear();
    Layout Lo;
    int rc = make_layout(jobs, n_jobs, Lo);
    if (rc != WS_OK) return rc;
    rc = check_advance(Lo, horizon, d_workspace, ws_bytes, d_results, results_bytes);
    if (rc != WS_OK) return rc;
    hipStream_t s = (hipStream_t)hip_stream;
    if (d_state_in) {
      rc = load_impl(jobs, n_jobs, Lo, d_workspace, d_state_in, state_in_bytes, s);
    } else {
      std::vector<uint8_t> img(Lo.off_state);
      rc = prepare_image(jobs, n_jobs, Lo, img.data(), d_workspace, s);
    }
    if (rc != WS_OK) return rc;
    rc = advance_impl(jobs, n_jobs, Lo, horizon, d_state_in ? 1 : 0, d_workspace, d_results,
                      nullptr, 0, s);
    if (rc != WS_OK) return rc;
    if (!d_state_out && !state_used) return WS_OK;
    return save_impl(jobs, n_jobs, Lo, d_workspace, d_state_out, state_out_bytes, state_used, s);
  });
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

int wait_sim_run_static(const ws_config *cfg, const ws_policy *pol, const ws_stream *streams,
                        int32_t n_replicas, int64_t horizon, void *d_results,
                        size_t results_bytes, void *hip_stream) {
  return guarded([&]() -> int {
    g_err.clear();
    ws_job jb;
    jb.cfg = cfg;
    jb.pol = pol;
    jb.streams = streams;
    jb.n = n_replicas;
    JobHost job;  // the layout's descriptor storage: no host allocation
    Layout Lo;
    int rc = make_layout(&jb, 1, Lo, &job);
    if (rc != WS_OK) return rc;
    if (Lo.total > WS_STATIC_WORKSPACE_BYTES)
      return fail(WS_EWORKSPACE,
                  "wait_sim_run_static: these replicas need more workspace than the "
                  "static workspace of WS_STATIC_WORKSPACE_BYTES holds; use wait_sim_run");
    void *ws = nullptr;
    rc = static_workspace(&ws);
    if (rc != WS_OK) return rc;
    rc = check_advance(Lo, horizon, ws, WS_STATIC_WORKSPACE_BYTES, d_results, results_bytes);
    if (rc != WS_OK) return rc;
    hipStream_t s = (hipStream_t)hip_stream;
    std::lock_guard<std::mutex> lock(static_mu);
    rc = prepare_image(&jb, 1, Lo, static_img, ws, s);
    if (rc != WS_OK) return rc;
    return advance_impl(&jb, 1, Lo, horizon, 0, ws, d_results, nullptr, 0, s);
  });
}

}  // extern "C"
