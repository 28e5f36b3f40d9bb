"""Python binding of the C ABI in include/wait_sim.h (argument marshalling only).

Every simulation step runs in the HIP library; this module only converts
workload descriptions into the C structs, allocates device buffers through
PyTorch and passes the current HIP stream.  It raises if the library is
missing instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Sequence

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
# another build of the library (e.g. the sanitizer build) may be named in
# WAIT_SIM_LIB
LIB_PATH = os.environ.get("WAIT_SIM_LIB") or os.path.join(PKG, "libwait_sim.so")

WS_OK, WS_EINVAL, WS_ENOMEM, WS_EDEVICE, WS_EWORKSPACE, WS_EUNSUPPORTED = 0, -1, -2, -3, -4, -5
WS_EINTERNAL = -6
WS_STATIC_WORKSPACE_BYTES = 64 << 20
WS_WAIT, WS_NESTED_WAIT, WS_FCFS, WS_WAIT_NOWAIT = 0, 1, 2, 3
WS_FLAG_CAPACITY, WS_FLAG_STALL, WS_FLAG_OVERFLOW, WS_FLAG_THIN_LIMIT = 1, 2, 4, 8
WS_ABI_VERSION = 4
WS_NI64, WS_NF64 = 12, 6
POLICY = {"wait": WS_WAIT, "nested": WS_NESTED_WAIT, "fcfs": WS_FCFS,
          "wait-nowait": WS_WAIT_NOWAIT}

I64_FIELDS = ["batches", "arrivals", "completions", "completed_tokens",
              "evictions", "evicted_tokens", "fallback_evictions",
              "batch_tokens_sum", "peak_mem", "waiting_end", "resident_end",
              "idle_waits"]
F64_FIELDS = ["t_end", "busy_time", "lat_area", "ttft_area",
              "lat_completed_sum", "mem_area"]


# ws_batch_rec (include/wait_sim.h)
BATCH_REC = np.dtype([("t_launch", np.float64), ("tau", np.float64)] + [
    (f, np.int64) for f in ("tokens", "prefills", "selected", "completions", "evict_pre",
                            "evict_post", "mem_after", "waiting_after", "resident_after",
                            "mplus")])


class WsConfig(C.Structure):
    _fields_ = [
        ("m", C.c_int32), ("prompt_len", C.c_void_p), ("lam", C.c_void_p),
        ("out_len", C.c_void_p), ("out_cap", C.c_int32),
        ("out_cdf_u32", C.c_void_p), ("d0", C.c_double), ("d1", C.c_double),
        ("C", C.c_int64), ("hist_edges", C.c_void_p), ("n_hist", C.c_int32),
        ("record_capacity", C.c_int32), ("trace_time", C.c_void_p),
        ("trace_type", C.c_void_p), ("trace_out_len", C.c_void_p),
        ("n_trace", C.c_int64), ("n_rate_pts", C.c_int32),
        ("rate_t", C.c_void_p), ("rate_f", C.c_void_p),
    ]


class WsPolicy(C.Structure):
    _fields_ = [("kind", C.c_int32), ("n", C.c_void_p), ("L", C.c_int32),
                ("seg_end", C.c_void_p), ("fcfs_reserve", C.c_double),
                ("fcfs_chunk", C.c_int32), ("stage_caps", C.c_void_p)]


class WsStream(C.Structure):
    _fields_ = [("seed", C.c_uint64), ("replica_id", C.c_uint32),
                ("reserved", C.c_uint32)]


class WsJob(C.Structure):
    _fields_ = [("cfg", C.POINTER(WsConfig)), ("pol", C.POINTER(WsPolicy)),
                ("streams", C.c_void_p), ("n", C.c_int32)]


class WaitSimError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"wait_sim error {code}: {msg}")
        self.code = code


_lib = None


def lib():
    """Load the HIP library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with paper_2504_11320_amd/build.py")
        L = C.CDLL(LIB_PATH)
        jp = C.POINTER(WsJob)
        L.wait_sim_workspace_bytes.argtypes = [jp, C.c_int32, C.POINTER(C.c_size_t)]
        L.wait_sim_results_bytes.argtypes = [jp, C.c_int32, C.POINTER(C.c_size_t),
                                             C.POINTER(C.c_int32)]
        L.wait_sim_prepare.argtypes = [jp, C.c_int32, C.c_void_p, C.c_size_t, C.c_void_p]
        L.wait_sim_advance.argtypes = [jp, C.c_int32, C.c_int64, C.c_int32, C.c_void_p,
                                       C.c_size_t, C.c_void_p, C.c_size_t, C.c_void_p]
        L.wait_sim_run.argtypes = [C.POINTER(WsConfig), C.POINTER(WsPolicy), C.c_void_p,
                                   C.c_int32, C.c_int64, C.c_void_p, C.c_size_t,
                                   C.c_void_p, C.c_size_t, C.c_void_p]
        L.wait_sim_run_batch.argtypes = [jp, C.c_int32, C.c_int64, C.c_void_p,
                                         C.c_size_t, C.c_void_p, C.c_size_t, C.c_void_p]
        L.wait_sim_advance_traced.argtypes = [jp, C.c_int32, C.c_int64, C.c_int32,
                                              C.c_void_p, C.c_size_t, C.c_void_p,
                                              C.c_size_t, C.c_void_p, C.c_int64, C.c_void_p]
        L.wait_sim_run_static.argtypes = [C.POINTER(WsConfig), C.POINTER(WsPolicy), C.c_void_p,
                                          C.c_int32, C.c_int64, C.c_void_p, C.c_size_t,
                                          C.c_void_p]
        L.wait_sim_save_state.argtypes = [jp, C.c_int32, C.c_void_p, C.c_size_t, C.c_void_p,
                                          C.c_size_t, C.POINTER(C.c_size_t), C.c_void_p]
        L.wait_sim_load_state.argtypes = [jp, C.c_int32, C.c_void_p, C.c_size_t, C.c_void_p,
                                          C.c_size_t, C.c_void_p]
        L.wait_sim_run_batch_ex.argtypes = [jp, C.c_int32, C.c_int64, C.c_void_p, C.c_size_t,
                                            C.c_void_p, C.c_size_t, C.c_void_p, C.c_void_p,
                                            C.c_size_t, C.c_void_p, C.c_size_t,
                                            C.POINTER(C.c_size_t)]
        L.wait_sim_last_error.restype = C.c_char_p
        L.wait_sim_abi_version.restype = C.c_int
        if L.wait_sim_abi_version() != WS_ABI_VERSION:
            raise RuntimeError(f"{LIB_PATH} has ABI version {L.wait_sim_abi_version()}, "
                               f"this binding needs {WS_ABI_VERSION}: rebuild it")
        _lib = L
    return _lib


def _check(rc: int):
    if rc != WS_OK:
        raise WaitSimError(rc, lib().wait_sim_last_error().decode())


class JobArray:
    """C structs for a list of jobs; keeps the host arrays alive."""

    def __init__(self, jobs: Sequence):
        self.keep = []
        self.cfgs = []
        self.pols = []
        self.n_jobs = len(jobs)
        self.arr = (WsJob * max(1, len(jobs)))()
        self.replicas = 0
        for i, job in enumerate(jobs):
            wl = job.wl
            cfg = WsConfig()
            cfg.m = wl.m
            cfg.prompt_len = self._a(wl.prompt_len, np.int32)
            cfg.lam = self._a(wl.lam, np.float64)
            cfg.out_len = None if wl.out_len is None else self._a(wl.out_len, np.int32)
            cfg.out_cap = int(wl.out_cap)
            cfg.out_cdf_u32 = None if wl.out_cdf is None else self._a(wl.out_cdf, np.uint32)
            cfg.d0, cfg.d1, cfg.C = float(wl.d0), float(wl.d1), int(wl.C)
            if wl.hist_edges is None:
                cfg.hist_edges, cfg.n_hist = None, 0
            else:
                cfg.hist_edges = self._a(wl.hist_edges, np.float64)
                cfg.n_hist = len(wl.hist_edges)
            cfg.record_capacity = int(wl.record_capacity)
            if wl.trace is not None:
                t, ty, L = wl.trace
                cfg.trace_time = self._a(t, np.float64)
                cfg.trace_type = self._a(ty, np.int32)
                cfg.trace_out_len = self._a(L, np.int32)
                cfg.n_trace = len(t)
            else:
                cfg.trace_time = cfg.trace_type = cfg.trace_out_len = None
                cfg.n_trace = 0
            if getattr(wl, "rate_t", None) is not None:
                P = len(wl.rate_t)
                cfg.n_rate_pts = P
                cfg.rate_t = self._a(wl.rate_t, np.float64)
                cfg.rate_f = self._a(np.asarray(wl.rate_f, dtype=np.float64).reshape(wl.m, P),
                                     np.float64)
            else:
                cfg.n_rate_pts, cfg.rate_t, cfg.rate_f = 0, None, None
            pol = WsPolicy()
            pol.kind = POLICY[wl.policy]
            pol.n = self._a(wl.n if len(wl.n) else [0], np.int32)
            pol.L = len(wl.seg_end) if wl.seg_end is not None else 0
            pol.seg_end = None if wl.seg_end is None else self._a(wl.seg_end, np.int32)
            pol.fcfs_reserve = float(wl.reserve)
            pol.fcfs_chunk = int(getattr(wl, "chunk", 0) or 0)
            caps = getattr(wl, "stage_caps", None)
            pol.stage_caps = None if caps is None else self._a(caps, np.int32)
            ids = np.asarray(job.replica_ids, dtype=np.uint32)
            st = (WsStream * max(1, len(ids)))()
            for x, rid in enumerate(ids):
                st[x].seed = int(job.seed)
                st[x].replica_id = int(rid)
                st[x].reserved = 0
            self.keep.append(st)
            self.cfgs.append(cfg)
            self.pols.append(pol)
            self.arr[i].cfg = C.pointer(cfg)
            self.arr[i].pol = C.pointer(pol)
            self.arr[i].streams = C.addressof(st)
            self.arr[i].n = len(ids)
            self.replicas += len(ids)

    def _a(self, x, dt):
        a = np.ascontiguousarray(np.asarray(x, dtype=dt))
        self.keep.append(a)
        return a.ctypes.data

    @property
    def ptr(self):
        return C.cast(self.arr, C.POINTER(WsJob))


def workspace_bytes(ja: JobArray) -> int:
    b = C.c_size_t()
    _check(lib().wait_sim_workspace_bytes(ja.ptr, ja.n_jobs, C.byref(b)))
    return int(b.value)


def results_bytes(ja: JobArray):
    b = C.c_size_t()
    h = C.c_int32()
    _check(lib().wait_sim_results_bytes(ja.ptr, ja.n_jobs, C.byref(b), C.byref(h)))
    return int(b.value), int(h.value)


def _stream_handle(torch, device):
    return C.c_void_p(torch.cuda.current_stream(device).cuda_stream)


class Simulation:
    """Device buffers for one set of jobs, advanced through the C ABI."""

    def __init__(self, jobs: Sequence, device: str = "cuda:0"):
        import torch
        self.torch = torch
        self.device = torch.device(device)
        self.ja = JobArray(jobs)
        self.ws_bytes = workspace_bytes(self.ja)
        self.res_bytes, self.hist_stride = results_bytes(self.ja)
        self.R = self.ja.replicas
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.device)
        self.res = torch.zeros(self.res_bytes, dtype=torch.uint8, device=self.device)
        self.prepared = False

    def prepare(self):
        with self.torch.cuda.device(self.device):
            _check(lib().wait_sim_prepare(self.ja.ptr, self.ja.n_jobs, self.ws.data_ptr(),
                                          self.ws_bytes, _stream_handle(self.torch, self.device)))
        self.prepared = True

    def advance(self, horizon: int, resume: bool = False):
        if not self.prepared:
            self.prepare()
        with self.torch.cuda.device(self.device):
            _check(lib().wait_sim_advance(self.ja.ptr, self.ja.n_jobs, int(horizon),
                                          1 if resume else 0, self.ws.data_ptr(),
                                          self.ws_bytes, self.res.data_ptr(), self.res_bytes,
                                          _stream_handle(self.torch, self.device)))

    def state_bytes(self) -> int:
        """Size of the checkpoint of the current state (wait_sim_save_state
        without a buffer)."""
        used = C.c_size_t()
        with self.torch.cuda.device(self.device):
            _check(lib().wait_sim_save_state(self.ja.ptr, self.ja.n_jobs, self.ws.data_ptr(),
                                             self.ws_bytes, None, 0, C.byref(used),
                                             _stream_handle(self.torch, self.device)))
        return int(used.value)

    def checkpoint(self, to_host: bool = False):
        """The checkpoint of every replica's live state after the calls issued
        so far (wait_sim_save_state): a device uint8 tensor of exactly its
        size, or a host copy with to_host."""
        torch = self.torch
        used = C.c_size_t(self.state_bytes())
        buf = torch.empty(used.value, dtype=torch.uint8, device=self.device)
        with torch.cuda.device(self.device):
            _check(lib().wait_sim_save_state(self.ja.ptr, self.ja.n_jobs, self.ws.data_ptr(),
                                             self.ws_bytes, buf.data_ptr(), used.value,
                                             C.byref(used), _stream_handle(torch, self.device)))
        return buf.cpu() if to_host else buf

    def restore(self, state) -> None:
        """Load a checkpoint of a Simulation of the same jobs
        (wait_sim_load_state); continue with advance(..., resume=True)."""
        torch = self.torch
        d = state.to(self.device).contiguous()
        with torch.cuda.device(self.device):
            _check(lib().wait_sim_load_state(self.ja.ptr, self.ja.n_jobs, self.ws.data_ptr(),
                                             self.ws_bytes, d.data_ptr(), d.numel(),
                                             _stream_handle(torch, self.device)))
        self.prepared = True

    def run_ex(self, horizon: int, state_in=None, state_out=None) -> int:
        """wait_sim_run_batch_ex: advance by `horizon` batches from the empty
        system or from the checkpoint `state_in` (a device uint8 tensor), and
        write the checkpoint of the state it leaves into `state_out` (a device
        uint8 tensor at least that large) if given.  Returns the checkpoint's
        size in bytes."""
        torch = self.torch
        used = C.c_size_t()
        sin = state_in.contiguous() if state_in is not None else None
        with torch.cuda.device(self.device):
            _check(lib().wait_sim_run_batch_ex(
                self.ja.ptr, self.ja.n_jobs, int(horizon), self.ws.data_ptr(), self.ws_bytes,
                self.res.data_ptr(), self.res_bytes, _stream_handle(torch, self.device),
                sin.data_ptr() if sin is not None else None,
                sin.numel() if sin is not None else 0,
                state_out.data_ptr() if state_out is not None else None,
                state_out.numel() if state_out is not None else 0, C.byref(used)))
        self.prepared = True
        return int(used.value)

    def advance_traced(self, horizon: int, btrace_cap: int, resume: bool = False) -> np.ndarray:
        """advance() that also returns the per-batch trace: a structured array
        [replicas][btrace_cap] of ws_batch_rec (records of batches not run are
        zero)."""
        if not self.prepared:
            self.prepare()
        torch = self.torch
        nbytes = BATCH_REC.itemsize * self.R * int(btrace_cap)
        buf = torch.zeros(max(nbytes, 1), dtype=torch.uint8, device=self.device)
        with torch.cuda.device(self.device):
            _check(lib().wait_sim_advance_traced(
                self.ja.ptr, self.ja.n_jobs, int(horizon), 1 if resume else 0,
                self.ws.data_ptr(), self.ws_bytes, self.res.data_ptr(), self.res_bytes,
                buf.data_ptr(), int(btrace_cap), _stream_handle(torch, self.device)))
        host = buf.cpu().numpy()[:nbytes]
        return host.view(BATCH_REC).reshape(self.R, int(btrace_cap))

    def results(self) -> dict:
        """Per-replica results as numpy arrays (synchronises the stream)."""
        host = self.res.cpu().numpy()
        R = self.R
        out = {}
        i64 = host[: 8 * WS_NI64 * R].view(np.int64).reshape(WS_NI64, R)
        for k, f in enumerate(I64_FIELDS):
            out[f] = i64[k].copy()
        f64 = host[8 * WS_NI64 * R: 8 * (WS_NI64 + WS_NF64) * R].view(np.float64)
        f64 = f64.reshape(WS_NF64, R)
        for k, f in enumerate(F64_FIELDS):
            out[f] = f64[k].copy()
        off = 8 * (WS_NI64 + WS_NF64) * R
        out["flags"] = host[off: off + 4 * R].view(np.uint32).copy()
        hoff = (off + 4 * R + 7) // 8 * 8
        out["hist"] = host[hoff: hoff + 4 * R * self.hist_stride].view(np.uint32).reshape(
            R, self.hist_stride).copy()
        return out


def run_batch(jobs: Sequence, horizon: int, device: str = "cuda:0") -> dict:
    """prepare + advance for a list of jobs; returns per-replica results."""
    sim = Simulation(jobs, device)
    sim.prepare()
    sim.advance(horizon, resume=False)
    return sim.results()


def run_static(job, horizon: int, device: str = "cuda:0") -> dict:
    """One job through wait_sim_run_static (the library's static workspace,
    no device allocation inside the call); the result buffer is allocated
    here, before the call."""
    import torch
    ja = JobArray([job])
    nbytes, _ = results_bytes(ja)
    dev = torch.device(device)
    res = torch.zeros(nbytes, dtype=torch.uint8, device=dev)
    sim = Simulation.__new__(Simulation)
    sim.torch, sim.device, sim.ja, sim.res, sim.R = torch, dev, ja, res, ja.replicas
    sim.res_bytes, sim.hist_stride = results_bytes(ja)
    with torch.cuda.device(dev):
        _check(lib().wait_sim_run_static(ja.arr[0].cfg, ja.arr[0].pol, ja.arr[0].streams,
                                         ja.arr[0].n, int(horizon), res.data_ptr(), nbytes,
                                         _stream_handle(torch, dev)))
    return sim.results()


def split_by_job(res: dict, jobs: Sequence) -> list:
    """Split per-replica result arrays into one dict per job."""
    out = []
    start = 0
    for job in jobs:
        n = len(job.replica_ids)
        out.append({k: v[start:start + n] for k, v in res.items()})
        start += n
    return out
