"""ctypes shim for the CPU oracle (test infrastructure).

Only tests, the smoke check and the benchmark's CPU-baseline leg may import
this module.  It builds and loads ``liboracle.so`` from ``wait_oracle.c`` in
this directory and shares nothing with the GPU library.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "wait_oracle.c")
HDR = os.path.join(HERE, "wait_oracle.h")
LIB = os.path.join(HERE, "liboracle.so")
# another build (e.g. the sanitizer build, build_sanitized()) may be named in
# WAIT_ORACLE_LIB
LIB_OVERRIDE = os.environ.get("WAIT_ORACLE_LIB")


def _stale() -> bool:
    return (not os.path.exists(LIB)
            or os.path.getmtime(LIB) < max(os.path.getmtime(SRC), os.path.getmtime(HDR)))

POLICY = {"wait": 0, "nested": 1, "fcfs": 2, "wait-nowait": 3}
FLAG_CAPACITY, FLAG_STALL, FLAG_OVERFLOW, FLAG_THIN_LIMIT = 1, 2, 4, 8

INT_FIELDS = ["batches", "arrivals", "completions", "completed_tokens",
              "evictions", "evicted_tokens", "fallback_evictions",
              "batch_tokens_sum", "peak_mem", "waiting_end", "resident_end",
              "idle_waits"]
F64_FIELDS = ["t_end", "busy_time", "lat_area", "ttft_area",
              "lat_completed_sum", "mem_area"]


class _Config(C.Structure):
    _fields_ = [
        ("m", C.c_int32), ("l", C.c_void_p), ("lam", C.c_void_p),
        ("lp", C.c_void_p), ("out_cap", C.c_int32), ("cdf", C.c_void_p),
        ("d0", C.c_double), ("d1", C.c_double), ("C", C.c_int64),
        ("edges", C.c_void_p), ("n_edges", C.c_int32),
        ("record_capacity", C.c_int64), ("tr_time", C.c_void_p),
        ("tr_type", C.c_void_p), ("tr_L", C.c_void_p), ("n_trace", C.c_int64),
        ("policy", C.c_int32), ("n", C.c_void_p), ("nseg", C.c_int32),
        ("seg_end", C.c_void_p), ("reserve", C.c_double),
        ("n_rate_pts", C.c_int32), ("rate_t", C.c_void_p), ("rate_f", C.c_void_p),
        ("chunk", C.c_int32), ("stage_caps", C.c_void_p),
    ]


class _Result(C.Structure):
    _fields_ = ([(f, C.c_int64) for f in INT_FIELDS]
                + [(f, C.c_double) for f in F64_FIELDS]
                + [("flags", C.c_uint32), ("pad", C.c_uint32)])


class _BatchRec(C.Structure):
    _fields_ = [("t_launch", C.c_double), ("tau", C.c_double)] + [
        (f, C.c_int64) for f in ("tokens", "prefills", "selected", "completions",
                                 "evict_pre", "evict_post", "mem_after",
                                 "waiting_after", "resident_after", "mplus")]


class _ReqLog(C.Structure):
    _fields_ = [("arr", C.c_void_p), ("done", C.c_void_p),
                ("first", C.c_void_p), ("cap", C.c_int64),
                ("ev_id", C.c_void_p), ("ev_batch", C.c_void_p),
                ("ev_kind", C.c_void_p), ("ev_cap", C.c_int64), ("n_ev", C.c_int64)]


# eviction kinds of the eviction log (wait_oracle.h)
EV_POST, EV_POST_FALLBACK, EV_PRE, EV_PRE_FALLBACK = 0, 1, 2, 3


_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle (plain C, -O2, no FP contraction, no fast-math)."""
    if force or _stale():
        cmd = ["gcc", "-O2", "-std=gnu11", "-Wall", "-ffp-contract=off",
               "-fno-fast-math", "-fPIC", "-shared", "-o", LIB + ".tmp", SRC,
               "-lpthread", "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(LIB + ".tmp", LIB)
    return LIB


def load(path: str):
    """Load an oracle library built from wait_oracle.c and declare its
    functions."""
    L = C.CDLL(path)
    L.oracle_run.argtypes = [C.POINTER(_Config), C.c_uint64, C.c_uint32,
                             C.c_int64, C.POINTER(_Result), C.c_void_p,
                             C.c_void_p, C.c_int64, C.c_void_p]
    L.oracle_run_many.argtypes = [C.POINTER(_Config), C.c_uint64, C.c_void_p,
                                  C.c_int32, C.c_int64, C.c_void_p,
                                  C.c_void_p, C.c_int32]
    L.oracle_philox4x32_10.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p]
    L.oracle_uniform.argtypes = [C.c_uint32, C.c_uint32]
    L.oracle_uniform.restype = C.c_double
    L.oracle_ln.argtypes = [C.c_double]
    L.oracle_ln.restype = C.c_double
    L.oracle_arrival_times.argtypes = [C.POINTER(_Config), C.c_uint64,
                                       C.c_uint32, C.c_int32, C.c_int64,
                                       C.c_void_p, C.c_void_p, C.c_void_p]
    L.oracle_arrival_times.restype = C.c_int
    L.oracle_draw.argtypes = [C.c_uint64, C.c_uint32, C.c_int32, C.c_uint32,
                              C.c_double, C.c_void_p, C.c_int32,
                              C.POINTER(C.c_double), C.POINTER(C.c_int32)]
    return L


def build_sanitized(out: str) -> str:
    """The oracle with AddressSanitizer and UndefinedBehaviorSanitizer (clang,
    shared ASan runtime: preload libclang_rt.asan when loading it)."""
    cc = "/opt/rocm/lib/llvm/bin/clang"
    cmd = [cc, "-O1", "-g", "-std=gnu11", "-Wall", "-ffp-contract=off", "-fno-fast-math",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-fno-omit-frame-pointer", "-shared-libasan", "-fPIC", "-shared", "-o", out,
           SRC, "-lpthread", "-lm"]
    subprocess.run(cmd, check=True)
    return out


def build_order_checked(out: str) -> str:
    """The oracle with the position-order counters of its Nested WAIT repairs
    (OR_CHECK_POSITION_ORDER): oracle_order_checks(kind) and
    oracle_order_misses(kind), kind 0 for boundary victims, 1 for interior."""
    cmd = ["gcc", "-O2", "-std=gnu11", "-Wall", "-ffp-contract=off", "-fno-fast-math",
           "-DOR_CHECK_POSITION_ORDER", "-fPIC", "-shared", "-o", out, SRC, "-lpthread", "-lm"]
    subprocess.run(cmd, check=True)
    L = load(out)
    for f in (L.oracle_order_checks, L.oracle_order_misses):
        f.argtypes = [C.c_int]
        f.restype = C.c_long
    return L


def lib():
    global _lib
    if _lib is None:
        if LIB_OVERRIDE:
            _lib = load(LIB_OVERRIDE)
            return _lib
        if _stale():
            build(force=True)
        _lib = load(LIB)
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


class _Pinned:
    """Keeps the numpy arrays behind a config alive."""

    def __init__(self, wl):
        self.keep = []
        c = _Config()
        c.m = wl.m

        def arr(x, dt):
            a = np.ascontiguousarray(np.asarray(x, dtype=dt))
            self.keep.append(a)
            return a

        c.l = _ptr(arr(wl.prompt_len, np.int32))
        c.lam = _ptr(arr(wl.lam, np.float64))
        c.lp = None if wl.out_len is None else _ptr(arr(wl.out_len, np.int32))
        c.out_cap = int(wl.out_cap)
        c.cdf = None if wl.out_cdf is None else _ptr(arr(wl.out_cdf, np.uint32))
        c.d0, c.d1, c.C = float(wl.d0), float(wl.d1), int(wl.C)
        if wl.hist_edges is None:
            c.edges, c.n_edges = None, 0
        else:
            c.edges = _ptr(arr(wl.hist_edges, np.float64))
            c.n_edges = len(wl.hist_edges)
        c.record_capacity = int(wl.record_capacity)
        if wl.trace is not None:
            t, ty, L = wl.trace
            c.tr_time = _ptr(arr(t, np.float64))
            c.tr_type = _ptr(arr(ty, np.int32))
            c.tr_L = _ptr(arr(L, np.int32))
            c.n_trace = len(t)
        else:
            c.tr_time = c.tr_type = c.tr_L = None
            c.n_trace = 0
        c.policy = POLICY[wl.policy]
        c.n = _ptr(arr(wl.n if len(wl.n) else [0], np.int32))
        if wl.seg_end is not None:
            c.seg_end = _ptr(arr(wl.seg_end, np.int32))
            c.nseg = len(wl.seg_end)
        else:
            c.seg_end, c.nseg = None, 0
        c.reserve = float(wl.reserve)
        c.chunk = int(getattr(wl, "chunk", 0) or 0)
        caps = getattr(wl, "stage_caps", None)
        c.stage_caps = None if caps is None else _ptr(arr(caps, np.int32))
        if getattr(wl, "rate_t", None) is not None:
            rt = arr(wl.rate_t, np.float64)
            rf = arr(np.asarray(wl.rate_f, dtype=np.float64).reshape(wl.m, len(rt)),
                     np.float64)
            c.n_rate_pts, c.rate_t, c.rate_f = len(rt), _ptr(rt), _ptr(rf)
        else:
            c.n_rate_pts, c.rate_t, c.rate_f = 0, None, None
        self.cfg = c


def _to_dict(res_arr, hist):
    out = {}
    for f in INT_FIELDS:
        out[f] = np.array([getattr(r, f) for r in res_arr], dtype=np.int64)
    for f in F64_FIELDS:
        out[f] = np.array([getattr(r, f) for r in res_arr], dtype=np.float64)
    out["flags"] = np.array([r.flags for r in res_arr], dtype=np.uint32)
    out["hist"] = hist
    return out


def run(wl, seed: int, replica_ids, horizon: int, threads: int = 0, library=None) -> dict:
    """Simulate every replica of a workload; returns arrays per field.
    `library`: another build of the oracle (a handle from load())."""
    L = library if library is not None else lib()
    pin = _Pinned(wl)
    ids = np.ascontiguousarray(np.asarray(replica_ids, dtype=np.uint32))
    n = len(ids)
    res = (_Result * n)()
    nb = (len(wl.hist_edges) if wl.hist_edges is not None else 0) + 1
    hist = np.zeros((n, nb), dtype=np.uint32)
    if threads <= 0:
        threads = min(os.cpu_count() or 1, 16)
    L.oracle_run_many(C.byref(pin.cfg), C.c_uint64(seed), ids.ctypes.data, n,
                      horizon, C.addressof(res), hist.ctypes.data, threads)
    return _to_dict(res, hist)


def run_job(job, horizon: int, threads: int = 0) -> dict:
    return run(job.wl, job.seed, job.replica_ids, horizon, threads)


def run_one(wl, seed: int, replica_id: int, horizon: int, btrace_cap: int = 0,
            rlog_cap: int = 0, evlog_cap: int = 0, library=None) -> dict:
    """One replica with optional per-batch trace, per-request log and
    eviction log (a list of (batch, request id, kind) in eviction order).
    `library`: another build of the oracle (a handle from load())."""
    L = library if library is not None else lib()
    pin = _Pinned(wl)
    res = _Result()
    nb = (len(wl.hist_edges) if wl.hist_edges is not None else 0) + 1
    hist = np.zeros(nb, dtype=np.uint32)
    bt = (_BatchRec * max(btrace_cap, 1))()
    rl = None
    logs = None
    ev = None
    if rlog_cap > 0 or evlog_cap > 0:
        n = max(rlog_cap, 1)
        logs = [np.full(n, -2.0), np.full(n, -2.0), np.full(n, -2.0)]
        ev = [np.zeros(max(evlog_cap, 1), np.int64), np.zeros(max(evlog_cap, 1), np.int64),
              np.zeros(max(evlog_cap, 1), np.int32)]
        rl = _ReqLog(logs[0].ctypes.data, logs[1].ctypes.data,
                     logs[2].ctypes.data, rlog_cap, ev[0].ctypes.data, ev[1].ctypes.data,
                     ev[2].ctypes.data, evlog_cap, 0)
    L.oracle_run(C.byref(pin.cfg), C.c_uint64(seed), C.c_uint32(replica_id),
                 horizon, C.byref(res), hist.ctypes.data,
                 C.addressof(bt) if btrace_cap > 0 else None, btrace_cap,
                 C.addressof(rl) if rl is not None else None)
    out = {f: getattr(res, f) for f in INT_FIELDS + F64_FIELDS}
    out["flags"] = res.flags
    out["hist"] = hist
    if btrace_cap > 0:
        nbt = min(btrace_cap, res.batches)
        out["batches_trace"] = [
            {f: getattr(bt[i], f) for f, _ in _BatchRec._fields_ if f != "pad"}
            for i in range(nbt)]
    if rlog_cap > 0:
        out["req_arr"], out["req_done"], out["req_first"] = logs
    if evlog_cap > 0:
        n_ev = min(rl.n_ev, evlog_cap)
        out["evictions_log"] = [(int(ev[1][i]), int(ev[0][i]), int(ev[2][i]))
                                for i in range(n_ev)]
    return out


# -------------------------------------------------------- RNG pieces ----


def philox(ctr, key) -> np.ndarray:
    L = lib()
    c = np.ascontiguousarray(np.asarray(ctr, dtype=np.uint32))
    k = np.ascontiguousarray(np.asarray(key, dtype=np.uint32))
    o = np.zeros(4, dtype=np.uint32)
    L.oracle_philox4x32_10(c.ctypes.data, k.ctypes.data, o.ctypes.data)
    return o


def uniform(w0: int, w1: int) -> float:
    return lib().oracle_uniform(w0, w1)


def ln(u: float) -> float:
    return lib().oracle_ln(u)


def draw(seed: int, replica_id: int, j: int, k: int, lam: float,
         cdf_row: Optional[np.ndarray] = None, out_cap: int = 0):
    L = lib()
    g = C.c_double()
    Lout = C.c_int32(0)
    row = None if cdf_row is None else np.ascontiguousarray(cdf_row, dtype=np.uint32)
    L.oracle_draw(C.c_uint64(seed), replica_id, j, k, lam, _ptr(row), out_cap,
                  C.byref(g), C.byref(Lout))
    return g.value, Lout.value


def arrival_times(wl, seed: int, replica_id: int, j: int, n: int):
    """First n arrival times of type j (inf once it has stopped), their output
    lengths and Philox counters, and the result flags."""
    L = lib()
    pin = _Pinned(wl)
    t = np.zeros(n, dtype=np.float64)
    Ls = np.zeros(n, dtype=np.int32)
    k = np.zeros(n, dtype=np.uint32)
    fl = L.oracle_arrival_times(C.byref(pin.cfg), C.c_uint64(seed), replica_id, j, n,
                                t.ctypes.data, Ls.ctypes.data, k.ctypes.data)
    return t, Ls, k, fl
