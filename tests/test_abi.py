"""The C-ABI library: loads, exports every declared symbol, validates input.

These run without a GPU: sizing and validation are host-only."""
import ctypes
import os
import re

import numpy as np
import pytest

import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "wait_sim.h")).read()
    return sorted(set(re.findall(r"^\w[\w\s\*]*?\b(wait_sim_\w+)\s*\(", src, re.M)))


def test_library_exports_header_symbols():
    from paper_2504_11320_amd import binding as B
    lib = B.lib()
    names = _declared()
    assert "wait_sim_run" in names and "wait_sim_advance" in names
    for n in names:
        assert hasattr(lib, n), n
    assert lib.wait_sim_abi_version() == B.WS_ABI_VERSION == 4


def _err(jobs):
    from paper_2504_11320_amd import binding as B
    with pytest.raises(B.WaitSimError) as e:
        B.workspace_bytes(B.JobArray(jobs))
    return e.value


def _job(**kw):
    wl = W.config2(replicas=2, rate_index=[3])[0].wl
    for k, v in kw.items():
        setattr(wl, k, v)
    return [W.Job(wl, 0, W.ids(2))]


def test_validation_errors():
    from paper_2504_11320_amd import binding as B
    assert _err(_job(d0=0.0)).code == B.WS_EINVAL
    assert _err(_job(d1=-1.0)).code == B.WS_EINVAL
    assert _err(_job(prompt_len=[0, 512, 1024])).code == B.WS_EINVAL
    assert _err(_job(lam=[-1.0, 0.1, 0.1])).code == B.WS_EINVAL
    assert _err(_job(n=[0, 1, 1])).code == B.WS_EINVAL
    assert _err(_job(record_capacity=1000)).code == B.WS_EINVAL
    # atomic feasibility: l_j + l'_j <= C
    assert _err(_job(C=1500)).code == B.WS_EINVAL
    assert _err(_job(hist_edges=np.array([1.0, 1.0]))).code == B.WS_EINVAL
    # Nested: the last segment must end at the largest output length
    assert _err(_job(policy="nested", seg_end=[64, 256])).code == B.WS_EINVAL
    assert _err(_job(policy="nested", seg_end=[64, 64, 512])).code == B.WS_EINVAL
    # a well-formed job sizes without error
    ja = B.JobArray(_job())
    assert B.workspace_bytes(ja) > 0
    nb, hs = B.results_bytes(ja)
    assert hs == 193 and nb >= 2 * (8 * 18 + 4 + 4 * 193)


def test_fcfs_reserve_validation():
    from paper_2504_11320_amd import binding as B
    jobs = W.config4(replicas=1, grid=1, n_rates=2)
    fc = [j for j in jobs if j.wl.policy == "fcfs"][:1]
    fc[0].wl.reserve = 1.0
    assert _err(fc).code == B.WS_EINVAL


def test_type_limits():
    """Every policy takes up to 64 request types; more than 64 is invalid.
    WAIT with more than 16 types takes constant rates only."""
    from paper_2504_11320_amd import binding as B

    def model(m, policy):
        kw = dict(prompt_len=[16] * m, lam=[0.01] * m, d0=5.0, d1=0.01, C=4096,
                  policy=policy, hist_edges=W.default_edges(5.0, 50))
        if policy == "nested":
            cap = 32
            kw.update(n=[1, 1], out_cap=cap, seg_end=[8, cap],
                      out_cdf=np.stack([W.geometric_cdf_table(8.0, cap)] * m))
        else:
            kw.update(out_len=[8] * m, n=[1] * m if policy == "wait" else [])
        return [W.Job(W.Workload(**kw), 0, W.ids(2))]

    for policy in ("wait", "fcfs", "nested"):
        assert B.workspace_bytes(B.JobArray(model(16, policy))) > 0
        assert _err(model(65, policy)).code == B.WS_EINVAL
    for policy in ("wait", "fcfs", "nested"):
        assert B.workspace_bytes(B.JobArray(model(64, policy))) > 0
    tv = model(17, "wait")
    rt, rf = W.diurnal_profile(17, 1e6, points=5)
    tv[0].wl.rate_t, tv[0].wl.rate_f = rt, rf
    assert _err(tv).code == B.WS_EUNSUPPORTED


def test_rate_profile_validation():
    """Time-varying rates: points strictly increasing and finite, factors
    finite and >= 0, at most WS_MAX_RATE_PTS points, no arrival list beside
    them; a valid profile sizes without error."""
    from paper_2504_11320_amd import binding as B
    m = 3

    def prof(t, f, **kw):
        return _job(rate_t=np.asarray(t, float), rate_f=np.asarray(f, float), **kw)

    ok = prof([0.0, 1000.0], [[1.0, 2.0]] * m)
    assert B.workspace_bytes(B.JobArray(ok)) > 0
    assert _err(prof([0.0, 0.0], [[1.0, 2.0]] * m)).code == B.WS_EINVAL
    assert _err(prof([1.0, 0.0], [[1.0, 2.0]] * m)).code == B.WS_EINVAL
    assert _err(prof([0.0, np.inf], [[1.0, 2.0]] * m)).code == B.WS_EINVAL
    assert _err(prof([0.0, 1.0], [[1.0, -2.0]] * m)).code == B.WS_EINVAL
    assert _err(prof([0.0, 1.0], [[1.0, np.nan]] * m)).code == B.WS_EINVAL
    assert _err(prof([0.0, 1.0], [[1.0, 1e308]] * m, lam=[10.0, 0.1, 0.1])).code == B.WS_EINVAL
    P = 33
    assert _err(prof(np.arange(P), np.ones((m, P)))).code == B.WS_EINVAL
    assert B.workspace_bytes(B.JobArray(prof(np.arange(32), np.ones((m, 32))))) > 0
    tr = W.trace_workload("wait", [16], [4], 5.0, 0.01, 1000, [1], [0.0], [0])
    tr.rate_t, tr.rate_f = np.array([0.0]), np.array([[1.0]])
    assert _err([W.Job(tr, 0, W.ids(1))]).code == B.WS_EINVAL


def test_chunk_validation():
    """fcfs_chunk >= 0, FCFS only."""
    from paper_2504_11320_amd import binding as B
    fc = _job(policy="fcfs", n=[], chunk=-1)
    assert _err(fc).code == B.WS_EINVAL
    assert _err(_job(chunk=64)).code == B.WS_EINVAL        # WAIT
    assert B.workspace_bytes(B.JobArray(_job(policy="fcfs", n=[], chunk=64))) > 0


def test_fcfs_drawn_lengths_validation():
    """FCFS with output lengths drawn per request is accepted (its own
    kernel); with chunked prefill or a rate profile it is WS_EUNSUPPORTED."""
    from paper_2504_11320_amd import binding as B
    wl = W.config3(replicas=2, rate_index=[3])[0].wl
    fc = W.Workload(**{**wl.__dict__, "policy": "fcfs", "n": [], "seg_end": None})
    assert B.workspace_bytes(B.JobArray([W.Job(fc, 0, W.ids(2))])) > 0
    ch = W.Workload(**{**fc.__dict__, "chunk": 256})
    assert _err([W.Job(ch, 0, W.ids(2))]).code == B.WS_EUNSUPPORTED
    rt, rf = W.diurnal_profile(3, 1e6, points=5)
    tv = W.with_profile(fc, rt, rf)
    assert _err([W.Job(tv, 0, W.ids(2))]).code == B.WS_EUNSUPPORTED


def test_wait_admission_bound():
    """WAIT: one batch may admit sum_j n_j (l_j + 1) tokens; at 2^29 or more the
    library's 32-bit resident-memory counters could overflow:
    WS_EUNSUPPORTED."""
    from paper_2504_11320_amd import binding as B
    assert _err(_job(n=[1 << 22, 1, 1])).code == B.WS_EUNSUPPORTED   # 2^22 x 129
    assert B.workspace_bytes(B.JobArray(_job(n=[1000, 1, 1]))) > 0


def test_static_entry_validates_on_the_host():
    """wait_sim_run_static checks the model and the size of its static
    workspace before touching the device: an invalid job gives WS_EINVAL, a
    job whose workspace exceeds WS_STATIC_WORKSPACE_BYTES gives
    WS_EWORKSPACE with a message naming the static workspace."""
    from paper_2504_11320_amd import binding as B
    L = B.lib()

    def call(jobs):
        ja = B.JobArray(jobs)
        a = ja.arr[0]
        return L.wait_sim_run_static(a.cfg, a.pol, a.streams, a.n, 10, None, 0, None)

    assert call(_job(d0=0.0)) == B.WS_EINVAL
    big = W.config2(replicas=1024, rate_index=[3])
    assert B.workspace_bytes(B.JobArray(big)) > B.WS_STATIC_WORKSPACE_BYTES
    assert call(big) == B.WS_EWORKSPACE
    assert b"static workspace" in L.wait_sim_last_error()


def test_checkpoint_entries_validate_on_the_host():
    """The checkpoint entry points reject bad arguments before any device
    call: NULL workspace or checkpoint buffers, a workspace smaller than the
    jobs need, a save with neither a buffer nor a size out-parameter, an
    invalid job."""
    from paper_2504_11320_amd import binding as B
    L = B.lib()
    ja = B.JobArray(_job())
    need = B.workspace_bytes(ja)
    used = ctypes.c_size_t()
    fake = ctypes.c_void_p(1 << 40)  # never dereferenced: the checks come first
    assert L.wait_sim_save_state(ja.ptr, ja.n_jobs, None, need, None, 0, ctypes.byref(used),
                                 None) == B.WS_EINVAL
    assert L.wait_sim_save_state(ja.ptr, ja.n_jobs, fake, need - 1, None, 0,
                                 ctypes.byref(used), None) == B.WS_EWORKSPACE
    assert L.wait_sim_save_state(ja.ptr, ja.n_jobs, fake, need, None, 0, None,
                                 None) == B.WS_EINVAL
    assert L.wait_sim_load_state(ja.ptr, ja.n_jobs, fake, need, None, 0, None) == B.WS_EINVAL
    assert L.wait_sim_load_state(ja.ptr, ja.n_jobs, None, need, fake, 1 << 20,
                                 None) == B.WS_EINVAL
    assert L.wait_sim_load_state(ja.ptr, ja.n_jobs, fake, need - 1, fake, 1 << 20,
                                 None) == B.WS_EWORKSPACE
    res, _ = B.results_bytes(ja)
    assert L.wait_sim_run_batch_ex(ja.ptr, ja.n_jobs, 10, fake, need - 1, fake, res, None,
                                   None, 0, None, 0, None) == B.WS_EWORKSPACE
    assert L.wait_sim_run_batch_ex(ja.ptr, ja.n_jobs, -1, fake, need, fake, res, None,
                                   None, 0, None, 0, None) == B.WS_EINVAL
    bad = B.JobArray(_job(d0=0.0))
    assert L.wait_sim_run_batch_ex(bad.ptr, bad.n_jobs, 10, fake, need, fake, res, None,
                                   None, 0, None, 0, None) == B.WS_EINVAL


def test_stage_caps_validation():
    """Per-stage caps: Nested WAIT only, >= 0, >= 1 in segment 1, and n[k]
    the largest cap of segment k."""
    from paper_2504_11320_amd import binding as B
    base = W.config_p512_mix(replicas=2, rates=[0.02])
    ja = B.JobArray(base)
    assert B.workspace_bytes(ja) > 0

    def with_caps(caps, n=None, policy="nested"):
        j = base[0]
        wl = W.Workload(**{**j.wl.__dict__, "stage_caps": caps})
        if n is not None:
            wl.n = n
        if policy != "nested":
            wl = W.config2(replicas=2, rate_index=[3])[0].wl
            wl.stage_caps = caps
        return [W.Job(wl, 0, W.ids(2))]

    # WAIT: l'_j + 1 caps per type, each >= 1, n_j the largest; not WAIT-no-wait
    wt = W.config2(replicas=2, rate_index=[3])[0].wl
    wcaps = sum(([1] * (lp + 1) for lp in wt.out_len), [])
    ok = W.Workload(**{**wt.__dict__, "stage_caps": wcaps})
    assert B.workspace_bytes(B.JobArray([W.Job(ok, 0, W.ids(2))])) > 0
    zero = W.Workload(**{**wt.__dict__, "stage_caps": [0] + wcaps[1:]})
    assert _err([W.Job(zero, 0, W.ids(2))]).code == B.WS_EINVAL
    big = W.Workload(**{**wt.__dict__, "stage_caps": [2] + wcaps[1:]})  # n_1 = 1 < 2
    assert _err([W.Job(big, 0, W.ids(2))]).code == B.WS_EINVAL
    nw = W.Workload(**{**wt.__dict__, "stage_caps": wcaps, "policy": "wait-nowait"})
    assert _err([W.Job(nw, 0, W.ids(2))]).code == B.WS_EINVAL

    caps = list(W.P512MIX_CAPS_TL30)
    assert _err(with_caps(caps[:20] + [-1] + caps[21:])).code == B.WS_EINVAL
    assert _err(with_caps([0] + caps[1:])).code == B.WS_EINVAL  # segment 1 needs >= 1
    assert _err(with_caps(caps, n=[1, 1])).code == B.WS_EINVAL  # n_1 is not the largest
    assert _err(with_caps(caps, policy="wait")).code == B.WS_EINVAL  # wrong length for WAIT


def test_host_allocation_failure_is_an_error_code():
    """No C++ exception crosses the C ABI: a job count whose host-side
    descriptors cannot be allocated returns WS_ENOMEM."""
    from paper_2504_11320_amd import binding as B
    try:
        overcommit = open("/proc/sys/vm/overcommit_memory").read().strip()
    except OSError:
        overcommit = "?"
    if overcommit != "0" and overcommit != "2":
        pytest.skip("the kernel may grant any allocation (overcommit_memory != 0, 2)")
    if os.environ.get("WAIT_SIM_SANITIZED"):
        pytest.skip("under AddressSanitizer its allocator, not the C++ one, answers")
    L = B.lib()
    ja = B.JobArray(_job())
    size = ctypes.c_size_t()
    rc = L.wait_sim_workspace_bytes(ja.ptr, (1 << 31) - 1, ctypes.byref(size))
    assert rc == B.WS_ENOMEM
    assert b"allocation" in L.wait_sim_last_error()
