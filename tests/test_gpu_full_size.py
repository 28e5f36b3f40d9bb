"""Full-size launches of the Nested WAIT, policy-sweep, heavy-tailed, cyclic
time-varying, chunked-prefill FCFS and decode-only workloads, exactly as configured (every replica, the full horizon, one
launch): properties that hold for every replica are checked on all of them,
and sampled replicas are recomputed one by one by the oracle and compared
field by field (integers exact, fp64 within 1e-12 relative)."""
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import workloads as W
from tests.parity_util import compare

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

CAP, STALL, OVERFLOW = 1, 2, 4


@pytest.fixture(scope="module")
def B():
    from tests.gpu_util import sim_module
    return sim_module()


def _run(B, jobs, horizon, ctx):
    import torch
    print(f"[gpu] {ctx}: {len(jobs)} jobs, {sum(j.n for j in jobs)} replicas, "
          f"horizon {horizon}", flush=True)
    t0 = time.perf_counter()
    g = B.run_batch(jobs, horizon)
    torch.cuda.synchronize()
    print(f"[gpu] {ctx}: launch done in {time.perf_counter() - t0:.1f} s", flush=True)
    return g


def _invariants(g, horizon, ctx):
    stopped = (g["flags"] & (CAP | STALL)) != 0
    assert np.all(g["batches"][~stopped] == horizon), ctx
    # request conservation: every arrival completed, waits, or is resident
    assert np.array_equal(g["arrivals"],
                          g["completions"] + g["waiting_end"] + g["resident_end"]), ctx
    assert np.array_equal(g["hist"].sum(axis=1).astype(np.int64), g["completions"]), ctx
    assert np.all(g["busy_time"] <= g["t_end"]), ctx
    assert np.all(g["evicted_tokens"] >= 0) and np.all(g["fallback_evictions"] <= g["evictions"]), ctx


def _sampled(g, jobs, horizon, picks, ctx):
    """picks: (job index, replica position within the job)."""
    from oracle import oracle as O
    starts = np.cumsum([0] + [j.n for j in jobs])
    sub = [W.Job(jobs[ji].wl, jobs[ji].seed,
                 np.array([jobs[ji].replica_ids[pos]], dtype=np.uint32)) for ji, pos in picks]
    with ThreadPoolExecutor(min(len(sub), 16)) as ex:
        outs = list(ex.map(lambda jb: O.run_job(jb, horizon, threads=1), sub))
    width = max(o["hist"].shape[1] for o in outs)
    for o in outs:
        o["hist"] = np.pad(o["hist"], ((0, 0), (0, width - o["hist"].shape[1])))
    o = {k: np.concatenate([x[k] for x in outs]) for k in outs[0]}
    idx = np.array([starts[ji] + pos for ji, pos in picks])
    gsub = {k: v[idx] for k, v in g.items()}
    gsub["hist"] = gsub["hist"][:, :width]
    st = compare(gsub, o, ctx)
    print(f"[gpu] {ctx}: {len(picks)} sampled replicas ok, fp64 bit-exact "
          f"{st['f64_bit_exact']}/{st['f64_total']}", flush=True)


def test_config3_full_size(B):
    """Nested WAIT, geometric outputs: 32 rates x 1024 replicas x 1e5 batches."""
    jobs = W.config3()
    g = _run(B, jobs, 100000, "config3 full size")
    _invariants(g, 100000, "config3")
    picks = [(ri, pos) for ri in (0, 15, 31) for pos in (0, 1023)]
    _sampled(g, jobs, 100000, picks, "config3 full size")


def test_config4_full_size(B):
    """Policy sweep: 16 rates x 16x16 WAIT thresholds x 16 replicas plus FCFS on
    the same streams, 1e5 batches, one launch."""
    jobs = W.config4()
    g = _run(B, jobs, 100000, "config4 full size")
    _invariants(g, 100000, "config4")
    n_wait = 16 * 256
    picks = [(0, 0), (17, 5), (255, 15), (256 * 8 + 128, 3), (n_wait - 1, 15),
             (n_wait, 0), (n_wait + 8, 7), (n_wait + 15, 15)]
    _sampled(g, jobs, 100000, picks, "config4 full size")
    # the WAIT cells and FCFS share replica streams: same arrival processes
    # (arrivals differ only through the queue-capacity stop)
    assert g["arrivals"].min() > 0


def test_config5_full_size(B):
    """Heavy-tailed 10-type mix, Nested WAIT with 6 segments: 8192 replicas x
    1e6 batches."""
    jobs = W.config5()
    g = _run(B, jobs, 1000000, "config5 full size")
    _invariants(g, 1000000, "config5")
    _sampled(g, jobs, 1000000, [(0, 0), (0, 4095), (0, 8191)], "config5 full size")


def test_cyclic_full_size(B):
    """Llama-shaped WAIT sweep with cyclic time-varying rates (two cycles of
    lam_j (1 + 0.5 sin(.)) over 8e8 ms, phases 2 pi j / 3): 32 rates x 1024
    replicas x 1e5 batches, the benchmark's launch."""
    jobs = W.config_cyclic()
    g = _run(B, jobs, 100000, "cyclic full size")
    _invariants(g, 100000, "cyclic")
    picks = [(0, 0), (0, 1023), (15, 511), (31, 7), (31, 1000)]
    _sampled(g, jobs, 100000, picks, "cyclic full size")


def test_fcfs_chunked_full_size(B):
    """FCFS with a 1 % reserve and 512-token chunked prefill on the
    Llama-shaped mix: 32 rates x 1024 replicas x 1e5 batches, the benchmark's
    launch."""
    jobs = W.config_chunked()
    g = _run(B, jobs, 100000, "fcfs-chunked full size")
    _invariants(g, 100000, "fcfs-chunked")
    picks = [(0, 0), (16, 512), (31, 1023)]
    _sampled(g, jobs, 100000, picks, "fcfs-chunked full size")


def test_pd_decode_full_size(B):
    """Decode-only p630d20, WAIT and FCFS at 9 rates x 1024 replicas x 1e5
    batches."""
    jobs = W.config_pd()
    g = _run(B, jobs, 100000, "pd-decode full size")
    _invariants(g, 100000, "pd-decode")
    picks = [(0, 0), (8, 1023), (9, 5), (17, 700)]
    _sampled(g, jobs, 100000, picks, "pd-decode full size")
