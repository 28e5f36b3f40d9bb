"""Checkpoints of the live state through the C ABI (wait_sim_run_batch_ex,
wait_sim_save_state, wait_sim_load_state).

A run cut into two calls, with the state between them saved to a checkpoint,
copied through host memory and restored into a fresh workspace, must end
exactly where one uninterrupted call ends: every counter, fp64 sum, flag and
histogram bin bit for bit, for every policy kind and for jobs that mix them.
The checkpoint must hold only the live records (its record bytes follow the
queue and resident counts the results report), and restoring one that does
not belong to the jobs, or is damaged, must be refused.
"""
import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu

HDR_USED, HDR_DIR, HDR_BLOB = 16, 48, 56  # byte offsets in the 256-byte header
W_FLAG_CAPACITY = 1


@pytest.fixture(scope="module")
def B():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2504_11320_amd import binding
    binding.lib()
    return binding


def _u64(host, off):
    return int(host[off:off + 8].view(np.uint64)[0])


def _random_mix():
    from tests.test_gpu_random import random_workload
    rng = np.random.default_rng(2024)
    return [W.Job(random_workload(rng), 5, W.ids(7)) for _ in range(10)]


CASES = {
    "wait-c2": (lambda: W.config2(replicas=70, rate_index=[0, 31]), 1500, 2500),
    "fcfs-chunked": (lambda: W.config_chunked(replicas=40, n_rates=2), 1000, 1500),
    "nested-c3": (lambda: W.config3(replicas=40, rate_index=[16, 31]), 1000, 1500),
    "nested-heavytail": (lambda: W.config5(replicas=48, record_capacity=1 << 14), 800, 1200),
    "wait-timevarying": (lambda: W.config_cyclic(replicas=40, rate_index=[20]), 1000, 1500),
    "pd-wait-and-fcfs": (lambda: W.config_pd(replicas=16), 600, 900),
    "random-mix": (_random_mix, 400, 600),
}


def _same(ref, got, ctx):
    for k in ref:
        assert np.array_equal(ref[k], got[k]), f"{ctx}: field {k} differs"


@pytest.mark.parametrize("name", list(CASES))
def test_run_batch_ex_resumes_bit_exact(B, name):
    import torch
    build, h1, h2 = CASES[name]
    jobs = build()
    print(f"[gpu] checkpoint {name}: {sum(j.n for j in jobs)} replicas, {h1}+{h2}", flush=True)
    ref = B.Simulation(jobs)
    ref.run_ex(h1 + h2)
    want = ref.results()

    a = B.Simulation(jobs)
    need = a.run_ex(h1)  # sizes the checkpoint without writing one
    buf = torch.zeros(need + 4096, dtype=torch.uint8, device="cuda")
    used = a.run_ex(h1, state_out=buf)  # the same h1 batches again, from t = 0
    assert used == need
    assert a.state_bytes() == used
    first = a.results()
    host = buf[:used].cpu()  # through host memory
    c = B.Simulation(jobs)
    c.run_ex(h2, state_in=host.to("cuda"))
    _same(want, c.results(), name)
    # saving does not disturb the saved workspace
    a.advance(h2, resume=True)
    _same(want, a.results(), name + " (saved workspace continued)")

    # the checkpoint holds the live state only
    hb = host.numpy()
    assert _u64(hb, HDR_USED) == used and used < a.ws_bytes
    dir_off, blob_off = _u64(hb, HDR_DIR), _u64(hb, HDR_BLOB)
    R = a.R
    starts = hb[dir_off:dir_off + 8 * R].view(np.uint64).astype(np.int64)
    sizes = np.diff(np.append(starts, used - blob_off))
    assert starts[0] == 0 and (sizes >= 0).all()
    print(f"[gpu] checkpoint {name}: {used} bytes ({used / a.ws_bytes:.2e} of the workspace)",
          flush=True)
    per_job = B.split_by_job(first, jobs)
    pos = 0
    for job, res in zip(jobs, per_job):
        s = sizes[pos:pos + job.n]
        pos += job.n
        if (res["flags"] & W_FLAG_CAPACITY).any():
            continue
        w, r = res["waiting_end"], res["resident_end"]
        if job.wl.policy in ("wait", "wait-nowait"):
            assert np.array_equal(s, 8 * w + 16 * r), name
        elif job.wl.policy == "fcfs":
            # a partially prefilled prompt (chunked prefill) lives in the
            # state slots, not in a resident record
            assert ((s <= 16 * (w + r)) & (s >= 16 * (w + r - 1))).all(), name
        else:
            seg = job.wl.seg_end
            entry = [0] + [e + 1 for e in seg[:-1]]
            fixed = sum((e - b + 1) * (32 * n + 4) for b, e, n in zip(entry, seg, job.wl.n))
            assert ((s >= fixed + 16 * w) & (s <= fixed + 16 * w + 32 * r)).all(), name


def test_checkpoint_chains(B):
    """Three calls, each resuming from the previous call's checkpoint, end
    where one call ends."""
    import torch
    jobs = W.config3(replicas=24, rate_index=[31])
    ref = B.Simulation(jobs)
    ref.run_ex(1800)
    want = ref.results()
    ck = None
    for i, h in enumerate((500, 700, 600)):
        s = B.Simulation(jobs)
        out = torch.empty(64 << 20, dtype=torch.uint8, device="cuda")
        used = s.run_ex(h, state_in=ck, state_out=out)
        ck = out[:used].clone()
        print(f"[gpu] checkpoint chain step {i}: {used} bytes", flush=True)
    _same(want, s.results(), "chain")


def test_checkpoint_refusals(B):
    """A checkpoint of other jobs, a damaged one, a truncated one and a blob
    directory that points past the checkpoint are refused with WS_EINVAL; a
    buffer too small for the checkpoint gives WS_EWORKSPACE and the size."""
    import torch
    jobs = W.config2(replicas=40, rate_index=[31])
    a = B.Simulation(jobs)
    a.run_ex(800)
    ck = a.checkpoint()
    used = ck.numel()

    def refused(sim, state, code):
        with pytest.raises(B.WaitSimError) as e:
            sim.restore(state)
        assert e.value.code == code, str(e.value)
        return str(e.value)

    other = [W.Job(j.wl, j.seed + 1, j.replica_ids) for j in jobs]
    assert "fingerprint" in refused(B.Simulation(other), ck, B.WS_EINVAL)
    bad = ck.clone()
    bad[0] ^= 1
    assert "magic" in refused(B.Simulation(jobs), bad, B.WS_EINVAL)
    refused(B.Simulation(jobs), ck[:used - 4].clone(), B.WS_EINVAL)
    host = ck.cpu().numpy()
    dir_off = _u64(host, HDR_DIR)
    R = a.R
    past = host.copy()
    past[dir_off + 8 * (R - 1): dir_off + 8 * R] = np.array([used], dtype=np.uint64).view(np.uint8)
    msg = refused(B.Simulation(jobs), torch.from_numpy(past).cuda(), B.WS_EINVAL)
    assert "blobs" in msg
    # the intact checkpoint still restores after the refusals
    b = B.Simulation(jobs)
    b.restore(ck)
    b.advance(300, resume=True)
    a.advance(300, resume=True)
    _same(a.results(), b.results(), "after refusals")
    # too small a buffer
    s = B.Simulation(jobs)
    small = torch.empty(1024, dtype=torch.uint8, device="cuda")
    with pytest.raises(B.WaitSimError) as e:
        s.run_ex(800, state_out=small)
    assert e.value.code == B.WS_EWORKSPACE and "needs" in str(e.value)
    assert s.state_bytes() == used
