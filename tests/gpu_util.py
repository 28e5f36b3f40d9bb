"""Shared helpers of the GPU parity tests."""
import numpy as np
import pytest

from tests.parity_util import compare


def sim_module():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2504_11320_amd import binding as B
    B.lib()
    return B


def oracle_results(jobs, horizon):
    """Oracle results of several jobs, histograms zero-padded to one width."""
    from oracle import oracle as O
    outs = [O.run_job(j, horizon) for j in jobs]
    width = max(o["hist"].shape[1] for o in outs)
    for o in outs:
        h = o["hist"]
        o["hist"] = np.pad(h, ((0, 0), (0, width - h.shape[1])))
    return {k: np.concatenate([o[k] for o in outs]) for k in outs[0]}


def check(B, jobs, horizon, ctx):
    print(f"[gpu] {ctx}: {len(jobs)} jobs, {sum(j.n for j in jobs)} replicas, "
          f"horizon {horizon}", flush=True)
    g = B.run_batch(jobs, horizon)
    o = oracle_results(jobs, horizon)
    st = compare(g, o, ctx)
    print(f"[gpu] {ctx}: ok, fp64 bit-exact {st['f64_bit_exact']}/{st['f64_total']}",
          flush=True)
    return g, o
