"""The host-side calibration and analysis helpers of the package, checked
against the paper's worked example, closed forms, and the oracle (an
independent implementation of the fluid formulas and exact per-request
latencies)."""
import json
import os

import numpy as np
import pytest

import workloads as W
from paper_2504_11320_amd import analysis as A
from paper_2504_11320_amd import calibrate as K

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_calibration_worked_example():
    """Section 6: segments 1-20 and 21-50, continuation 0.3, tl = 30 gives
    segment caps of about 21 and 9."""
    g = json.load(open(os.path.join(GOLD, "calibration_two_segment.json")))
    r = K.calibrate_nested(g["tl"], [20, 50], g["p"], g["eta"])
    assert r["segment_caps"] == g["caps_rounded"]
    assert abs(20 * r["n"][0] + 30 * r["n"][1] - 30) < 1e-12
    assert abs(r["n"][1] / r["n"][0] - 0.3) < 1e-12
    assert [sum(c) for c in r["stage_caps"]] == g["caps_rounded"]
    assert len(r["stage_caps"][0]) == 20 and max(r["stage_caps"][0]) - min(r["stage_caps"][0]) <= 1


def test_calibration_matches_oracle_formula():
    from oracle import fluid as F
    rng = np.random.default_rng(7)
    for _ in range(50):
        L = int(rng.integers(1, 7))
        seg_end = np.cumsum(rng.integers(1, 200, L)).tolist()
        widths = [seg_end[0]] + [seg_end[k] - seg_end[k - 1] for k in range(1, L)]
        p = rng.uniform(0.0, 1.0, L - 1).tolist()
        tl, eta = float(rng.uniform(10, 500)), float(rng.choice([0.0, 0.05, 0.2]))
        a = K.calibrate_nested(tl, seg_end, p, eta)
        b = F.calibrate(tl, widths, p, eta)
        assert np.allclose(a["n"], b["n"], rtol=1e-12)
        assert a["segment_caps"] == [int(round(x)) for x in b["B"]]


def test_wait_calibration():
    r = K.calibrate_wait(21, 20)   # 21 over the prefill and 20 decode stages
    assert r["stage_caps"] == [1] * 21 and r["threshold"] == 1
    assert K.calibrate_wait(22, 20)["stage_caps"] == [2] + [1] * 20
    assert K.calibrate_wait(100, 9)["threshold"] == 10


def test_fluid_boundary_of_the_workloads():
    """The rate scales of the configured sweeps are the fluid boundaries."""
    from oracle import fluid as F
    es2 = K.mean_stage_work(W.C2_PROMPTS, W.C2_MIX, out_len=W.C2_OUTPUTS)
    lam2 = K.fluid_boundary(es2, 15.0, 0.05, 131072)
    assert abs(lam2 / W.LAM_STAR_C2 - 1) < 1e-12
    assert abs(lam2 / F.lambda_star(es2, 15.0, 0.05, 131072) - 1) < 1e-15
    # at Lambda* the fluid memory requirement is exactly C
    assert abs(F.fluid_mean_work(es2, lam2, 15.0, 0.05) / 131072 - 1) < 1e-12
    # distribution-mode rate scales were derived from the exact laws; the u32
    # CDF tables quantize each value to 2^-32 (a few 1e-9 relative in E[S])
    wl3 = W.config3(replicas=1, rate_index=[0])[0].wl
    es3 = K.mean_stage_work(wl3.prompt_len, W.C2_MIX, cdf=wl3.out_cdf, cap=wl3.out_cap)
    assert abs(K.fluid_boundary(es3, 15.0, 0.05, 131072) / W.LAM_STAR_C3 - 1) < 1e-8
    wl5 = W.config5(replicas=1)[0].wl
    m = len(wl5.prompt_len)
    es5 = K.mean_stage_work(wl5.prompt_len, [1.0 / m] * m, cdf=wl5.out_cdf, cap=wl5.out_cap)
    assert abs(K.fluid_boundary(es5, 15.0, 0.05, 262144) / W.LAM_STAR_C5 - 1) < 1e-8


def test_length_law_and_segments():
    """Geometric outputs (mean mu, capped): P(L > r) = (1 - 1/mu)^r below the
    cap; the segment rates and continuation probabilities follow."""
    cap = 2048
    mus = (64.0, 256.0, 512.0)
    cdf = np.stack([W.geometric_cdf_table(mu, cap) for mu in mus])
    for j, mu in enumerate(mus):
        pmf = K.length_pmf(cdf[j], cap)
        assert abs(pmf.sum() - 1) < 1e-12
        for r in (1, 64, 256, 1024):
            assert abs(pmf[r + 1:].sum() - (1 - 1 / mu) ** r) < 1e-8
    lam = [0.5, 0.3, 0.2]
    seg_end = [64, 256, 1024, 2048]
    rates = K.segment_rates(lam, seg_end, cdf=cdf, cap=cap)
    assert abs(sum(rates) - 1.0) < 1e-12
    tail = lambda r: sum(w * (1 - 1 / mu) ** r for w, mu in zip(lam, mus))
    p = K.continuation_probabilities(rates)
    assert abs(p[0] - tail(64)) < 1e-8
    assert abs(p[1] - tail(256) / tail(64)) < 1e-8
    assert abs(p[2] - tail(1024) / tail(256)) < 1e-8
    # known lengths: all mass in the segment holding l'
    assert K.segment_rates([1.0, 2.0], [10, 20], out_len=[10, 11]) == [1.0, 2.0]


def test_hist_percentile_brackets_exact_latency(oracle_lib):
    """The percentile from a histogram row is the upper edge of the bin that
    holds the exact empirical quantile of the completed latencies."""
    from oracle import oracle as O
    wl = W.config1()[0].wl
    r = O.run_one(wl, 0, 3, 4000, rlog_cap=200000)
    done = r["req_done"] >= 0
    lat = np.sort((r["req_done"] - r["req_arr"])[done])
    assert len(lat) == r["completions"]
    edges = wl.hist_edges
    for q in (0.1, 0.5, 0.9, 0.99):
        k = int(np.ceil(q * len(lat))) - 1
        exact = lat[max(k, 0)]
        up = A.hist_percentile(r["hist"], edges, q)
        b = int(np.searchsorted(edges, up))
        lo = edges[b - 1] if b > 0 else -np.inf
        assert lo <= exact < up, (q, exact, lo, up)


def test_summaries_and_lambda_hat(oracle_lib):
    from oracle import oracle as O
    jobs = W.config2(replicas=4, rate_index=[0, 31])
    res = [O.run_job(j, 3000) for j in jobs]
    s = [A.summarize(x) for x in res]
    for x, y in zip(res, s):
        assert np.allclose(y["completion_rate"], x["completions"] / x["t_end"])
        assert np.all(y["busy_fraction"] <= 1.0)
    means = A.job_means(np.concatenate([y["completion_rate"] for y in s]), [4, 4])
    assert len(means) == 2 and all(np.isfinite(m) for m, _ in means)
    rates = [1.0, 2.0, 3.0, 4.0]
    assert A.lambda_hat(rates, [1.0, 1.97, 2.5, 4.0], tol=0.05) == 2.0
    assert A.lambda_hat(rates, [0.5, 2.0, 3.0, 4.0]) == 0.0
    assert A.lambda_hat(rates[::-1], [4.0, 3.0, 2.0, 1.0]) == 4.0
