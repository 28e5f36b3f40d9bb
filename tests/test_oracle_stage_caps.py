"""Per-stage caps of Nested WAIT and WAIT (Section 6, "WAIT and Nested WAIT
settings"), in the oracle.

The experiments turn a system-wide batch-size cap tl into segment caps B_k
and spread each over the segment's decode stages, so caps inside a segment
differ by one.  Reading A29: segment k takes its stages' caps in turn, one
per service, as the size of the entering cohort (its threshold for that
service).  Pinned by a hand trace (golden/nested_stage_caps.json: caps
(2, 1) and (1, 0) on two segments, batch by batch), by the reduction to the
one-threshold policy when every cap of a segment equals n_k, by the prefill
sequence of the tl = 30 calibration, and by copies of the oracle with a
planted misreading that the hand trace rejects.  WAIT (one type: tl spread over
its prefill and decode stages) has the same four kinds of pins
(golden/wait_stage_caps.json, caps (2, 1, 1)).
"""
import json
import os
import subprocess

import numpy as np
import pytest

import workloads as W

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                    "nested_stage_caps.json")
FIELDS = ("tokens", "prefills", "selected", "completions", "evict_pre", "evict_post",
          "mem_after", "waiting_after", "resident_after", "mplus")


def _gold():
    with open(GOLD) as f:
        return json.load(f)


def _workload(g):
    i = g["instance"]
    times = [a[0] for a in i["arrivals"]]
    lengths = [a[1] for a in i["arrivals"]]
    return W.trace_workload("nested", [i["prompt_len"]], None, i["d0"], i["d1"], i["C"],
                            i["n"], times, [0] * len(times), lengths=lengths,
                            seg_end=i["seg_end"], out_cap=i["out_cap"],
                            stage_caps=i["stage_caps"])


def _mismatches(r, g):
    bad = []
    bt = r["batches_trace"]
    if len(bt) != len(g["batches"]):
        bad.append(f"{len(bt)} batches")
    for b, (got, want) in enumerate(zip(bt, g["batches"])):
        for f in FIELDS + ("t_launch",):
            if got[f] != want[f]:
                bad.append(f"batch {b} {f}: {got[f]} != {want[f]}")
    for k, v in g["final"].items():
        if r[k] != v:
            bad.append(f"{k}: {r[k]} != {v}")
    return bad


def _run(O, g, library=None):
    h = g["instance"]["horizon"]
    return O.run_one(_workload(g), 0, 0, h, btrace_cap=h, library=library)


def test_golden_arithmetic_is_consistent():
    g = _gold()
    caps = g["instance"]["stage_caps"]
    r1 = g["instance"]["seg_end"][0]
    # every batch serves segment 1, whose cohorts take its caps in turn
    for b, want in enumerate(g["batches"]):
        assert want["prefills"] == caps[b % r1]
    fin = g["final"]
    assert fin["batch_tokens_sum"] == sum(b["tokens"] for b in g["batches"])
    assert fin["completions"] == sum(b["completions"] for b in g["batches"])
    assert fin["arrivals"] == len(g["instance"]["arrivals"])
    assert fin["resident_end"] == g["batches"][-1]["resident_after"]


def test_stage_caps_hand_trace(oracle_lib):
    g = _gold()
    assert _mismatches(_run(oracle_lib, g), g) == []


def _random_nested(rng):
    m = int(rng.integers(1, 4))
    cap = int(rng.integers(3, 30))
    nseg = int(rng.integers(1, min(4, cap) + 1))
    cuts = sorted(rng.choice(np.arange(1, cap), size=nseg - 1, replace=False).tolist())
    seg_end = [int(c) for c in cuts] + [cap]
    n = [int(x) for x in rng.integers(1, 4, nseg)]
    l = [int(x) for x in rng.integers(1, 40, m)]
    cdf = np.stack([W.geometric_cdf_table(float(rng.uniform(1.5, cap)), cap) for _ in range(m)])
    C = int((max(l) + cap) * rng.uniform(1.0, 6.0))
    return W.Workload(prompt_len=l, lam=[float(x) for x in rng.uniform(0.02, 1.0, m)],
                      d0=float(rng.uniform(0.5, 5.0)), d1=float(rng.uniform(0.0, 0.02)),
                      C=C, policy="nested", n=n, out_cap=cap, out_cdf=cdf, seg_end=seg_end,
                      hist_edges=W.default_edges(1.0, 64), record_capacity=1 << 14)


def test_uniform_caps_are_the_one_threshold_policy(oracle_lib):
    """Caps all equal to n_k in segment k give the policy without caps, bit
    for bit (random models, evictions included)."""
    O = oracle_lib
    rng = np.random.default_rng(31)
    for _ in range(12):
        wl = _random_nested(rng)
        caps = []
        lo = 0
        for e, nk in zip(wl.seg_end, wl.n):
            caps += [nk] * (e - lo)
            lo = e
        a = O.run(wl, 4, W.ids(4), 1500)
        wl.stage_caps = caps
        b = O.run(wl, 4, W.ids(4), 1500)
        for k in a:
            assert np.array_equal(a[k], b[k]), k


def test_tl30_calibration_sets_the_prefill_sequence(oracle_lib):
    """On the two-type p512 mix with the caps tl = 30 gives, every batch
    admits into segment 1 exactly the cap of the segment's stage its service
    count points at: prefills follow (2, 1, ..., 1) with period 20."""
    from paper_2504_11320_amd import calibrate as Cal
    cal = Cal.calibrate_nested(30, W.P512MIX_SEG_END, [0.3], eta=0.0)
    assert cal["segment_caps"] == [21, 9]
    assert sum(cal["stage_caps"], []) == W.P512MIX_CAPS_TL30
    job = W.config_p512_mix(replicas=1, rates=[0.022])[0]
    r = oracle_lib.run_one(job.wl, 0, 0, 400, btrace_cap=400)
    pre = [b["prefills"] for b in r["batches_trace"]]
    assert pre == [W.P512MIX_CAPS_TL30[b % 20] for b in range(400)]


# ------------------------------------------------- planted misreadings ----

MUTATIONS = {
    # the x-th service takes the cap of stage r_{k-1} + 1 + x mod width
    "cap_offset": ("return c->stage_caps[lo + (int32_t)(S->nsvc[k] % width)];",
                   "return c->stage_caps[lo + (int32_t)((S->nsvc[k] + 1) % width)];"),
    # interior cells limited by the cap of the current service
    "cell_limit": ("select_by_stage(S, lo, i, -1, tokens);",
                   "select_by_stage(S, lo, i, nk, tokens);"),
    # the caps are not taken in turn: every service uses the first
    "no_rotation": ("    S->nsvc[k]++;\n", "\n"),
    # one threshold per segment (the largest cap)
    "segment_max": ("  if (!c->stage_caps) return c->n[k - 1];",
                    "  if (c->stage_caps) return c->n[k - 1];"),
}


def _mutant(O, tmp_path, name):
    src = open(O.SRC).read()
    old, new = MUTATIONS[name]
    assert src.count(old) == 1, name
    path = tmp_path / f"wait_oracle_{name}.c"
    path.write_text(src.replace(old, new))
    lib = tmp_path / f"liboracle_{name}.so"
    subprocess.run(["gcc", "-O2", "-std=gnu11", "-ffp-contract=off", "-fno-fast-math",
                    "-fPIC", "-shared", "-I", os.path.dirname(O.SRC), "-o", str(lib),
                    str(path), "-lpthread", "-lm"], check=True)
    return O.load(str(lib))


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_hand_trace_rejects_planted_misreading(oracle_lib, tmp_path, name):
    g = _gold()
    lib = _mutant(oracle_lib, tmp_path, name)
    assert _mismatches(_run(oracle_lib, g, library=lib), g), name


# ----------------------------------------------------------------- WAIT ----

WAIT_GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                         "wait_stage_caps.json")
WAIT_FIELDS = tuple(f for f in FIELDS if f != "mplus")


def _wait_gold():
    with open(WAIT_GOLD) as f:
        return json.load(f)


def _wait_workload(g):
    i = g["instance"]
    n = len(i["arrivals"])
    return W.trace_workload("wait", [i["prompt_len"]], [i["out_len"]], i["d0"], i["d1"], i["C"],
                            i["n"], i["arrivals"], [0] * n, stage_caps=i["stage_caps"])


def _wait_mismatches(r, g):
    bad = []
    bt = r["batches_trace"]
    if len(bt) != len(g["batches"]):
        bad.append(f"{len(bt)} batches")
    for b, (got, want) in enumerate(zip(bt, g["batches"])):
        for f in WAIT_FIELDS + ("t_launch",):
            if got[f] != want[f]:
                bad.append(f"batch {b} {f}: {got[f]} != {want[f]}")
    for k, v in g["final"].items():
        if r[k] != v:
            bad.append(f"{k}: {r[k]} != {v}")
    return bad


def _wait_run(O, g, library=None):
    h = g["instance"]["horizon"]
    return O.run_one(_wait_workload(g), 0, 0, h, btrace_cap=h, library=library)


def test_wait_golden_is_consistent():
    g = _wait_gold()
    fin = g["final"]
    assert fin["batch_tokens_sum"] == sum(b["tokens"] for b in g["batches"])
    assert fin["completions"] == sum(b["completions"] for b in g["batches"])
    assert fin["arrivals"] == len(g["instance"]["arrivals"])


def test_wait_stage_caps_hand_trace(oracle_lib):
    g = _wait_gold()
    assert _wait_mismatches(_wait_run(oracle_lib, g), g) == []


def _random_wait(rng):
    m = int(rng.integers(1, 4))
    l = [int(x) for x in rng.integers(1, 40, m)]
    lp = [int(x) for x in rng.integers(1, 20, m)]
    n = [int(x) for x in rng.integers(1, 4, m)]
    C = int(max(a + b for a, b in zip(l, lp)) * rng.uniform(1.0, 5.0))
    return W.Workload(prompt_len=l, lam=[float(x) for x in rng.uniform(0.02, 1.0, m)],
                      d0=float(rng.uniform(0.5, 5.0)), d1=float(rng.uniform(0.0, 0.02)),
                      C=C, policy="wait", n=n, out_len=lp,
                      hist_edges=W.default_edges(1.0, 64), record_capacity=1 << 14)


def test_wait_uniform_caps_are_the_one_threshold_policy(oracle_lib):
    """Caps all equal to n_j over type j's l'_j + 1 stages reproduce WAIT
    without caps, bit for bit (random models, evictions included)."""
    O = oracle_lib
    rng = np.random.default_rng(41)
    for _ in range(12):
        wl = _random_wait(rng)
        a = O.run(wl, 4, W.ids(4), 1500)
        wl.stage_caps = sum(([nj] * (lpj + 1) for nj, lpj in zip(wl.n, wl.out_len)), [])
        b = O.run(wl, 4, W.ids(4), 1500)
        for k in a:
            assert np.array_equal(a[k], b[k]), k


def test_wait_tl30_calibration_sets_the_prefill_sequence(oracle_lib):
    """Single-type p512d20 WAIT with the caps tl = 30 gives (30 over 21
    stages: 2 on the first nine, 1 on the rest): while the queue never runs
    short of the next cap, the admissions follow the caps with period 21."""
    from paper_2504_11320_amd import calibrate as Cal
    cal = Cal.calibrate_wait(30, 20)
    assert cal["stage_caps"] == [2] * 9 + [1] * 12
    wl = W.config_p512d20(replicas=1)[6].wl  # the boundary rate under WAIT
    wl.stage_caps = cal["stage_caps"]
    wl.n = [2]
    wl.lam = [0.5]  # a queue that never empties
    r = oracle_lib.run_one(wl, 0, 0, 300, btrace_cap=300)
    pre = [b["prefills"] for b in r["batches_trace"]]
    assert pre == [cal["stage_caps"][b % 21] for b in range(300)]


WAIT_MUTATIONS = {
    "wait_cap_offset": ("return c->stage_caps[lo + S->nsvc[j] % (c->lp[j] + 1)];",
                        "return c->stage_caps[lo + (S->nsvc[j] + 1) % (c->lp[j] + 1)];"),
    "wait_no_rotation": ("    select_by_stage(S, 0, cnt, -1, tokens);\n    S->nsvc[j]++;\n",
                         "    select_by_stage(S, 0, cnt, -1, tokens);\n"),
    "wait_cell_limit": ("    select_by_stage(S, 0, cnt, -1, tokens);\n    S->nsvc[j]++;\n",
                        "    select_by_stage(S, 0, cnt, cap, tokens);\n    S->nsvc[j]++;\n"),
    "wait_one_threshold": ("  if (!c->stage_caps) return c->n[j];",
                           "  if (c->stage_caps) return c->n[j];"),
}


@pytest.mark.parametrize("name", sorted(WAIT_MUTATIONS))
def test_wait_hand_trace_rejects_planted_misreading(oracle_lib, tmp_path, name):
    g = _wait_gold()
    src = open(oracle_lib.SRC).read()
    old, new = WAIT_MUTATIONS[name]
    assert src.count(old) == 1, name
    path = tmp_path / f"wait_oracle_{name}.c"
    path.write_text(src.replace(old, new))
    lib = tmp_path / f"liboracle_{name}.so"
    subprocess.run(["gcc", "-O2", "-std=gnu11", "-ffp-contract=off", "-fno-fast-math",
                    "-fPIC", "-shared", "-I", os.path.dirname(oracle_lib.SRC), "-o", str(lib),
                    str(path), "-lpthread", "-lm"], check=True)
    assert _wait_mismatches(_wait_run(oracle_lib, g, library=oracle_lib.load(str(lib))), g), name
