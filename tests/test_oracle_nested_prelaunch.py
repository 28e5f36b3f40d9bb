"""Hand traces of Nested WAIT's pre-launch repair (Algorithm 4, Appendix B.1).

Before a batch launches, Nested WAIT projects the state Q+ that the batch
would leave if no selected prompt completed early, and while M_res(Q+) > C it
evicts unselected resident boundary prompts, most recently admitted first.
The instances in golden/nested_prelaunch_repair.json were traced by hand from
that definition, the M_res formula of Section 5.1 and the readings A1-A3,
A11, A15 and A20 (the file states each batch's arithmetic).  They fix, batch
by batch, Q+ before and after the repair, the number of evictions, which
prompt is evicted and of what kind, the interior fallback and the OVERFLOW
flag.

The second half builds copies of the oracle with one plausible misreading
planted in each (on the CPU) and checks that the hand traces reject every one
of them: a survivor charged l + r_k + 1, the selected prefills left out of
Q+, a boundary prompt projected one stage short, FIFO instead of LIFO victim
choice.
"""
import json
import os
import subprocess

import pytest

from workloads import trace_workload

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                    "nested_prelaunch_repair.json")
FIELDS = ("tokens", "prefills", "selected", "completions", "evict_pre", "evict_post",
          "mem_after", "waiting_after", "resident_after")
FLAG_OVERFLOW = 4


def _instances():
    with open(GOLD) as f:
        return json.load(f)["instances"]


def _workload(g):
    times = [a[0] for a in g["arrivals"]]
    types = [a[1] for a in g["arrivals"]]
    lengths = [a[2] for a in g["arrivals"]]
    return trace_workload("nested", g["prompt_len"], None, g["d0"], g["d1"], g["C"], g["n"],
                          times, types, lengths=lengths, seg_end=g["seg_end"],
                          out_cap=g["out_cap"])


def _run(O, g, library=None):
    h = g["horizon"]
    return O.run_one(_workload(g), 0, 0, h, btrace_cap=h, evlog_cap=64, library=library)


def _mismatches(r, g):
    """Every way the oracle's run differs from the hand trace."""
    bad = []
    bt = r["batches_trace"]
    if len(bt) != len(g["batches"]):
        bad.append(f"{len(bt)} batches, want {len(g['batches'])}")
    for b, (got, want) in enumerate(zip(bt, g["batches"])):
        for f in FIELDS:
            if got[f] != want[f]:
                bad.append(f"batch {b} {f}: {got[f]} != {want[f]}")
        if got["mplus"] != want["mplus_after"]:
            bad.append(f"batch {b} M_res(Q+) after repair: {got['mplus']} != {want['mplus_after']}")
        if got["tau"] != g["d0"] + g["d1"] * want["tokens"]:
            bad.append(f"batch {b} tau {got['tau']}")
    victims = [tuple(v[:3]) for v in g["victims"]]
    if r["evictions_log"] != victims:
        bad.append(f"victims {r['evictions_log']} != {victims}")
    for k, v in g["final"].items():
        if k == "overflow":
            if bool(r["flags"] & FLAG_OVERFLOW) != v:
                bad.append(f"overflow flag {r['flags']}")
        elif r[k] != v:
            bad.append(f"{k}: {r[k]} != {v}")
    return bad


def test_golden_arithmetic_is_consistent():
    """The stored trace is self-consistent: Q+ falls by exactly the charges of
    the batch's victims, the victims count as that batch's pre-launch
    evictions, and the totals add up."""
    for name, g in _instances().items():
        for b, want in enumerate(g["batches"]):
            freed = sum(v[3] for v in g["victims"] if v[0] == b)
            assert want["mplus_before"] - want["mplus_after"] == freed, (name, b)
            assert want["evict_pre"] == sum(1 for v in g["victims"] if v[0] == b), (name, b)
            assert want["mplus_after"] <= g["C"] or g["final"]["overflow"], (name, b)
        fin = g["final"]
        assert fin["batch_tokens_sum"] == sum(b["tokens"] for b in g["batches"]), name
        assert fin["completions"] == sum(b["completions"] for b in g["batches"]), name
        assert fin["evictions"] == sum(b["evict_pre"] + b["evict_post"] for b in g["batches"])
        assert fin["fallback_evictions"] == sum(1 for v in g["victims"] if v[2] == 3), name
        assert fin["waiting_end"] == g["batches"][-1]["waiting_after"], name
        assert fin["resident_end"] == g["batches"][-1]["resident_after"], name


@pytest.mark.parametrize("name", ["boundary_lifo", "interior_fallback",
                                  "fallback_then_overflow", "three_segments"])
def test_prelaunch_repair_hand_trace(oracle_lib, name):
    g = _instances()[name]
    r = _run(oracle_lib, g)
    assert _mismatches(r, g) == []


# ------------------------------------------------- planted misreadings ----

MUTATIONS = {
    # a prompt selected at the end r_k of segment k < L is projected into the
    # next boundary queue at l + r_k + 1 instead of l + r_k
    "survivor_charge": ("return k < c->nseg ? l + c->seg_end[k - 1] : 0;",
                        "return k < c->nseg ? l + c->seg_end[k - 1] + 1 : 0;"),
    # the selected prefills are left out of M_res(Q+)
    "prefills_missing": ("if (r->sp == 0) mplus += projected_charge(c, c->l[r->j], 1, 0);",
                         "if (0) mplus += projected_charge(c, c->l[r->j], 1, 0);"),
    # a selected boundary prompt is projected one stage short (l + r_{k-1} + 1)
    "boundary_stage": ("mplus += r->sel ? projected_charge(c, c->l[r->j], k, r->sp)",
                       "mplus += r->sel ? projected_charge(c, c->l[r->j], k, r->sp - 1)"),
    # the pre-launch repair evicts the oldest unselected boundary prompt
    "fifo_victim": ("        if (S->R[r].sel) continue;\n"
                    "        if (best < 0 || key_less(&S->R[best], &S->R[r])) best = r;",
                    "        if (S->R[r].sel) continue;\n"
                    "        if (best < 0 || key_less(&S->R[r], &S->R[best])) best = r;"),
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
def test_hand_traces_reject_planted_misreading(oracle_lib, tmp_path, name):
    O = oracle_lib
    lib = _mutant(O, tmp_path, name)
    bad = []
    for g in _instances().values():
        bad += _mismatches(_run(O, g, library=lib), g)
    assert bad, f"the misreading {name} passes every hand trace"
