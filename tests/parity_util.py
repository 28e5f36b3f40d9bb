"""Comparison of GPU results with the oracle's, field by field."""
import numpy as np

INT_FIELDS = ["batches", "arrivals", "completions", "completed_tokens",
              "evictions", "evicted_tokens", "fallback_evictions",
              "batch_tokens_sum", "peak_mem", "waiting_end", "resident_end",
              "idle_waits"]
F64_FIELDS = ["t_end", "busy_time", "lat_area", "ttft_area",
              "lat_completed_sum", "mem_area"]

# fp64 accumulators: the two sides perform the same IEEE operations in the
# same order, so they normally agree bit for bit; the bound allows reordering
# of a sum of at most ~1e4 terms.
RTOL = 1e-12


def compare(gpu: dict, ora: dict, ctx: str = "", rtol: float = RTOL) -> dict:
    """Assert integer fields equal and fp64 fields within rtol; return stats."""
    n = len(ora["batches"])
    for f in INT_FIELDS:
        g = np.asarray(gpu[f])[:n]
        o = np.asarray(ora[f])[:n]
        bad = np.nonzero(g != o)[0]
        assert bad.size == 0, (f"{ctx}: {f} differs at replicas {bad[:8].tolist()}: "
                               f"gpu {g[bad[:8]].tolist()} oracle {o[bad[:8]].tolist()}")
    g = np.asarray(gpu["flags"])[:n]
    o = np.asarray(ora["flags"])[:n]
    assert np.array_equal(g, o), f"{ctx}: flags {g[:8]} vs {o[:8]}"
    nb = ora["hist"].shape[1]
    assert np.array_equal(np.asarray(gpu["hist"])[:n, :nb], ora["hist"]), f"{ctx}: histogram"
    if gpu["hist"].shape[1] > nb:
        assert not np.any(np.asarray(gpu["hist"])[:n, nb:]), f"{ctx}: histogram padding"
    exact = 0
    total = 0
    for f in F64_FIELDS:
        g = np.asarray(gpu[f])[:n]
        o = np.asarray(ora[f])[:n]
        den = np.maximum(np.abs(o), 1e-300)
        rel = np.abs(g - o) / den
        rel[(g == o)] = 0.0
        worst = int(np.argmax(rel))
        assert rel[worst] <= rtol, (f"{ctx}: {f} rel err {rel[worst]:.3e} at replica {worst}: "
                                    f"gpu {g[worst]!r} oracle {o[worst]!r}")
        exact += int(np.sum(g.view(np.uint64) == o.view(np.uint64)))
        total += n
    return {"f64_bit_exact": exact, "f64_total": total}
