"""Comparison rules between the oracle and a device result (test infrastructure).

Block selection is decided by floating-point scores, and the device sums them
in fp32 in another order than the oracle's float64, so two blocks whose
scores differ by less than the rounding can swap places at the top-n
threshold. The rule: the device set has exactly n ids, ascending and unique,
contains the forced local blocks, and every id in the symmetric difference
with the oracle's set has an oracle score within ``tol`` of the threshold
(the smallest finite score the oracle kept).
"""
from __future__ import annotations

import numpy as np


def check_selection(dev_idx, ref_idx, ref_scores, n, n_local, tol=1e-3):
    """Returns the number of near-tie swaps; raises AssertionError on a violation."""
    dev = [int(x) for x in dev_idx]
    ref = [int(x) for x in ref_idx]
    M = len(ref_scores)
    assert len(dev) == n, f"device kept {len(dev)} blocks, expected {n}"
    assert dev == sorted(set(dev)), "device ids not ascending and unique"
    assert all(0 <= m < M for m in dev), "device id out of range"
    forced = set(range(max(M - n_local, 0), M))
    assert forced <= set(dev), "a forced local block is missing"
    diff = set(dev) ^ set(ref)
    if not diff:
        return 0
    finite = [ref_scores[m] for m in ref if m not in forced]
    assert finite, "sets differ although every kept block is forced"
    tau = min(finite)
    for m in diff:
        assert abs(ref_scores[m] - tau) <= tol, (
            f"block {m}: score {ref_scores[m]:.6f} is {abs(ref_scores[m] - tau):.3e} from the "
            f"threshold {tau:.6f} (tolerance {tol})")
    return len(diff) // 2


def max_abs_err(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    both_inf = np.isneginf(a) & np.isneginf(b)
    d = np.where(both_inf, 0.0, np.abs(a - b))
    return float(np.max(d)) if d.size else 0.0
