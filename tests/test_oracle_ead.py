"""Pins of Section 2's accounting against the paper's worked examples and the
propositions' closed forms."""
import json
import os

import numpy as np
import pytest

from oracle import ead

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))


def test_exploration_example():
    g = GOLD["exploration_example"]
    assert ead.ceil_x(g["ead"], g["X"]) == g["ceil"]
    assert ead.exploration_overhead(g["ead"], g["X"]) == g["overhead"]
    assert ead.resolution(g["X"], g["L"]) == g["resolution"]


def test_selection_example():
    g = GOLD["selection_example"]
    L, e = g["L"], g["ead"]
    c = g["conservative"]
    assert ead.selection_overhead(L, c["s"], 1.0, [], e) == c["overhead"]
    a = g["aggressive"]
    # a failed aggressive exit charges L + s_t + s_{t+1} + s_{t+2}
    for s1, s2 in [(4, 4), (3, 9), (0, 0)]:
        cost = ead.selection_cost(L, a["s"], 0.0, [a["s"], s1, s2])
        assert cost == a["charged_constant"] + s1 + s2


def test_stable_ead():
    acc = ead.acceptance([5, 9, 9, 5, 9, 9, 9], 9)
    assert ead.ead(acc) == 2
    assert ead.ead_stable(acc) == 5
    assert ead.ead_stable(ead.acceptance([1, 2, 3], 7)) == 3       # only the final depth


@pytest.mark.parametrize("L", [8, 20, 32])
def test_speedup_bounds_and_monotonicity(L):
    rng = np.random.default_rng(L)
    eads = [int(x) for x in rng.integers(1, L + 1, size=200)]
    Xc = sorted({L, L // 2, L // 4} - {0})
    Xf = sorted(set(Xc) | {L // 8 or 1, 3 * L // 4})
    lo, sx, hi = ead.speedup_bounds(L, eads, Xc)
    assert 1.0 <= lo <= sx <= hi
    _, sxf, _ = ead.speedup_bounds(L, eads, Xf)
    assert sx <= sxf <= hi
    # X = [L] reaches the EAD oracle
    _, s_all, s_ead = ead.speedup_bounds(L, eads, list(range(1, L + 1)))
    assert s_all == s_ead
    for e in eads:
        assert 0 <= ead.exploration_overhead(e, Xc) <= ead.resolution(Xc, L)
