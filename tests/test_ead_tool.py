"""CPU: the EAD tool's accounting (paper_2606_29223_amd/ead.py) against the
paper's worked example and, on random acceptance matrices, against the
oracle's independent implementation of Definitions 1, 3, 4 and
Proposition 3."""
import json
import os

import numpy as np
import pytest

from oracle import ead as oead
from paper_2606_29223_amd import ead as tool

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))


def test_exploration_example():
    g = GOLD["exploration_example"]
    assert tool.ceil_x(g["ead"], g["X"]) == g["ceil"]
    assert tool.resolution(g["X"], g["L"]) == g["resolution"]


@pytest.mark.parametrize("L,seed", [(4, 0), (12, 1), (32, 2)])
def test_accounting_matches_oracle(L, seed):
    rng = np.random.default_rng(seed)
    acc = (rng.random((300, L)) < 0.6).astype(np.int8)
    acc[:, -1] = 1
    for a in acc[:50]:
        lst = [int(x) for x in a]
        assert tool.ead(a) == oead.ead(lst)
        assert tool.ead_stable(a) == oead.ead_stable(lst)
    X = sorted({L, max(1, L // 2), max(1, L // 4)})
    out = tool.accounting(acc, X, L)
    es = [oead.ead_stable([int(x) for x in a]) for a in acc]
    lo, sx, hi = oead.speedup_bounds(L, es, X)
    assert out["S_X"] == pytest.approx(sx, rel=1e-12)
    assert out["S_EAD"] == pytest.approx(hi, rel=1e-12)
    assert out["S_lower"] == pytest.approx(lo, rel=1e-12)
    assert out["bounds_hold"] and out["overhead_in_bounds"]
    assert out["resolution"] == oead.resolution(X, L)
