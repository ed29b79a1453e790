"""Oracle: the depth-side accounting of Section 2 (used as test pins).

TEST INFRASTRUCTURE ONLY (see oracle/model.py).

  * Definition 1: acceptance Omega(t, l), earliest available depth EAD and its
    stable version (accepted at l and at every deeper depth).
  * Definition 2 / Proposition 1: expected layer cost of depth selection and
    its overhead over the EAD oracle.
  * Definition 3: depth ceiling ceil_X(l) and resolution Delta(X).
  * Definition 4 / Proposition 2: exploration workload W_X(t) = ceil_X(EAD(t)).
  * Proposition 3: depth-side speedup S = L T / sum_t W(t).
"""

from __future__ import annotations

import numpy as np


def ceil_x(l: int, X) -> int:
    """Smallest explored depth >= l."""
    return min(d for d in X if d >= l)


def resolution(X, L: int) -> int:
    """Largest upward rounding ceil_X(l) - l over l in [1, L]."""
    return max(ceil_x(l, X) - l for l in range(1, L + 1))


def acceptance(depth_tokens, final_token) -> list:
    """Omega(t, l) for l = 1..L under greedy decoding: the depth-l argmax equals
    the final-depth token; Omega(t, L) = 1 by construction."""
    acc = [int(t == final_token) for t in depth_tokens]
    acc[-1] = 1
    return acc


def ead(acc) -> int:
    """Earliest accepted depth (1-based)."""
    return 1 + acc.index(1)


def ead_stable(acc) -> int:
    """Earliest depth accepted at itself and at every deeper depth."""
    L = len(acc)
    e = L
    for l in range(L, 0, -1):
        if acc[l - 1]:
            e = l
        else:
            break
    return e


def selection_cost(L: int, s_t: int, p_acc: float, discarded) -> float:
    """Expected layer cost charged to a position by depth selection
    (Proposition 1's workload): p s_t + (1-p) (L + sum of discarded exits)."""
    return p_acc * s_t + (1.0 - p_acc) * (L + sum(discarded))


def selection_overhead(L: int, s_t: int, p_acc: float, discarded, ead_t: int) -> float:
    return selection_cost(L, s_t, p_acc, discarded) - ead_t


def exploration_workload(ead_t: int, X) -> int:
    return ceil_x(ead_t, X)


def exploration_overhead(ead_t: int, X) -> int:
    return ceil_x(ead_t, X) - ead_t


def speedup(L: int, workloads) -> float:
    return L * len(workloads) / float(sum(workloads))


def speedup_bounds(L: int, eads, X):
    """(lower, S_X, upper) of Proposition 3."""
    D = resolution(X, L)
    lower = speedup(L, [min(e + D, L) for e in eads])
    sx = speedup(L, [ceil_x(e, X) for e in eads])
    upper = speedup(L, list(eads))
    return lower, sx, upper


def depth_argmaxes(logits_all_depths: np.ndarray) -> np.ndarray:
    """[T, L, V] -> [T, L] argmax with lowest-id ties."""
    return np.argmax(logits_all_depths, axis=-1)
