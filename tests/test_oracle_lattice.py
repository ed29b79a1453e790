"""Pins of the oracle's lattice bookkeeping with a scripted (fake) exit head.

No model: each node's candidate is dictated by a script that knows the true
token sequence and a chosen match depth k*_t per commit, so every outcome
pattern can be exercised.  Checked against what the paper prints
(Section 3.2: 2^q - 1 tokens at state q, the buffer ETK_0..ETK_14 at state 4
with ETK_1 the depth child and ETK_2 the position child of ETK_0; Appendix E:
2^K - 1 tokens per cycle and a largest batch of 128 at K = 8) and against the
closed-form round count of an uncapped lattice.
"""
import itertools
import json
import os

import numpy as np
import pytest

from oracle.lattice import Lattice

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))
P = 5  # prompt length (positions of the scripted sequences)


def _prefix(lat, slot, committed):
    chain = slot.ancestors()
    return committed + [a.x for a in chain[1:]] + ([slot.x] if slot is not lat.anchor else [])


def _scripted_token(prefix, stage, mask, truth, pattern, N, vocab=10_000):
    pos = len(prefix) - 1
    t = pos + 1 - P
    on_path = prefix[P:] == truth[: len(prefix) - P]
    if on_path and t < len(truth):
        if stage == N - 1:
            return truth[t]
        k = pattern[t] if t < len(pattern) else N - 1
        if stage == k:
            return truth[t]
        if stage < k:
            d = 0
            while d in mask or d == truth[t]:
                d += 1
            return d
    h = hash((tuple(prefix), stage)) % vocab + 1000
    while h in mask:
        h += 1
    return h


def run_scripted(N, W, decs, truth, pattern, max_context=10 ** 9, on_round=None):
    """Drive a Lattice with the scripted head.  truth[0] is the prefill token."""
    committed = list(range(100, 100 + P)) + [truth[0]]
    lat = Lattice(N, W, decs, max_context, truth[0], P)
    rounds, kst, rows_log = 0, [], []
    while len(committed) - P < len(truth):
        rows = lat.begin_round()
        for r in rows:   # eligibility: ancestors' keys at this stage exist from earlier rounds
            for a in r.slot.ancestors():
                assert a.c > r.stage or (r.new and r.stage == 0 and a.c >= 1)
        toks = [_scripted_token(_prefix(lat, r.slot, committed), r.stage, lat.mask(r.slot, r.stage),
                                truth, pattern, N) for r in rows]
        if on_round:
            on_round(lat, rows)
        rows_log.append([(lat.index(r.slot), r.stage) for r in rows])
        cm = lat.end_round(rows, toks)
        rounds += 1
        if cm is not None:
            assert cm.token == truth[len(committed) - P]
            committed.append(cm.token)
            kst.append(cm.kstar)
    return rounds, kst, rows_log


def test_fsm_counts_and_heap_numbering_printed_in_paper():
    g = GOLD["lattice_fsm"]
    N = g["explorers"]
    truth = list(range(50, 60))
    heap = {}
    sizes = []

    def on_round(lat, rows):
        for r in rows:
            s = r.slot
            if r.new:
                parent_node = heap[(s.parent.uid, s.fork_stage)]
                heap[(s.uid, 0)] = 2 * parent_node + 2
            elif r.stage == 0:
                heap[(s.uid, 0)] = 0
            else:
                heap[(s.uid, r.stage)] = 2 * heap[(s.uid, r.stage - 1)] + 1
        sizes.append(len(heap))

    # no reuse in the first cycle: k* = N-1 at the first commit
    run_scripted(N, 0, True, truth[:2], [None, N - 1], on_round=on_round)
    assert sizes == [2 ** q - 1 for q in range(1, N + 1)]
    assert sorted(heap.values()) == g["buffer_at_state_4"]
    assert heap[(0, 1)] == g["depth_child_of_0"]
    anchors = [heap[(0, k)] for k in range(N)]
    assert anchors == [0, 1, 3, 7]


@pytest.mark.parametrize("kstar", [0, 1, 2, 3])
def test_collapse_keeps_subtree_of_matched_branch(kstar):
    N = 4
    truth = list(range(50, 60))
    kept = {}

    lat_holder = {}

    def on_round(lat, rows):
        lat_holder["lat"] = lat

    rounds, kst, _ = run_scripted(N, 0, True, truth[:2], [None, kstar], on_round=on_round)
    lat = lat_holder["lat"]
    assert kst == [kstar]
    # nodes retained: completed stages of every kept slot
    nodes = sum(s.c for s in lat.slots)
    if kstar <= N - 2:
        assert nodes == 2 ** (N - 1 - kstar) - 1
        assert lat.q == N - 1 - kstar            # FSM resumes at the matched child's depth
    else:
        assert nodes == 0 and lat.q == 0


def test_expansion_growth_K8():
    g = GOLD["expansion_growth"]
    K = g["explorers"]
    sizes = []
    run_scripted(K, 0, True, [7, 8], [None, K - 1], on_round=lambda lat, rows: sizes.append(len(rows)))
    assert sizes == [2 ** r for r in range(K)]
    assert sum(sizes) == 2 ** K - 1
    assert max(sizes) == g["largest_batch"]


@pytest.mark.parametrize("N", [2, 3, 4, 5])
def test_uncapped_rounds_closed_form(N):
    rng = np.random.default_rng(N)
    for trial in range(20):
        T = 12
        truth = list(range(3000, 3000 + T))
        pattern = [None] + [int(x) for x in rng.integers(0, N, size=T - 1)]
        rounds, kst, _ = run_scripted(N, 0, True, truth, pattern)
        assert kst == pattern[1:]
        assert rounds == N + sum(k + 1 for k in pattern[1:T - 1])


@pytest.mark.parametrize("N", [2, 3, 4])
def test_wide_cap_reproduces_uncapped_lattice(N):
    rng = np.random.default_rng(10 + N)
    T = 10
    truth = list(range(3000, 3000 + T))
    pattern = [None] + [int(x) for x in rng.integers(0, N, size=T - 1)]
    a = run_scripted(N, 0, True, truth, pattern)
    b = run_scripted(N, 2 ** (N - 1), True, truth, pattern)
    assert a == b


@pytest.mark.parametrize("N,W", [(4, 1), (4, 2), (4, 4), (8, 8), (16, 16), (16, 4)])
def test_capped_lattice_invariants(N, W):
    rng = np.random.default_rng(N * 100 + W)
    T = 24
    truth = list(range(5000, 5000 + T))
    pattern = [None] + [int(x) for x in rng.integers(0, N, size=T - 1)]
    log = []

    def on_round(lat, rows):
        assert rows[0].slot is lat.anchor and rows[0].stage == lat.anchor.c
        assert len(rows) <= W
        assert len({id(r.slot) for r in rows}) == len(rows)      # one stage per slot per round
        log.append(len(rows))

    rounds, kst, _ = run_scripted(N, W, True, truth, pattern, on_round=on_round)
    assert len(kst) == T - 1
    # a width-1 lattice is plain one-row-per-round decoding of the anchor
    if W == 1:
        assert rounds == N * (T - 1)
    # never slower than no reuse, never faster than one commit per round
    assert T - 1 <= rounds <= N * (T - 1)


def test_single_exit_reduction():
    """X = {d, L} (N = 2) is single-exit draft/verify: a commit takes one round
    when the exit-d draft matched the final token and two otherwise."""
    rng = np.random.default_rng(3)
    T = 30
    truth = list(range(100, 100 + T))
    pattern = [None] + [int(x) for x in rng.integers(0, 2, size=T - 1)]
    rounds, kst, _ = run_scripted(2, 0, True, truth, pattern)
    assert kst == pattern[1:]
    assert rounds == 2 + sum(k + 1 for k in pattern[1:T - 1])


def test_vanilla_skips_duplicate_forks():
    lat = Lattice(4, 0, False, 10 ** 9, 1, P)
    lat.anchor.u = [7, 7, 9]
    lat.anchor.c = 3
    items = lat.eligible()
    forks = [f for kind, s, f in items if kind == "fork"]
    assert forks == [0, 2]
    lat2 = Lattice(4, 0, True, 10 ** 9, 1, P)
    assert lat2.mask(lat2.anchor, 0) == ()
    lat2.anchor.u = [3, 4, 5]
    lat2.anchor.c = 3
    assert lat2.mask(lat2.anchor, 2) == (3, 4)
    assert lat2.mask(lat2.anchor, 3) == ()           # final-depth reference is never masked


def test_capacity_stops_forks():
    lat = Lattice(4, 0, True, P + 1, 1, P)             # anchor at the last position
    lat.anchor.u = [3]
    lat.anchor.c = 1
    assert [k for k, s, f in lat.eligible()] == ["advance"]
