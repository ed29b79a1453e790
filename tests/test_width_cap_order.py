"""Pin of the width-cap priority against hand-derived lattice states.

The paper fixes no pruning rule (Appendix E names branch pruning as future
work).  The rule both implementations follow -- anchor first, then the
lowest (hypothesis cost, path length, path) with paths as depth/position
step strings, depth step before position step -- is written out in
tests/golden/width_cap_order.json together with, for each state, the item
order derived by hand from that statement.  The oracle's Lattice.select and
the engine's planner (through the host-only dex_debug_plan tap) must both
reproduce every list, and the pin must reject a permuted sort key, an
inverted depth/position order and fork-stage tuples in place of step strings.
"""
import json
import os

import pytest

from oracle import lattice as olat
from oracle.lattice import Lattice, Slot

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "width_cap_order.json")))
POS0 = 40


def build_state(st, width_cap=None):
    """Lattice of the golden state: slot i = [parent, fork_stage, c, u]."""
    N = st["N"]
    W = st["W"] if width_cap is None else width_cap
    spec = st["slots"]
    lat = Lattice(N, W, True, 10 ** 6, 7, POS0)
    slots = []
    for i, (par, f, c, u) in enumerate(spec):
        if par < 0:
            s = lat.anchor
        else:
            p = slots[par]
            s = Slot(p.u[f], p.pos + 1, p, f, 1000 + i)
            p.children[f] = s
        s.c = c
        s.u = list(u)
        slots.append(s)
    lat.slots = slots
    return lat


def as_list(lat, items):
    return [[k, lat.index(s), f] for k, s, f in items]


@pytest.mark.parametrize("st", GOLD["states"], ids=[s["name"] for s in GOLD["states"]])
def test_oracle_select_matches_hand_derivation(st):
    lat = build_state(st)
    assert as_list(lat, lat.select()) == st["kept"]
    latu = build_state(st, width_cap=0)
    assert as_list(latu, latu.select()[1:]) == st["order"]
    if "kept_W5" in st:
        lat5 = build_state(st, width_cap=5)
        assert as_list(lat5, lat5.select()) == st["kept_W5"]


def _golden_fails(priority):
    """True if some golden state catches the planted priority."""
    for st in GOLD["states"]:
        for w, key in ((None, "kept"), (0, None), (5, "kept_W5")):
            if key is not None and key not in st:
                continue
            lat = build_state(st, width_cap=w)
            lat.priority = priority.__get__(lat, Lattice)
            got = as_list(lat, lat.select())
            want = st[key] if key else [["advance", 0, None]] + st["order"]
            if got != want:
                return True
    return False


def test_pin_rejects_planted_orders():
    def permuted(self, item):            # path length before hypothesis cost
        steps = self.item_steps(item)
        return (len(steps), olat.hypothesis_cost(self.item_forks(item)), steps)

    def inverted(self, item):            # position step before depth step
        steps = tuple(1 - x for x in self.item_steps(item))
        return (olat.hypothesis_cost(self.item_forks(item)), len(steps), steps)

    def fork_tuples(self, item):         # path read as the tuple of fork stages
        forks = self.item_forks(item)
        return (olat.hypothesis_cost(forks), len(forks), forks)

    def no_length(self, item):           # cost, then the step string alone
        steps = self.item_steps(item)
        return (olat.hypothesis_cost(self.item_forks(item)), steps)

    for bad in (permuted, inverted, fork_tuples, no_length):
        assert _golden_fails(bad), bad.__name__
    assert not _golden_fails(Lattice.priority)


def test_wide_cap_keeps_every_item():
    for st in GOLD["states"]:
        n_items = len(st["order"]) + 1
        lat = build_state(st, width_cap=n_items)
        assert len(lat.select()) == n_items


def _engine_plan(st, width_cap):
    from paper_2606_29223_amd import dexlib
    if not os.path.exists(dexlib.LIB_PATH):
        pytest.skip("libdex.so not built")
    slots = []
    pos = {0: POS0}
    for i, (par, f, c, u) in enumerate(st["slots"]):
        if par >= 0:
            pos[i] = pos[par] + 1
        slots.append((par, f, c, pos[i], u))
    got = dexlib.dex_debug_plan(st["N"], width_cap, 1, 10 ** 6, slots)
    return [["advance" if k == 0 else "fork", s, None if k == 0 else f] for k, s, f in got]


@pytest.mark.parametrize("st", GOLD["states"], ids=[s["name"] for s in GOLD["states"]])
def test_engine_planner_matches_hand_derivation(st):
    """The engine's host planner (the code dex_step runs) on the same states."""
    assert _engine_plan(st, st["W"]) == st["kept"]
    assert _engine_plan(st, 0)[1:] == st["order"]
    if "kept_W5" in st:
        assert _engine_plan(st, 5) == st["kept_W5"]


def test_engine_planner_rejects_malformed_states():
    from paper_2606_29223_amd import dexlib
    if not os.path.exists(dexlib.LIB_PATH):
        pytest.skip("libdex.so not built")
    bad = [
        [(0, -1, 1, 5, [3])],                             # anchor with a parent
        [(-1, -1, 2, 5, [3, 4]), (-1, 0, 0, 6, [])],       # second root
        [(-1, -1, 2, 5, [3, 4]), (0, 2, 0, 6, [])],        # fork past the parent's completed stages
        [(-1, -1, 2, 5, [3, 4]), (0, 0, 0, 6, []), (0, 0, 0, 6, [])],   # two children at one stage
        [(-1, -1, 5, 5, [1, 2, 3, 4])],                   # c above N
    ]
    for slots in bad:
        with pytest.raises(dexlib.DexError):
            dexlib.dex_debug_plan(4, 0, 1, 10 ** 6, slots)
