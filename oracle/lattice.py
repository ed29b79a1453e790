"""Oracle: the depth-position lattice of DEX as pure bookkeeping (no model).

TEST INFRASTRUCTURE ONLY (see oracle/model.py).

Follows Algorithm 1 (expand / DECS / insert / validate-and-commit / collapse /
advance) and Section 3.2 (lattice expansion, commit process, FSM and
collapse), with Algorithm 2 (DECS, greedy mode) deciding the masks.

Terms.  A *slot* is one branch-conditioned next token: an input token x at
absolute position pos whose prefix is the committed context followed by the
inputs of its ancestor slots.  Running stage k (layers (d_{k-1}, d_k]) on a
slot produces one lattice node (an exploration token) and its candidate
u[k] = DECS-argmax of the exit logits at depth d_k.  c counts the stages a
slot has completed; the anchor is the slot of the commit position under the
committed prefix and its c is the FSM state q.

One round:
  * work items: advance(anchor) always; advance(s) for a non-anchor slot when
    every ancestor had completed more stages than s at round start (so the
    ancestor's keys/values at the stage s runs were produced in an earlier
    round, as on the paper's one-explorer-per-device pipeline); and
    fork(s, f) for every completed stage f <= N-2 of s not yet forked: a new
    slot with input u_s[f] at pos_s + 1 that runs stage 0 (position
    expansion).  Without a width cap these are exactly the depth and position
    children of the previous round's nodes, so the lattice is the paper's
    binary expansion (2^q - 1 nodes after q rounds).
  * width cap W (not in the paper, which names branch pruning as future
    work): keep the anchor item and the W-1 others of lowest
    (hypothesis cost, path length, path).  The lattice is the binary tree of
    Section 3.2 rooted at the anchor's stage-0 node: a depth step D goes from
    a slot's stage-k node to its stage-(k+1) node, a position step P from a
    slot's stage-f node to the stage-0 node of the slot forked there.  An
    item's path is the step string from the root to the node it evaluates
    (advance(s): s's stage c_s node; fork(s, f): the new slot's stage-0
    node), its length the number of steps, and paths of equal length compare
    lexicographically with D before P.  Path length then lexicographic order
    is the paper's node numbering (depth child 2i+1, position child 2i+2)
    read relative to the current anchor.  The hypothesis cost is
    sum(f + 1) over the fork stages f on the path (each P step costs one
    plus the D steps taken in its slot before it), i.e. the length of the
    path up to its last P step.  The paper fixes no pruning rule; the order
    is pinned by hand-derived lattice states (tests/golden/
    width_cap_order.json) and, for W >= 2^(N-1), by the paper's uncapped
    lattice, which the rule must reproduce exactly.
  * DECS (greedy): a node's candidate is the argmax with the tokens already
    proposed by shallower nodes of the same slot masked out, except the
    anchor's final-depth node, which is never masked.  decs=False masks
    nothing and then skips a fork whose token repeats a shallower fork of
    the same slot (its states would be identical).
  * commit, once the anchor completes stage N-1: y = u[N-1] is appended;
    k* is the shallowest j <= N-2 with u[j] == y, else N-1.
  * collapse: the anchor's keys/values become committed position pos; the
    fork child(anchor, k*) -- if it exists -- becomes the new anchor and
    its subtree is kept (the only slots whose prefix equals the new
    committed prefix); every other slot is discarded.  With no such child
    the new anchor is a fresh slot (y, pos+1) with c = 0.
  * canonical slot order is creation order; collapse keeps the relative
    order of the retained slots (the collapse map lists their old indices).
"""

from __future__ import annotations

from dataclasses import dataclass, field


class Slot:
    __slots__ = ("x", "pos", "parent", "fork_stage", "c", "u", "children", "uid", "state")

    def __init__(self, x: int, pos: int, parent, fork_stage: int, uid: int):
        self.x = x
        self.pos = pos
        self.parent = parent
        self.fork_stage = fork_stage
        self.c = 0
        self.u = []
        self.children = {}
        self.uid = uid
        self.state = {}

    def ancestors(self):
        """Ancestor slots from the anchor down to the parent."""
        out = []
        p = self.parent
        while p is not None:
            out.append(p)
            p = p.parent
        out.reverse()
        return out

    def path(self):
        """Fork stages from the anchor down to this slot."""
        out = []
        s = self
        while s.parent is not None:
            out.append(s.fork_stage)
            s = s.parent
        out.reverse()
        return tuple(out)


def hypothesis_cost(path) -> int:
    """sum(f + 1) over the fork stages f of a path (the width-cap priority)."""
    return sum(f + 1 for f in path)


DEPTH_STEP, POSITION_STEP = 0, 1     # lexicographic order: depth step first


def steps_of_forks(forks) -> tuple:
    """Step string from the anchor's stage-0 node to the stage-0 node of the
    slot reached by forking at stages `forks` (anchor first): each fork at
    stage f is f depth steps inside its slot, then one position step."""
    out = []
    for f in forks:
        out += [DEPTH_STEP] * f + [POSITION_STEP]
    return tuple(out)


@dataclass
class Row:
    slot: Slot
    stage: int
    new: bool          # the slot was created by a fork this round


@dataclass
class Commit:
    token: int
    kstar: int
    collapse_map: list          # old canonical indices of retained slots, in order
    old_anchor: Slot
    fresh_anchor: bool


@dataclass
class Lattice:
    n_explored: int
    width_cap: int              # 0 = uncapped
    decs: bool
    max_context: int
    anchor_token: int
    anchor_pos: int
    slots: list = field(default_factory=list)
    _uid: int = 0

    def __post_init__(self):
        self.slots = [self._new_slot(self.anchor_token, self.anchor_pos, None, -1)]

    def _new_slot(self, x, pos, parent, f):
        s = Slot(x, pos, parent, f, self._uid)
        self._uid += 1
        return s

    @property
    def anchor(self) -> Slot:
        return self.slots[0]

    @property
    def q(self) -> int:
        return self.anchor.c

    def index(self, s: Slot) -> int:
        return self.slots.index(s)

    # ------------------------------------------------------------- planning
    def eligible(self):
        """All work items: ('advance', slot, None) / ('fork', slot, f)."""
        N = self.n_explored
        A = self.anchor
        items = []
        for s in self.slots:
            if s is A:
                items.append(("advance", s, None))
            elif all(a.c > s.c for a in s.ancestors()):
                items.append(("advance", s, None))
            if s.pos + 1 > self.max_context - 1:
                continue
            for f in range(min(s.c, N - 1)):
                if f in s.children:
                    continue
                if not self.decs and s.u[f] in s.u[:f]:
                    continue
                items.append(("fork", s, f))
        return items

    @staticmethod
    def item_forks(item):
        """Fork stages from the anchor down to the item's slot (a fork item's
        own fork last)."""
        kind, s, f = item
        return s.path() + ((f,) if kind == "fork" else ())

    @staticmethod
    def item_steps(item):
        """Step string from the anchor's stage-0 node to the item's node."""
        kind, s, f = item
        if kind == "fork":
            return steps_of_forks(s.path() + (f,))
        return steps_of_forks(s.path()) + (DEPTH_STEP,) * s.c

    def priority(self, item):
        steps = self.item_steps(item)
        return (hypothesis_cost(self.item_forks(item)), len(steps), steps)

    def select(self):
        items = self.eligible()
        first = items[0]
        assert first[0] == "advance" and first[1] is self.anchor
        rest = items[1:]
        rest.sort(key=self.priority)
        if self.width_cap > 0:
            rest = rest[: self.width_cap - 1]
        return [first] + rest

    def begin_round(self):
        """Pick this round's items and create the forked slots.  Returns the
        rows (slot, stage) in priority order (anchor first)."""
        rows = []
        for kind, s, f in self.select():
            if kind == "advance":
                rows.append(Row(s, s.c, False))
            else:
                child = self._new_slot(s.u[f], s.pos + 1, s, f)
                s.children[f] = child
                self.slots.append(child)
                rows.append(Row(child, 0, True))
        return rows

    def mask(self, s: Slot, stage: int):
        """DECS mask set Prior(node) for running `stage` on slot s."""
        if not self.decs:
            return ()
        if s is self.anchor and stage == self.n_explored - 1:
            return ()
        return tuple(s.u[:stage])

    # ------------------------------------------------------- commit/collapse
    def end_round(self, rows, tokens):
        """Insert the decoded candidates; commit and collapse if the anchor
        reached the final depth.  Returns a Commit or None."""
        for r, t in zip(rows, tokens):
            assert r.stage == r.slot.c
            r.slot.u.append(int(t))
            r.slot.c += 1
        N = self.n_explored
        A = self.anchor
        if A.c < N:
            return None
        y = A.u[N - 1]
        kstar = N - 1
        for j in range(N - 1):
            if A.u[j] == y:
                kstar = j
                break
        child = A.children.get(kstar) if kstar <= N - 2 else None
        if child is not None:
            keep = []
            for i, s in enumerate(self.slots):
                t = s
                while t is not None and t is not child:
                    t = t.parent
                if t is child:
                    keep.append(i)
            child.parent = None
            child.fork_stage = -1
            self.slots = [self.slots[i] for i in keep]
            return Commit(y, kstar, keep, A, False)
        self.slots = [self._new_slot(y, A.pos + 1, None, -1)]
        return Commit(y, kstar, [], A, True)
