"""Oracle: Depth Exploration Decoding (Algorithm 1) on the synthetic model.

TEST INFRASTRUCTURE ONLY (see oracle/model.py).

The loop of Algorithm 1, one iteration per round: expand (run each selected
lattice node through its stage, one row at a time), DECS (Algorithm 2,
greedy) on the node's exit logits, insert into the explore buffer, and when
the anchor reaches the final depth validate-and-commit then collapse (the
bookkeeping lives in lattice.py).  Attention for a node at layer l covers
the committed keys [0, n-1) followed by the layer-l keys of its ancestor
slots in position order and its own.

The initial state is the prompt prefill; it commits y_0 (the final-depth
argmax at the last prompt position), so T generated tokens need T-1 commits
from the loop.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import adapter as adapter_mod
from .ar import Cache
from .gumbel import decode
from .lattice import Lattice
from .model import Model


@dataclass
class RoundTrace:
    q: int                              # FSM state (anchor's completed stages) at round start
    rows: list                          # (canonical slot index, stage, pos, input token)
    rows_per_stage: list
    tokens: list                        # decoded candidate per row
    commit: tuple | None = None         # (token, kstar, collapse_map, fresh)


@dataclass
class DexResult:
    tokens: list
    rounds: int
    trace: list = field(default_factory=list)
    layers_streamed: int = 0            # sum over rounds of layers in stages with >= 1 row
    row_layers: int = 0                 # sum over rows of the layers they ran
    kstars: list = field(default_factory=list)


def stages_of(explored, L):
    """Stage k covers the layers (d_{k-1}, d_k] (0-based layer ids)."""
    prev = 0
    out = []
    for d in explored:
        out.append(list(range(prev, d)))
        prev = d
    assert prev == L
    return out


def validate_explored(explored, L):
    """Definition 3: strictly increasing depths in [1, L], last one L."""
    if not explored or explored[-1] != L:
        raise ValueError("explored depths must end at the final depth")
    if any(b <= a for a, b in zip(explored, explored[1:])) or explored[0] < 1:
        raise ValueError("explored depths must be strictly increasing in [1, L]")


def dex_generate(model: Model, prompt, explored, width_cap: int, decs: bool, T: int,
                 max_context: int | None = None, force=None, prefill=None, keep_trace=True,
                 check=None, temperature: float = 0.0, seed: int = 0, seq: int = 0, adapters=None):
    """Run DEX until T tokens are generated (y_0 from the prefill included).

    temperature > 0 selects Algorithm 2's sampling mode: every node decodes
    argmax(l / temperature + G) with the Gumbel row of (seed, seq, its
    position) (oracle/gumbel.py); 0 is greedy.
    adapters: None, or one inducing adapter per non-final stage (dicts of
    oracle/adapter.PARTS); a node at stage k < N-1 decodes h + dh_k(h).

    force(prefix_tokens, stage, natural_token, mask) may return a token that
    replaces a node's candidate (used by the brute-force test to steer the
    outcome of nodes on the true prefix); None keeps the natural one.
    check(lattice, cache, n_committed) is called after every round."""
    L = model.L
    validate_explored(explored, L)
    N = len(explored)
    stages = stages_of(explored, L)
    P = len(prompt)
    max_context = P + T if max_context is None else max_context
    Ks, Vs, h_last = prefill if prefill is not None else model.prefill(prompt)
    cache = Cache(model, Ks, Vs, max_context)
    committed = list(int(t) for t in prompt)
    y0 = decode(model.exit_logits(h_last), (), temperature, seed, seq, P - 1)
    committed.append(y0)
    out = [y0]
    lat = Lattice(N, width_cap, bool(decs), max_context, y0, P)
    res = DexResult(tokens=out, rounds=0)
    while len(out) < T:
        n = len(committed)                  # committed tokens; keys cached for [0, n-1)
        q = lat.q
        rows = lat.begin_round()
        toks = []
        for r in rows:
            s, k = r.slot, r.stage
            chain = s.ancestors()
            h = model.embed(s.x) if k == 0 else s.state["h"]
            for l in stages[k]:
                past_k = [cache.K[l][: n - 1]] + [a.state["k"][l][None] for a in chain]
                past_v = [cache.V[l][: n - 1]] + [a.state["v"][l][None] for a in chain]
                h, kk, vv = model.layer_row(l, h, s.pos, np.concatenate(past_k), np.concatenate(past_v))
                s.state.setdefault("k", {})[l] = kk
                s.state.setdefault("v", {})[l] = vv
            s.state["h"] = h
            if adapters is not None and k < N - 1:
                z = model.exit_logits(h + adapter_mod.delta(adapters[k], h, model.eps))
            else:
                z = model.exit_logits(h)
            m = lat.mask(s, k)
            tok = decode(z, m, temperature, seed, seq, s.pos)
            if force is not None:
                prefix = committed + [a.x for a in chain[1:]] + ([s.x] if s is not lat.anchor else [])
                # prefix ends with the slot's own input (the anchor's input is committed[-1])
                ft = force(prefix, k, tok, m)
                if ft is not None:
                    tok = int(ft)
            toks.append(tok)
        res.row_layers += sum(len(stages[r.stage]) for r in rows)
        per_stage = [0] * N
        for r in rows:
            per_stage[r.stage] += 1
        res.layers_streamed += sum(len(stages[k]) for k in range(N) if per_stage[k] > 0)
        tr = RoundTrace(q, [(lat.index(r.slot), r.stage, r.slot.pos, r.slot.x) for r in rows],
                        per_stage, list(toks))
        cm = lat.end_round(rows, toks)
        res.rounds += 1
        if cm is not None:
            A = cm.old_anchor
            for l in range(L):
                cache.K[l][A.pos] = A.state["k"][l]
                cache.V[l][A.pos] = A.state["v"][l]
            committed.append(cm.token)
            out.append(cm.token)
            res.kstars.append(cm.kstar)
            tr.commit = (cm.token, cm.kstar, list(cm.collapse_map), cm.fresh_anchor)
        if keep_trace:
            res.trace.append(tr)
        if check is not None:
            check(lat, cache, len(committed))
    return res
