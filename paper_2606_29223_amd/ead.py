"""Earliest available depth on the GPU (Definition 1) and the depth-side
accounting built on it (Definitions 3-4, Propositions 2-3).

Measurement: the library decodes with every depth explored (X = {1..L}),
width 1 and no DECS mask.  Each round then advances the anchor by one layer
and decodes its exit, so when a position commits, its anchor holds the
final-depth rule's candidate at every depth 1..L, computed on exactly the
states of plain decoding (the committed tokens are AR's).  Acceptance is
Omega(t, l) = [candidate at depth l == committed token] (greedy rule;
Omega(t, L) = 1), EAD the earliest accepted depth, stable EAD the earliest
depth accepted at itself and every deeper depth.

Accounting for an explored set X: W_X(t) = ceil_X(stable EAD(t)),
c(t) = W_X(t) - EAD^stab(t) in [0, Delta(X)], S_X = L T / sum_t W_X(t) with
the bounds of Proposition 3.  mean_t W_X(t) is the depth-side prediction of
DEX's critical-path layers per committed token, (L / N) rounds / commit.

    python3 -m paper_2606_29223_amd.ead --config NAME --tokens T
"""

from __future__ import annotations

import argparse
import json
import os
import sys

import numpy as np


def ceil_x(l: int, X) -> int:
    """Smallest explored depth >= l (Definition 3)."""
    return min(d for d in X if d >= l)


def resolution(X, L: int) -> int:
    """Delta(X) = max over l of ceil_X(l) - l (Definition 3)."""
    return max(ceil_x(l, X) - l for l in range(1, L + 1))


def ead(acc) -> int:
    """Earliest accepted depth, 1-based (acc[L-1] is 1)."""
    return 1 + int(np.flatnonzero(np.asarray(acc))[0])


def ead_stable(acc) -> int:
    """Earliest depth accepted at itself and at every deeper depth."""
    bad = np.flatnonzero(np.asarray(acc) == 0)
    return 1 if bad.size == 0 else int(bad[-1]) + 2


def measure(cfg: dict, dev_weights: dict, prompts, T: int, max_context: int | None = None):
    """Run the all-depth decoder for T tokens per sequence.  Returns
    (tokens [B][T], acceptance [B][T-1][L] int8) -- acceptance for the
    tokens committed by decode rounds (y_0 comes from the prefill, which
    exits at the final depth only)."""
    from . import dexlib
    L = cfg["n_layers"]
    prompts = np.asarray(prompts, dtype=np.int32)
    B, P = prompts.shape
    dec = dexlib.Decoder(cfg, dev_weights, explored=list(range(1, L + 1)), width_cap=1, decs=0, batch=B,
                         max_context=max_context or P + T)
    try:
        first = dec.prefill(prompts)
        toks = [[int(first[b])] for b in range(B)]
        cands = [dict() for _ in range(B)]          # stage -> candidate of the current anchor
        acc = [[] for _ in range(B)]
        while min(len(t) for t in toks) < T:
            c = dec.step()
            inf = dec.info
            for r in range(inf.n_rows):
                b, slot, stage = inf.row_seq[r], inf.row_slot[r], inf.row_stage[r]
                if slot == 0:
                    cands[b][stage] = inf.row_token[r]
            for b in range(B):
                if c[b] >= 0:
                    if len(toks[b]) < T:
                        u = [cands[b][k] for k in range(L)]
                        acc[b].append([int(x == int(c[b])) for x in u])
                        toks[b].append(int(c[b]))
                    cands[b] = {}
    finally:
        dec.close()
    return np.array(toks), np.array(acc, dtype=np.int8)


def accounting(acc: np.ndarray, X, L: int) -> dict:
    """Definitions 3-4 and Propositions 2-3 over acceptance rows acc[t][l]."""
    e = np.array([ead(a) for a in acc])
    es = np.array([ead_stable(a) for a in acc])
    W = np.array([ceil_x(int(x), X) for x in es])
    dx = resolution(X, L)
    T = len(acc)
    s_x = L * T / W.sum()
    s_ead = L * T / es.sum()
    lower = L * T / np.minimum(es + dx, L).sum()
    return {
        "X": list(X), "tokens": T, "resolution": dx,
        "mean_ead": float(e.mean()), "mean_stable_ead": float(es.mean()),
        "mean_W_X": float(W.mean()),
        "overhead_in_bounds": bool(np.all((W - es >= 0) & (W - es <= dx))),
        "S_X": float(s_x), "S_EAD": float(s_ead), "S_lower": float(lower),
        "bounds_hold": bool(1.0 <= lower <= s_x <= s_ead),
        "stable_ead_hist": {int(k): int(v) for k, v in zip(*np.unique(es, return_counts=True))},
    }


def main():
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    if root not in sys.path:
        sys.path.insert(0, root)
    from synth import configs, gen

    from . import dexlib
    ap = argparse.ArgumentParser()
    ap.add_argument("--config", default=configs.HEADLINE)
    ap.add_argument("--tokens", type=int, default=64)
    args = ap.parse_args()
    cfg = configs.get(args.config)
    dev = dexlib.device_weights(cfg, gen.generate_model(cfg))
    toks, acc = measure(cfg, dev, gen.prompts(cfg), args.tokens)
    out = accounting(acc.reshape(-1, cfg["n_layers"]), cfg["explored"], cfg["n_layers"])
    out["predicted_critical_path_layers_per_commit"] = out["mean_W_X"]
    out["config"] = cfg["name"]
    print(json.dumps(out))


if __name__ == "__main__":
    main()
