"""Oracle: plain greedy autoregressive decoding and teacher-forced exit logits.

TEST INFRASTRUCTURE ONLY (see oracle/model.py).

Greedy AR (Section 2.1; the decoding rule every DEX commit must reproduce,
Section 3.2 "Lossless invariant"): y_0 = argmax z_L at the last prompt
position; y_t = argmax z_L at position P+t-1 after feeding y_{t-1}.  The
generated list holds T tokens y_0..y_{T-1}.
"""

from __future__ import annotations

import numpy as np

from .model import Model, argmax_lowest


class Cache:
    """Committed per-layer keys/values for positions [0, n)."""

    def __init__(self, model: Model, Ks, Vs, capacity: int):
        n = Ks[0].shape[0]
        self.K = [np.zeros((capacity, model.Hkv, model.hd)) for _ in range(model.L)]
        self.V = [np.zeros((capacity, model.Hkv, model.hd)) for _ in range(model.L)]
        for l in range(model.L):
            self.K[l][:n] = Ks[l]
            self.V[l][:n] = Vs[l]
        self.n = n


def decode_row(model: Model, cache: Cache, token: int, pos: int, layers=None, h=None, write=True):
    """Run one row (input `token` at position `pos`) through `layers` (default:
    all) against cache positions [0, pos); optionally append its K/V.
    Returns the hidden state after every layer run, as a list."""
    layers = range(model.L) if layers is None else layers
    if h is None:
        h = model.embed(token)
    hs = []
    for l in layers:
        h, k, v = model.layer_row(l, h, pos, cache.K[l][:pos], cache.V[l][:pos])
        if write:
            cache.K[l][pos] = k
            cache.V[l][pos] = v
        hs.append(h)
    return hs


def ar_generate(model: Model, prompt, T: int, prefill=None, temperature: float = 0.0, seed: int = 0,
                seq: int = 0):
    """Plain AR: greedy, or (temperature > 0) Gumbel-max sampling with the row
    of (seed, seq, position) at every position (oracle/gumbel.py).  Returns
    the T generated tokens y_0..y_{T-1}."""
    from .gumbel import decode
    P = len(prompt)
    Ks, Vs, h_last = prefill if prefill is not None else model.prefill(prompt)
    cache = Cache(model, Ks, Vs, P + T)
    toks = [decode(model.exit_logits(h_last), (), temperature, seed, seq, P - 1)]
    for t in range(1, T):
        pos = P + t - 1
        hs = decode_row(model, cache, toks[-1], pos)
        toks.append(decode(model.exit_logits(hs[-1]), (), temperature, seed, seq, pos))
    return toks


def depth_logits(model: Model, prompt, seq, depths, prefill=None, adapters=None):
    """Teacher-forced exit logits.  For t = 1..len(seq)-1 the row at position
    P+t-1 has input seq[t-1] and prefix prompt || seq[:t-1]; returns an array
    [len(seq)-1, len(depths), V] of z_d for d in `depths` (1-based).
    adapters: None, or the inducing adapters of depths[:-1] (decoded as
    h + dh, oracle/adapter.py)."""
    from .adapter import delta
    P = len(prompt)
    Ks, Vs, _ = prefill if prefill is not None else model.prefill(prompt)
    cache = Cache(model, Ks, Vs, P + len(seq))
    out = np.empty((len(seq) - 1, len(depths), model.V))
    for t in range(1, len(seq)):
        pos = P + t - 1
        hs = decode_row(model, cache, seq[t - 1], pos)
        for j, d in enumerate(depths):
            h = hs[d - 1]
            if adapters is not None and j < len(depths) - 1:
                h = h + delta(adapters[j], h, model.eps)
            out[t - 1, j] = model.exit_logits(h)
    return out


def prefill_token(model: Model, prefill) -> int:
    """y_0 from a prefill result."""
    return argmax_lowest(model.exit_logits(prefill[2]))
