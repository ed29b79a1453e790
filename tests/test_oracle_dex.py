"""Pins of the oracle's DEX procedure on real (synthetic) models.

  * losslessness (Section 3.2): DEX tokens equal greedy AR for every
    explored set, width cap and DECS mode;
  * X = {L} is plain AR and X = {d, L} single-exit draft/verify;
  * the uncapped trace in closed form: k*_t recomputed independently from
    teacher-forced per-depth logits with DECS masks, rounds
    = N + sum_{t=1}^{T-2} (k*_t + 1);
  * d_{k*_t} <= ceil_X(stable EAD(t)) (Definitions 1, 3, 4);
  * brute force on the 4-layer model: every outcome pattern of k* forced on
    the true prefix; tokens, rounds and every live node's hidden state and
    keys/values equal a from-scratch recomputation of that node's prefix.
"""
import itertools

import numpy as np
import pytest

import oracle
from oracle import ar, dex, ead
from oracle.model import argmax_lowest
from synth import configs, gen


@pytest.fixture(scope="module")
def tiny():
    cfg = configs.get("tiny-4L-d128-fp32")
    m = oracle.load(cfg)
    prompt = [int(t) for t in gen.prompts(cfg)[0]]
    pf = m.prefill(prompt)
    ar_toks = ar.ar_generate(m, prompt, cfg["gen_len"], prefill=pf)
    return cfg, m, prompt, pf, ar_toks


@pytest.mark.parametrize("X,W,decs", [
    ([1, 2, 3, 4], 0, True), ([1, 2, 3, 4], 0, False), ([1, 2, 3, 4], 3, True),
    ([1, 2, 3, 4], 2, False), ([2, 4], 0, True), ([1, 3, 4], 5, True), ([4], 1, True),
    ([1, 2, 3, 4], 1, True)])
def test_lossless_tiny(tiny, X, W, decs):
    cfg, m, prompt, pf, ar_toks = tiny
    T = cfg["gen_len"]
    r = dex.dex_generate(m, prompt, X, W, decs, T, prefill=pf, keep_trace=False)
    assert r.tokens == ar_toks
    if X == [4]:
        assert r.rounds == T - 1 and r.row_layers == 4 * (T - 1)


def test_lossless_gqa_fine_exploration():
    base = configs.get("llama-32L-d4096-x2-w16")
    cfg = configs.scaled_down(base, n_layers=8, d_model=128, d_ffn=256, vocab=700)
    cfg.update(n_heads=4, n_kv_heads=2, head_dim=32, prompt_len=20)
    assert cfg["explored"] == [1, 2, 3, 4, 5, 6, 7, 8]
    m = oracle.load(cfg)
    prompt = [int(t) for t in gen.prompts(cfg)[0]]
    pf = m.prefill(prompt)
    T = 24
    want = ar.ar_generate(m, prompt, T, prefill=pf)
    for W in (16, 5):
        r = dex.dex_generate(m, prompt, cfg["explored"], W, True, T, prefill=pf, keep_trace=True)
        assert r.tokens == want
        assert max(sum(t.rows_per_stage) for t in r.trace) <= W


def test_lossless_small_truncated():
    cfg = configs.get("small-12L-d768-bf16")
    m = oracle.load(cfg)
    prompt = [int(t) for t in gen.prompts(cfg)[0]][:32]
    pf = m.prefill(prompt)
    T = 10
    want = ar.ar_generate(m, prompt, T, prefill=pf)
    r = dex.dex_generate(m, prompt, cfg["explored"], cfg["width_cap"], True, T, prefill=pf)
    assert r.tokens == want


def _decs_kstars(m, prompt, pf, toks, X, decs=True):
    """k*_t from teacher-forced exit logits at the explored depths."""
    z = ar.depth_logits(m, prompt, toks, X, prefill=pf)      # [T-1, N, V]
    N = len(X)
    out = []
    for t in range(1, len(toks)):
        y = toks[t]
        prior = []
        k = N - 1
        for j in range(N - 1):
            u = argmax_lowest(z[t - 1, j], prior if decs else ())
            prior.append(u)
            if u == y:
                k = j
                break
        assert argmax_lowest(z[t - 1, N - 1]) == y
        out.append(k)
    return out


@pytest.mark.parametrize("X,decs", [([1, 2, 3, 4], True), ([1, 2, 3, 4], False), ([1, 3, 4], True),
                                    ([2, 4], True)])
def test_uncapped_trace_closed_form(tiny, X, decs):
    cfg, m, prompt, pf, ar_toks = tiny
    T = 40
    toks = ar_toks[:T]
    ks = _decs_kstars(m, prompt, pf, toks, X, decs)
    r = dex.dex_generate(m, prompt, X, 0, decs, T, prefill=pf, keep_trace=False)
    assert r.kstars == ks
    N = len(X)
    assert r.rounds == N + sum(k + 1 for k in ks[:-1])


def test_match_depth_bounded_by_stable_ead(tiny):
    cfg, m, prompt, pf, ar_toks = tiny
    L = cfg["n_layers"]
    T = 40
    toks = ar_toks[:T]
    zall = ar.depth_logits(m, prompt, toks, list(range(1, L + 1)), prefill=pf)
    for X in ([1, 2, 3, 4], [2, 4], [3, 4]):
        for decs in (True, False):
            ks = _decs_kstars(m, prompt, pf, toks, X, decs)
            for t in range(1, T):
                acc = ead.acceptance([argmax_lowest(zall[t - 1, l]) for l in range(L)], toks[t])
                assert X[ks[t - 1]] <= ead.ceil_x(ead.ead_stable(acc), X)


def _recompute_check(m, pf, prompt, stages):
    """check(lattice, cache, n): every live slot's boundary hidden state and
    per-layer keys/values equal a from-scratch recomputation."""
    P = len(prompt)

    def check(lat, cache, n_committed):
        for s in lat.slots:
            if s.c == 0:
                continue
            # inputs at positions P .. pos: committed tokens up to n-2, then the
            # slot chain (anchor first) down to the slot itself
            chain_inputs = [a.x for a in s.ancestors()] + [s.x]
            toks = check.committed[P:n_committed - 1] + chain_inputs
            fresh = ar.Cache(m, pf[0], pf[1], s.pos + 1)
            for i, p in enumerate(range(P, s.pos + 1)):
                hs = ar.decode_row(m, fresh, toks[i], p)
            last_layer = stages[s.c - 1][-1]
            assert np.array_equal(hs[last_layer], s.state["h"])
            for k in range(s.c):
                for l in stages[k]:
                    assert np.array_equal(fresh.K[l][s.pos], s.state["k"][l])
                    assert np.array_equal(fresh.V[l][s.pos], s.state["v"][l])
        # the committed cache itself equals plain AR's
        for l in range(m.L):
            assert np.array_equal(cache.K[l][:n_committed - 1], check.ar_cache.K[l][:n_committed - 1])

    return check


def test_brute_force_outcomes_tiny(tiny):
    cfg, m, prompt, pf, ar_toks = tiny
    X = cfg["explored"]
    N = len(X)
    stages = dex.stages_of(X, m.L)
    P = len(prompt)
    full = prompt + ar_toks
    m_len = 5                                    # commits whose outcome is forced
    T = m_len + 1
    ar_cache = ar.Cache(m, pf[0], pf[1], P + T)
    for p in range(P, P + T - 1):
        ar.decode_row(m, ar_cache, full[p], p)
    patterns = list(itertools.product(range(N), repeat=m_len))
    for idx, pattern in enumerate(patterns):
        def force(prefix, stage, natural, mask):
            pos = len(prefix) - 1
            t = pos + 1 - P
            if prefix != full[: pos + 1] or t >= T or t < 1:
                return None
            y = ar_toks[t]
            if stage == N - 1:
                assert natural == y                # the final depth is the AR token
                return None
            k = pattern[t - 1]
            if stage == k:
                return y
            if stage < k:
                d = 0
                while d in mask or d == y:
                    d += 1
                return d
            return None

        check = None
        if idx % 16 == 0:                          # full state recomputation on a subset
            check = _recompute_check(m, pf, prompt, stages)
            check.committed = full
            check.ar_cache = ar_cache
        r = dex.dex_generate(m, prompt, X, 0, True, T, prefill=pf, force=force, keep_trace=False,
                             check=check)
        assert r.tokens == ar_toks[:T], pattern
        assert r.kstars == list(pattern), pattern
        assert r.rounds == N + sum(k + 1 for k in pattern[:-1])
