"""GPU: edge cases of the C ABI on a live context.

  * argument and order errors (step before prefill, an empty or over-long
    prompt, token ids outside the vocabulary) are reported without
    poisoning the context, which then decodes normally;
  * decoding right up to max_context: forks never reach past the last
    position, every sequence stops with exactly max_context - prompt_len
    generated tokens (sequences of one batch reach it in different rounds),
    the tokens equal plain AR's, and further steps report DEX_E_CAPACITY;
  * a round at the row capacity: 32 sequences of width 8 make up to
    DEX_MAX_ROWS = 256 rows a round (stage GEMMs over several 64-row
    blocks, the exit head over every row, many attention groups), and the
    tokens are still plain AR's;
  * the degenerate lattice of width 1: only the anchor advances, so every
    commit takes exactly N rounds from a fresh anchor, and the tokens are
    still AR's (Algorithm 1 with no parallel branch is sequential
    early-exit verification at every depth);
  * the binding's generate helper and the generation module.
"""
import numpy as np
import pytest

import oracle
from oracle import dex
from synth import configs, gen
from tests.gpu_common import decoder, host_weights, run, torch_cuda

pytestmark = pytest.mark.gpu

TINY = "tiny-4L-d128-fp32"


def _collect(dec, prompts, max_ctx):
    """Prefill, then step until the library reports every sequence full.
    Returns (tokens per sequence, rounds, deepest row position seen)."""
    from paper_2606_29223_amd import dexlib
    B = dec.batch
    first = dec.prefill(prompts)
    toks = [[int(first[b])] for b in range(B)]
    rounds, deepest = 0, -1
    while True:
        try:
            c = dec.step()
        except dexlib.DexError as e:
            assert e.status == dexlib.DEX_E_CAPACITY, e
            break
        rounds += 1
        assert rounds < 64 * max_ctx, "decoding did not stop at max_context"
        inf = dec.info
        for r in range(inf.n_rows):
            deepest = max(deepest, inf.row_pos[r])
        for b in range(B):
            if c[b] >= 0:
                toks[b].append(int(c[b]))
    return toks, rounds, deepest


def test_errors_do_not_poison_the_context():
    torch_cuda()
    from paper_2606_29223_amd import dexlib
    cfg, _ = host_weights(TINY)
    P, T = cfg["prompt_len"], 8
    prompt = gen.prompts(cfg)
    dec = decoder(TINY, max_context=P + T)

    def status(fn):
        with pytest.raises(dexlib.DexError) as e:
            fn()
        return e.value.status

    assert status(dec.step) == dexlib.DEX_E_STATE
    assert status(lambda: dec.prefill(np.zeros((1, 0), dtype=np.int32))) == dexlib.DEX_E_INVAL
    assert status(lambda: dec.prefill(np.zeros((1, P + T), dtype=np.int32))) == dexlib.DEX_E_CAPACITY
    for bad in (cfg["vocab"], -1):
        p2 = prompt.copy()
        p2[0, 3] = bad
        assert status(lambda: dec.prefill(p2)) == dexlib.DEX_E_INVAL
    toks, _, _ = _collect(dec, prompt, P + T)
    dec.close()
    ar_dec = decoder(TINY, explored=[cfg["n_layers"]], width_cap=1, max_context=P + T)
    ar_toks, _, _ = _collect(ar_dec, prompt, P + T)
    ar_dec.close()
    assert toks == ar_toks and len(toks[0]) == T


@pytest.mark.parametrize("X,W", [([1, 2, 3, 4], 0), ([1, 2, 3, 4], 3), ([2, 4], 2)])
def test_decoding_stops_exactly_at_max_context(X, W):
    torch_cuda()
    cfg = configs.get(TINY)
    P, T = cfg["prompt_len"], 12
    prompts = np.stack([gen.tokens(gen.mix64(s), P, cfg["vocab"]) for s in (31, 32, 33)])
    dec = decoder(TINY, explored=X, width_cap=W, batch=3, max_context=P + T)
    toks, rounds, deepest = _collect(dec, prompts, P + T)
    dec.close()
    assert deepest <= P + T - 1
    assert all(len(t) == T for t in toks)
    ar_dec = decoder(TINY, explored=[cfg["n_layers"]], width_cap=1, batch=3, max_context=P + T)
    ar_toks, ar_rounds, _ = _collect(ar_dec, prompts, P + T)
    ar_dec.close()
    assert toks == ar_toks
    assert ar_rounds == T - 1                     # AR commits once per round
    assert rounds > ar_rounds


@pytest.mark.parametrize("name,X", [(TINY, [1, 2, 3, 4]), ("small-12L-d768-bf16", [3, 6, 9, 12])])
def test_rows_per_round_at_the_maximum(name, X):
    torch_cuda()
    cfg = configs.get(name)
    B, W, T = 32, 8, 10
    assert B * W == 256                           # DEX_MAX_ROWS
    P = cfg["prompt_len"]
    prompts = np.stack([gen.tokens(gen.mix64(900 + s), P, cfg["vocab"]) for s in range(B)])
    dec = decoder(name, explored=X, width_cap=W, batch=B, max_context=P + 4 * T)
    toks, rounds = run(dec, prompts, T)
    dec.close()
    most = max(len(r["rows"]) for r in rounds)
    assert most == B * W                          # a round at the capacity
    ar_dec = decoder(name, explored=[cfg["n_layers"]], width_cap=1, batch=B, max_context=P + 4 * T)
    ar_toks, _ = run(ar_dec, prompts, T)
    ar_dec.close()
    assert np.array_equal(toks, ar_toks)


def test_width_one_commits_every_n_rounds():
    torch_cuda()
    cfg, w = host_weights(TINY)
    X, T = [1, 2, 3, 4], 16
    P = cfg["prompt_len"]
    prompt = gen.prompts(cfg)
    dec = decoder(TINY, explored=X, width_cap=1, max_context=P + T)
    toks, rounds, _ = _collect(dec, prompt, P + T)
    dec.close()
    assert rounds == len(X) * (T - 1)
    m = oracle.Model(cfg, gen.model_as_f64(cfg, w))
    pl = [int(t) for t in prompt[0]]
    res = dex.dex_generate(m, pl, X, 1, True, T, keep_trace=False)
    assert res.tokens == toks[0] and res.rounds == rounds


def test_generate_helper_and_cli(capsys, monkeypatch):
    """Decoder.generate and the generation module: DEX tokens equal the
    same library's AR tokens and the oracle's greedy AR, with one commit
    per generated token after y_0."""
    torch_cuda()
    import json

    from oracle import ar
    from paper_2606_29223_amd import generate as gen_cli
    cfg, w = host_weights(TINY)
    T = 16
    prompt = gen.prompts(cfg)
    dec = decoder(TINY, max_context=cfg["prompt_len"] + T)
    toks, st = dec.generate(prompt, T)
    dec.close()
    m = oracle.Model(cfg, gen.model_as_f64(cfg, w))
    assert toks[0] == ar.ar_generate(m, [int(t) for t in prompt[0]], T)
    assert len(st["kstar"]) == T - 1 and st["rounds"] >= T - 1
    monkeypatch.setattr("sys.argv", ["generate", "--config", TINY, "--tokens", str(T), "--ar"])
    gen_cli.main()
    out = json.loads(capsys.readouterr().out.strip().splitlines()[-1])
    assert out["equals_ar"] and out["tokens"] == toks and out["commits"] == T - 1
