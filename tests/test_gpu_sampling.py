"""GPU: DECS sampling mode (Algorithm 2's Gumbel branch) through the C ABI.

  * the library's Gumbel rows equal the oracle's generator within binary32
    rounding;
  * sampled DEX commits exactly the tokens of the same library's sampled AR
    (same seed): the committed token is the Gumbel-max of the unmasked
    final-depth logits with the row of its position, whatever the lattice
    did; the lattice trace equals the oracle lattice's on the GPU's
    candidates;
  * the sampled tokens follow the float64 oracle re-scoring the GPU's own
    prefix (argmax of logits / tau + G), except within 1e-2 / tau of a tie.
"""
import numpy as np
import pytest

import oracle
from oracle import ar, gumbel
from synth import configs, gen
from tests.gpu_common import GAP, device_weights, host_weights, torch_cuda
from tests.test_gpu_decode import _replay, _run

pytestmark = pytest.mark.gpu

TINY = "tiny-4L-d128-fp32"
SMALL = "small-12L-d768-bf16"
C3 = "llama-32L-d4096-x8-w4"


def test_gumbel_rows_match_oracle():
    torch = torch_cuda()
    from paper_2606_29223_amd import dexlib
    lib = dexlib.load()
    V = 32000
    out = torch.empty(V, dtype=torch.float32, device="cuda")
    for seed, seq, pos in [(0, 0, 0), (1, 0, 5), (12345, 3, 8191), (2 ** 63 + 7, 7, 100000)]:
        assert lib.dex_debug_gumbel(seed, seq, pos, V, out.data_ptr(), torch.cuda.current_stream().cuda_stream) == 0
        torch.cuda.synchronize()
        g = out.cpu().numpy().astype(np.float64)
        ref = gumbel.gumbel_row(seed, seq, pos, V)
        assert np.max(np.abs(g - ref) / (1.0 + np.abs(ref))) < 2e-6, (seed, seq, pos)


def _check_sampled(z_final, seq_tokens, tau, seed, seq, P):
    """z_final[t-1]: oracle final-depth logits at position P+t-1 on the GPU's
    prefix; the GPU's token t must be the Gumbel-max there (or a near tie)."""
    flips = 0
    for t in range(1, len(seq_tokens)):
        pos = P + t - 1
        s = z_final[t - 1] / tau + gumbel.gumbel_row(seed, seq, pos, len(z_final[t - 1]))
        y = int(seq_tokens[t])
        best = int(np.argmax(s))
        if y != best:
            assert s[best] - s[y] < GAP / tau, (t, y, best)
            flips += 1
    return flips


@pytest.mark.parametrize("name,tau,seed", [(TINY, 1.0, 11), (TINY, 0.6, 12), (SMALL, 1.0, 21)])
def test_sampled_dex_equals_sampled_ar_and_oracle(name, tau, seed):
    torch = torch_cuda()
    from paper_2606_29223_amd import dexlib
    cfg, w = host_weights(name)
    P = cfg["prompt_len"]
    T = 40
    prompt = gen.prompts(cfg)
    dev = device_weights(name)
    ar_dec = dexlib.Decoder(cfg, dev, explored=[cfg["n_layers"]], width_cap=1, max_context=P + T,
                            temperature=tau, seed=seed)
    ar_toks, _ = _run(ar_dec, prompt, T, collapse=False)
    ar_dec.close()
    dec = dexlib.Decoder(cfg, dev, max_context=P + T, temperature=tau, seed=seed)
    toks, rounds = _run(dec, prompt, T)
    dec.close()
    assert np.array_equal(toks, ar_toks)
    _replay(rounds, len(cfg["explored"]), cfg["width_cap"], cfg["decs"], P + T, toks[0][0], P)
    greedy = dexlib.Decoder(cfg, dev, explored=[cfg["n_layers"]], width_cap=1, max_context=P + T)
    g_toks, _ = _run(greedy, prompt, T, collapse=False)
    greedy.close()
    assert not np.array_equal(g_toks, toks)           # sampling changed the sequence
    m = oracle.Model(cfg, gen.model_as_f64(cfg, w))
    pl = [int(t) for t in prompt[0]]
    pf = m.prefill(pl)
    seq = [int(t) for t in toks[0]]
    s0 = m.exit_logits(pf[2]) / tau + gumbel.gumbel_row(seed, 0, P - 1, cfg["vocab"])
    assert seq[0] == int(np.argmax(s0)) or s0.max() - s0[seq[0]] < GAP / tau
    z = ar.depth_logits(m, pl, seq, [cfg["n_layers"]], prefill=pf)
    assert _check_sampled(z[:, 0], seq, tau, seed, 0, P) <= 2


def test_sampled_dex_equals_sampled_ar_full_size():
    torch = torch_cuda()
    from paper_2606_29223_amd import dexlib
    cfg = configs.get(C3)
    P, T = cfg["prompt_len"], 24
    dev = dexlib.device_weights(cfg, gen.generate_model(cfg))
    prompt = gen.prompts(cfg)
    ar_dec = dexlib.Decoder(cfg, dev, explored=[cfg["n_layers"]], width_cap=1, max_context=P + T,
                            temperature=1.0, seed=5)
    ar_toks, _ = _run(ar_dec, prompt, T, collapse=False)
    ar_dec.close()
    dec = dexlib.Decoder(cfg, dev, max_context=P + T, temperature=1.0, seed=5)
    toks, rounds = _run(dec, prompt, T)
    dec.close()
    assert np.array_equal(toks, ar_toks)
    _replay(rounds, len(cfg["explored"]), cfg["width_cap"], cfg["decs"], P + T, toks[0][0], P)
    del dev
    torch.cuda.empty_cache()
