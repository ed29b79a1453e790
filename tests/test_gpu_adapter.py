"""GPU: inducing adapters at the non-final explored depths (Section 3.4 and
its appendix) through the C ABI, with synthetic adapter weights.

  * DEX with adapters commits exactly the same library's plain AR tokens
    (the final depth is never adapted), while its intermediate candidates
    differ from DEX without adapters;
  * the lattice trace equals the oracle lattice's on the GPU's candidates;
  * every anchor row's exit logits -- adapted below the final depth -- agree
    with the float64 oracle's within 2e-2 (max relative), teacher-forced.
"""
import numpy as np
import pytest

import oracle
from oracle import ar
from synth import configs, gen
from tests.gpu_common import LOGIT_RTOL, device_weights, host_weights, max_rel_err, torch_cuda
from tests.test_gpu_decode import _replay, _run

pytestmark = pytest.mark.gpu

TINY = "tiny-4L-d128-fp32"
SMALL = "small-12L-d768-bf16"
C3 = "llama-32L-d4096-x8-w4"


@pytest.mark.parametrize("name,alpha", [(TINY, 0.8), (SMALL, 0.5)])
def test_adapters_lossless_and_oracle_logits(name, alpha):
    torch = torch_cuda()
    from paper_2606_29223_amd import dexlib
    cfg, w = host_weights(name)
    P, T = cfg["prompt_len"], 40
    prompt = gen.prompts(cfg)
    dev = device_weights(name)
    ad = gen.generate_adapters(cfg, alpha)
    dev_ad = dexlib.device_weights(cfg, ad)
    ar_dec = dexlib.Decoder(cfg, dev, explored=[cfg["n_layers"]], width_cap=1, max_context=P + T)
    ar_toks, _ = _run(ar_dec, prompt, T, collapse=False)
    ar_dec.close()
    plain = dexlib.Decoder(cfg, dev, max_context=P + T)
    p_toks, p_rounds = _run(plain, prompt, T)
    plain.close()
    dec = dexlib.Decoder(cfg, dev, max_context=P + T, adapters=dev_ad)
    tap = torch.empty((dec.batch * 8, cfg["vocab"]), dtype=torch.float32, device="cuda")
    dec.set_logits_tap(tap)
    toks, rounds = _run(dec, prompt, T, tap=tap)
    dec.close()
    assert np.array_equal(toks, ar_toks) and np.array_equal(p_toks, ar_toks)
    cand = lambda rs: [r[4] for rd in rs for r in rd["rows"]]  # noqa: E731
    assert cand(rounds) != cand(p_rounds)
    _replay(rounds, len(cfg["explored"]), cfg["width_cap"], cfg["decs"], P + T, toks[0][0], P)
    m = oracle.Model(cfg, gen.model_as_f64(cfg, w))
    ads = gen.adapters_as_f64(cfg, ad)
    pl = [int(t) for t in prompt[0]]
    pf = m.prefill(pl)
    seq = [int(t) for t in toks[0]]
    z = ar.depth_logits(m, pl, seq, cfg["explored"], prefill=pf, adapters=ads)
    worst, seen = 0.0, 0
    for rd in rounds:
        for r, (s, slot, stage, pos, tok) in enumerate(rd["rows"]):
            if slot == 0 and pos - P < len(seq) - 1:
                worst = max(worst, max_rel_err(rd["logits"][r], z[pos - P, stage]))
                seen += 1
    assert seen > 10
    assert worst <= LOGIT_RTOL, worst


def test_adapters_lossless_full_size():
    torch = torch_cuda()
    from paper_2606_29223_amd import dexlib
    cfg = configs.get(C3)
    P, T = cfg["prompt_len"], 24
    dev = dexlib.device_weights(cfg, gen.generate_model(cfg))
    dev_ad = dexlib.device_weights(cfg, gen.generate_adapters(cfg, 0.5))
    prompt = gen.prompts(cfg)
    ar_dec = dexlib.Decoder(cfg, dev, explored=[cfg["n_layers"]], width_cap=1, max_context=P + T)
    ar_toks, _ = _run(ar_dec, prompt, T, collapse=False)
    ar_dec.close()
    dec = dexlib.Decoder(cfg, dev, max_context=P + T, adapters=dev_ad)
    toks, rounds = _run(dec, prompt, T)
    dec.close()
    assert np.array_equal(toks, ar_toks)
    _replay(rounds, len(cfg["explored"]), cfg["width_cap"], cfg["decs"], P + T, toks[0][0], P)
    del dev, dev_ad
    torch.cuda.empty_cache()
