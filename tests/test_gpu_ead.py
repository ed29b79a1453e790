"""GPU: the earliest-available-depth tool (Definition 1) on the synthetic
models, and the invariants the paper derives from it.

  * the all-depth decoder commits exactly plain AR's tokens, and its
    acceptance rows equal the float64 oracle's (the oracle re-scores every
    depth of the GPU's own prefix; a depth may differ only at a near tie);
  * Proposition 2 (0 <= ceil_X(EAD) - EAD <= Delta(X)) and Proposition 3's
    bounds hold on the measured EADs;
  * a DEX run with the workload's X commits at matched depths that never
    exceed the X-ceiling of the position's stable EAD: d_{k*} <=
    ceil_X(EAD^stab(t)).
"""
import numpy as np
import pytest

import oracle
from oracle import ar
from paper_2606_29223_amd import ead as tool
from synth import configs, gen
from tests.gpu_common import GAP, device_weights, host_weights, torch_cuda
from tests.test_gpu_decode import _run

pytestmark = pytest.mark.gpu

TINY = "tiny-4L-d128-fp32"
SMALL = "small-12L-d768-bf16"
C3 = "llama-32L-d4096-x8-w4"


def _kstar_check(cfg, dev, prompt, T, acc):
    from paper_2606_29223_amd import dexlib
    P = cfg["prompt_len"]
    dec = dexlib.Decoder(cfg, dev, max_context=P + T)
    toks, rounds = _run(dec, prompt, T, collapse=False)
    dec.close()
    X = cfg["explored"]
    ks = [rd["kstar"][0] for rd in rounds if rd["kstar"][0] >= 0]
    assert len(ks) >= T - 1
    for t, k in enumerate(ks[: T - 1]):
        assert X[k] <= tool.ceil_x(tool.ead_stable(acc[t]), X), (t, k)
    return toks


@pytest.mark.parametrize("name,T", [(TINY, 48), (SMALL, 40)])
def test_ead_tool_matches_oracle_and_invariants(name, T):
    torch_cuda()
    from paper_2606_29223_amd import dexlib
    cfg, w = host_weights(name)
    L, P = cfg["n_layers"], cfg["prompt_len"]
    dev = device_weights(name)
    prompt = gen.prompts(cfg)
    toks, acc = tool.measure(cfg, dev, prompt, T)
    ar_dec = dexlib.Decoder(cfg, dev, explored=[L], width_cap=1, max_context=P + T)
    ar_toks, _ = _run(ar_dec, prompt, T, collapse=False)
    ar_dec.close()
    assert np.array_equal(toks, ar_toks)
    acc = acc[0]
    assert acc.shape == (T - 1, L) and np.all(acc[:, -1] == 1)
    m = oracle.Model(cfg, gen.model_as_f64(cfg, w))
    pl = [int(t) for t in prompt[0]]
    seq = [int(t) for t in toks[0]]
    z = ar.depth_logits(m, pl, seq, list(range(1, L + 1)), prefill=m.prefill(pl))   # [T-1, L, V]
    diff = 0
    for t in range(T - 1):
        for l in range(L):
            o = int(np.argmax(z[t, l]) == seq[t + 1])
            if o != acc[t, l]:
                srt = np.sort(z[t, l])
                assert srt[-1] - srt[-2] < GAP, (t, l)
                diff += 1
    assert diff <= 2
    out = tool.accounting(acc, cfg["explored"], L)
    assert out["overhead_in_bounds"] and out["bounds_hold"]
    dex_toks = _kstar_check(cfg, dev, prompt, T, acc)
    assert np.array_equal(dex_toks, toks)


def test_ead_invariant_full_size():
    torch = torch_cuda()
    from paper_2606_29223_amd import dexlib
    cfg = configs.get(C3)
    T = 20
    dev = dexlib.device_weights(cfg, gen.generate_model(cfg))
    prompt = gen.prompts(cfg)
    toks, acc = tool.measure(cfg, dev, prompt, T)
    out = tool.accounting(acc[0], cfg["explored"], cfg["n_layers"])
    assert out["overhead_in_bounds"] and out["bounds_hold"]
    dex_toks = _kstar_check(cfg, dev, prompt, T, acc[0])
    assert np.array_equal(dex_toks, toks)
    del dev
    torch.cuda.empty_cache()
