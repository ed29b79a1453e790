"""CPU pins of the oracle's inducing adapter (Section 3.4 and its appendix).

  * the parameter count reproduces the paper's three printed totals;
  * closed forms: alpha = 0 is the identity; W2 = 0 leaves alpha * b2; W1 = 0
    leaves alpha * (W2 silu(b1) + b2); RMSNorm makes dh invariant to scaling
    h -- a dropped gate, bias, activation or norm fails one of them;
  * DEX with adapters commits exactly AR's tokens (the final depth is never
    adapted) while its intermediate candidates, and so its trace, change.
"""
import json
import os

import numpy as np
import pytest

from oracle import adapter, ar, dex
from oracle.model import Model, silu
from synth import configs, gen

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")


def test_parameter_count_matches_printed_totals():
    g = json.load(open(GOLDEN))["adapter_sizes"]
    p = adapter.param_count(g["hidden"])
    assert p == 4 * g["hidden"] ** 2 + 4 * g["hidden"] + 1 == 268468225
    for c in g["cases"]:
        tot = c["non_final_depths"] * p
        if "printed_params_millions" in c:
            assert round(tot / 1e6, 1) == c["printed_params_millions"]
        else:
            assert round(tot / 1e9, 2) == c["printed_params_billions"]


def _random_adapter(rng, h, m, alpha=0.7):
    return {"norm": 1 + 0.05 * rng.standard_normal(h), "w1": rng.standard_normal((m, h)) / np.sqrt(h),
            "b1": 0.1 * rng.standard_normal(m), "w2": rng.standard_normal((h, m)) / np.sqrt(m),
            "b2": 0.1 * rng.standard_normal(h), "alpha": np.array([alpha])}


def test_closed_forms():
    rng = np.random.default_rng(0)
    h, m, eps = 24, 48, 1e-5
    ad = _random_adapter(rng, h, m)
    x = 3.0 * rng.standard_normal(h)
    z = dict(ad, alpha=np.array([0.0]))
    assert np.array_equal(adapter.delta(z, x, eps), np.zeros(h))
    w2z = dict(ad, w2=np.zeros((h, m)))
    assert np.allclose(adapter.delta(w2z, x, eps), 0.7 * ad["b2"], rtol=0, atol=1e-15)
    w1z = dict(ad, w1=np.zeros((m, h)))
    assert np.allclose(adapter.delta(w1z, x, eps), 0.7 * (ad["w2"] @ silu(ad["b1"]) + ad["b2"]), atol=1e-14)
    # RMSNorm: scaling h leaves dh (nearly) unchanged, a missing norm would not
    d1, d2 = adapter.delta(ad, x, eps), adapter.delta(ad, 50.0 * x, eps)
    assert np.max(np.abs(d1 - d2)) < 1e-5 * np.max(np.abs(d1))
    assert np.max(np.abs(d1)) > 0.05
    # linear in alpha
    assert np.allclose(adapter.delta(dict(ad, alpha=np.array([1.4])), x, eps), 2 * d1, atol=1e-14)


def test_synthetic_adapters_shapes_and_determinism():
    cfg = configs.get("small-12L-d768-bf16")
    a = gen.generate_adapters(cfg, 0.5)
    b = gen.generate_adapters(cfg, 0.5)
    assert set(a) == set(b)
    for k in range(len(cfg["explored"]) - 1):
        assert a[f"adapters.{k}.w1"].shape == (1536, 768) and a[f"adapters.{k}.w1"].dtype == np.uint16
        assert a[f"adapters.{k}.w2"].shape == (768, 1536)
        assert np.array_equal(a[f"adapters.{k}.w1"], b[f"adapters.{k}.w1"])
    assert not np.array_equal(a["adapters.0.w1"], a["adapters.1.w1"])


@pytest.mark.parametrize("X,W", [([1, 2, 3, 4], 0), ([2, 4], 2), ([1, 3, 4], 3)])
def test_dex_with_adapters_is_lossless(X, W):
    cfg = configs.get("tiny-4L-d128-fp32", explored=X)
    m = Model(cfg, gen.model_as_f64(cfg, gen.generate_model(cfg)))
    prompt = [int(t) for t in gen.prompts(cfg)[0]]
    pf = m.prefill(prompt)
    ads = gen.adapters_as_f64(cfg, gen.generate_adapters(cfg, 0.8))
    T = 40
    ref = ar.ar_generate(m, prompt, T, prefill=pf)
    plain = dex.dex_generate(m, prompt, X, W, True, T, prefill=pf)
    adapted = dex.dex_generate(m, prompt, X, W, True, T, prefill=pf, adapters=ads)
    assert plain.tokens == ref and adapted.tokens == ref
    cand = lambda r: [t for tr in r.trace for t in tr.tokens]  # noqa: E731
    assert cand(plain) != cand(adapted)
