"""CPU pins of the oracle's DECS sampling mode (Algorithm 2, sampling branch).

  * the generator reproduces SplitMix64's published outputs;
  * the uniforms are exact binary32 values in (0, 1) and the Gumbel rows have
    the Gumbel(0, 1) mean (Euler's constant) and variance (pi^2 / 6);
  * Gumbel-max over many positions samples softmax(l / tau) (the trick the
    paper relies on for exactness) -- a sign, scale or temperature mistake
    shifts the frequencies far outside the tolerance;
  * DEX in sampling mode commits exactly the tokens of AR sampling with the
    same seed (lossless), with and without DECS, capped and uncapped;
  * non-final nodes never repeat a shallower node's token of their slot
    chain under DECS (the mask applies in sampling mode too).
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import ar, dex, gumbel
from oracle.model import Model
from synth import configs, gen

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "splitmix64.json")


def test_splitmix64_published_outputs():
    g = json.load(open(GOLDEN))
    out = gumbel.stream(g["seed"], len(g["outputs_hex"]))
    assert [int(x) for x in out] == [int(h, 16) for h in g["outputs_hex"]]
    assert gumbel.mix64(gumbel.GAMMA) == int(g["outputs_hex"][0], 16)


def test_uniforms_exact_and_gumbel_moments():
    u = np.concatenate([gumbel.uniforms(11, s, p, 4096) for s in range(4) for p in range(16)])
    assert u.min() > 0.0 and u.max() < 1.0
    assert np.array_equal(u.astype(np.float32).astype(np.float64), u)     # exact in binary32
    assert abs(u.mean() - 0.5) < 4 * math.sqrt(1 / 12 / u.size)
    g = np.concatenate([gumbel.gumbel_row(11, s, p, 4096) for s in range(4) for p in range(16)])
    n = g.size
    assert abs(g.mean() - 0.5772156649015329) < 4 * math.sqrt(math.pi ** 2 / 6 / n)
    assert abs(g.var() - math.pi ** 2 / 6) < 0.05
    # rows differ across positions, sequences and seeds
    a = gumbel.gumbel_row(1, 0, 5, 64)
    assert not np.array_equal(a, gumbel.gumbel_row(1, 0, 6, 64))
    assert not np.array_equal(a, gumbel.gumbel_row(1, 1, 5, 64))
    assert not np.array_equal(a, gumbel.gumbel_row(2, 0, 5, 64))
    assert np.array_equal(a, gumbel.gumbel_row(1, 0, 5, 64))


@pytest.mark.parametrize("tau", [0.5, 1.0, 2.0])
def test_gumbel_max_samples_softmax(tau):
    z = np.array([1.0, 0.2, -0.5, 0.9, -2.0])
    n = 30000
    counts = np.zeros(len(z))
    for pos in range(n):
        counts[gumbel.decode(z, (), tau, 1234, 0, pos)] += 1
    p = np.exp(z / tau - (z / tau).max())
    p /= p.sum()
    f = counts / n
    assert np.all(np.abs(f - p) < 5 * np.sqrt(p * (1 - p) / n) + 1e-3), (f, p)
    # masking removes an id and renormalises the rest
    counts = np.zeros(len(z))
    for pos in range(n // 2):
        counts[gumbel.decode(z, (0,), tau, 99, 1, pos)] += 1
    q = p.copy()
    q[0] = 0
    q /= q.sum()
    f = counts / (n // 2)
    assert counts[0] == 0
    assert np.all(np.abs(f - q) < 5 * np.sqrt(q * (1 - q) / (n // 2)) + 1e-3), (f, q)


def test_temperature_zero_is_greedy():
    z = np.array([0.1, 3.0, 3.0, -1.0])
    assert gumbel.decode(z, (), 0.0, 5, 0, 7) == 1
    assert gumbel.decode(z, (1,), 0.0, 5, 0, 7) == 2


@pytest.fixture(scope="module")
def tiny():
    cfg = configs.get("tiny-4L-d128-fp32")
    m = Model(cfg, gen.model_as_f64(cfg, gen.generate_model(cfg)))
    prompt = [int(t) for t in gen.prompts(cfg)[0]]
    return cfg, m, prompt, m.prefill(prompt)


@pytest.mark.parametrize("X,W,decs,tau,seed", [([1, 2, 3, 4], 0, 1, 1.0, 7), ([2, 4], 2, 1, 0.7, 8),
                                               ([1, 2, 3, 4], 3, 0, 1.3, 9), ([1, 3, 4], 0, 1, 0.4, 10)])
def test_sampling_dex_equals_ar_sampling(tiny, X, W, decs, tau, seed):
    cfg, m, prompt, pf = tiny
    T = 40
    ref = ar.ar_generate(m, prompt, T, prefill=pf, temperature=tau, seed=seed)
    greedy = ar.ar_generate(m, prompt, T, prefill=pf)
    assert ref != greedy                         # the noise changes the sequence
    r = dex.dex_generate(m, prompt, X, W, bool(decs), T, prefill=pf, temperature=tau, seed=seed)
    assert r.tokens == ref
    # a different seed gives a different sample
    assert ar.ar_generate(m, prompt, T, prefill=pf, temperature=tau, seed=seed + 100) != ref


def test_sampling_decs_masks_prior_tokens(tiny):
    cfg, m, prompt, pf = tiny
    seen = {"checked": 0}

    def check(lat, cache, n):
        for s in lat.slots:
            u = s.u
            for j in range(len(u)):
                final_ref = (s is lat.anchor and j == len(cfg["explored"]) - 1)
                if j > 0 and not final_ref:
                    assert u[j] not in u[:j]
                    seen["checked"] += 1

    dex.dex_generate(m, prompt, [1, 2, 3, 4], 0, True, 30, prefill=pf, temperature=1.0, seed=3, check=check)
    assert seen["checked"] > 20
