"""Seeded inputs: the C generator and its numpy twin agree bit for bit."""
import numpy as np

from synth import configs, gen


def test_c_and_numpy_twins_agree():
    for bf16 in (False, True):
        for scale, off in ((0.3, 0.0), (0.05, 1.0), (3.0, 0.0)):
            a = gen.uniform(987654321, 50_001, scale, off, bf16=bf16, start=17)
            b = gen.uniform(987654321, 50_001, scale, off, bf16=bf16, start=17, force_numpy=True)
            assert a.dtype == b.dtype
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8))
    t1 = gen.tokens(42, 10_000, 32000)
    t2 = gen.tokens(42, 10_000, 32000, force_numpy=True)
    assert np.array_equal(t1, t2) and t1.min() >= 0 and t1.max() < 32000


def test_uniform_moments_and_range():
    v = gen.uniform(5, 1 << 20, 1.0)
    assert -1.0 < v.min() and v.max() < 1.0
    assert abs(v.mean()) < 5e-3 and abs(v.var() - 1.0 / 3.0) < 5e-3


def test_bf16_rounding_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1e-30], dtype=np.float32)
    b = gen.f32_to_bf16_bits(x)
    back = gen.bf16_bits_to_f32(b)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: even mantissa wins (1.0)
    assert back[0] == 1.0 and back[1] == 1.0 and back[2] == np.float32(1.0 + 2 ** -6)
    assert back[3] == -2.5


def test_model_tensors_shapes_and_determinism():
    cfg = configs.get("tiny-4L-d128-fp32")
    w1 = gen.generate_model(cfg)
    w2 = gen.generate_model(cfg, force_numpy=True)
    assert set(w1) == set(w2)
    for k in w1:
        assert np.array_equal(w1[k], w2[k]), k
    assert w1["layers.0.wq"].shape == (128, 128) and w1["layers.3.w_down"].shape == (128, 344)
    p = gen.prompts(cfg)
    assert p.shape == (1, 16) and p.dtype == np.int32
    cfg2 = configs.get("small-12L-d768-bf16")
    specs = gen.tensor_specs(cfg2)
    assert sum(int(np.prod(s)) for _, s, _ in specs) > 100_000_000
