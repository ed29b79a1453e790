"""Pins of the oracle's model (no GPU).

The oracle's forward is checked against things other than itself:
  * Hugging Face Transformers' Llama implementation (a third-party library
    routine) loaded with the same weights -- the per-layer residual scale
    alpha_l is folded into o_proj and down_proj, which is exact algebra;
    this fixes RMSNorm, RoPE (rotate-half), GQA head grouping, SiLU gating and
    the shared exit head at every depth;
  * RoPE against complex multiplication and its relative-position property;
  * closed forms for attention special cases;
  * the per-row (cached) decode against the matrix-form prefill.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import ar
from oracle.model import Model, argmax_lowest, rmsnorm, rope
from synth import configs, gen


def _hf_model(cfg, w64):
    from transformers import LlamaConfig, LlamaForCausalLM
    hc = LlamaConfig(
        vocab_size=cfg["vocab"], hidden_size=cfg["d_model"], intermediate_size=cfg["d_ffn"],
        num_hidden_layers=cfg["n_layers"], num_attention_heads=cfg["n_heads"],
        num_key_value_heads=cfg["n_kv_heads"], head_dim=cfg["head_dim"], rms_norm_eps=cfg["rms_eps"],
        rope_theta=cfg["rope_theta"], max_position_embeddings=4096, tie_word_embeddings=False,
        attention_bias=False, mlp_bias=False, hidden_act="silu")
    hc._attn_implementation = "eager"
    m = LlamaForCausalLM(hc).to(torch.float64).eval()
    L = cfg["n_layers"]
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a))
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(T(w64["embed"]))
        m.model.norm.weight.copy_(T(w64["final_norm"]))
        m.lm_head.weight.copy_(T(w64["lm_head"]))
        for l in range(L):
            a = cfg["residual_scale"] * (l + 1) / L
            lay = m.model.layers[l]
            p = f"layers.{l}."
            lay.input_layernorm.weight.copy_(T(w64[p + "attn_norm"]))
            lay.post_attention_layernorm.weight.copy_(T(w64[p + "ffn_norm"]))
            lay.self_attn.q_proj.weight.copy_(T(w64[p + "wq"]))
            lay.self_attn.k_proj.weight.copy_(T(w64[p + "wk"]))
            lay.self_attn.v_proj.weight.copy_(T(w64[p + "wv"]))
            lay.self_attn.o_proj.weight.copy_(T(a * w64[p + "wo"]))
            lay.mlp.gate_proj.weight.copy_(T(w64[p + "w_gate"]))
            lay.mlp.up_proj.weight.copy_(T(w64[p + "w_up"]))
            lay.mlp.down_proj.weight.copy_(T(a * w64[p + "w_down"]))
    return m


def _hf_depth_logits(hf, seq):
    """z_l at every position for l = 1..L from the library's own forward."""
    with torch.no_grad():
        out = hf(torch.tensor([seq]), output_hidden_states=True, use_cache=False)
        hs = out.hidden_states              # embeddings, layer 1 .. layer L (last one normed)
        L = len(hs) - 1
        zs = [hf.lm_head(hf.model.norm(hs[l]))[0] for l in range(1, L)]
        zs.append(out.logits[0])
    return torch.stack(zs, dim=1).numpy()   # [n, L, V]


GQA_TINY = dict(n_layers=3, d_model=64, n_heads=4, n_kv_heads=2, head_dim=16, d_ffn=96, vocab=97,
                dtype="f32", rope_theta=1.0e4, rms_eps=1.0e-5, residual_scale=0.3, model_seed=11,
                explored=[1, 2, 3], width_cap=0, decs=1, batch=1, prompt_len=9, gen_len=12,
                prompt_seeds=[7])


@pytest.mark.parametrize("which", ["tiny", "gqa", "bf16"])
def test_forward_matches_transformers_llama(which):
    if which == "tiny":
        cfg = configs.get("tiny-4L-d128-fp32")
    elif which == "gqa":
        cfg = dict(GQA_TINY, name="gqa")
    else:  # bf16 family at reduced size (exact bf16 values upcast)
        cfg = configs.scaled_down(configs.get("llama-32L-d4096-x8-w4"), n_layers=4, d_model=256,
                                  d_ffn=512, vocab=1000)
        cfg.update(n_heads=4, n_kv_heads=2, head_dim=64, prompt_len=12)
    w = gen.generate_model(cfg)
    w64 = gen.model_as_f64(cfg, w)
    m = Model(cfg, w64)
    prompt = [int(t) for t in gen.prompts(cfg)[0]]
    toks = ar.ar_generate(m, prompt, 8)
    seq = prompt + toks[:-1]
    hf = _hf_model(cfg, w64)
    z_ref = _hf_depth_logits(hf, seq)                       # [n, L, V]
    L = cfg["n_layers"]
    # teacher-forced per-row decode, every depth, generated positions
    z_row = ar.depth_logits(m, prompt, toks, list(range(1, L + 1)))
    P = len(prompt)
    ref = z_ref[P:P + len(toks) - 1]
    # The library computes RoPE angles and RMSNorm statistics in float32 even
    # for a float64 model, so agreement is at float32 level; a dropped term, a
    # wrong sign or a mis-grouped head moves logits by O(1).
    tol = dict(rtol=1e-5, atol=2e-5)
    assert np.allclose(z_row, ref, **tol), np.abs(z_row - ref).max()
    # matrix-form prefill: last-position final logits and keys
    Ks, Vs, h_last = m.prefill(prompt)
    assert np.allclose(m.exit_logits(h_last), z_ref[P - 1, L - 1], **tol)
    # greedy AR equals the library's argmax chain (ties are not expected here)
    assert toks[1:] == [int(np.argmax(z_ref[P + i, L - 1])) for i in range(len(toks) - 1)]


def test_rope_is_complex_rotation_and_relative():
    rng = np.random.default_rng(0)
    hd, theta = 8, 1.0e4
    x = rng.standard_normal((3, hd))
    for pos in (0, 1, 7, 123):
        r = rope(x, pos, theta)
        c = x[:, : hd // 2] + 1j * x[:, hd // 2:]
        ang = pos * theta ** (-2.0 * np.arange(hd // 2) / hd)
        c2 = c * np.exp(1j * ang)
        assert np.allclose(r, np.concatenate([c2.real, c2.imag], axis=1), atol=1e-12)
    q, k = rng.standard_normal((1, hd)), rng.standard_normal((1, hd))
    d1 = float(rope(q, 10, theta)[0] @ rope(k, 3, theta)[0])
    d2 = float(rope(q, 110, theta)[0] @ rope(k, 103, theta)[0])
    assert abs(d1 - d2) < 1e-9
    assert np.allclose(rope(x, 0, theta), x)


def test_rmsnorm_and_argmax_conventions():
    x = np.array([3.0, -4.0])
    g = np.array([1.0, 2.0])
    y = rmsnorm(x, g, 0.0)
    assert np.allclose(y, [3.0 / math.sqrt(12.5), -8.0 / math.sqrt(12.5)])
    assert np.allclose(rmsnorm(5.0 * x, g, 0.0), y)
    z = np.array([0.0, 2.0, 2.0, 1.0])
    assert argmax_lowest(z) == 1
    assert argmax_lowest(z, masked=(1,)) == 2
    assert argmax_lowest(z, masked=(1, 2)) == 3


def test_attention_special_cases():
    cfg = dict(GQA_TINY)
    m = oracle.load(cfg)
    rng = np.random.default_rng(1)
    q = rng.standard_normal((m.H, m.hd))
    # one key: output is its value
    k1 = rng.standard_normal((1, m.Hkv, m.hd))
    v1 = rng.standard_normal((1, m.Hkv, m.hd))
    o = m.attend_row(q, k1, v1)
    for h in range(m.H):
        assert np.allclose(o[h], v1[0, h // (m.H // m.Hkv)])
    # identical keys: output is the mean of the values
    kk = np.repeat(k1, 5, axis=0)
    vv = rng.standard_normal((5, m.Hkv, m.hd))
    o = m.attend_row(q, kk, vv)
    for h in range(m.H):
        assert np.allclose(o[h], vv[:, h // (m.H // m.Hkv)].mean(axis=0))


def test_cached_rows_match_prefill():
    cfg = configs.get("tiny-4L-d128-fp32")
    m = oracle.load(cfg)
    prompt = [int(t) for t in gen.prompts(cfg)[0]]
    Ks, Vs, h_last = m.prefill(prompt)
    # rebuild the prompt's cache row by row
    cache = ar.Cache(m, [k[:1] for k in Ks], [v[:1] for v in Vs], len(prompt))
    h0 = ar.decode_row(m, cache, prompt[0], 0, write=True)
    for p in range(1, len(prompt)):
        hs = ar.decode_row(m, cache, prompt[p], p)
    for l in range(m.L):
        assert np.allclose(cache.K[l][: len(prompt)], Ks[l], atol=1e-10)
        assert np.allclose(cache.V[l][: len(prompt)], Vs[l], atol=1e-10)
    assert np.allclose(hs[-1], h_last, atol=1e-10)
