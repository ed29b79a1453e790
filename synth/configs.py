"""The five synthetic decode workloads (model shape, explored depths, lattice
width cap, batch, prompt and generation lengths, seeds).

These stand in for the paper's evaluation models and prompt sets (Section 4
setup): greedy decoding at batch 1 with a few hundred new tokens, uniform
depth partitions DEX-1/K.  Weights are random (seeded), prompts are tokens
drawn uniformly over the vocabulary.
"""

from __future__ import annotations

import copy

_LLAMA32 = dict(
    n_layers=32, d_model=4096, n_heads=32, n_kv_heads=8, head_dim=128,
    d_ffn=14336, vocab=32000, dtype="bf16", rope_theta=1.0e4, rms_eps=1.0e-5,
    residual_scale=0.3, model_seed=3,
)

CONFIGS = {
    # 4 layers, d=128, fp32; exit at every depth; uncapped lattice.
    "tiny-4L-d128-fp32": dict(
        n_layers=4, d_model=128, n_heads=4, n_kv_heads=4, head_dim=32,
        d_ffn=344, vocab=512, dtype="f32", rope_theta=1.0e4, rms_eps=1.0e-5,
        residual_scale=0.3, model_seed=1,
        explored=[1, 2, 3, 4], width_cap=0, decs=1, batch=1,
        prompt_len=16, gen_len=64, prompt_seeds=[101],
    ),
    # 12 layers, d=768, bf16; exits {3,6,9,12}; width cap 4.
    "small-12L-d768-bf16": dict(
        n_layers=12, d_model=768, n_heads=12, n_kv_heads=12, head_dim=64,
        d_ffn=2048, vocab=32000, dtype="bf16", rope_theta=1.0e4, rms_eps=1.0e-5,
        residual_scale=0.3, model_seed=2,
        explored=[3, 6, 9, 12], width_cap=4, decs=1, batch=1,
        prompt_len=128, gen_len=256, prompt_seeds=[201],
    ),
    # Llama-shaped 32 layers, d=4096, GQA 32/8; exits {8,16,24,32}; cap 4.
    "llama-32L-d4096-x8-w4": dict(
        _LLAMA32, explored=[8, 16, 24, 32], width_cap=4, decs=1, batch=1,
        prompt_len=512, gen_len=512, prompt_seeds=[301],
    ),
    # Same model, exits every 2 layers; cap 16 (GEMMs at M up to 16).
    "llama-32L-d4096-x2-w16": dict(
        _LLAMA32, explored=list(range(2, 33, 2)), width_cap=16, decs=1, batch=1,
        prompt_len=512, gen_len=512, prompt_seeds=[401],
    ),
    # Same model, exits every 4 layers; cap 8 per lattice; 8 sequences with
    # 8192-token prompts decoded as one batch of lattices.
    "llama-32L-d4096-x4-w8-b8-ctx8192": dict(
        _LLAMA32, explored=list(range(4, 33, 4)), width_cap=8, decs=1, batch=8,
        prompt_len=8192, gen_len=1024, prompt_seeds=list(range(501, 509)),
    ),
}

# The configuration the headline throughput is quoted on.
HEADLINE = "llama-32L-d4096-x8-w4"
SMALLEST = "tiny-4L-d128-fp32"


def get(name: str, **overrides) -> dict:
    """A copy of a named workload, with optional field overrides."""
    cfg = copy.deepcopy(CONFIGS[name])
    cfg["name"] = name
    cfg.update(overrides)
    return cfg


def ar_variant(cfg: dict) -> dict:
    """The same workload decoded plainly: the only explored depth is L."""
    out = copy.deepcopy(cfg)
    out["explored"] = [cfg["n_layers"]]
    out["width_cap"] = 1
    return out


def scaled_down(cfg: dict, n_layers: int | None = None, d_model: int | None = None,
                d_ffn: int | None = None, vocab: int | None = None) -> dict:
    """A smaller model of the same family (used by fast parity tests)."""
    out = copy.deepcopy(cfg)
    if n_layers is not None:
        old = cfg["n_layers"]
        out["n_layers"] = n_layers
        out["explored"] = sorted({max(1, (d * n_layers) // old) for d in cfg["explored"]} | {n_layers})
    if d_model is not None:
        out["d_model"] = d_model
    if d_ffn is not None:
        out["d_ffn"] = d_ffn
    if vocab is not None:
        out["vocab"] = vocab
    return out
