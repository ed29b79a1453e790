"""Seeded synthetic weights and prompts for both the oracle and the GPU path.

Every value comes from the counter-based generator documented in
``_synth.c`` (SplitMix64 finaliser over a per-tensor key).  ``libsynth.so``
fills large tensors quickly; ``_np_*`` below computes exactly the same bits
with numpy and is used when the library is not built and by the test that
checks the two agree.

Initialisation (the paper trains real models; these stand in for them):
  * every projection matrix W[out, in]: uniform with variance 1/in, except
    the query and key projections, variance 4/in (sharper attention, so the
    next token depends on context rather than only on the current token);
  * the embedding: uniform with variance 9 (standard deviation 3: the
    residual stream is dominated by the token embedding, so intermediate
    exits often agree with the final depth);
  * the LM head [V, d]: uniform with variance 1/d;
  * RMSNorm gains: 1 + 0.05 * uniform(-1, 1);
  * bf16 models store matrices and the embedding rounded to bfloat16
    (round-to-nearest-even); gains are always float32.
"""

from __future__ import annotations

import ctypes
import math
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_GAMMA = 0x9E3779B97F4A7C15
_MASK = (1 << 64) - 1

LAYER_PARAMS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")

_lib = None


def _load():
    global _lib
    if _lib is None and os.path.exists(_LIB_PATH):
        lib = ctypes.CDLL(_LIB_PATH)
        u64, i64, f32 = ctypes.c_uint64, ctypes.c_int64, ctypes.c_float
        vp = ctypes.c_void_p
        lib.synth_mix64.restype = u64
        lib.synth_mix64.argtypes = [u64]
        lib.synth_uniform_f32.argtypes = [u64, u64, i64, f32, f32, vp]
        lib.synth_uniform_bf16.argtypes = [u64, u64, i64, f32, f32, vp]
        lib.synth_tokens.argtypes = [u64, u64, i64, ctypes.c_uint32, vp]
        lib.synth_bf16_to_f64.argtypes = [vp, i64, vp]
        _lib = lib
    return _lib


def build_lib(verbose: bool = False) -> str:
    """Compile libsynth.so with gcc (OpenMP, no FMA contraction)."""
    import subprocess
    src = os.path.join(_HERE, "_synth.c")
    tmp = _LIB_PATH + ".tmp"
    cmd = ["gcc", "-O3", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off", src, "-o", tmp]
    subprocess.run(cmd, check=True, capture_output=not verbose)
    os.replace(tmp, _LIB_PATH)
    global _lib
    _lib = None
    return _LIB_PATH


# --------------------------------------------------------------------------
# numpy twins (bit-identical to _synth.c)

def mix64(z: int) -> int:
    z &= _MASK
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK
    return z ^ (z >> 31)


def _np_mix64(z: np.ndarray) -> np.ndarray:
    z = z ^ (z >> np.uint64(30))
    z *= np.uint64(0xBF58476D1CE4E5B9)
    z ^= z >> np.uint64(27)
    z *= np.uint64(0x94D049BB133111EB)
    z ^= z >> np.uint64(31)
    return z


def _np_stream(key: int, start: int, n: int) -> np.ndarray:
    with np.errstate(over="ignore"):
        i = np.arange(start + 1, start + 1 + n, dtype=np.uint64)
        z = np.uint64(key) + i * np.uint64(_GAMMA)
        return _np_mix64(z)


def _np_uniform_f32(key: int, start: int, n: int, scale: float, offset: float) -> np.ndarray:
    z = _np_stream(key, start, n)
    u = (z >> np.uint64(40)).astype(np.int64)
    w = (2 * u + 1 - 16777216).astype(np.float32) / np.float32(16777216.0)
    s = np.float32(scale) * w
    return (np.float32(offset) + s).astype(np.float32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest-even), returned as uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _np_tokens(key: int, start: int, n: int, vocab: int) -> np.ndarray:
    z = _np_stream(key, start, n)
    with np.errstate(over="ignore"):
        return (((z >> np.uint64(32)) * np.uint64(vocab)) >> np.uint64(32)).astype(np.int32)


# --------------------------------------------------------------------------
# fills (library when present, numpy otherwise)

def uniform(key: int, n: int, scale: float, offset: float = 0.0, bf16: bool = False,
            start: int = 0, force_numpy: bool = False) -> np.ndarray:
    lib = None if force_numpy else _load()
    if lib is None:
        v = _np_uniform_f32(key, start, n, scale, offset)
        return f32_to_bf16_bits(v) if bf16 else v
    out = np.empty(n, dtype=np.uint16 if bf16 else np.float32)
    fn = lib.synth_uniform_bf16 if bf16 else lib.synth_uniform_f32
    fn(key, start, n, scale, offset, out.ctypes.data)
    return out


def tokens(key: int, n: int, vocab: int, force_numpy: bool = False) -> np.ndarray:
    lib = None if force_numpy else _load()
    if lib is None:
        return _np_tokens(key, 0, n, vocab)
    out = np.empty(n, dtype=np.int32)
    lib.synth_tokens(key, 0, n, vocab, out.ctypes.data)
    return out


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    lib = _load()
    b = np.ascontiguousarray(b, dtype=np.uint16)
    if lib is None:
        return bf16_bits_to_f32(b).astype(np.float64)
    out = np.empty(b.shape, dtype=np.float64)
    lib.synth_bf16_to_f64(b.ctypes.data, b.size, out.ctypes.data)
    return out


# --------------------------------------------------------------------------
# model tensors

def tensor_specs(cfg: dict):
    """[(name, shape, kind)] in a fixed order; kind is 'gain', 'embed' or 'matrix'."""
    d, H, Hkv, hd, F, V = (cfg["d_model"], cfg["n_heads"], cfg["n_kv_heads"], cfg["head_dim"],
                           cfg["d_ffn"], cfg["vocab"])
    specs = [("embed", (V, d), "embed"), ("final_norm", (d,), "gain"), ("lm_head", (V, d), "matrix")]
    for l in range(cfg["n_layers"]):
        specs += [
            (f"layers.{l}.attn_norm", (d,), "gain"),
            (f"layers.{l}.wq", (H * hd, d), "matrix"),
            (f"layers.{l}.wk", (Hkv * hd, d), "matrix"),
            (f"layers.{l}.wv", (Hkv * hd, d), "matrix"),
            (f"layers.{l}.wo", (d, H * hd), "matrix"),
            (f"layers.{l}.ffn_norm", (d,), "gain"),
            (f"layers.{l}.w_gate", (F, d), "matrix"),
            (f"layers.{l}.w_up", (F, d), "matrix"),
            (f"layers.{l}.w_down", (d, F), "matrix"),
        ]
    return specs


def tensor_key(model_seed: int, index: int) -> int:
    return mix64((mix64(model_seed) + index) & _MASK)


def generate_model(cfg: dict, force_numpy: bool = False) -> dict:
    """name -> numpy array.  bf16 models: matrices/embedding as uint16 bf16 bits;
    fp32 models: float32.  Gains are float32 in both cases."""
    bf16 = cfg["dtype"] == "bf16"
    out = {}
    for idx, (name, shape, kind) in enumerate(tensor_specs(cfg)):
        key = tensor_key(cfg["model_seed"], idx)
        n = int(np.prod(shape))
        if kind == "gain":
            arr = uniform(key, n, 0.05, 1.0, bf16=False, force_numpy=force_numpy)
        else:
            if kind == "embed":
                var = 9.0
            elif name.endswith(".wq") or name.endswith(".wk"):
                var = 4.0 / shape[1]
            else:
                var = 1.0 / shape[1]
            a = math.sqrt(3.0 * var)
            arr = uniform(key, n, a, 0.0, bf16=bf16, force_numpy=force_numpy)
        out[name] = arr.reshape(shape)
    return out


def adapter_specs(cfg: dict):
    """[(name, shape, kind)] of the inducing adapters, one per non-final
    explored depth (index k of the explored list), hidden width m = 2d."""
    d = cfg["d_model"]
    m = 2 * d
    specs = []
    for k in range(len(cfg["explored"]) - 1):
        specs += [
            (f"adapters.{k}.norm", (d,), "gain"),
            (f"adapters.{k}.w1", (m, d), "matrix"),
            (f"adapters.{k}.b1", (m,), "bias"),
            (f"adapters.{k}.w2", (d, m), "matrix"),
            (f"adapters.{k}.b2", (d,), "bias"),
        ]
    return specs


def generate_adapters(cfg: dict, alpha: float, force_numpy: bool = False) -> dict:
    """Synthetic inducing adapters (the paper trains them; these stand in):
    matrices uniform with variance 1/in (bf16 bits for bf16 models), norm
    gains 1 + 0.05 * uniform(-1, 1), biases uniform(-0.1, 0.1) float32, and
    the gate alpha (float32 [1]) set to `alpha` at every depth."""
    bf16 = cfg["dtype"] == "bf16"
    out = {}
    base = mix64((cfg["model_seed"] + 0xADA97E) & _MASK)
    for idx, (name, shape, kind) in enumerate(adapter_specs(cfg)):
        key = mix64((base + idx) & _MASK)
        n = int(np.prod(shape))
        if kind == "gain":
            arr = uniform(key, n, 0.05, 1.0, bf16=False, force_numpy=force_numpy)
        elif kind == "bias":
            arr = uniform(key, n, 0.1, 0.0, bf16=False, force_numpy=force_numpy)
        else:
            a = math.sqrt(3.0 / shape[1])
            arr = uniform(key, n, a, 0.0, bf16=bf16, force_numpy=force_numpy)
        out[name] = arr.reshape(shape)
    for k in range(len(cfg["explored"]) - 1):
        out[f"adapters.{k}.alpha"] = np.array([alpha], dtype=np.float32)
    return out


def adapters_as_f64(cfg: dict, ad: dict) -> list:
    """Per non-final depth, the adapter tensors as exact binary64 (oracle)."""
    f = model_as_f64(cfg, ad)
    return [{p: f[f"adapters.{k}.{p}"] for p in ("norm", "w1", "b1", "w2", "b2", "alpha")}
            for k in range(len(cfg["explored"]) - 1)]


def prompts(cfg: dict, force_numpy: bool = False) -> np.ndarray:
    """int32 [batch, prompt_len], uniform over the vocabulary."""
    rows = []
    for s in cfg["prompt_seeds"][: cfg["batch"]]:
        key = mix64((mix64(s) + 0x5EED) & _MASK)
        rows.append(tokens(key, cfg["prompt_len"], cfg["vocab"], force_numpy=force_numpy))
    return np.stack(rows).astype(np.int32)


def model_as_f64(cfg: dict, weights: dict) -> dict:
    """Exact binary64 copies of the generated tensors (what the oracle computes on)."""
    out = {}
    for name, arr in weights.items():
        if arr.dtype == np.uint16:
            out[name] = bf16_bits_to_f64(arr)
        else:
            out[name] = arr.astype(np.float64)
    return out
