"""Oracle: the synthetic decoder and its exit heads, in float64 numpy.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this
package; only the tests, the smoke check and the CPU-baseline leg of the
benchmark do.  It shares no code with the GPU path.

Model (Llama-family decoder, the backbone family of the paper's Section 4
setup; one shared final RMSNorm and LM head decode every explored depth, as
the inducing-adapter appendix states):

  h^0_p = E[x_p]
  for layer l = 1..L, with alpha_l = residual_scale * l / L:
    a      = RMSNorm(h^{l-1}_p; g^attn_l)
    q,k,v  = Wq a, Wk a, Wv a; q and k rotated by RoPE at position p
    o_h    = sum_{j<=p} softmax_j(q_h . k_{j,g(h)} / sqrt(hd)) v_{j,g(h)},  g(h) = h // (H/H_kv)
    h'     = h^{l-1}_p + alpha_l * Wo concat_h(o_h)
    b      = RMSNorm(h'; g^ffn_l)
    h^l_p  = h' + alpha_l * W_down (SiLU(W_gate b) * (W_up b))
  exit logits at depth l: z_l(p) = W_head RMSNorm(h^l_p; g^final)

RMSNorm(x; g) = g * x / sqrt(mean(x^2) + eps).  RoPE pairs element i with
i + hd/2 (rotate-half) at angle p * theta^(-2i/hd).  argmax ties resolve to
the lowest token id.

Every decode-time quantity is computed one row (one position of one branch)
at a time, so that a row's bits never depend on which other rows exist.
"""

from __future__ import annotations

import math

import numpy as np


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """g * x / sqrt(mean(x^2) + eps) over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return g * (x / np.sqrt(ms + eps))


def rope(x: np.ndarray, pos, theta: float) -> np.ndarray:
    """Rotate-half RoPE.  x: [..., n_heads, hd]; pos: scalar or [rows] broadcast
    against the leading axis."""
    hd = x.shape[-1]
    half = hd // 2
    i = np.arange(half, dtype=np.float64)
    inv_freq = theta ** (-2.0 * i / hd)
    pos = np.asarray(pos, dtype=np.float64)
    ang = pos[..., None] * inv_freq                      # [..., half]
    cos = np.cos(ang)[..., None, :]
    sin = np.sin(ang)[..., None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def argmax_lowest(z: np.ndarray, masked=()) -> int:
    """argmax over the vocabulary with masked ids at -inf; ties -> lowest id."""
    if masked:
        z = z.copy()
        z[list(masked)] = -np.inf
    return int(np.argmax(z))      # numpy returns the first maximal index


class Model:
    """The synthetic decoder with float64 weights (exact upcasts of the
    generated values)."""

    def __init__(self, cfg: dict, weights64: dict):
        self.cfg = cfg
        self.L = cfg["n_layers"]
        self.d = cfg["d_model"]
        self.H = cfg["n_heads"]
        self.Hkv = cfg["n_kv_heads"]
        self.hd = cfg["head_dim"]
        self.V = cfg["vocab"]
        self.eps = cfg["rms_eps"]
        self.theta = cfg["rope_theta"]
        self.w = weights64
        self.layers = []
        for l in range(self.L):
            p = f"layers.{l}."
            self.layers.append({k: weights64[p + k] for k in
                                ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")})

    def alpha(self, l: int) -> float:
        """Residual-branch scale of 0-based layer l (1-based depth l+1)."""
        return self.cfg["residual_scale"] * (l + 1) / self.L

    # ---------------------------------------------------------------- rows
    def embed(self, token: int) -> np.ndarray:
        return self.w["embed"][token].copy()

    def qkv_row(self, l: int, h: np.ndarray, pos: int):
        P = self.layers[l]
        a = rmsnorm(h, P["attn_norm"], self.eps)
        q = (P["wq"] @ a).reshape(self.H, self.hd)
        k = (P["wk"] @ a).reshape(self.Hkv, self.hd)
        v = (P["wv"] @ a).reshape(self.Hkv, self.hd)
        return rope(q, pos, self.theta), rope(k, pos, self.theta), v

    def attend_row(self, q: np.ndarray, keys: np.ndarray, vals: np.ndarray) -> np.ndarray:
        """q [H, hd]; keys/vals [n, Hkv, hd] in logical position order 0..pos."""
        group = self.H // self.Hkv
        out = np.empty((self.H, self.hd))
        scale = 1.0 / math.sqrt(self.hd)
        for h in range(self.H):
            g = h // group
            s = (keys[:, g, :] @ q[h]) * scale
            s = s - s.max()
            p = np.exp(s)
            p = p / p.sum()
            out[h] = p @ vals[:, g, :]
        return out

    def layer_row(self, l: int, h: np.ndarray, pos: int, past_k: np.ndarray, past_v: np.ndarray):
        """One layer for one row.  past_k/past_v: [pos, Hkv, hd] keys/values at
        positions 0..pos-1 of this row's own prefix.  Returns (h_out, k, v)."""
        P = self.layers[l]
        al = self.alpha(l)
        q, k, v = self.qkv_row(l, h, pos)
        keys = np.concatenate([past_k, k[None]], axis=0)
        vals = np.concatenate([past_v, v[None]], axis=0)
        o = self.attend_row(q, keys, vals).reshape(-1)
        h1 = h + al * (P["wo"] @ o)
        b = rmsnorm(h1, P["ffn_norm"], self.eps)
        f = P["w_down"] @ (silu(P["w_gate"] @ b) * (P["w_up"] @ b))
        return h1 + al * f, k, v

    def exit_logits(self, h: np.ndarray) -> np.ndarray:
        """Shared exit head: z = W_head RMSNorm(h; g_final)."""
        return self.w["lm_head"] @ rmsnorm(h, self.w["final_norm"], self.eps)

    # -------------------------------------------------------------- prefill
    def prefill(self, prompt):
        """Causal forward over the whole prompt (matrix form).  Returns
        (K, V, h_last): K/V lists over layers of [P, Hkv, hd]; h_last the
        final hidden state of the last prompt position."""
        x = np.asarray(prompt, dtype=np.int64)
        n = len(x)
        h = self.w["embed"][x].copy()
        pos = np.arange(n)
        group = self.H // self.Hkv
        scale = 1.0 / math.sqrt(self.hd)
        causal = np.triu(np.ones((n, n), dtype=bool), k=1)
        Ks, Vs = [], []
        for l in range(self.L):
            P = self.layers[l]
            al = self.alpha(l)
            a = rmsnorm(h, P["attn_norm"], self.eps)
            q = rope((a @ P["wq"].T).reshape(n, self.H, self.hd), pos, self.theta)
            k = rope((a @ P["wk"].T).reshape(n, self.Hkv, self.hd), pos, self.theta)
            v = (a @ P["wv"].T).reshape(n, self.Hkv, self.hd)
            o = np.empty((n, self.H, self.hd))
            for hh in range(self.H):
                g = hh // group
                s = (q[:, hh, :] @ k[:, g, :].T) * scale
                s[causal] = -np.inf
                s = s - s.max(axis=1, keepdims=True)
                p = np.exp(s)
                p = p / p.sum(axis=1, keepdims=True)
                o[:, hh, :] = p @ v[:, g, :]
            h = h + al * (o.reshape(n, -1) @ P["wo"].T)
            b = rmsnorm(h, P["ffn_norm"], self.eps)
            h = h + al * ((silu(b @ P["w_gate"].T) * (b @ P["w_up"].T)) @ P["w_down"].T)
            Ks.append(k)
            Vs.append(v)
        return Ks, Vs, h[-1].copy()

    def exit_depth_states(self, h: np.ndarray, pos: int, Ks, Vs, n_past: int):
        """Run one row through all layers against a committed cache of n_past
        positions; returns (hidden after every layer [L, d], k list, v list)."""
        hs = []
        ks, vs = [], []
        for l in range(self.L):
            h, k, v = self.layer_row(l, h, pos, Ks[l][:n_past], Vs[l][:n_past])
            hs.append(h)
            ks.append(k)
            vs.append(v)
        return np.stack(hs), ks, vs
