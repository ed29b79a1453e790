"""Oracle: the Gumbel source of DECS sampling mode (Algorithm 2).

TEST INFRASTRUCTURE ONLY (see oracle/model.py).

In sampling mode Algorithm 2 decodes a lattice node as
    y = argmax_v ( l_v / tau + G[r(i), v] )
with l the node's logits after the DECS mask (masked ids at -inf), tau the
temperature and G one row of standard Gumbel noise per sampling slot, drawn
once and shared by every depth of the slot chain.  The final-depth node of
the anchor is never masked, so by the Gumbel-max trick its token is an exact
sample of softmax(l / tau): the committed distribution is the target one.

Reading (the paper does not say how rows are drawn): the row of a slot is a
function of (seed, sequence, position of the slot's input token) only, drawn
from a counter-based generator, so that plain autoregressive sampling at the
same position draws the same row.  Slots of different branches at one
position therefore share noise; the committed branch at each position is
decided by earlier rows only, so the committed sample stays exact.

Generator: the SplitMix64 stream (Steele, Lea and Flood, "Fast splittable
pseudorandom number generators", OOPSLA 2014): with gamma = 0x9E3779B97F4A7C15
and the finaliser
    mix64(z):  z ^= z >> 30;  z *= 0xBF58476D1CE4E5B9;
               z ^= z >> 27;  z *= 0x94D049BB133111EB;  z ^= z >> 31
(all mod 2^64), output i >= 1 of the stream seeded with s is
mix64(s + i * gamma).  Per row
    key   = mix64(seed XOR mix64(seq * 2^32 + pos))
    z_v   = output v + 1 of the stream seeded with key
    u_v   = (floor(z_v / 2^41) + 1/2) / 2^23           (exact in binary32)
    G_v   = -ln(-ln u_v)                                 (float64 here)
"""

from __future__ import annotations

import numpy as np

from .model import argmax_lowest

GAMMA = 0x9E3779B97F4A7C15
_MASK = (1 << 64) - 1


def mix64(z: int) -> int:
    """SplitMix64 finaliser on a Python int (mod 2^64)."""
    z &= _MASK
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK
    return z ^ (z >> 31)


def stream(seed: int, n: int) -> np.ndarray:
    """Outputs 1..n of the SplitMix64 stream seeded with `seed` (uint64)."""
    i = np.arange(1, n + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(seed & _MASK) + i * np.uint64(GAMMA)
        z = z ^ (z >> np.uint64(30))
        z = z * np.uint64(0xBF58476D1CE4E5B9)
        z = z ^ (z >> np.uint64(27))
        z = z * np.uint64(0x94D049BB133111EB)
        z = z ^ (z >> np.uint64(31))
    return z


def row_key(seed: int, seq: int, pos: int) -> int:
    return mix64((seed & _MASK) ^ mix64((seq << 32) + pos))


def uniforms(seed: int, seq: int, pos: int, V: int) -> np.ndarray:
    z = stream(row_key(seed, seq, pos), V)
    return ((z >> np.uint64(41)).astype(np.float64) + 0.5) / 8388608.0


def gumbel_row(seed: int, seq: int, pos: int, V: int) -> np.ndarray:
    """G[v] ~ Gumbel(0, 1) for the slot of sequence `seq` at position `pos`."""
    return -np.log(-np.log(uniforms(seed, seq, pos, V)))


def decode(z: np.ndarray, masked, temperature: float, seed: int, seq: int, pos: int) -> int:
    """Algorithm 2 for one node: greedy (temperature <= 0) or Gumbel-max
    sampling, masked ids at -inf, lowest id on ties."""
    if temperature <= 0.0:
        return argmax_lowest(z, masked)
    return argmax_lowest(z / temperature + gumbel_row(seed, seq, pos, len(z)), masked)
