"""Oracle: the inducing adapter at a non-final explored depth (Section 3.4,
Appendix "Inducing adapter").

TEST INFRASTRUCTURE ONLY (see oracle/model.py).

At each explored depth l in X \\ {L} a residual MLP maps the hidden state
h_l to h~_l = h_l + dh_l, which the shared final norm and LM head decode;
the final depth decodes h_L itself, and the backbone continues from h_l
(the adapter only changes which intermediate candidates are proposed).

Reading: the printed formula omits biases while the printed parameter count
includes two linear layers with biases, an RMSNorm scale and the scalar
gate, so
    dh = alpha * ( W2 silu( W1 RMSNorm(h; g) + b1 ) + b2 ),
W1 [m, h], b1 [m], W2 [h, m], b2 [h], g [h], alpha scalar, m = 2h, and
silu is the backbone's activation.
"""

from __future__ import annotations

import numpy as np

from .model import rmsnorm, silu

PARTS = ("norm", "w1", "b1", "w2", "b2", "alpha")


def delta(ad: dict, h: np.ndarray, eps: float) -> np.ndarray:
    """dh for one hidden state (or a batch over the leading axis)."""
    u = ad["w1"] @ rmsnorm(h, ad["norm"], eps) + ad["b1"]
    alpha = float(np.asarray(ad["alpha"], dtype=np.float64).reshape(-1)[0])
    return alpha * (ad["w2"] @ silu(u) + ad["b2"])


def param_count(h: int, m: int | None = None) -> int:
    """hm + mh + m + 2h + 1 (two biased linear layers, the norm scale and the
    gate); 4h^2 + 4h + 1 at the default m = 2h."""
    m = 2 * h if m is None else m
    return h * m + m * h + m + 2 * h + 1
