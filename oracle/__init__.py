"""Plain CPU oracle of Depth Exploration Decoding (float64 numpy).

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the GPU library; both read the same seeded inputs from synth/.

Modules: model (the synthetic decoder and exit heads), ar (AR decoding and
teacher-forced exit logits), lattice (Algorithm 1 / Section 3.2 bookkeeping
with Algorithm 2's masks), dex (the full procedure on the model), gumbel
(Algorithm 2's sampling-mode noise and decode rule), adapter (the inducing
adapter of non-final depths), ead (Section 2's accounting, used as test
pins).
"""
from . import adapter, ar, dex, ead, gumbel, lattice, model  # noqa: F401
from .model import Model  # noqa: F401


def load(cfg, weights=None):
    """Build the oracle model for a workload config (weights from synth)."""
    from synth import gen
    if weights is None:
        weights = gen.generate_model(cfg)
    return Model(cfg, gen.model_as_f64(cfg, weights))
