"""The GPU tests' node oracle (tests/gpu_common.NodeOracle) against plain
teacher-forced decoding: a lattice node's exit logits are those of ordinary
decoding of its own token prefix, at every depth, whatever order the
prefixes are asked for in."""
import numpy as np

import oracle
from oracle import ar
from synth import configs, gen
from tests.gpu_common import NodeOracle, node_key


def test_node_oracle_equals_teacher_forced_decoding():
    cfg = configs.get("tiny-4L-d128-fp32")
    w = gen.generate_model(cfg)
    m = oracle.Model(cfg, gen.model_as_f64(cfg, w))
    prompt = [int(t) for t in gen.prompts(cfg)[0]]
    P = len(prompt)
    pf = m.prefill(prompt)
    no = NodeOracle(m, P, pf)
    rng = np.random.default_rng(5)
    base = [int(t) for t in rng.integers(0, cfg["vocab"], size=6)]
    # branches sharing the first tokens, asked deep-first and shallow-first
    keys = [tuple(base), tuple(base[:3]), tuple(base[:3] + [7, 9]), tuple(base[:1]), tuple(base[:4] + [11])]
    for key in keys:
        seq = list(key) + [0]                         # depth_logits scores positions of seq[:-1]
        z = ar.depth_logits(m, prompt, seq, [1, 2, 3, 4], prefill=pf)[-1]
        for j, d in enumerate([1, 2, 3, 4]):
            got = no.logits(key, d)
            assert np.allclose(got, z[j], rtol=1e-12, atol=1e-12), (key, d)


def test_node_key_follows_the_slot_chain():
    from oracle.lattice import Lattice
    P = 10
    lat = Lattice(4, 0, True, 100, 50, P + 2)        # anchor at position P + 2 with input 50
    lat.anchor.u = [60, 61]
    lat.anchor.c = 2
    rows = lat.begin_round()
    child = [r.slot for r in rows if r.new and r.slot.fork_stage == 1][0]
    generated = [40, 41, 50, 999]
    assert node_key(generated, lat.anchor, P) == (40, 41, 50)
    assert node_key(generated, child, P) == (40, 41, 50, 61)
