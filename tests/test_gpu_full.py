"""GPU: the 32-layer d4096 GQA workloads at full size, in the configuration
the benchmark times (prompt length, explored depths, width caps).

The batch-8 workload with 8192-token prompts is too large for the float64
oracle's prefill; it is checked through the properties alone.
Properties that hold at any size are checked exhaustively: DEX committed
tokens equal the same library's plain AR tokens bit for bit, the lattice
trace equals the oracle lattice driven by the GPU's candidates, and the
key/value collapse gather is bit-exact.  The float64 oracle re-scores a few
sampled positions of the GPU's sequence one by one (teacher-forced tokens and
per-depth exit logits).
"""
import numpy as np
import pytest

import oracle
from oracle import ar
from synth import configs, gen
from tests.gpu_common import LOGIT_RTOL, check_tokens_teacher_forced, max_rel_err, torch_cuda
from tests.test_gpu_decode import _replay, _run, _snapshot

pytestmark = pytest.mark.gpu

C3 = "llama-32L-d4096-x8-w4"
C4 = "llama-32L-d4096-x2-w16"
C5 = "llama-32L-d4096-x4-w8-b8-ctx8192"


@pytest.fixture(scope="module")
def llama():
    torch_cuda()
    from paper_2606_29223_amd import dexlib
    cfg = configs.get(C3)
    w = gen.generate_model(cfg)
    return cfg, w, dexlib.device_weights(cfg, w)


def _decoder(cfg, dev_w, **kw):
    from paper_2606_29223_amd import dexlib
    return dexlib.Decoder(cfg, dev_w, **kw)


@pytest.mark.parametrize("name,T", [(C3, 40), (C4, 24)])
def test_dex_equals_ar_full_size(llama, name, T):
    torch = torch_cuda()
    _, _, dev_w = llama
    cfg = configs.get(name)
    P = cfg["prompt_len"]
    prompt = gen.prompts(cfg)
    ar_dec = _decoder(cfg, dev_w, explored=[cfg["n_layers"]], width_cap=1, max_context=P + T)
    ar_toks, _ = _run(ar_dec, prompt, T, collapse=False)
    ar_dec.close()
    dec = _decoder(cfg, dev_w, max_context=P + T)
    toks, rounds = _run(dec, prompt, T)
    dec.close()
    assert np.array_equal(toks, ar_toks)
    _replay(rounds, len(cfg["explored"]), cfg["width_cap"], cfg["decs"], P + T, toks[0][0], P)
    assert max(len(rd["rows"]) for rd in rounds) <= cfg["width_cap"]
    torch.cuda.empty_cache()


def test_dex_equals_ar_batch8_ctx8192(llama):
    """Eight sequences with 8192-token prompts (explored depths 4..32 step 4,
    width 8): every sequence's DEX tokens equal its plain AR tokens bit for
    bit, and every sequence's lattice trace equals the oracle lattice's."""
    torch = torch_cuda()
    _, _, dev_w = llama
    cfg = configs.get(C5)
    P, T, B = cfg["prompt_len"], 12, cfg["batch"]
    prompt = gen.prompts(cfg)
    ar_dec = _decoder(cfg, dev_w, explored=[cfg["n_layers"]], width_cap=1, max_context=P + T)
    ar_toks, _ = _run(ar_dec, prompt, T, collapse=False)
    ar_dec.close()
    dec = _decoder(cfg, dev_w, max_context=P + T)
    toks, rounds = _run(dec, prompt, T)
    dec.close()
    assert toks.shape == (B, T)
    assert np.array_equal(toks, ar_toks)
    for b in range(B):
        _replay(rounds, len(cfg["explored"]), cfg["width_cap"], cfg["decs"], P + T, toks[b][0], P, seq=b)
    torch.cuda.empty_cache()


def test_kv_collapse_full_size(llama):
    torch = torch_cuda()
    cfg, _, dev_w = llama
    P = cfg["prompt_len"]
    dec = _decoder(cfg, dev_w, max_context=P + 24)
    dec.prefill(gen.prompts(cfg))
    checked = 0
    for _ in range(12):
        base = dec.slot_entry(0, 0)
        c = dec.step()
        if c[0] < 0:
            continue
        after_k, after_v = _snapshot(dec, torch)
        keep, fresh, cpos = dec.last_collapse(0)
        new_entries = [dec.slot_entry(0, j) for j in range(len(keep))]
        for ak in (after_k, after_v):
            assert np.array_equal(ak[:, 0, :, cpos, :], ak[:, 0, :, base, :])
            for j, old in enumerate(keep):
                assert np.array_equal(ak[:, 0, :, new_entries[j], :], ak[:, 0, :, base + old, :])
        checked += 1
        del after_k, after_v
    dec.close()
    assert checked >= 3


@pytest.mark.parametrize("name", [C3, C4])
def test_oracle_sampled_positions_full_size(llama, name):
    """The float64 oracle re-scores sampled positions of the GPU's sequence:
    the committed token is its argmax (or a near tie) and every explored
    depth's exit logits agree within 2e-2 (max relative) -- four depths at
    width 4, sixteen at width 16."""
    torch = torch_cuda()
    _, w, dev_w = llama
    cfg = configs.get(name)
    P = cfg["prompt_len"]
    T = 12
    prompt = gen.prompts(cfg)
    dec = _decoder(cfg, dev_w, max_context=P + T)
    tap = torch.empty((cfg["width_cap"], cfg["vocab"]), dtype=torch.float32, device="cuda")
    dec.set_logits_tap(tap)
    toks, rounds = _run(dec, prompt, T, tap=tap)
    dec.close()
    seq = [int(t) for t in toks[0]]
    m = oracle.Model(cfg, gen.model_as_f64(cfg, w))
    pl = [int(t) for t in prompt[0]]
    pf = m.prefill(pl)
    # sampled positions: the first three generated tokens after y_0
    n_pos = 3
    z = ar.depth_logits(m, pl, seq[: n_pos + 1], cfg["explored"], prefill=pf)   # [n_pos, N, V]
    check_tokens_teacher_forced(z[:, -1], seq[: n_pos + 1])
    worst, seen = 0.0, 0
    for rd in rounds:
        for r, (s, slot, stage, pos, tok) in enumerate(rd["rows"]):
            t = pos + 1 - P
            if slot == 0 and 1 <= t <= n_pos:
                worst = max(worst, max_rel_err(rd["logits"][r], z[t - 1, stage]))
                seen += 1
    assert seen >= n_pos
    assert worst <= LOGIT_RTOL, worst
