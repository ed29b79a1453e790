"""GPU: the DEX decode step through the C ABI against the oracle.

  * DEX committed tokens are bit-identical to the GPU's own plain
    autoregressive path (same library, X = {L}, width 1);
  * tokens equal the oracle's greedy AR except where the oracle's top-2 gap
    is below 1e-2 (teacher-forced: the oracle re-scores the GPU's prefix);
  * every anchor row's exit logits (before the DECS mask) are within max
    relative error 2e-2 of the oracle's at that depth and position;
  * the lattice trace -- rows per round, commits, match depths, collapse
    maps and slot tables -- equals the oracle lattice's on the same
    candidate tokens, and (fp32 model) the oracle's own full DEX trace;
  * the key/value collapse gather is bit-exact.
"""
import numpy as np
import pytest

import oracle
from oracle import ar, dex
from oracle.lattice import Lattice
from synth import configs, gen
from tests.gpu_common import (GAP, LOGIT_RTOL, NodeOracle, check_tokens_teacher_forced, decoder, device_weights,
                              host_weights, max_rel_err, node_key, torch_cuda)

pytestmark = pytest.mark.gpu

TINY = "tiny-4L-d128-fp32"
SMALL = "small-12L-d768-bf16"


def _run(dec, prompts, T, tap=None, collapse=True):
    torch = torch_cuda()
    B = dec.batch
    first = dec.prefill(prompts)
    toks = [[int(first[b])] for b in range(B)]
    rounds = []
    while min(len(t) for t in toks) < T:
        c = dec.step()
        inf = dec.info
        rows = [(inf.row_seq[r], inf.row_slot[r], inf.row_stage[r], inf.row_pos[r], inf.row_token[r])
                for r in range(inf.n_rows)]
        rd = dict(rows=rows, kstar=[inf.kstar[b] for b in range(B)], committed=[int(x) for x in c],
                  layers=inf.layers_streamed)
        if tap is not None:
            torch.cuda.synchronize()
            rd["logits"] = tap[: inf.n_rows].cpu().numpy().copy()
        if collapse:
            rd["collapse"] = [dec.last_collapse(b) if c[b] >= 0 else None for b in range(B)]
            rd["lattice"] = [dec.lattice(b) for b in range(B)]
        rounds.append(rd)
        for b in range(B):
            if c[b] >= 0 and len(toks[b]) < T:
                toks[b].append(int(c[b]))
    return np.array(toks), rounds


def _replay(rounds, N, W, decs, max_ctx, y0, P, seq=0, on_row=None):
    """Feed the GPU's candidate tokens to the oracle lattice; every planning
    and collapse decision must agree.  on_row(round, gpu_row_index,
    oracle_row) is called for each of the sequence's rows before the round's
    candidates are inserted (the oracle row's slot chain is then the node's)."""
    lat = Lattice(N, W, bool(decs), max_ctx, int(y0), P)
    for i, rd in enumerate(rounds):
        if not any(r[0] == seq for r in rd["rows"]):
            break
        rows = lat.begin_round()
        orc = [(lat.index(r.slot), r.stage, r.slot.pos) for r in rows]
        order = sorted(range(len(orc)), key=lambda j: orc[j][1])
        gpu = [(r[1], r[2], r[3], r[4]) for r in rd["rows"] if r[0] == seq]
        assert [orc[j] for j in order] == [g[:3] for g in gpu], f"round {i}"
        if on_row is not None:
            gidx = [r for r, row in enumerate(rd["rows"]) if row[0] == seq]
            for k, j in enumerate(order):
                on_row(i, gidx[k], rows[j])
        toks = [0] * len(rows)
        for k, j in enumerate(order):
            toks[j] = gpu[k][3]
        cm = lat.end_round(rows, toks)
        assert (cm is not None) == (rd["kstar"][seq] >= 0), f"round {i}"
        if cm is not None:
            assert cm.kstar == rd["kstar"][seq] and cm.token == rd["committed"][seq]
            gmap, gfresh, gpos = rd["collapse"][seq]
            assert list(cm.collapse_map) == list(gmap) and int(cm.fresh_anchor) == gfresh
            assert gpos == cm.old_anchor.pos
        tab = rd["lattice"][seq]
        assert len(tab) == len(lat.slots)
        for j, s in enumerate(lat.slots):
            par = lat.index(s.parent) if s.parent is not None else -1
            row = [s.x, s.pos, par, s.fork_stage, s.c] + (s.u + [-1] * (N - len(s.u)))
            assert list(tab[j]) == row, f"round {i} slot {j}"
    return lat


@pytest.fixture(scope="module")
def tiny_oracle():
    cfg, w = host_weights(TINY)
    m = oracle.Model(cfg, gen.model_as_f64(cfg, w))
    prompt = [int(t) for t in gen.prompts(cfg)[0]]
    pf = m.prefill(prompt)
    return cfg, m, prompt, pf


def test_tiny_dex_equals_ar_and_oracle(tiny_oracle):
    torch = torch_cuda()
    cfg, m, prompt, pf = tiny_oracle
    T = cfg["gen_len"]
    P = len(prompt)
    ar_dec = decoder(TINY, explored=[cfg["n_layers"]], width_cap=1)
    ar_toks, ar_rounds = _run(ar_dec, [prompt], T, collapse=False)
    ar_dec.close()
    dec = decoder(TINY)
    tap = torch.empty((dec.batch * 8, cfg["vocab"]), dtype=torch.float32, device="cuda")
    dec.set_logits_tap(tap)
    toks, rounds = _run(dec, [prompt], T, tap=tap)
    dec.close()
    assert np.array_equal(toks, ar_toks)
    assert all(len(r["rows"]) == 1 for r in ar_rounds)
    # oracle: teacher-forced final-depth logits and exit logits on the GPU's prefix
    seq = [int(t) for t in toks[0]]
    X = cfg["explored"]
    z = ar.depth_logits(m, prompt, seq, X, prefill=pf)
    check_tokens_teacher_forced(z[:, -1], seq)
    assert seq == ar.ar_generate(m, prompt, T, prefill=pf)
    worst = 0.0
    for rd in rounds:
        for r, (s, slot, stage, pos, tok) in enumerate(rd["rows"]):
            if slot != 0:
                continue
            t = pos + 1 - P
            worst = max(worst, max_rel_err(rd["logits"][r], z[t - 1, stage]))
    assert worst <= LOGIT_RTOL
    assert worst < 1e-4          # fp32 model: agreement at float32 level
    # trace: the oracle lattice on the GPU's tokens, then the oracle's own run
    _replay(rounds, len(X), cfg["width_cap"], cfg["decs"], P + T, seq[0], P)
    res = dex.dex_generate(m, prompt, X, cfg["width_cap"], True, T, prefill=pf)
    assert res.tokens == seq
    assert res.rounds == len(rounds)
    for tr, rd in zip(res.trace, rounds):
        orc = sorted([(a[1], a[0], a[2], tk) for a, tk in zip(tr.rows, tr.tokens)], key=lambda v: v[0])
        gpu = [(st, sl, p, tk) for (_, sl, st, p, tk) in rd["rows"]]
        assert orc == gpu
        if tr.commit is not None:
            assert tr.commit[1] == rd["kstar"][0] and tr.commit[2] == list(rd["collapse"][0][0])


@pytest.mark.parametrize("X,W,decs", [([1, 2, 3, 4], 0, 0), ([1, 2, 3, 4], 3, 1), ([2, 4], 0, 1),
                                      ([1, 3, 4], 2, 0)])
def test_tiny_variants_lossless_and_trace(tiny_oracle, X, W, decs):
    cfg, m, prompt, pf = tiny_oracle
    T = 40
    P = len(prompt)
    ar_dec = decoder(TINY, explored=[4], width_cap=1, max_context=P + T)
    ar_toks, _ = _run(ar_dec, [prompt], T, collapse=False)
    ar_dec.close()
    dec = decoder(TINY, explored=X, width_cap=W, decs=decs, max_context=P + T)
    toks, rounds = _run(dec, [prompt], T)
    dec.close()
    assert np.array_equal(toks, ar_toks)
    _replay(rounds, len(X), W, decs, P + T, toks[0][0], P)
    res = dex.dex_generate(m, prompt, X, W, bool(decs), T, prefill=pf, keep_trace=False)
    assert res.tokens == [int(t) for t in toks[0]] and res.rounds == len(rounds)


def test_tiny_batch_of_lattices_matches_single():
    cfg = configs.get(TINY)
    prompts = np.stack([gen.tokens(gen.mix64(s), cfg["prompt_len"], cfg["vocab"]) for s in (11, 12, 13)])
    T = 24
    dec = decoder(TINY, batch=3, max_context=cfg["prompt_len"] + T)
    toks, rounds = _run(dec, prompts, T)
    dec.close()
    for b in range(3):
        one = decoder(TINY, batch=1, max_context=cfg["prompt_len"] + T)
        t1, r1 = _run(one, prompts[b:b + 1], T)
        one.close()
        assert np.array_equal(toks[b], t1[0])
        _replay(rounds, 4, 0, 1, cfg["prompt_len"] + T, toks[b][0], cfg["prompt_len"], seq=b)


def _snapshot(dec, torch):
    from paper_2606_29223_amd import dexlib
    k, v, E = dec.kv_layout()
    cfg = dec.cfg
    es = 2 if cfg["dtype"] == "bf16" else 4
    nbytes = cfg["n_layers"] * dec.batch * cfg["n_kv_heads"] * E * cfg["head_dim"] * es
    out = []
    for base in (k, v):
        buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        assert dexlib.load().dex_debug_copy(buf.data_ptr(), base, nbytes, dec.stream.cuda_stream) == 0
        torch.cuda.synchronize()
        out.append(buf.cpu().numpy().view(np.uint16 if es == 2 else np.uint32).reshape(
            cfg["n_layers"], dec.batch, cfg["n_kv_heads"], E, cfg["head_dim"]))
    return out


@pytest.mark.parametrize("name", [TINY, SMALL])
def test_kv_collapse_gather_bitexact(name):
    torch = torch_cuda()
    cfg, _ = host_weights(name)
    P = 24
    prompt = gen.prompts(cfg)[:, :P]
    dec = decoder(name, max_context=P + 40)
    dec.prefill(prompt)
    checked = 0
    for _ in range(30):
        before_k, before_v = _snapshot(dec, torch)
        base = dec.slot_entry(0, 0)       # slot j of the current half lives at base + j
        c = dec.step()
        after_k, after_v = _snapshot(dec, torch)
        if c[0] < 0:
            continue
        keep, fresh, cpos = dec.last_collapse(0)
        new_entries = [dec.slot_entry(0, j) for j in range(len(keep))]
        # the anchor's keys/values (entry of slot 0 before the step, as written
        # during the step) land on committed position cpos
        anchor_e = base
        for (bk, ak) in ((before_k, after_k), (before_v, after_v)):
            assert np.array_equal(ak[:, 0, :, cpos, :], ak[:, 0, :, anchor_e, :])
            assert np.array_equal(ak[:, 0, :, :cpos, :], bk[:, 0, :, :cpos, :])   # older positions untouched
            for j, old in enumerate(keep):
                assert np.array_equal(ak[:, 0, :, new_entries[j], :], ak[:, 0, :, base + old, :])
        checked += 1
    dec.close()
    assert checked >= 5


def test_small_bf16_lossless_and_oracle():
    torch = torch_cuda()
    cfg, w = host_weights(SMALL)
    P = cfg["prompt_len"]
    T = 48
    prompt = gen.prompts(cfg)
    ar_dec = decoder(SMALL, explored=[cfg["n_layers"]], width_cap=1, max_context=P + T)
    ar_toks, _ = _run(ar_dec, prompt, T, collapse=False)
    ar_dec.close()
    dec = decoder(SMALL, max_context=P + T)
    tap = torch.empty((4, cfg["vocab"]), dtype=torch.float32, device="cuda")
    dec.set_logits_tap(tap)
    toks, rounds = _run(dec, prompt, T, tap=tap)
    dec.close()
    assert np.array_equal(toks, ar_toks)
    _replay(rounds, 4, cfg["width_cap"], 1, P + T, toks[0][0], P)
    m = oracle.Model(cfg, gen.model_as_f64(cfg, w))
    seq = [int(t) for t in toks[0]]
    pl = [int(t) for t in prompt[0]]
    pf = m.prefill(pl)
    z = ar.depth_logits(m, pl, seq, cfg["explored"], prefill=pf)
    flips = check_tokens_teacher_forced(z[:, -1], seq)
    assert len(flips) <= 2
    worst = 0.0
    for rd in rounds:
        for r, (s, slot, stage, pos, tok) in enumerate(rd["rows"]):
            if slot == 0:
                worst = max(worst, max_rel_err(rd["logits"][r], z[pos - P, stage]))
    assert worst <= LOGIT_RTOL, worst


def test_small_bf16_every_row_logits():
    """Every row of every round -- speculative nodes included, whose
    attention reads their ancestor slots' keys/values -- against the float64
    oracle recomputing that node from its own prefix (committed tokens, then
    the inputs of its slot chain) at its stage's depth: max relative error of
    the exit logits (before the DECS mask) within 2e-2 (12-layer bf16 model,
    explored depths {3,6,9,12}, width 4, 48 tokens)."""
    torch = torch_cuda()
    cfg, w = host_weights(SMALL)
    P, T = cfg["prompt_len"], 48
    prompt = gen.prompts(cfg)
    dec = decoder(SMALL, max_context=P + T)
    tap = torch.empty((cfg["width_cap"], cfg["vocab"]), dtype=torch.float32, device="cuda")
    dec.set_logits_tap(tap)
    toks, rounds = _run(dec, prompt, T, tap=tap)
    dec.close()
    m = oracle.Model(cfg, gen.model_as_f64(cfg, w))
    pl = [int(t) for t in prompt[0]]
    no = NodeOracle(m, P, m.prefill(pl))
    seq = [int(t) for t in toks[0]]
    X = cfg["explored"]
    stats = {"worst": 0.0, "rows": 0, "speculative": 0}

    def on_row(i, r, orow):
        key = node_key(seq, orow.slot, P)
        z = no.logits(key, X[orow.stage])
        stats["worst"] = max(stats["worst"], max_rel_err(rounds[i]["logits"][r], z))
        stats["rows"] += 1
        stats["speculative"] += orow.slot.parent is not None

    _replay(rounds, len(X), cfg["width_cap"], cfg["decs"], P + T, seq[0], P, on_row=on_row)
    assert stats["rows"] == sum(len(rd["rows"]) for rd in rounds)
    assert stats["speculative"] >= 40, stats
    assert stats["worst"] <= LOGIT_RTOL, stats


@pytest.mark.parametrize("X,W,decs", [([2, 4, 6, 8, 10, 12], 8, 1), ([6, 12], 2, 1), ([3, 6, 9, 12], 4, 0),
                                      ([1, 12], 0, 1), ([4, 8, 12], 16, 1)])
def test_small_bf16_explored_sets(X, W, decs):
    """Other explored sets, width caps and vanilla mode on the 12-layer bf16
    model (batch 2): DEX equals plain AR bit for bit and every round's plan,
    commit and collapse equals the oracle lattice's on the GPU's candidates."""
    torch_cuda()
    cfg = configs.get(SMALL)
    P, T = 64, 32
    prompts = np.stack([gen.tokens(gen.mix64(s), P, cfg["vocab"]) for s in (7101, 7102)])
    ar_dec = decoder(SMALL, explored=[cfg["n_layers"]], width_cap=1, batch=2, max_context=P + T)
    ar_toks, _ = _run(ar_dec, prompts, T, collapse=False)
    ar_dec.close()
    dec = decoder(SMALL, explored=X, width_cap=W, decs=decs, batch=2, max_context=P + T)
    toks, rounds = _run(dec, prompts, T)
    dec.close()
    assert np.array_equal(toks, ar_toks)
    for b in range(2):
        _replay(rounds, len(X), W, decs, P + T, toks[b][0], P, seq=b)


def test_small_bf16_lossless_over_seeds():
    """Losslessness over more seeded prompts: six prompt sets of three
    sequences (prompt lengths 24 to 109), each decoded by DEX under one of
    three explored-set / width-cap / DECS settings (two sets each), equal
    plain AR token for token."""
    torch_cuda()
    cfg = configs.get(SMALL)
    T = 40
    cases = [([3, 6, 9, 12], 4, 1), ([2, 5, 8, 12], 3, 1), ([4, 12], 0, 0)]
    for seed in range(6):
        P = 24 + 17 * seed
        prompts = np.stack([gen.tokens(gen.mix64(9000 + 10 * seed + b), P, cfg["vocab"]) for b in range(3)])
        ar_dec = decoder(SMALL, explored=[cfg["n_layers"]], width_cap=1, batch=3, max_context=P + T)
        ar_toks, _ = _run(ar_dec, prompts, T, collapse=False)
        ar_dec.close()
        X, W, decs = cases[seed % len(cases)]
        dec = decoder(SMALL, explored=X, width_cap=W, decs=decs, batch=3, max_context=P + T)
        toks, _ = _run(dec, prompts, T, collapse=False)
        dec.close()
        assert np.array_equal(toks, ar_toks), (seed, X, W, decs)


@pytest.mark.parametrize("P", [1, 45, 97])
def test_small_bf16_prefill_ragged_prompts(P):
    """Prompt lengths that are not a multiple of the 32-query / 64-key tiles
    of the matrix-core prompt attention (and the one-token prompt), at batch
    2: y_0 and the next tokens follow the float64 oracle (near ties aside) and
    the exit logits of every decoded row agree within 2e-2 (max relative)."""
    torch = torch_cuda()
    from paper_2606_29223_amd import dexlib
    cfg = configs.get(SMALL, prompt_len=P, batch=2, prompt_seeds=[7001, 7002])
    _, w = host_weights(SMALL)
    T = 5
    dec = dexlib.Decoder(cfg, device_weights(SMALL), explored=[cfg["n_layers"]], width_cap=1,
                         max_context=P + T)
    tap = torch.empty((8, cfg["vocab"]), dtype=torch.float32, device="cuda")
    dec.set_logits_tap(tap)
    prompt = gen.prompts(cfg)
    toks, rounds = _run(dec, prompt, T, tap=tap, collapse=False)
    dec.close()
    m = oracle.Model(cfg, gen.model_as_f64(cfg, w))
    for b in range(2):
        pl = [int(t) for t in prompt[b]]
        seq = [int(t) for t in toks[b]]
        pf = m.prefill(pl)
        z0 = m.exit_logits(pf[2])
        if seq[0] != int(np.argmax(z0)):
            srt = np.sort(z0)
            assert srt[-1] - srt[-2] < GAP and z0.max() - z0[seq[0]] < GAP
        z = ar.depth_logits(m, pl, seq, [cfg["n_layers"]], prefill=pf)
        check_tokens_teacher_forced(z[:, -1], seq)
        seen = 0
        for rd in rounds:
            for r, (s, slot, stage, pos, tok) in enumerate(rd["rows"]):
                if s == b and pos - P < len(seq) - 1:
                    assert max_rel_err(rd["logits"][r], z[pos - P, 0]) <= LOGIT_RTOL
                    seen += 1
        assert seen == T - 1


def test_large_prompt_batch_prefill_matches_batch_one():
    """Two 1100-token prompts make 2200 prompt rows, so the gate/up prompt
    GEMM gets 144 256 x 256 workgroups and runs on the LDS-staged kernel;
    one prompt alone (80 such workgroups) runs the 128 x 128 kernel.  Both
    feed the MFMA tiles the same operands in the same k-step order and share
    the epilogues (RoPE and cache write, residual and norm partials, SwiGLU),
    so sequence 0's prompt keys/values, y_0 and the next tokens are the same
    bits either way."""
    torch = torch_cuda()
    from paper_2606_29223_amd import dexlib
    P, T = 1100, 4
    cfg2 = configs.get(SMALL, prompt_len=P, batch=2, prompt_seeds=[7101, 7102])
    cfg1 = configs.get(SMALL, prompt_len=P, batch=1, prompt_seeds=[7101])
    prompt = gen.prompts(cfg2)
    assert np.array_equal(gen.prompts(cfg1)[0], prompt[0])
    res = []
    for cfg, pr in ((cfg2, prompt), (cfg1, prompt[:1])):
        dec = dexlib.Decoder(cfg, device_weights(SMALL), max_context=P + T)
        first = dec.prefill(pr)
        k, v = _snapshot(dec, torch)
        kv = (k[:, 0, :, :P, :].copy(), v[:, 0, :, :P, :].copy())
        toks = [int(first[0])]
        while len(toks) < T:
            c = dec.step()
            if c[0] >= 0:
                toks.append(int(c[0]))
        dec.close()
        res.append((kv, toks))
    (kv2, t2), (kv1, t1) = res
    assert np.array_equal(kv2[0], kv1[0]) and np.array_equal(kv2[1], kv1[1])
    assert t2 == t1


@pytest.mark.parametrize("P,G", [(1, 4), (45, 4), (97, 4), (300, 4), (3100, 4), (97, 1), (300, 2), (45, 8),
                                 (300, 8)])
def test_gqa128_prefill_ragged_prompts(P, G):
    """The 32-layer model's attention shape (head_dim 128, four query heads
    per kv head; also one, two and eight) on a 2-layer model small enough for
    the float64 oracle, with prompt lengths that are not multiples of the
    32-query / 64-key blocks of the prompt attention (and the one-token
    prompt), at batch 2: y_0 and the
    next tokens follow the oracle (near ties aside) and every decoded row's
    exit logits agree within 2e-2 (max relative).  At 2 x 3100 prompt rows
    all four prompt GEMMs (QKV with RoPE and the cache write, O and down with
    the residual, gate/up with SwiGLU) take the 256 x 256 LDS-staged form
    (150, 100, 400 and 100 workgroups)."""
    torch = torch_cuda()
    from paper_2606_29223_amd import dexlib
    cfg = configs.scaled_down(configs.get("llama-32L-d4096-x8-w4"), n_layers=2, d_model=1024, d_ffn=2048,
                              vocab=4096)
    cfg.update(n_heads=2 * G, n_kv_heads=2, head_dim=128, prompt_len=P, batch=2, prompt_seeds=[7201, 7202])
    w = gen.generate_model(cfg)
    T = 5
    dec = dexlib.Decoder(cfg, dexlib.device_weights(cfg, w), explored=[cfg["n_layers"]], width_cap=1,
                         max_context=P + T)
    tap = torch.empty((8, cfg["vocab"]), dtype=torch.float32, device="cuda")
    dec.set_logits_tap(tap)
    prompt = gen.prompts(cfg)
    toks, rounds = _run(dec, prompt, T, tap=tap, collapse=False)
    dec.close()
    m = oracle.Model(cfg, gen.model_as_f64(cfg, w))
    for b in range(2):
        pl = [int(t) for t in prompt[b]]
        seq = [int(t) for t in toks[b]]
        pf = m.prefill(pl)
        z0 = m.exit_logits(pf[2])
        if seq[0] != int(np.argmax(z0)):
            srt = np.sort(z0)
            assert srt[-1] - srt[-2] < GAP and z0.max() - z0[seq[0]] < GAP
        z = ar.depth_logits(m, pl, seq, [cfg["n_layers"]], prefill=pf)
        check_tokens_teacher_forced(z[:, -1], seq)
        seen = 0
        for rd in rounds:
            for r, (s, slot, stage, pos, tok) in enumerate(rd["rows"]):
                if s == b and pos - P < len(seq) - 1:
                    assert max_rel_err(rd["logits"][r], z[pos - P, 0]) <= LOGIT_RTOL
                    seen += 1
        assert seen == T - 1


@pytest.mark.parametrize("name", [SMALL, TINY])
def test_stage_schedules_do_not_change_results(name):
    """Grouped launches (a lane's stages in step, each kernel launched once
    per layer step for all of them) on one lane and on three, and per-stage
    launches on one stream and spread over four, change only the schedule:
    tokens, lattice traces and every row's exit logits are the same bits
    (batch 3; the bf16 model takes the grouped matrix-core attention, the
    fp32 model one attention launch per stage inside the grouped sweep)."""
    torch = torch_cuda()
    from paper_2606_29223_amd import dexlib
    cfg = configs.get(name, batch=3, prompt_seeds=[8101, 8102, 8103])
    prompt = gen.prompts(cfg)
    T = 24
    W = cfg["width_cap"] or 2 ** (len(cfg["explored"]) - 1)
    out = []
    for grouping, lanes in ((0, 1), (0, 3), (-1, 1), (-1, 4)):
        dec = dexlib.Decoder(cfg, device_weights(name), max_context=cfg["prompt_len"] + T, stage_streams=lanes,
                             stage_grouping=grouping)
        tap = torch.empty((dec.batch * W, cfg["vocab"]), dtype=torch.float32, device="cuda")
        dec.set_logits_tap(tap)
        out.append(_run(dec, prompt, T, tap=tap))
        dec.close()
    t0, r0 = out[0]
    for t1, r1 in out[1:]:
        assert np.array_equal(t0, t1)
        assert len(r0) == len(r1)
        for a, b in zip(r0, r1):
            assert a["rows"] == b["rows"] and a["kstar"] == b["kstar"] and a["collapse"] == b["collapse"]
            assert all(np.array_equal(x, y) for x, y in zip(a["lattice"], b["lattice"]))
            assert np.array_equal(a["logits"].view(np.uint32), b["logits"].view(np.uint32))


def test_grouped_lane_longer_than_one_launch():
    """Every layer of the 12-layer model explored (12 stages, width 16,
    batch 2) on one grouped lane: a layer step's segment list outgrows what
    one launch takes and goes out as several launches.  Tokens, lattice
    traces and every exit logit equal per-stage launches bit for bit, and
    the committed tokens equal plain AR's."""
    torch = torch_cuda()
    from paper_2606_29223_amd import dexlib
    cfg = configs.get(SMALL, batch=2, explored=list(range(1, 13)), width_cap=16, prompt_seeds=[8201, 8202])
    prompt = gen.prompts(cfg)
    T = 20
    out, most = [], 0
    for grouping in (0, -1):
        dec = dexlib.Decoder(cfg, device_weights(SMALL), max_context=cfg["prompt_len"] + T, stage_streams=1,
                             stage_grouping=grouping)
        tap = torch.empty((dec.batch * 16, cfg["vocab"]), dtype=torch.float32, device="cuda")
        dec.set_logits_tap(tap)
        toks, rounds = _run(dec, prompt, T, tap=tap)
        dec.close()
        out.append((toks, rounds))
        most = max(most, max(len({r[2] for r in rd["rows"]}) for rd in rounds))
    assert most > 8                     # some round ran more stages than one launch takes
    (t0, r0), (t1, r1) = out
    assert np.array_equal(t0, t1) and len(r0) == len(r1)
    for a, b in zip(r0, r1):
        assert a["rows"] == b["rows"] and a["kstar"] == b["kstar"]
        assert np.array_equal(a["logits"].view(np.uint32), b["logits"].view(np.uint32))
    ar = dexlib.Decoder(cfg, device_weights(SMALL), explored=[cfg["n_layers"]], width_cap=1,
                        max_context=cfg["prompt_len"] + T)
    ar_toks, _ = _run(ar, prompt, T, collapse=False)
    ar.close()
    assert np.array_equal(t0, ar_toks)


def test_small_bf16_long_context_merged_blocks():
    """A 2600-token prompt (41 key splits, several beyond one wave's reach of
    64 rows' groups): DEX still equals plain AR bit for bit, and the tokens
    and exit logits follow the float64 oracle at long context."""
    torch = torch_cuda()
    from paper_2606_29223_amd import dexlib
    cfg = configs.get(SMALL, prompt_len=2600, prompt_seeds=[9001])
    _, w = host_weights(SMALL)
    P, T = cfg["prompt_len"], 16
    prompt = gen.prompts(cfg)
    dev = device_weights(SMALL)
    ar_dec = dexlib.Decoder(cfg, dev, explored=[cfg["n_layers"]], width_cap=1, max_context=P + T)
    ar_toks, _ = _run(ar_dec, prompt, T, collapse=False)
    ar_dec.close()
    dec = dexlib.Decoder(cfg, dev, max_context=P + T)
    tap = torch.empty((8, cfg["vocab"]), dtype=torch.float32, device="cuda")
    dec.set_logits_tap(tap)
    toks, rounds = _run(dec, prompt, T, tap=tap)
    dec.close()
    assert np.array_equal(toks, ar_toks)
    _replay(rounds, len(cfg["explored"]), cfg["width_cap"], cfg["decs"], P + T, toks[0][0], P)
    m = oracle.Model(cfg, gen.model_as_f64(cfg, w))
    pl = [int(t) for t in prompt[0]]
    pf = m.prefill(pl)
    seq = [int(t) for t in toks[0]]
    z = ar.depth_logits(m, pl, seq, cfg["explored"], prefill=pf)
    check_tokens_teacher_forced(z[:, -1], seq)
    worst, seen = 0.0, 0
    for rd in rounds:
        for r, (s, slot, stage, pos, tok) in enumerate(rd["rows"]):
            if slot == 0 and pos - P < len(seq) - 1:
                worst = max(worst, max_rel_err(rd["logits"][r], z[pos - P, stage]))
                seen += 1
    assert seen >= T
    assert worst <= LOGIT_RTOL, worst
