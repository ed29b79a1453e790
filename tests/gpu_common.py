"""Shared helpers for the GPU tests: weights on the device, contexts, and the
two comparison rules against the oracle (teacher-forced tokens with a top-2
gap exemption; per-row max relative logit error)."""
from __future__ import annotations

import functools

import numpy as np

from synth import configs, gen

GAP = 1e-2          # tokens may differ from the oracle only where its top-2 gap is below this
LOGIT_RTOL = 2e-2   # max_v |z_gpu - z_oracle| / max_v |z_oracle| per row


def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        import pytest
        pytest.skip("no GPU")
    return torch


@functools.lru_cache(maxsize=4)
def host_weights(name: str, **over):
    cfg = configs.get(name, **over)
    return cfg, gen.generate_model(cfg)


@functools.lru_cache(maxsize=2)
def device_weights(name: str):
    torch_cuda()
    from paper_2606_29223_amd import dexlib
    cfg, w = host_weights(name)
    return dexlib.device_weights(cfg, w)


def decoder(name: str, **kw):
    torch_cuda()
    from paper_2606_29223_amd import dexlib
    cfg, _ = host_weights(name)
    return dexlib.Decoder(cfg, device_weights(name), **kw)


def run(dec, prompts, T):
    """Prefill then step until every sequence has T generated tokens.  Returns
    (tokens [B][T], per-round infos as dicts)."""
    B = dec.batch
    first = dec.prefill(prompts)
    toks = [[int(first[b])] for b in range(B)]
    rounds = []
    while min(len(t) for t in toks) < T:
        c = dec.step()
        inf = dec.info
        rows = [(inf.row_seq[r], inf.row_slot[r], inf.row_stage[r], inf.row_pos[r], inf.row_token[r])
                for r in range(inf.n_rows)]
        rounds.append(dict(rows=rows, kstar=[inf.kstar[b] for b in range(B)],
                           committed=[int(x) for x in c], q=[inf.q[b] for b in range(B)],
                           layers=inf.layers_streamed, per_stage=list(inf.rows_per_stage[: dec.N])))
        for b in range(B):
            if c[b] >= 0 and len(toks[b]) < T:
                toks[b].append(int(c[b]))
    return np.array(toks), rounds


def check_tokens_teacher_forced(z_oracle_final: np.ndarray, gpu_tokens) -> list:
    """z_oracle_final [T-1, V]: oracle final-depth logits re-scoring the GPU's
    own prefix.  Returns the list of positions where the GPU token is not the
    oracle argmax (each must be a near tie)."""
    flips = []
    for t in range(1, len(gpu_tokens)):
        z = z_oracle_final[t - 1]
        y = int(gpu_tokens[t])
        best = int(np.argmax(z))
        if y != best:
            srt = np.sort(z)
            gap = srt[-1] - srt[-2]
            assert gap < GAP and z[best] - z[y] < GAP, (t, y, best, gap)
            flips.append(t)
    return flips


def max_rel_err(z_gpu: np.ndarray, z_ref: np.ndarray) -> float:
    return float(np.max(np.abs(z_gpu - z_ref)) / np.max(np.abs(z_ref)))
