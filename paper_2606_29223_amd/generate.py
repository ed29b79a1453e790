"""Greedy (or sampled) DEX generation on a synthetic workload, through the
C ABI: prefill, then one dex_step per round until the requested number of
tokens, with the lattice statistics of the run and, optionally, the same
library's plain AR decoding (X = {L}, width 1) to show the tokens agree.

    python3 -m paper_2606_29223_amd.generate --config NAME --tokens T [--ar] [--temperature TAU]
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time


def main():
    ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    if ROOT not in sys.path:
        sys.path.insert(0, ROOT)
    from synth import configs, gen

    ap = argparse.ArgumentParser()
    ap.add_argument("--config", default=configs.SMALLEST)
    ap.add_argument("--tokens", type=int, default=32)
    ap.add_argument("--explored", default=None, help="comma-separated explored depths (default: the workload's)")
    ap.add_argument("--width-cap", type=int, default=None)
    ap.add_argument("--temperature", type=float, default=0.0)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--ar", action="store_true", help="also decode with X = {L} and compare")
    args = ap.parse_args()

    import torch

    from paper_2606_29223_amd import dexlib

    cfg = configs.get(args.config)
    dev_w = dexlib.device_weights(cfg, gen.generate_model(cfg))
    prompts = gen.prompts(cfg)
    X = [int(x) for x in args.explored.split(",")] if args.explored else None
    max_ctx = cfg["prompt_len"] + args.tokens
    samp = dict(temperature=args.temperature, seed=args.seed)
    dec = dexlib.Decoder(cfg, dev_w, explored=X, width_cap=args.width_cap, max_context=max_ctx, **samp)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    toks, st = dec.generate(prompts, args.tokens)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    L, N = cfg["n_layers"], dec.N
    commits = len(st["kstar"])
    out = {"workload": cfg["name"], "explored": dec.explored, "tokens": toks,
           "rounds": st["rounds"], "commits": commits, "seconds": round(dt, 4),
           "rounds_per_commit": round(st["rounds"] / max(commits, 1), 4),
           "critical_path_layers_per_commit": round(L / N * st["rounds"] / max(commits, 1), 3),
           "weight_layers_per_commit": round(st["layers_streamed"] / max(commits, 1), 3),
           "matched_depth_hist": {str(k): st["kstar"].count(k) for k in sorted(set(st["kstar"]))}}
    dec.close()
    if args.ar:
        ar = dexlib.Decoder(cfg, dev_w, explored=[L], width_cap=1, max_context=max_ctx, **samp)
        ar_toks, _ = ar.generate(prompts, args.tokens)
        ar.close()
        out["equals_ar"] = ar_toks == toks
    print(json.dumps(out))


if __name__ == "__main__":
    main()
