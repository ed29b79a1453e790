"""Launch sequence for hardware traffic counters (run under rocprofv3 --pmc).

Runs a plain device copy of a known size (the calibration reference), then
either back-to-back launches of the decode GEMM classes on the named
workload at one row per stage, so that FETCH_SIZE / WRITE_SIZE per dispatch
can be compared with each kernel's algorithmic bytes, or (--decode-steps N)
the decode itself: --warmup rounds, then N rounds whose dispatches the
summary adds up, with the algorithmic bytes of those rounds (weights of the
stages each round ran, the exit head, and the attention's key/value reads):

  rocprofv3 --pmc FETCH_SIZE --output-format csv -d OUT -- \
      python3 -m paper_2606_29223_amd.traffic_run [--decode-steps 128]
"""

from __future__ import annotations

import argparse
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

COPY_BYTES = 1 << 30


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--config", default=None)
    ap.add_argument("--reps", type=int, default=8)
    ap.add_argument("--rows", type=int, default=1)
    ap.add_argument("--decode-steps", type=int, default=0)
    ap.add_argument("--warmup", type=int, default=8)
    args = ap.parse_args()
    import torch

    from paper_2606_29223_amd import dexlib
    from synth import configs, gen

    cfg = configs.get(args.config or configs.HEADLINE)
    lib = dexlib.load()
    src = torch.empty(COPY_BYTES, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1)
    torch.cuda.synchronize()
    for _ in range(4):
        assert lib.dex_debug_copy(dst.data_ptr(), src.data_ptr(), COPY_BYTES, None) == 0
    torch.cuda.synchronize()
    del src, dst
    dev_w = dexlib.device_weights(cfg, gen.generate_model(cfg))
    if args.decode_steps > 0:
        decode(cfg, dev_w, args)
        return
    dec = dexlib.Decoder(cfg, dev_w, max_context=cfg["prompt_len"] + 8)
    dec.prefill(gen.prompts(cfg))
    out = {"copy_bytes": COPY_BYTES, "config": cfg["name"], "rows": args.rows, "kernels": {}}
    for cls in (3, 4, 5, 6):
        us, b = dec.time_kernel(cls, args.rows, reps=args.reps)
        out["kernels"][dexlib.KERNEL_CLASSES[cls]] = {"avg_us": us, "algorithmic_bytes": b}
    dec.close()
    print(json.dumps(out))


def decode(cfg, dev_w, args):
    """Warm-up rounds, then the measured rounds with per-kernel byte counts
    (timing mode: one stream, which the counters serialise anyway)."""
    import torch

    from paper_2606_29223_amd import dexlib
    from synth import gen

    P = cfg["prompt_len"]
    dec = dexlib.Decoder(cfg, dev_w, max_context=P + max(cfg["gen_len"], args.warmup + args.decode_steps + 2))
    dec.prefill(gen.prompts(cfg))
    for _ in range(args.warmup):
        dec.step()
    torch.cuda.synchronize()
    dec.set_timing(True)
    layers = commits = 0
    for _ in range(args.decode_steps):
        c = dec.step()
        layers += dec.info.layers_streamed
        commits += int((c >= 0).sum())
    torch.cuda.synchronize()
    _, _, nbytes = dec.kernel_times()
    dec.close()
    es = 2 if cfg["dtype"] == "bf16" else 4
    d, F, V = cfg["d_model"], cfg["d_ffn"], cfg["vocab"]
    layer_bytes = es * (d * (cfg["n_heads"] + 2 * cfg["n_kv_heads"]) * cfg["head_dim"]
                        + cfg["n_heads"] * cfg["head_dim"] * d + 3 * d * F)
    n = args.decode_steps
    alg = (layers * layer_bytes + n * es * V * d + nbytes[1]) / n
    print(json.dumps({"copy_bytes": COPY_BYTES, "config": cfg["name"], "warmup": args.warmup, "rounds": n,
                      "commits": commits, "weight_layers": layers, "attention_bytes": nbytes[1],
                      "algorithmic_bytes_per_round": alg}))


if __name__ == "__main__":
    main()
