"""Launch sequence for hardware traffic counters (run under rocprofv3 --pmc).

Runs a plain device copy of a known size (the calibration reference), then
back-to-back launches of the decode GEMM classes on the named workload at
one row per stage, so that FETCH_SIZE / WRITE_SIZE per dispatch can be
compared with each kernel's algorithmic bytes:

  rocprofv3 --pmc FETCH_SIZE --output-format csv -d OUT -- \
      python3 -m paper_2606_29223_amd.traffic_run
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
    dec = dexlib.Decoder(cfg, dev_w, max_context=cfg["prompt_len"] + 8)
    dec.prefill(gen.prompts(cfg))
    out = {"copy_bytes": COPY_BYTES, "config": cfg["name"], "rows": args.rows, "kernels": {}}
    for cls in (3, 4, 5, 6):
        us, b = dec.time_kernel(cls, args.rows, reps=args.reps)
        out["kernels"][dexlib.KERNEL_CLASSES[cls]] = {"avg_us": us, "algorithmic_bytes": b}
    dec.close()
    print(json.dumps(out))


if __name__ == "__main__":
    main()
