"""Turn rocprofv3 CSV output into the short text summaries kept in profiles/.

  python3 -m paper_2606_29223_amd.profile_summary stats STATS.csv TRACE.csv \
      --command "..." --out profiles/NAME.txt
  python3 -m paper_2606_29223_amd.profile_summary traffic FETCH_DIR WRITE_DIR \
      --command "..." --out-json profiles/traffic.json --out profiles/NAME.txt
  python3 -m paper_2606_29223_amd.profile_summary step FETCH_DIR WRITE_DIR \
      --run-json RUN.json --bench-json BENCH.json --command "..." --out profiles/NAME.txt
  python3 -m paper_2606_29223_amd.profile_summary mfma PMC_DIR --command "..." \
      --out profiles/NAME.txt

`stats` lists the kernels by total time and, for the decode GEMMs and the
attention kernels, the median duration of their decode launches.  `traffic`
reads the FETCH_SIZE and WRITE_SIZE passes over `traffic_run`, derives the
scale factor from the plain copy kernel (known bytes read and written) and
reports bytes per launch for each decode GEMM class next to its algorithmic
bytes.  `step` adds up the counters over whole decode rounds of
`traffic_run --decode-steps` and sets them against the rounds' algorithmic
bytes and, with an unprofiled bench line, against the time per round.
The traffic JSON records a hash of the GEMM kernel source so that a later
change of the kernel invalidates the measurement.
"""

from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import statistics

PKG = os.path.dirname(os.path.abspath(__file__))
SHORT = {
    "gemm_kernel<unsigned short, 1, 1,": "qkv (bf16, M<=16)",
    "gemm_kernel<unsigned short, 2, 1,": "o-proj / down (bf16, M<=16)",
    "gemm_kernel<unsigned short, 3, 1,": "gate/up (bf16, M<=16)",
    "gemm_kernel<unsigned short, 4, 1,": "lm-head (bf16, M<=16)",
}
# grouped launches (one segment per stage on grid z): listed per segment
SHORT_SEG = {
    "gemm_seg_kernel<unsigned short, 1, 1,": "qkv grouped, per segment",
    "gemm_seg_kernel<unsigned short, 2, 1,": "o-proj / down grouped, per segment",
    "gemm_seg_kernel<unsigned short, 3, 1,": "gate/up grouped, per segment",
}


def code_text(src: str) -> str:
    """C/C++/HIP source with comments removed and whitespace runs collapsed:
    what the compiler sees, so a comment edit leaves a measurement valid."""
    out, i, n = [], 0, len(src)
    while i < n:
        c = src[i]
        if c in "\"'":                       # string or character literal
            j = i + 1
            while j < n and src[j] != c:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        elif src.startswith("//", i):
            j = src.find("\n", i)
            i = n if j < 0 else j
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def gemm_source_hash() -> str:
    """Hash of the decode GEMM kernel code and of its argument struct."""
    h = hashlib.sha1()
    h.update(code_text(open(os.path.join(PKG, "csrc", "gemm.hip")).read()).encode())
    hdr = open(os.path.join(PKG, "csrc", "dex_kernels.h")).read()
    start = hdr.index("struct GemmArgs {")
    h.update(code_text(hdr[start:hdr.index("};", start)]).encode())
    return h.hexdigest()[:16]


def csrc_source_hash() -> str:
    """Hash of every kernel and engine source's code (comments and spacing
    aside): whole-round traffic depends on all of them."""
    h = hashlib.sha1()
    for f in sorted(glob.glob(os.path.join(PKG, "csrc", "*"))):
        h.update(os.path.basename(f).encode())
        h.update(code_text(open(f).read()).encode())
    return h.hexdigest()[:16]


def _short(name: str) -> str:
    name = name.replace("(anonymous namespace)::", "")
    base = name.split("(")[0].replace("void ", "").replace("dex::", "")
    return base


def stats(args):
    rows = list(csv.DictReader(open(args.stats_csv)))
    trace = list(csv.DictReader(open(args.trace_csv))) if args.trace_csv else []
    lines = [f"command: {args.command}", "", "rocprofv3 kernel statistics (all dispatches of the run)", ""]
    lines.append(f"{'kernel':58s} {'calls':>7s} {'avg_us':>9s} {'total_ms':>9s} {'pct':>6s}")
    for r in rows[: args.top]:
        lines.append(f"{_short(r['Name'])[:58]:58s} {r['Calls']:>7s} {float(r['AverageNs']) / 1e3:9.2f} "
                     f"{float(r['TotalDurationNs']) / 1e6:9.2f} {float(r['Percentage']):6.1f}")
    if trace:
        lines += ["", "decode launches (median duration; decode = M <= 16 GEMMs and the decode attention kernels;",
                  "a grouped GEMM launch counts once per segment, at its duration / segments)"]
        groups = {}
        for t in trace:
            n = _short(t["Kernel_Name"])
            dur = (int(t["End_Timestamp"]) - int(t["Start_Timestamp"])) / 1e3
            key = None
            for k, v in SHORT.items():
                if n.startswith(k):
                    key = v
            for k, v in SHORT_SEG.items():
                if n.startswith(k):
                    key = v
                    segs = max(int(t.get("Grid_Size_Z") or 1), 1)
                    groups.setdefault(key, []).extend([dur / segs] * segs)
                    key = None
            if n.startswith("attn_mfma_kernel") or (n.startswith("attn_kernel") and int(t["Grid_Size_X"]) <= 256 * 64):
                key = "attention (decode)"
            if n.startswith("attn_mfma_seg_kernel"):
                key = "attention grouped, per launch"
            if n.startswith("combine_kernel") and int(t["Grid_Size_X"]) <= 256 * 64:
                key = "attention combine (decode)"
            if key:
                groups.setdefault(key, []).append(dur)
        for k in sorted(groups):
            v = groups[k]
            lines.append(f"  {k:34s} launches={len(v):6d} median_us={statistics.median(v):8.2f}")
    if args.out_json and trace:
        # average duration of every launch of each decode GEMM class (the
        # instantiation the benchmark's workload uses), for bench.py's
        # roofline next to its own timing
        cls_of = {"gemm_kernel<unsigned short, 1,": "qkv", "gemm_kernel<unsigned short, 3,": "gate_up",
                  "gemm_kernel<unsigned short, 4,": "lm_head", "gemm_kernel<unsigned short, 2,": "o_proj+down"}
        # a launch ran alone when no other kernel of the run was active at
        # any point of its span (launches of concurrent stage lanes share HBM)
        span = sorted((int(t["Start_Timestamp"]), int(t["End_Timestamp"]), i) for i, t in enumerate(trace))
        alone = [True] * len(trace)
        far_end, far_i = -1, -1
        for s0, e0, i in span:
            if s0 < far_end:
                alone[i] = False
                alone[far_i] = False
            if e0 > far_end:
                far_end, far_i = e0, i
        per, per_alone = {}, {}
        for i, t in enumerate(trace):
            n = _short(t["Kernel_Name"])
            dur = (int(t["End_Timestamp"]) - int(t["Start_Timestamp"])) / 1e3
            for k, c in cls_of.items():
                if n.startswith(k):
                    per.setdefault(c, {}).setdefault(n, []).append(dur)
                    if alone[i]:
                        per_alone.setdefault(c, {}).setdefault(n, []).append(dur)
        classes = {}
        for c, insts in per.items():
            n, v = max(insts.items(), key=lambda kv: len(kv[1]))     # the most launched instantiation
            classes[c] = {"kernel": n, "launches": len(v), "avg_us": statistics.fmean(v),
                          "median_us": statistics.median(v)}
            va = per_alone.get(c, {}).get(n, [])
            if va:
                classes[c].update({"launches_alone": len(va), "avg_alone_us": statistics.fmean(va),
                                   "median_alone_us": statistics.median(va)})
        lines += ["", "decode GEMM classes, most launched instantiation: mean over all launches, and over the",
                  "launches that ran alone (no other kernel active during their span)"]
        for c in sorted(classes):
            e = classes[c]
            lines.append(f"  {c:12s} {e['kernel']:42s} all {e['launches']:6d} x {e['avg_us']:7.2f} us"
                         + (f"   alone {e['launches_alone']:6d} x {e['avg_alone_us']:7.2f} us" if "avg_alone_us" in e
                            else ""))
        json.dump({"source": csrc_source_hash(), "config": args.config, "command": args.command,
                   "classes": classes}, open(args.out_json, "w"), indent=1)
    os.makedirs(os.path.dirname(args.out) or ".", exist_ok=True)
    open(args.out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _counter_rows(d):
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    rows = list(csv.DictReader(open(files[0])))
    rows.sort(key=lambda r: int(r.get("Dispatch_Id", r.get("Correlation_Id", 0))))
    return rows


def _per_dispatch(rows, counter):
    out = []
    for r in rows:
        if r["Counter_Name"] == counter:
            out.append((_short(r["Kernel_Name"]), float(r["Counter_Value"])))
    return out


def traffic(args):
    run = json.load(open(args.run_json)) if args.run_json else None
    reps = args.reps
    res = {}
    for counter, d in (("FETCH_SIZE", args.fetch_dir), ("WRITE_SIZE", args.write_dir)):
        disp = _per_dispatch(_counter_rows(d), counter)
        copies = [v for n, v in disp if n.startswith("copy_kernel")]
        res[counter] = {"copy_kib": statistics.median(copies)}
        # the decode GEMM launches of traffic_run: (reps + 1) per class, in class order
        seq = {"o_proj": ("gemm_kernel<unsigned short, 2, 1,", 0),
               "down": ("gemm_kernel<unsigned short, 2, 1,", 1),
               "gate_up": ("gemm_kernel<unsigned short, 3, 1,", 0),
               "lm_head": ("gemm_kernel<unsigned short, 4, 1,", 0)}
        for cls, (name, idx) in seq.items():
            vals = [v for n, v in disp if n.startswith(name)]
            groups = {"gemm_kernel<unsigned short, 2, 1,": 2}.get(name, 1)
            vals = vals[-groups * (reps + 1):]
            vals = vals[idx * (reps + 1) + 1:(idx + 1) * (reps + 1)]   # drop the warm-up launch
            res[counter][cls] = statistics.median(vals) if vals else None
    copy_bytes = 1 << 30
    f_scale = copy_bytes / (res["FETCH_SIZE"]["copy_kib"] * 1024.0)
    w_scale = copy_bytes / (res["WRITE_SIZE"]["copy_kib"] * 1024.0)
    out = {"gemm_source": gemm_source_hash(), "fetch_scale": f_scale, "write_scale": w_scale,
           "command": args.command, "rows": 1}
    cfg = args.config
    out[cfg] = {}
    lines = [f"command: {args.command}", "",
             f"calibration: plain copy of {copy_bytes} bytes read FETCH_SIZE={res['FETCH_SIZE']['copy_kib']:.0f} KiB, "
             f"WRITE_SIZE={res['WRITE_SIZE']['copy_kib']:.0f} KiB -> scale fetch {f_scale:.4f}, write {w_scale:.4f}", "",
             f"{'kernel':10s} {'fetch_MB':>10s} {'write_MB':>10s} {'traffic_MB':>11s} {'algorithmic_MB':>15s}"]
    for cls in ("o_proj", "gate_up", "down", "lm_head"):
        fk, wk = res["FETCH_SIZE"][cls], res["WRITE_SIZE"][cls]
        if fk is None or wk is None:
            continue
        fb, wb = fk * 1024.0 * f_scale, wk * 1024.0 * w_scale
        alg = run["kernels"][cls]["algorithmic_bytes"] if run else None
        out[cfg][cls] = {"bytes_per_launch": fb + wb, "fetch_bytes": fb, "write_bytes": wb, "algorithmic_bytes": alg}
        lines.append(f"{cls:10s} {fb / 1e6:10.2f} {wb / 1e6:10.3f} {(fb + wb) / 1e6:11.2f} "
                     f"{(alg or 0) / 1e6:15.2f}")
    json.dump(out, open(args.out_json, "w"), indent=1)
    open(args.out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def step(args):
    """HBM traffic of whole decode rounds: FETCH_SIZE and WRITE_SIZE of every
    dispatch of traffic_run's measured rounds (the rounds are delimited by
    the argmax launch that ends each exit head; the prompt's is the first),
    scaled by the copy calibration, against the rounds' algorithmic bytes;
    with the unprofiled bench's time per round, the counters' GB/s."""
    run = json.load(open(args.run_json))
    bench = json.load(open(args.bench_json)) if args.bench_json else None
    tot = {}
    for counter, d in (("FETCH_SIZE", args.fetch_dir), ("WRITE_SIZE", args.write_dir)):
        disp = _per_dispatch(_counter_rows(d), counter)
        copies = [v for n, v in disp if n.startswith("copy_kernel")]
        scale = run["copy_bytes"] / (statistics.median(copies) * 1024.0)
        ends = [i for i, (n, _) in enumerate(disp) if n.startswith("argmax_kernel")]
        w, n = run["warmup"], run["rounds"]
        lo, hi = ends[w] + 1, ends[w + n] + 1          # dispatches of the measured rounds
        tot[counter] = sum(v for _, v in disp[lo:hi]) * 1024.0 * scale
    per_round = (tot["FETCH_SIZE"] + tot["WRITE_SIZE"]) / run["rounds"]
    alg = run["algorithmic_bytes_per_round"]
    lines = [f"command: {args.command}", "",
             f"workload {run['config']}: rounds {run['warmup'] + 1}..{run['warmup'] + run['rounds']} after the prompt, "
             f"{run['commits']} commits, {run['weight_layers']} weight-layers streamed",
             f"counted HBM bytes per round   {per_round / 1e9:8.3f} GB (fetch {tot['FETCH_SIZE'] / run['rounds'] / 1e9:.3f},"
             f" write {tot['WRITE_SIZE'] / run['rounds'] / 1e9:.3f})",
             f"algorithmic bytes per round   {alg / 1e9:8.3f} GB (weights of the stages run, exit head, K/V reads)",
             f"counted / algorithmic         {per_round / alg:8.4f}"]
    out = {"source": csrc_source_hash(), "command": args.command, "config": run["config"],
           "warmup": run["warmup"], "rounds": run["rounds"], "counted_bytes_per_round": per_round,
           "fetch_bytes_per_round": tot["FETCH_SIZE"] / run["rounds"],
           "write_bytes_per_round": tot["WRITE_SIZE"] / run["rounds"], "algorithmic_bytes_per_round": alg}
    if bench is not None and bench["config"]["workload"] == run["config"]:
        ms = bench["ms_per_step"]
        gbs = per_round / (ms * 1e-3) / 1e9
        lines.append(f"unprofiled bench: {ms:.4f} ms per round -> {gbs:8.1f} GB/s counted = "
                     f"{100 * gbs / 8000:.1f} % of 8 TB/s")
        out.update({"ms_per_round": ms, "counted_GBps": gbs})
    if args.out_json:
        json.dump(out, open(args.out_json, "w"), indent=1)
    open(args.out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def mfma(args):
    """Matrix-core utilisation per kernel from one --pmc pass with
    SQ_VALU_MFMA_BUSY_CYCLES, SQ_INSTS_VALU_MFMA_MOPS_BF16 and
    GRBM_GUI_ACTIVE: busy cycles summed over the SIMDs over active cycles x
    SIMDs (GRBM_GUI_ACTIVE reads as the sum of the per-XCD instances, hence
    the division by --xcds), and achieved bf16 matrix flops (MOPS x 512) over
    the kernels' duration."""
    rows = _counter_rows(args.pmc_dir)
    per = {}
    for r in rows:
        key = (r["Dispatch_Id"], _short(r["Kernel_Name"]))
        d = per.setdefault(key, {"dur": (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9})
        d[r["Counter_Name"]] = float(r["Counter_Value"])
    agg = {}
    for (_, name), d in per.items():
        a = agg.setdefault(name, {"n": 0, "busy": 0.0, "gui": 0.0, "mops": 0.0, "dur": 0.0})
        a["n"] += 1
        a["busy"] += d.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
        a["gui"] += d.get("GRBM_GUI_ACTIVE", 0.0)
        a["mops"] += d.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0)
        a["dur"] += d["dur"]
    simds = args.simds
    lines = [f"command: {args.command}", "",
             f"matrix-core utilisation per kernel ({simds} SIMDs; util = MFMA busy cycles / (active cycles x SIMDs),",
             f"active cycles = GRBM_GUI_ACTIVE / {args.xcds} XCD instances;",
             "bf16 TFLOP/s = SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 / kernel time; dense bf16 peak 2500 TFLOP/s)", "",
             f"{'kernel':44s} {'launches':>8s} {'time_ms':>9s} {'mfma_util_%':>11s} {'bf16_TFLOP/s':>12s}"]
    for name, a in sorted(agg.items(), key=lambda kv: -kv[1]["dur"])[: args.top]:
        util = 100.0 * a["busy"] / (a["gui"] / args.xcds * simds) if a["gui"] else 0.0
        tf = a["mops"] * 512 / a["dur"] / 1e12 if a["dur"] else 0.0
        lines.append(f"{name[:44]:44s} {a['n']:8d} {a['dur'] * 1e3:9.2f} {util:11.2f} {tf:12.2f}")
    open(args.out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("stats_csv")
    s.add_argument("trace_csv", nargs="?")
    s.add_argument("--command", required=True)
    s.add_argument("--out", required=True)
    s.add_argument("--top", type=int, default=16)
    s.add_argument("--out-json", default=None)
    s.add_argument("--config", default="llama-32L-d4096-x8-w4")
    t = sub.add_parser("traffic")
    t.add_argument("fetch_dir")
    t.add_argument("write_dir")
    t.add_argument("--run-json", default=None)
    t.add_argument("--reps", type=int, default=8)
    t.add_argument("--config", default="llama-32L-d4096-x8-w4")
    t.add_argument("--command", required=True)
    t.add_argument("--out-json", required=True)
    t.add_argument("--out", required=True)
    st = sub.add_parser("step")
    st.add_argument("fetch_dir")
    st.add_argument("write_dir")
    st.add_argument("--run-json", required=True)
    st.add_argument("--bench-json", default=None)
    st.add_argument("--command", required=True)
    st.add_argument("--out", required=True)
    st.add_argument("--out-json", default=None)
    m = sub.add_parser("mfma")
    m.add_argument("pmc_dir")
    m.add_argument("--command", required=True)
    m.add_argument("--out", required=True)
    m.add_argument("--simds", type=int, default=1024)
    m.add_argument("--xcds", type=int, default=8)
    m.add_argument("--top", type=int, default=12)
    a = ap.parse_args()
    {"stats": stats, "traffic": traffic, "step": step, "mfma": mfma}[a.cmd](a)


if __name__ == "__main__":
    main()
