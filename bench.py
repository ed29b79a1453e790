"""Benchmark of the DEX decode step on one MI355X.

A step is one dex_step call: one round of Algorithm 1 (every stage that has
lattice rows streams its layers once, then the batched exit head, verify /
commit and the key/value collapse).  The value is committed tokens per
second over the timed steps, inputs and weights already resident in HBM.

Prints one JSON line.  Besides the contract fields it carries
  roofline     for the dominant kernel (most time in an event-instrumented
               rerun of the timed steps): algorithmic bytes per launch over its
               mean duration, measured with HIP events on the decode stream
               around back-to-back launches at the most common rows-per-stage,
               against the 8 TB/s HBM peak;
  dex          lattice statistics: rounds and layers per committed token,
               matched-depth histogram, algorithmic bytes per commit (weights
               of the stages each round ran, the exit head, and the
               attention's key/value reads) and the resulting HBM-roofline
               tokens/s of this schedule;
  e2e          committed tokens/s including the prefill (y_0 counts);
  step_traffic HBM bytes per round of this run's own rounds: its algorithmic
               bytes (weights of the stages each round ran, the exit head,
               the attention's key/value reads) times the counted/algorithmic
               ratio that rocprofv3 measured over whole decode rounds of the
               same workload (FETCH_SIZE + WRITE_SIZE, profiles/
               step_traffic_<workload>.json, only while the kernel and
               engine sources are unchanged), over this run's time per round;
  cpu_baseline the oracle (float64 numpy) running the same decode on the host
               cores for a bounded sample, DEX and plain AR timed separately.
"""

from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from synth import configs, gen  # noqa: E402

PEAK_HBM_GBS = 8000.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=128)
    p.add_argument("--warmup", type=int, default=8)
    p.add_argument("--config", default=configs.HEADLINE)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=20.0)
    p.add_argument("--no-ar", action="store_true", help="skip the plain AR reference rate")
    p.add_argument("--temperature", type=float, default=0.0,
                   help="> 0: Algorithm 2's sampling mode (Gumbel-max, seed --seed); 0: greedy")
    p.add_argument("--seed", type=int, default=0)
    p.add_argument("--stage-grouping", type=int, default=0, choices=(0, 1, -1),
                   help="0/1: each lane's stages in step, one launch per kernel and layer step; "
                        "-1: launches per stage")
    p.add_argument("--stage-streams", type=int, default=0, help="lanes (0: the library default)")
    p.add_argument("--adapter-alpha", type=float, default=None,
                   help="attach synthetic inducing adapters with this gate to the non-final depths")
    p.add_argument("--traffic-json", default=os.path.join(ROOT, "profiles", "traffic.json"))
    p.add_argument("--step-traffic-json", default=None,
                   help="default: profiles/step_traffic_<workload>.json")
    p.add_argument("--kernel-stats-json", default=None,
                   help="default: profiles/kernel_stats_<workload>.json")
    return p.parse_args()


def cpu_baseline(cfg, weights, prompts, budget_s, temperature=0.0, seed=0):
    """The oracle as it stands, timed on this host after its prefill of
    sequence 0 (prefill untimed): DEX rounds (the value), then plain greedy
    AR over a budget of a third of DEX's."""
    import oracle
    from oracle import ar, dex
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas_threads = None
    m = oracle.Model(cfg, gen.model_as_f64(cfg, weights))
    prompt = [int(t) for t in prompts[0]]
    pf = m.prefill(prompt)

    def grow(run, budget):
        # run for growing T until the budget is used; report the last full run
        T = 2
        while True:
            t0 = time.perf_counter()
            extra = run(T)
            dt = time.perf_counter() - t0
            if dt * 2.5 > budget or T >= cfg["gen_len"]:
                return T - 1, dt, extra
            T = min(cfg["gen_len"], T * 2)

    commits, t_used, rounds = grow(
        lambda T: dex.dex_generate(m, prompt, cfg["explored"], cfg["width_cap"], bool(cfg["decs"]), T,
                                   prefill=pf, keep_trace=False, temperature=temperature, seed=seed).rounds,
        budget_s)
    ar_commits, ar_used, _ = grow(
        lambda T: ar.ar_generate(m, prompt, T, prefill=pf, temperature=temperature, seed=seed), budget_s / 3)
    cores = len(os.sched_getaffinity(0))
    return {
        "value": commits / t_used, "unit": "committed tokens/s", "cores": blas_threads or cores,
        "kind": "oracle",
        "ar_value": ar_commits / ar_used,
        "sample": f"float64 oracle on sequence 0 of {cfg['name']} after its {cfg['prompt_len']}-token prompt "
                  f"(prefill untimed): DEX {commits} commits in {rounds} rounds, {t_used:.1f} s; plain AR "
                  f"{ar_commits} tokens in {ar_used:.1f} s (ar_value); host affinity {cores} cores",
    }


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the decode step runs on one GPU (no multi-GPU path); --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import torch
    from paper_2606_29223_amd import dexlib

    cfg = configs.get(args.config)
    if args.step_traffic_json is None:
        args.step_traffic_json = os.path.join(ROOT, "profiles", f"step_traffic_{cfg['name']}.json")
    if args.kernel_stats_json is None:
        args.kernel_stats_json = os.path.join(ROOT, "profiles", f"kernel_stats_{cfg['name']}.json")
    t0 = time.time()
    weights = gen.generate_model(cfg)
    prompts = gen.prompts(cfg)
    dev_w = dexlib.device_weights(cfg, weights)
    torch.cuda.synchronize()
    setup_s = time.time() - t0

    P = cfg["prompt_len"]
    max_ctx = P + cfg["gen_len"]
    # warm-up, the timed steps, the round-timing pass and the instrumented
    # pass all decode on the same context (at most one commit per sequence
    # and round)
    need = args.warmup + 3 * args.steps + 2
    if need > cfg["gen_len"]:
        max_ctx = P + need

    samp = dict(temperature=args.temperature, seed=args.seed, stage_grouping=args.stage_grouping,
                stage_streams=args.stage_streams)
    dev_ad = None
    if args.adapter_alpha is not None:
        dev_ad = dexlib.device_weights(cfg, gen.generate_adapters(cfg, args.adapter_alpha))
        torch.cuda.synchronize()
    dec = dexlib.Decoder(cfg, dev_w, max_context=max_ctx, adapters=dev_ad, **samp)
    torch.cuda.synchronize()
    tp = time.perf_counter()
    dec.prefill(prompts)
    torch.cuda.synchronize()
    prefill_s = time.perf_counter() - tp
    B = dec.batch

    m_hist = {}
    kstar_hist = {}
    stages_hist = {}    # stages with rows per round (how much a round can overlap)

    ad_runs = [0]       # non-final stages with exit rows: each streams its adapter

    attn_total = [0.0]  # algorithmic bytes of the attention launches

    def run(n):
        """n rounds; each round's commits and step info are copied out and
        tallied after the loop, so the timed loop holds only the steps."""
        outs = np.empty((n, B), np.int32)
        infos = (dexlib.DexStepInfo * n)()
        size = ctypes.sizeof(dexlib.DexStepInfo)
        src = ctypes.addressof(dec.info)
        for i in range(n):
            outs[i] = dec.step()
            ctypes.memmove(ctypes.addressof(infos[i]), src, size)
        return outs, infos

    def tally(outs, infos):
        commits = int((outs >= 0).sum())
        rounds = layers = row_layers = 0
        for inf in infos:
            rounds += 1
            layers += inf.layers_streamed
            row_layers += inf.row_layers
            attn_total[0] += inf.attn_bytes
            ns = sum(1 for k in range(dec.N) if inf.rows_per_stage[k])
            stages_hist[ns] = stages_hist.get(ns, 0) + 1
            for k in range(dec.N):
                mk = inf.rows_per_stage[k]
                if mk:
                    m_hist[mk] = m_hist.get(mk, 0) + 1
                    if k < dec.N - 1:
                        ad_runs[0] += 1
            for b in range(B):
                ks = inf.kstar[b]
                if ks >= 0:
                    kstar_hist[ks] = kstar_hist.get(ks, 0) + 1
        return commits, rounds, layers, row_layers

    def steps(n):
        return tally(*run(n))

    tw = time.perf_counter()
    warm_commits = steps(args.warmup)[0]
    torch.cuda.synchronize()
    warm_s = time.perf_counter() - tw
    m_hist.clear()
    kstar_hist.clear()
    stages_hist.clear()
    ad_runs[0] = 0
    attn_total[0] = 0.0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    timed = run(args.steps)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    commits, rounds, layers, row_layers = tally(*timed)
    value = commits / elapsed
    # end to end as the paper counts it: y_0 of every sequence from the
    # prefill plus every commit, over prefill and all decode rounds so far
    e2e = (B + warm_commits + commits) / (prefill_s + warm_s + elapsed)
    kstar_timed = dict(kstar_hist)
    stages_timed = dict(stages_hist)
    m_timed = dict(m_hist)
    ad_runs_timed = ad_runs[0]
    attn_bytes_per_round = attn_total[0] / max(rounds, 1)   # K/V, q and outputs of the attention

    # a pass of the same length with events at the round boundaries only
    # (the schedule of the timed steps): where a round's wall time goes,
    # including the gap between rounds
    dec.set_round_timing(True)
    tr0 = time.perf_counter()
    steps(args.steps)
    torch.cuda.synchronize()
    tr_wall = (time.perf_counter() - tr0) / args.steps * 1e3
    rt_ms, rt_n = dec.round_times()
    dec.set_round_timing(False)
    round_phases = {"wall_ms_per_round": round(tr_wall, 4), "rounds": rt_n}
    for i, nm in enumerate(dexlib.ROUND_PHASES):
        cnt = rt_n - 1 if nm in ("commit_collapse", "gap_before_round") else rt_n
        round_phases[nm + "_ms"] = round(rt_ms[i] / max(cnt, 1), 4)

    # instrumented run of the same length: per-kernel HIP event durations
    # (each launch bracketed by events; includes the event overhead)
    dec.set_timing(True)
    steps(args.steps)
    torch.cuda.synchronize()
    ms, n, nbytes = dec.kernel_times()
    dec.set_timing(False)
    names = dexlib.KERNEL_CLASSES
    per_kernel = {names[i]: {"ms": round(ms[i], 3), "launches": int(n[i]),
                             "avg_us_event": round(ms[i] / max(n[i], 1) * 1e3, 2),
                             "GBps_event": round(nbytes[i] / max(ms[i], 1e-9) / 1e6, 1) if nbytes[i] else None}
                  for i in range(8)}
    # roofline of the dominant weight-streaming kernel: mean duration of
    # back-to-back launches on the decode stream (HIP events around the whole
    # run, layers cycled so no launch re-reads a matrix from cache), at the
    # most common rows-per-stage of the timed steps
    dom = max((3, 4, 5, 6), key=lambda i: ms[i])
    m_mode = max(m_hist.items(), key=lambda kv: kv[1])[0] if m_hist else 1
    avg_us, bytes_per = dec.time_kernel(dom, m_mode, reps=96)
    dec.close()
    achieved = bytes_per / (avg_us * 1e-6) / 1e9
    traffic = None
    if os.path.exists(args.traffic_json):
        # counters taken for the current GEMM kernel source only
        from paper_2606_29223_amd.profile_summary import gemm_source_hash
        try:
            tj = json.load(open(args.traffic_json))
            ent = tj.get(cfg["name"], {}).get(names[dom])
            if ent and tj.get("gemm_source") == gemm_source_hash() and tj.get("rows") == m_mode:
                traffic = ent.get("bytes_per_launch")
        except (OSError, ValueError):
            traffic = None
    roofline = {"bound": "hbm", "kernel": names[dom], "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": traffic,
                "frac_source": "mean of 96 back-to-back launches of the class at the most common rows per "
                               "stage (HIP events on the decode stream, layers cycled)",
                "bytes_per_launch": bytes_per, "avg_launch_us": round(avg_us, 2), "rows": m_mode}
    # the same class inside the steps: events around each launch of the
    # instrumented rerun (all stages on one stream), and, when a kernel trace
    # of this benchmark's own command exists for the current sources, the
    # rocprofv3 average duration of the class
    if n[dom]:
        ev_us = ms[dom] / n[dom] * 1e3
        ev_bytes = nbytes[dom] / n[dom]
        roofline["in_step_events"] = {"avg_launch_us": round(ev_us, 2),
                                      "frac": round(ev_bytes / (ev_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
    if os.path.exists(args.kernel_stats_json):
        from paper_2606_29223_amd.profile_summary import csrc_source_hash
        try:
            ks = json.load(open(args.kernel_stats_json))
            ent = ks.get("classes", {}).get(names[dom])
            if ent and ks.get("source") == csrc_source_hash() and ks.get("config") == cfg["name"]:
                roofline["rocprof"] = {"avg_launch_us": round(ent["avg_us"], 2), "launches": ent["launches"],
                                       "frac": round(bytes_per / (ent["avg_us"] * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
                                       "median_launch_us": round(ent["median_us"], 2),
                                       "median_frac": round(bytes_per / (ent["median_us"] * 1e-6) / 1e9
                                                            / PEAK_HBM_GBS, 4),
                                       "note": "single-layer launches of the class in the traced run; launches "
                                               "of concurrent stage lanes overlap and share HBM, which lengthens "
                                               "some (the mean) but not the typical one (the median); 'alone': "
                                               "the launches during which no other kernel ran",
                                       "profile": os.path.relpath(args.kernel_stats_json, ROOT)}
                if "avg_alone_us" in ent:
                    roofline["rocprof"].update({
                        "alone_launches": ent["launches_alone"],
                        "alone_avg_launch_us": round(ent["avg_alone_us"], 2),
                        "alone_frac": round(bytes_per / (ent["avg_alone_us"] * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)})
        except (OSError, ValueError, KeyError):
            pass

    # whole-round traffic: this run's algorithmic bytes per round times the
    # counted/algorithmic ratio measured over whole rounds with the current
    # sources
    step_traffic = None
    L, N = cfg["n_layers"], len(cfg["explored"])
    es = 2 if cfg["dtype"] == "bf16" else 4
    d, F, V = cfg["d_model"], cfg["d_ffn"], cfg["vocab"]
    layer_bytes = es * (d * (cfg["n_heads"] + 2 * cfg["n_kv_heads"]) * cfg["head_dim"]
                        + cfg["n_heads"] * cfg["head_dim"] * d + 3 * d * F)
    ad_bytes = (ad_runs_timed * 2 * d * (2 * d) * es) if args.adapter_alpha is not None else 0
    alg_per_round = (layers * layer_bytes + rounds * es * V * d + ad_bytes) / max(rounds, 1) + attn_bytes_per_round
    if os.path.exists(args.step_traffic_json) and args.adapter_alpha is None:
        from paper_2606_29223_amd.profile_summary import csrc_source_hash
        try:
            st = json.load(open(args.step_traffic_json))
            if st.get("source") == csrc_source_hash() and st.get("config") == cfg["name"]:
                ratio = st["counted_bytes_per_round"] / st["algorithmic_bytes_per_round"]
                counted = ratio * alg_per_round
                gbs = counted / (elapsed / args.steps) / 1e9
                step_traffic = {"counted_over_algorithmic": round(ratio, 5),
                                "ratio_measured_over": f"rounds {st['warmup'] + 1}..{st['warmup'] + st['rounds']} "
                                                       f"of {st['config']} ({os.path.relpath(args.step_traffic_json, ROOT)})",
                                "algorithmic_bytes_per_round": alg_per_round,
                                "counted_bytes_per_round": counted,
                                "achieved_GBps": round(gbs, 1), "frac": round(gbs / PEAK_HBM_GBS, 4)}
        except (OSError, ValueError, KeyError, ZeroDivisionError):
            step_traffic = None

    ar_value = None
    if not args.no_ar:
        ar = dexlib.Decoder(cfg, dev_w, explored=[cfg["n_layers"]], width_cap=1, max_context=max_ctx, **samp)
        ar.prefill(prompts)
        for _ in range(args.warmup):
            ar.step()
        torch.cuda.synchronize()
        ta = time.perf_counter()
        na = 0
        for _ in range(args.steps):
            na += int((ar.step() >= 0).sum())
        torch.cuda.synchronize()
        ar_value = na / (time.perf_counter() - ta)
        ar.close()

    bytes_per_commit = (layers * layer_bytes + rounds * es * V * d + ad_bytes) / max(commits, 1)
    hbm_bytes_per_commit = bytes_per_commit + attn_bytes_per_round * rounds / max(commits, 1)
    cpu = None
    if not args.no_cpu_baseline:
        del dev_w
        torch.cuda.empty_cache()
        cpu = cpu_baseline(cfg, weights, prompts, args.cpu_seconds, args.temperature, args.seed)

    out = {
        "metric": "committed tokens/s at batch 1 (32L d4096 bf16) + achieved HBM GB/s vs peak",
        "value": round(value, 3),
        "unit": "committed tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg["dtype"] == "bf16" else "f32",
        "data": "synthetic (seeded random weights and uniform prompts)",
        "config": {"workload": cfg["name"], "explored": cfg["explored"], "width_cap": cfg["width_cap"],
                   "batch": B, "prompt_len": P, "parallelism": "single GPU",
                   "stage_launches": "grouped" if args.stage_grouping >= 0 else "per stage",
                   "decoding": (f"sampling, temperature {args.temperature}, seed {args.seed}"
                                if args.temperature > 0 else "greedy"),
                   "adapters": (f"synthetic, gate {args.adapter_alpha}" if args.adapter_alpha is not None
                                else None)},
        "roofline": roofline,
        "step_traffic": step_traffic,
        "cpu_baseline": cpu,
        "dex": {"commits": commits, "rounds": rounds, "rounds_per_commit": round(rounds / max(commits, 1), 4),
                "weight_layers_streamed_per_commit": round(layers / max(commits, 1), 3),
                "row_layers_per_commit": round(row_layers / max(commits, 1), 3),
                "critical_path_layers_per_commit": round(L / N * rounds / max(commits, 1), 3),
                "ar_layers_per_commit": L,
                "rows_per_stage_hist": {str(k): v for k, v in sorted(m_timed.items())},
                "stages_per_round_hist": {str(k): v for k, v in sorted(stages_timed.items())},
                "matched_depth_hist": {str(k): v for k, v in sorted(kstar_timed.items())},
                "weight_bytes_per_commit": bytes_per_commit,
                "hbm_bytes_per_commit": hbm_bytes_per_commit,
                "roofline_tokens_per_s": round(PEAK_HBM_GBS * 1e9 / hbm_bytes_per_commit, 2),
                "frac_of_schedule_roofline": round(value * hbm_bytes_per_commit / (PEAK_HBM_GBS * 1e9), 4),
                "achieved_GBps": round(value * hbm_bytes_per_commit / 1e9, 1)},
        "round_phases": round_phases,
        "prefill_s": round(prefill_s, 3),
        "e2e_tokens_per_s": round(e2e, 3),
        "ar_tokens_per_s": round(ar_value, 3) if ar_value else None,
        "kernels": per_kernel,
        "setup_s": round(setup_s, 1),
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
