#!/usr/bin/env python3
"""Sparse decode-step throughput on one MI355X.

Default workload: the hierarchical 128k-context layer (B=64, 32 query / 8
KV heads, head_dim 128, 8192 blocks of 16 tokens per sequence, top-k 128
blocks, all KV in a pinned DRAM pool, an HBM block cache of 25% of each
sequence's blocks, queries drifting 0.3 per step).  One step is the whole
decode path of that layer: block scoring, top-k selection, the host-side
cache resolve (--resolve device runs it on the GPU instead), the gather of
missed blocks from DRAM and sparse attention.
Inputs are resident (pool in pinned DRAM, metadata and cache in HBM) when
timing starts.  The workload's cache state is fixed: the timed steps start
from a cache that holds exactly the previous step's selection (one cold
fill step right before them).  Warm-up steps beyond that one run first on
a throwaway cache state, which is then emptied, so --warmup changes what is
warmed (kernels, streams, host threads), never the timed workload.
The same run then measures the full 32-layer decode step with ragged
lengths (reported under "layers32"; --no-layers32 skips it), by default
with the sequence groups pipelined across layers and the slot tables on
the GPU (ss_decode_step_dev), and again with them on host threads
(ss_decode_step, under "other_resolve").

Prints one JSON line on stdout (progress goes to stderr):
  value      = B * steps / wall time of the timed steps (tokens/s)
  roofline   = the step's dominant kernel, the gather over the PCIe 5.0 x16
               host link (63.0 GB/s per direction): missed-record bytes per
               step / the link's busy time (the union of the HIP-event
               intervals of the step's gather launches in the timed region)
  rooflines_isolated = scoring, top-k and attention each launched alone on
               the same data, against the HBM peak (8 TB/s)
  cpu_baseline = the CPU oracle on a bounded sample of the same workload
  host       = the negotiated PCIe link of the GPU and the host's CPUs.
"""
import argparse
import json
import math
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

HBM_PEAK_GBS = 8000.0
LINK_PEAK_GBS = 32.0 * 16 * 128 / 130 / 8  # PCIe 5.0 x16, one direction: 63.0 GB/s
D = 128


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default: the workload's)")
    ap.add_argument("--warmup", type=int, default=1,
                    help="untimed steps first: the last one fills the emptied cache (the workload's own warm-up "
                         "step); the ones before it run on a throwaway cache state")
    ap.add_argument("--config", default="2", help="workload index or name (see synth/configs.py)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--parts", default="auto",
                    help="sequence groups pipelined within a layer step: auto (B >= 40: seven groups that grow "
                         "then shrink, 2,4,10,20,18,8,2 at B=64; 8 <= B < 40: four growing groups, 2,3,5,6 at "
                         "B=16; smaller B: one or two; with the groups schedule four equal groups), N (equal), "
                         "tentN (small first/last), or comma-separated sizes")
    ap.add_argument("--cpu-seqs", type=int, default=64, help="sequences in the CPU-oracle sample")
    ap.add_argument("--cpu-steps", type=int, default=8, help="timed steps in the CPU-oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--pool-flags", type=int, default=0, help="0 coherent, 1 non-coherent pinned pool")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB copy kernel (the scale for HBM traffic counters) and exit")
    ap.add_argument("--summarize-pmc", nargs=4, metavar=("FETCH", "WRITE", "COPY_FETCH", "COPY_WRITE"),
                    help="rocprofv3 --pmc output folders of this script (FETCH_SIZE, WRITE_SIZE) and of "
                         "--calibrate-copy; prints the traffic summary and exits (no GPU)")
    ap.add_argument("--bench-json", help="with --summarize-pmc: the JSON line the profiled run printed")
    ap.add_argument("--resolve", choices=["auto", "host", "device"], default="auto",
                    help="the slot-table resolve on host threads (ss_decode_layer) or on the GPU "
                         "(ss_decode_layer_dev); auto: host for one layer, GPU for multi-layer workloads")
    ap.add_argument("--layers32-resolve", choices=["host", "device"], default="device",
                    help="the resolve of the 32-layer sub-record")
    ap.add_argument("--schedule", choices=["auto", "layers", "groups"], default="auto",
                    help="multi-layer workloads: each layer's step in turn (layers), or the sequence groups "
                         "pipelined across layers (groups: ss_decode_step with the host resolve, "
                         "ss_decode_step_dev with the device resolve); auto: groups for multi-layer workloads")
    ap.add_argument("--layers32-schedule", choices=["auto", "layers", "groups"], default="auto",
                    help="the schedule of the 32-layer sub-record")
    ap.add_argument("--layers32-parts", default="auto", help="the sequence groups of the 32-layer sub-record")
    ap.add_argument("--with-save", action="store_true",
                    help="every step also appends its new tokens (metadata on a fill) and saves them to DRAM "
                         "(FlashD2H); single-layer workloads, one warm-up step")
    ap.add_argument("--save-stream", choices=["own", "main"], default="own",
                    help="with --with-save: the FlashD2H copies on a stream of their own or on the main stream")
    ap.add_argument("--no-variants", action="store_true", help="skip the scoring-variant comparison")
    ap.add_argument("--no-working-set", action="store_true",
                    help="skip the working-set study and the batch-control comparison (Algorithm 1)")
    ap.add_argument("--no-prefill", action="store_true", help="skip the layer-segmented prefill measurement")
    ap.add_argument("--no-save-bandwidth", action="store_true", help="skip FlashD2H saving against block size")
    ap.add_argument("--comparisons", action="store_true",
                    help="also time the paper's comparison transfers: one hipMemcpyAsync per block for loading "
                         "and saving, and GPU-direct saving")
    ap.add_argument("--no-layers32", action="store_true", help="skip the 32-layer sub-record")
    ap.add_argument("--pool-budget-gib", type=float, default=56.0,
                    help="pinned DRAM for KV records; layers beyond it reuse earlier layers' records")
    return ap.parse_args()


def group_sizes(spec, B, H, schedule="layers"):
    if spec == "auto":
        return H.default_parts(B, schedule)
    if spec.startswith("tent"):
        return H.tent_parts(B, int(spec[4:]))
    if "," in spec:
        return [int(x) for x in spec.split(",")]
    return int(spec)


def main():
    args = parse()
    if args.summarize_pmc:
        summarize_pmc(args)
        return
    if args.calibrate_copy:
        calibrate_copy()
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU: the decode path has no cross-GPU step (every (sequence, KV head) "
              f"unit is independent); got --gpus {args.gpus}, WORLD_SIZE {world}.", file=sys.stderr)
        sys.exit(2)

    import torch

    import synth
    from paper_2509_24626_amd import binding as ss
    from paper_2509_24626_amd import harness as H

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    ss.lib()
    cfg = synth.get(int(args.config)) if args.config.isdigit() else synth.get(args.config)
    if cfg.placement != "host":
        print("bench.py times the hierarchical workloads (2, 3, 4); the all-HBM ones are parity cases",
              file=sys.stderr)
        sys.exit(2)
    if args.with_save and (cfg.layers != 1 or args.warmup > 1):
        print("--with-save runs single-layer workloads with one warm-up step", file=sys.stderr)
        sys.exit(2)
    steps = args.steps if args.steps is not None else cfg.steps
    warmup = max(args.warmup, 1)
    if args.resolve == "auto":
        # the host resolve (the paper's arrangement) for one layer; with many layers
        # each layer's ramp pays the host's reaction, and the GPU resolve measured
        # 2-3% more tokens/s on the 32-layer workload over seeds 0-2
        args.resolve = "device" if cfg.layers > 1 else "host"
    host = host_facts()
    log(f"host: {host}")

    schedule = pick_schedule(args.schedule, cfg, args.resolve)
    run = measure(cfg, args, steps, warmup, args.resolve, args.parts, torch, ss, H, synth, studies=True,
                  schedule=schedule)
    result = {
        "metric": "sparse decode-step tokens/sec at 1 GPU; % HBM roofline; gather host-link GB/s",
        "value": run["value"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": run["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": run["config"],
        "workload_conforms": True,
        "warmup_note": ("the timed steps start from a cache holding exactly the previous step's selection, "
                        "whatever --warmup is: warm-up steps before that fill step run on a throwaway cache "
                        "state, which is emptied before the fill step"),
        "roofline": run["roofline"],
        "pipeline_ms": run["pipeline_ms"],
        **({"pipeline_ms_per_step": run["pipeline_ms_per_step"]} if "pipeline_ms_per_step" in run else {}),
        "step_ms_events": run["step_ms_events"],
        "rooflines_isolated": run["rooflines_isolated"],
        "parts": run["parts"],
        "miss_rate": run["miss_rate"],
        "miss_rate_per_step": run["miss_rate_per_step"],
        "gather_GBps": run["roofline"]["achieved"],
        "hbm_frac": {"score": run["rooflines_isolated"]["score"]["frac"],
                     "attention": run["rooflines_isolated"]["attention"]["frac"]},
        "metadata_build": run["metadata_build"],
        "cpu_baseline": run.get("cpu_baseline"),
        "host": host,
    }
    for key in ("save_side", "save_bandwidth", "load_comparison", "working_set", "batch_control", "score_variants",
                "prefill"):
        if run.get(key) is not None:
            result[key] = run[key]

    # ------------------------------------- the full 32-layer decode step
    if cfg.layers == 1 and not args.with_save and not args.no_layers32:
        c3 = synth.get(3)
        sched3 = pick_schedule(args.layers32_schedule, c3, args.layers32_resolve)
        sub = measure(c3, args, c3.steps, warmup, args.layers32_resolve, args.layers32_parts, torch, ss, H, synth,
                      studies=False, schedule=sched3)
        result["layers32"] = {
            "workload": sub["config"]["workload"], "value": sub["value"], "unit": "tokens/s",
            "steps": c3.steps, "warmup": warmup, "ms_per_step": sub["ms_per_step"],
            "layers": c3.layers, "layers_with_own_dram_records": sub["config"]["layers_with_own_dram_records"],
            "resolve": args.layers32_resolve, "schedule": sched3, "parts": sub["parts"],
            "miss_rate": sub["miss_rate"],
            "gather": {k: sub["roofline"][k] for k in ("bound", "achieved", "peak", "unit", "frac",
                                                        "bytes_per_step", "link_busy_ms_per_step")},
            "pipeline_ms_per_layer": sub["pipeline_ms"], "step_ms_events": sub["step_ms_events"],
            **({"pipeline_ms_per_step": sub["pipeline_ms_per_step"]} if "pipeline_ms_per_step" in sub else {}),
            "rooflines_isolated": sub["rooflines_isolated"],
            "note": ("all 32 layers in every step; ragged lengths U[8k, 64k]; 30% cache per layer; " +
                     ("groups schedule: each sequence group runs its layers in order on its own stream, its "
                      "layer l+1 after its layer-l attention, and the next step starts after the whole step; "
                      "pipeline_ms_per_step from events on every gather, pipeline_ms_per_layer = per step / 32"
                      if sched3 == "groups" else
                      "layers schedule: each layer's step in turn; pipeline_ms is per layer (sampled on the "
                      "first and last layer of every step)"))}
        # the same step with the slot tables resolved the other way (host threads, the paper's cache
        # manager, when the default is the GPU), same schedule, same run
        other = "host" if args.layers32_resolve == "device" else "device"
        sub2 = measure(c3, args, c3.steps, warmup, other, args.layers32_parts, torch, ss, H, synth, studies=False,
                       schedule=pick_schedule(args.layers32_schedule, c3, other))
        result["layers32"]["other_resolve"] = {
            "resolve": other, "value": sub2["value"], "ms_per_step": sub2["ms_per_step"],
            "miss_rate": sub2["miss_rate"], "gather_frac": sub2["roofline"]["frac"],
            **({"pipeline_ms_per_step": sub2["pipeline_ms_per_step"]} if "pipeline_ms_per_step" in sub2 else {})}
    print(json.dumps(result), flush=True)
    exit_report()


def pick_schedule(spec, cfg, resolve):
    if spec == "auto":
        return "groups" if cfg.layers > 1 else "layers"
    return spec


def measure(cfg, args, steps, warmup, resolve, parts_spec, torch, ss, H, synth, studies, schedule="layers"):
    """Builds the workload, runs its warm-up, times `steps` steps and
    measures each HBM kernel alone; with `studies` also runs the studies
    and the CPU baseline on it.  Frees everything it allocated.
    schedule: "layers" (each layer's step in turn) or "groups" (the groups
    pipelined across layers, one ss_decode_step_dev call per step)."""
    lens = synth.gen.lengths(cfg, args.seed)
    nblk = (lens // cfg.blk).astype(np.int32)
    _, per_layer = H.pool_layout(cfg, nblk)
    budget = int(args.pool_budget_gib * 2**30)
    n_distinct = H.distinct_layers(cfg, nblk, budget)
    log(f"workload {cfg.name}: {cfg.layers} layer(s), {n_distinct} with DRAM records of their own, "
        f"pool {per_layer * n_distinct / 2**30:.2f} GiB pinned")
    parts = group_sizes(parts_spec, cfg.B, H, schedule)
    new_kv = None
    res = {}
    if args.with_save:
        reserve = (warmup + steps) // cfg.blk + 2
        off, total = H.pool_layout(cfg, nblk, reserve)
        pool = H.HostPool(total, args.pool_flags)
        L = H.build_hier_layer(cfg, args.seed, 0, pool, 0, nblk, progress=log, parts=parts, reserve=reserve)
        L.enable_save(threads=2, save_stream=torch.cuda.Stream() if args.save_stream == "own" else None)
        layers = [L]
        sK, sV = synth.gen.channel_scales(cfg.Hkv, D, args.seed, 0, "cuda")
        # the steps' new tokens, resident in HBM before timing (the layer's
        # projection would have produced them)
        new_kv = [synth.gen.new_tokens(cfg.B, cfg.Hkv, D, sK, sV, args.seed, 0, s, "cuda")
                  for s in range(warmup + steps)]
    else:
        # pinned memory freed by an earlier workload of this process may not all
        # be available again at once: a multi-layer model steps its budget down
        for b in (budget, budget - (8 << 30), budget - (16 << 30)) if cfg.layers > 1 else (budget,):
            try:
                pool, layers, n_distinct = H.build_hier_model(cfg, args.seed, nblk, args.pool_flags, b,
                                                              progress=log, parts=parts,
                                                              dev_cache=resolve == "device")
                break
            except ss.SparseServeError as e:
                if b == budget - (16 << 30) or cfg.layers == 1:
                    raise
                log(f"pool of {b / 2**30:.0f} GiB not available ({e}); trying a smaller one")
    try:
        # q index 0 is the workload's warm-up (cache fill) step, 1..steps the timed ones
        qstreams = [H.query_stream(cfg, args.seed, l, steps) for l in range(cfg.layers)]

        def run_step(L, l, s, events=None):
            if new_kv is None:
                L.step(s, qstreams[l][s][1], events)
            else:
                L.step_with_save(s, qstreams[l][s][1], new_kv[s], events)

        def run_studies():
            single = new_kv is None and cfg.layers == 1
            if single and not args.no_working_set:
                res["working_set"] = working_set_study(cfg, layers[0], qstreams[0][-1][0], steps + 1, args.seed, ss,
                                                       torch)
                res["batch_control"] = batch_control_study(cfg, layers[0], pool, ss, torch, H, args.seed)
            if single and not args.no_variants:
                res["score_variants"] = score_variants_study(cfg, layers[0], qstreams[0][-1][1], pool, ss, torch)
            if args.comparisons:
                res["load_comparison"] = load_comparison(cfg, layers[0], pool, ss, torch)
            if not args.no_save_bandwidth:
                res["save_bandwidth"] = save_bandwidth(ss, torch, H, comparisons=args.comparisons)
            if not args.no_prefill:
                res["prefill"] = prefill_study(ss, torch, H)
            if not args.no_cpu_baseline:
                res["cpu_baseline"] = cpu_baseline(cfg, pool, layers[0], qstreams[0], nblk, args)

        groups = schedule == "groups"
        assert not groups or new_kv is None

        res["metadata_build"] = metadata_build_rate(cfg, pool, layers[0], nblk, ss, torch)

        # --------------------------------------------------------- warm-up
        # extra warm-up steps run on a throwaway cache state (queries of a
        # separate stream), then every cache is emptied, so the fill step
        # below leaves exactly its selection in the cache
        if warmup > 1:
            qthrow = [H.query_stream(cfg, args.seed + 1000, l, warmup - 2) for l in range(cfg.layers)]
            for s in range(warmup - 1):
                if groups:
                    H.decode_step_groups(layers, s, [qthrow[l][s][1] for l in range(len(layers))])
                    continue
                for l, L in enumerate(layers):
                    L.step(s, qthrow[l][s][1])
            torch.cuda.synchronize()
            for L in layers:
                L.reset_cache()
        if groups:
            H.decode_step_groups(layers, 0, [qstreams[l][0][1] for l in range(len(layers))])
        else:
            for l, L in enumerate(layers):
                run_step(L, l, 0)
        torch.cuda.synchronize()
        log(f"warm-up done ({warmup} step(s), the last on an empty cache); timing {steps} step(s)")

        # ----------------------------------------------------------- timed
        P = layers[0].parts
        if groups:
            res.update(timed_groups(cfg, layers, qstreams, steps, resolve, args, torch, ss, H, lens, n_distinct))
            iso = isolated_rates(cfg, layers[0], qstreams[0][steps][1], ss, torch)
            key = (cfg.name, args.seed, steps, tuple(layers[0].part_sizes), resolve, schedule)
            for name in iso:
                iso[name]["traffic"] = traffic(name, key)
            res["rooflines_isolated"] = iso
            if studies:
                run_studies()
            return res
        ev = [[[torch.cuda.Event(enable_timing=True) for _ in range(7 * P)] for _ in layers] for _ in range(steps)]
        # every timing event is a barrier packet on its queue: events go only on the
        # first and the last layer of a step (the step's start and end), and there
        # only around each group's start, end and gather (the dominant kernel)
        sampled = sorted({0, len(layers) - 1})
        used = [False] * (7 * P)
        used[0] = used[7 * (P - 1) + 6] = True
        for p in range(P):
            used[7 * p + 3] = used[7 * p + 4] = True
        for row in ev:  # create the underlying events before timing
            for es in row:
                for e in es:
                    e.record()
        torch.cuda.synchronize()
        n_miss = np.zeros((steps, len(layers)), np.int64)
        dev_step = [[0] * len(layers) for _ in range(steps + 1)]
        dev_step[0] = [ss.ss_dev_cache_total_misses(L.dev) if L.dev is not None else 0 for L in layers]
        t0 = time.perf_counter()
        for i in range(steps):
            s = 1 + i
            for l, L in enumerate(layers):
                run_step(L, l, s, events=[e.cuda_event if used[j] else None for j, e in enumerate(ev[i][l])]
                         if l in sampled else None)
                n_miss[i, l] = L.last_n_miss or 0
        if new_kv is not None:
            for L in layers:  # the last step's save is part of the work
                ss.ss_kv_save_wait(L.saver)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        for l, L in enumerate(layers):
            if L.dev is not None:  # the device resolve counts its misses on the GPU: spread the total over the steps
                n_miss[:, l] = (ss.ss_dev_cache_total_misses(L.dev) - dev_step[0][l]) / steps

        # --------------------------------------------------- accounting
        # Gathers of consecutive groups overlap (two transfer streams), so the
        # link's busy time is the union of the gather intervals of a step.  Also
        # per step: the ramp before the first gather starts, idle gaps inside
        # the gather span, and the tail after the last gather ends.
        pipe = {"ramp": [], "link_busy": [], "link_gaps": [], "tail": []}
        gather_launch_ms = []
        for i in range(steps):
            for l in sampled:  # layers are alike (same lengths, shapes and drift): the sampled ones stand for all
                e = ev[i][l]
                iv = sorted((e[0].elapsed_time(e[7 * p + 3]), e[0].elapsed_time(e[7 * p + 4])) for p in range(P))
                gather_launch_ms += [b - a for a, b in iv]
                busy, cur_a, cur_b = 0.0, iv[0][0], iv[0][1]
                for a, b in iv[1:]:
                    if a > cur_b:
                        busy += cur_b - cur_a
                        cur_a, cur_b = a, b
                    else:
                        cur_b = max(cur_b, b)
                busy += cur_b - cur_a
                first, last = iv[0][0], max(b for _, b in iv)
                pipe["ramp"].append(first)
                pipe["link_busy"].append(busy)
                pipe["link_gaps"].append(last - first - busy)
                pipe["tail"].append(e[0].elapsed_time(e[7 * (P - 1) + 6]) - last)
        pipe = {k: round(float(np.mean(v)), 4) for k, v in pipe.items()}
        # each step on its own: from the first layer's first event to the last
        # layer's last (GPU time; the wall-clock mean above includes host time
        # between steps)
        step_ms = np.array([ev[i][0][0].elapsed_time(ev[i][-1][7 * (P - 1) + 6]) for i in range(steps)])
        units = cfg.B * cfg.Hkv
        # the gather's algorithmic bytes per step: the missed block records (mean
        # over the timed steps) over the host link, against the link's busy time
        gather_bytes = float(n_miss.sum()) / steps * cfg.record_bytes
        busy_ms = pipe["link_busy"] * len(layers)
        ach = gather_bytes / (busy_ms * 1e-3) / 1e9 if busy_ms > 0 else 0.0
        key = (cfg.name, args.seed, steps, tuple(layers[0].part_sizes), resolve)
        value = cfg.B * steps / wall
        miss_rate = float(n_miss.mean()) / (units * cfg.k)
        log(f"{cfg.name}: {value:.0f} tokens/s, {wall / steps * 1e3:.3f} ms/step; gather {ach:.1f} GB/s; "
            f"miss rate {miss_rate:.4f}; pipeline {pipe}")
        res.update({
            "value": round(value, 2), "ms_per_step": round(wall / steps * 1e3, 4),
            "config": {"workload": cfg.name, "batch": cfg.B, "q_heads": cfg.Hq, "kv_heads": cfg.Hkv, "head_dim": D,
                       "context": int(lens.max()), "block": cfg.blk, "topk_blocks": cfg.k,
                       "cache_frac": cfg.cache_frac, "layers": cfg.layers,
                       "layers_with_own_dram_records": n_distinct, "drift": cfg.drift, "seed": args.seed,
                       "resolve": resolve},
            "roofline": {"kernel": "gather", "bound": "host-link", "achieved": round(ach, 2),
                         "peak": round(LINK_PEAK_GBS, 2), "unit": "GB/s", "frac": round(ach / LINK_PEAK_GBS, 4),
                         "bytes_per_step": int(gather_bytes), "link_busy_ms_per_step": round(busy_ms, 4),
                         "launches_per_step": len(layers) * P,
                         "ms_per_launch": round(float(np.mean(gather_launch_ms)), 4),
                         "traffic": traffic("gather", key)},
            "pipeline_ms": pipe,
            "step_ms_events": {"median": round(float(np.median(step_ms)), 4), "min": round(float(step_ms.min()), 4),
                               "max": round(float(step_ms.max()), 4),
                               "p90": round(float(np.percentile(step_ms, 90)), 4)},
            "parts": layers[0].part_sizes,
            "miss_rate": round(miss_rate, 4),
            "miss_rate_per_step": [round(float(x), 4) for x in n_miss.mean(axis=1) / (units * cfg.k)],
        })
        if new_kv is not None:
            L = layers[0]
            res["config"]["with_save"] = True
            res["save_side"] = {"blocks_filled_per_sequence": int((L.nblk.cpu().numpy() - nblk).max()),
                                "overflow": int(L.overflow.item()),
                                "note": "each timed step also appends its new tokens (metadata on a fill) and "
                                        "saves them with FlashD2H; the last save is waited for inside the timed "
                                        "region"}

        # --------------------------------------- isolated kernel rates
        # Each kernel alone over the whole batch (one launch, nothing else on the
        # GPU), on the last timed step's data: the HBM kernels' own rates, which
        # the overlapped step hides behind the host-link gather.
        iso = isolated_rates(cfg, layers[0], qstreams[0][steps][1], ss, torch)
        for name in iso:
            iso[name]["traffic"] = traffic(name, key)
        res["rooflines_isolated"] = iso
        if not studies:
            return res
        run_studies()
        return res
    finally:
        for L in layers:
            L.close()
        pool.close()
        torch.cuda.synchronize()
        torch.cuda.empty_cache()


def union_ms(iv):
    """Busy time of a set of (start, end) intervals."""
    iv = sorted(iv)
    busy, a0, b0 = 0.0, iv[0][0], iv[0][1]
    for a, b in iv[1:]:
        if a > b0:
            busy += b0 - a0
            a0, b0 = a, b
        else:
            b0 = max(b0, b)
    return busy + b0 - a0


def timed_groups(cfg, layers, qstreams, steps, resolve, args, torch, ss, H, lens, n_distinct):
    """The timed steps with the sequence groups pipelined across layers (one
    ss_decode_step_dev call per step).  Every gather of every layer carries
    start/end events on its own dispatch; the step's start and end are
    events on the caller's stream around the call."""
    P = layers[0].parts
    n = len(layers)
    dev = layers[0].dev is not None
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2 * n * P + 2)] for _ in range(steps)]
    for row in ev:  # create the underlying events before timing
        for e in row:
            e.record()
    torch.cuda.synchronize()
    tot0 = [ss.ss_dev_cache_total_misses(L.dev) for L in layers] if dev else None
    host_miss = 0  # the host resolve returns its misses with each call
    t0 = time.perf_counter()
    for i in range(steps):
        s = 1 + i
        e = ev[i]
        e[-2].record()
        H.decode_step_groups(layers, s, [qstreams[l][s][1] for l in range(n)],
                             events=[x.cuda_event for x in e[:2 * n * P]])
        e[-1].record()
        if not dev:
            host_miss += sum(L.last_n_miss for L in layers)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    if dev:
        miss = sum(ss.ss_dev_cache_total_misses(L.dev) - m0 for L, m0 in zip(layers, tot0)) / steps
    else:
        miss = host_miss / steps
    pipe = {"ramp": [], "link_busy": [], "link_gaps": [], "tail": []}
    gather_launch_ms, step_ms = [], []
    for i in range(steps):
        e = ev[i]
        st = e[-2]
        iv = [(st.elapsed_time(e[2 * j]), st.elapsed_time(e[2 * j + 1])) for j in range(n * P)]
        gather_launch_ms += [b - a for a, b in iv]
        busy = union_ms(iv)
        first, last = min(a for a, _ in iv), max(b for _, b in iv)
        end = st.elapsed_time(e[-1])
        step_ms.append(end)
        pipe["ramp"].append(first)
        pipe["link_busy"].append(busy)
        pipe["link_gaps"].append(last - first - busy)
        pipe["tail"].append(end - last)
    per_step = {k: float(np.mean(v)) for k, v in pipe.items()}
    step_ms = np.array(step_ms)
    units = cfg.B * cfg.Hkv
    gather_bytes = miss * cfg.record_bytes
    busy_ms = per_step["link_busy"]
    ach = gather_bytes / (busy_ms * 1e-3) / 1e9 if busy_ms > 0 else 0.0
    value = cfg.B * steps / wall
    miss_rate = miss / (n * units * cfg.k)
    pipe_layer = {k: round(v / n, 4) for k, v in per_step.items()}
    log(f"{cfg.name} (groups across layers): {value:.0f} tokens/s, {wall / steps * 1e3:.3f} ms/step; gather "
        f"{ach:.1f} GB/s; miss rate {miss_rate:.4f}; per step {per_step}")
    return {
        "value": round(value, 2), "ms_per_step": round(wall / steps * 1e3, 4),
        "config": {"workload": cfg.name, "batch": cfg.B, "q_heads": cfg.Hq, "kv_heads": cfg.Hkv, "head_dim": D,
                   "context": int(lens.max()), "block": cfg.blk, "topk_blocks": cfg.k, "cache_frac": cfg.cache_frac,
                   "layers": cfg.layers, "layers_with_own_dram_records": n_distinct, "drift": cfg.drift,
                   "seed": args.seed, "resolve": resolve, "schedule": "groups"},
        "roofline": {"kernel": "gather", "bound": "host-link", "achieved": round(ach, 2),
                     "peak": round(LINK_PEAK_GBS, 2), "unit": "GB/s", "frac": round(ach / LINK_PEAK_GBS, 4),
                     "bytes_per_step": int(gather_bytes), "link_busy_ms_per_step": round(busy_ms, 4),
                     "launches_per_step": n * P, "ms_per_launch": round(float(np.mean(gather_launch_ms)), 4),
                     "traffic": None},
        "pipeline_ms": pipe_layer,
        "pipeline_ms_per_step": {k: round(v, 4) for k, v in per_step.items()},
        "step_ms_events": {"median": round(float(np.median(step_ms)), 4), "min": round(float(step_ms.min()), 4),
                           "max": round(float(step_ms.max()), 4), "p90": round(float(np.percentile(step_ms, 90)), 4)},
        "parts": layers[0].part_sizes,
        "miss_rate": round(miss_rate, 4),
        "miss_rate_per_step": None,
    }


def metadata_build_rate(cfg, pool, L0, nblk, ss, torch):
    """The metadata build (setup path, when blocks fill) timed alone on one
    sequence's records copied to HBM."""
    kv_one = torch.empty(cfg.Hkv * int(nblk[0]) * cfg.record_bytes, dtype=torch.uint8, device="cuda")
    kv_one.copy_(pool.t[int(L0.pool_off_host[0]):int(L0.pool_off_host[0]) + kv_one.numel()])
    off1 = torch.from_numpy(np.arange(cfg.Hkv, dtype=np.int64) * int(nblk[0]) * cfg.record_bytes).cuda()
    n1 = torch.tensor([int(nblk[0])], dtype=torch.int32, device="cuda")
    meta1 = torch.empty(cfg.Hkv, cfg.nblk_max, 2, D, dtype=torch.int16, device="cuda")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    meta_ms = []
    for _ in range(3):
        e0.record()
        ss.ss_build_metadata(kv_one, off1, n1, 1, cfg.Hkv, cfg.nblk_max, cfg.blk, D, meta1)
        e1.record()
        torch.cuda.synchronize()
        meta_ms.append(e0.elapsed_time(e1))
    meta_bytes = cfg.Hkv * int(nblk[0]) * (cfg.blk * D * 2 + 2 * D * 2)
    ms = float(np.median(meta_ms))
    return {"ms": round(ms, 4), "bytes": meta_bytes, "GBps": round(meta_bytes / (ms * 1e-3) / 1e9, 1),
            "note": "setup path (when blocks fill), one sequence, not in the step"}


def _read(path):
    try:
        with open(path) as fh:
            return fh.read().strip()
    except OSError:
        return None


def host_facts():
    """The GPU's PCIe link as negotiated (each device on the path from the
    GPU to the root port: speed and width now and at most) and the host's
    CPUs (count, affinity, cgroup quota, model)."""
    import ctypes
    facts = {}
    try:
        hip = ctypes.CDLL("libamdhip64.so")
        buf = ctypes.create_string_buffer(64)
        dev = ctypes.c_int(0)
        hip.hipGetDevice(ctypes.byref(dev))
        if hip.hipDeviceGetPCIBusId(buf, 64, dev) == 0:
            bus = buf.value.decode().lower()
            path = os.path.realpath(f"/sys/bus/pci/devices/{bus}")
            chain = []
            while os.path.basename(path).count(":") == 2:  # PCI addresses dddd:bb:dd.f
                chain.append({"device": os.path.basename(path),
                              "current_link_speed": _read(os.path.join(path, "current_link_speed")),
                              "current_link_width": _read(os.path.join(path, "current_link_width")),
                              "max_link_speed": _read(os.path.join(path, "max_link_speed")),
                              "max_link_width": _read(os.path.join(path, "max_link_width"))})
                path = os.path.dirname(path)
            facts["pcie_bus_id"] = bus
            facts["pcie_path_gpu_to_root"] = chain
    except OSError as e:
        facts["pcie_error"] = str(e)
    facts["os_cpu_count"] = os.cpu_count()
    facts["affinity_cpus"] = len(os.sched_getaffinity(0))
    quota = _read("/sys/fs/cgroup/cpu.max")
    if quota:
        facts["cgroup_cpu_max"] = quota
        q, per = quota.split()[:2]
        if q != "max":
            facts["cgroup_cpus"] = round(int(q) / int(per), 2)
    info = {}
    try:
        for line in open("/proc/cpuinfo"):
            if ":" not in line:
                if info:
                    break
                continue
            k, v = (x.strip() for x in line.split(":", 1))
            if k in ("vendor_id", "cpu family", "model", "model name", "stepping") and k not in info:
                info[k] = v
    except OSError:
        pass
    facts["cpu"] = info
    return facts


def exit_report():
    """Lists what is still alive as the script ends (child processes,
    threads), so a run that leaves anything behind shows it on stderr."""
    import threading
    try:
        import psutil
        kids = [f"{c.pid}:{c.name()}" for c in psutil.Process().children(recursive=True)]
    except Exception as e:  # psutil missing or a process gone meanwhile
        kids = [f"unknown ({e})"]
    threads = [t.name for t in threading.enumerate() if t is not threading.main_thread()]
    log(f"exit: child processes {kids or 'none'}; Python threads {threads or 'none'}")


# ------------------------------------------------------- HBM traffic
# Measured HBM bytes of the step's kernels: two rocprofv3 --pmc runs of this
# script with default arguments (FETCH_SIZE, then WRITE_SIZE, KiB per
# dispatch), each counter scaled by what it reads for a plain copy of known
# size (--calibrate-copy), written by --summarize-pmc.  A figure is reported
# only for the workload and arguments it was taken with, and only while the
# sources of its kernel hash as they did then; otherwise traffic is null.
KERNEL_SOURCES = {
    "gather": ["gather.hip", "decode.cpp"],
    "score": ["score.hip"],
    "topk": ["topk.hip"],
    "attention": ["attention.hip"],
}
# hierarchical 128k-context layer, seed 0, 20 timed steps (the driver's --steps 20 --warmup 5), groups
# 2,4,10,20,18,8,2, host resolve
_KEY = ["hier-b64-ctx128k-blk16-k128-cache25", 0, 20, [2, 4, 10, 20, 18, 8, 2], "host"]
TRAFFIC = {
    "gather": {"key": _KEY, "digest": "fc3ee5fdc0ce0be4", "bytes": 245801680, "fetch": 123714256,
              "write": 122087424},
    "score": {"key": _KEY, "digest": "c9510f2bf97a7ac5", "bytes": 2168521631, "fetch": 2151712671,
              "write": 16808960},
    "topk": {"key": _KEY, "digest": "1d38913edab606c6", "bytes": 17217148, "fetch": 16955004,
              "write": 262144},
    "attention": {"key": _KEY, "digest": "9e23bba1c2251224", "bytes": 539142308, "fetch": 538093732,
              "write": 1048576},
}


def source_digest(kernel):
    import hashlib
    h = hashlib.sha256()
    base = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2509_24626_amd", "csrc")
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(base, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic(kernel, key):
    rec = TRAFFIC.get(kernel)
    norm = lambda k: (k[0], int(k[1]), int(k[2]), tuple(int(x) for x in k[3]), k[4])
    if not rec or norm(rec["key"]) != norm(key):
        return None
    if rec["digest"] != source_digest(kernel):
        return None
    return rec["bytes"]


def calibrate_copy(reps=5):
    """A plain copy of known size for scaling the traffic counters: 1 GiB
    read and 1 GiB written per launch (an elementwise multiply by 1)."""
    import torch
    n = 1 << 28
    src = torch.empty(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1.0)
    for _ in range(reps):
        torch.mul(src, 1.0, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": n * 4, "launches": reps}), flush=True)


def _pmc_rows(folder, counter):
    """Per-dispatch (kernel name, grid size, value) of one counter, in
    dispatch order, from a rocprofv3 csv output folder."""
    import csv
    import glob
    files = sorted(glob.glob(os.path.join(folder, "**", "*counter_collection.csv"), recursive=True))
    if not files:
        raise SystemExit(f"no counter_collection.csv under {folder}")
    rows = {}
    for f in files:
        with open(f, newline="") as fh:
            for r in csv.DictReader(fh):
                if r.get("Counter_Name") != counter:
                    continue
                did = int(r["Dispatch_Id"])
                name, grid, val = r["Kernel_Name"], int(r.get("Grid_Size", 0) or 0), float(r["Counter_Value"])
                if did in rows:
                    val += rows[did][2]
                rows[did] = (name, grid, val)
    return [rows[k] for k in sorted(rows)]


def summarize_pmc(args):
    fetch_dir, write_dir, cf_dir, cw_dir = args.summarize_pmc
    with open(args.bench_json) as fh:
        bench = json.loads([ln for ln in fh if ln.startswith("{")][-1])
    scale = {}
    for c, folder in (("FETCH_SIZE", cf_dir), ("WRITE_SIZE", cw_dir)):
        vals = [v for n, _, v in _pmc_rows(folder, c) if "Mul" in n]
        if not vals:
            raise SystemExit(f"no copy kernel dispatches in {folder}")
        scale[c] = (1 << 30) / (float(np.median(vals)) * 1024)
    P = len(bench["parts"]) * bench["config"]["layers"]
    steps, warmup = bench["steps"], bench["warmup"]
    out = {}
    lines = []
    for c, folder in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        rows = _pmc_rows(folder, c)
        g = [v for n, _, v in rows if "gather_kernel" in n or "gather_units_kernel" in n]
        assert len(g) == (warmup + steps) * P, (len(g), warmup, steps, P)
        timed = g[warmup * P:]
        per_step = sum(timed) / steps * 1024 * scale[c]
        out.setdefault("gather", {})[c] = per_step
        for name, tag in (("score", "score_kernel"), ("topk", "topk_kernel"), ("attention", "attn_kernel")):
            # the isolated full-batch launches are each kernel's last 10 dispatches
            vals = [v for n, _, v in rows if tag in n][-10:]
            out.setdefault(name, {})[c] = float(np.median(vals)) * 1024 * scale[c]
    key = [bench["config"]["workload"], bench["config"]["seed"], steps, bench["parts"],
           bench["config"].get("resolve", "host")]
    algo = {"gather": bench["roofline"]["bytes_per_step"]}
    for name in ("score", "topk", "attention"):
        algo[name] = bench["rooflines_isolated"][name]["bytes_per_launch"]
    lines.append(f"copy-kernel scale: FETCH_SIZE x{scale['FETCH_SIZE']:.4f}, WRITE_SIZE x{scale['WRITE_SIZE']:.4f}")
    lines.append("")
    lines.append("| kernel | unit | fetched bytes | written bytes | traffic | algorithmic bytes | traffic / algorithmic |")
    lines.append("|---|---|---|---|---|---|---|")
    table = {}
    for name, v in out.items():
        t = v["FETCH_SIZE"] + v["WRITE_SIZE"]
        unit = "per step (all gather launches)" if name == "gather" else "per launch (isolated, full batch)"
        lines.append(f"| {name} | {unit} | {v['FETCH_SIZE']:.4g} | {v['WRITE_SIZE']:.4g} | {t:.4g} | {algo[name]:.4g} "
                     f"| {t / algo[name]:.3f} |")
        table[name] = {"key": key, "digest": source_digest(name), "bytes": int(round(t)),
                       "fetch": int(round(v["FETCH_SIZE"])), "write": int(round(v["WRITE_SIZE"]))}
    print("\n".join(lines))
    print()
    print("TRAFFIC = " + json.dumps(table, indent=1))


def score_variants_study(cfg, L, q, pool, ss, torch, reps=5):
    """The metadata kinds and GQA aggregations (Section 2.2).

    Speed: each scoring kernel alone over this layer's whole batch and
    query (after a cache flush; kernel-attached events).

    Quality: on the Llama-3-8B-shaped all-HBM layer (32 sequences, 32k
    context, 64 planted critical blocks per KV head; the timed workload's
    random keys have no critical blocks to find), the top-k of each variant
    against (a) the planted blocks and (b) the exact softmax attention mass
    of sampled (sequence, KV head) units (all tokens, each query head,
    averaged) that falls in the selected blocks; the exact top-k by block
    maximum max_h max_t q_h.k_t is the reference selection."""
    import synth
    from synth import gen
    import paper_2509_24626_amd.harness as Hm
    if L.meta_kind != 0:
        return None
    B, Hq, Hkv, k, blk = cfg.B, cfg.Hq, cfg.Hkv, cfg.k, cfg.blk
    nmax = L.nblk_max
    flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    flush.fill_(1.0)
    mean = torch.empty(B, Hkv, nmax, D, dtype=torch.int16, device="cuda")
    ss.ss_build_metadata_mean(pool.dev, L.pool_off, L.nblk, B, Hkv, nmax, blk, D, mean)  # from mapped DRAM
    metas = {0: L.meta, 1: mean}
    scores = torch.empty(B, Hkv, nmax, dtype=torch.float32, device="cuda")
    res = {}
    for kind, kname in ((0, "cuboid"), (1, "mean")):
        row_bytes = (2 if kind == 0 else 1) * D * 2
        nbytes = int(L.nblk_host.sum()) * Hkv * (row_bytes + 4) + B * Hq * D * 2
        for agg, aname in ((0, "max"), (1, "sum")):
            ts = []
            for _ in range(reps):
                flush.sum()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                e1.record()
                ss.ss_time_next_kernel(e0, e1)
                ss.ss_score_blocks_variant(q, metas[kind], kind, agg, L.nblk, B, Hq, Hkv, nmax, D, scores)
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1))
            ms = float(np.median(ts))
            res[f"{kname}-{aname}"] = {"ms": round(ms, 4), "GBps": round(nbytes / (ms * 1e-3) / 1e9, 1),
                                       "frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    del mean, metas, scores, flush

    qc = synth.get(1)
    seed = 0
    HL, _, qq = Hm.build_hbm_layer(qc, seed)
    Bq, G = qc.B, qc.G
    nq = qc.nblk_max
    mean = torch.empty(Bq, qc.Hkv, nq, D, dtype=torch.int16, device="cuda")
    ss.ss_build_metadata_mean(HL.kv, HL.unit_off, HL.nblk, Bq, qc.Hkv, nq, qc.blk, D, mean)
    metas = {0: HL.meta, 1: mean}
    sc = torch.empty(Bq, qc.Hkv, nq, dtype=torch.float32, device="cuda")
    sel = torch.empty(Bq, qc.Hkv, qc.k, dtype=torch.int32, device="cuda")
    qh = qq.float().cpu().numpy()
    refs = []
    for b, g in ((0, 0), (7, 3), (15, 5), (23, 1), (31, 7)):
        K = HL.kv[b, g, :, :qc.blk * D].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        Kf = (K.astype(np.uint32) << 16).view(np.float32).reshape(nq * qc.blk, D)
        z = qh[b, g * G:(g + 1) * G] @ Kf.T
        p = np.exp((z - z.max(axis=1, keepdims=True)) / math.sqrt(D))
        mass = (p / p.sum(axis=1, keepdims=True)).reshape(G, nq, qc.blk).sum(axis=2)
        best = z.reshape(G, nq, qc.blk).max(axis=2).max(axis=0)
        top = set(np.argsort(-best, kind="stable")[:qc.k].tolist())
        exact_mass = float(mass[:, sorted(top)].sum(axis=1).mean())
        refs.append((b, g, mass, top, exact_mass))
    planted = {(b, g): set(gen.planted_blocks(nq, qc.n_plant, seed, 0, b, g, "cuda").cpu().tolist())
               for b in range(Bq) for g in range(qc.Hkv)}
    for kind, kname in ((0, "cuboid"), (1, "mean")):
        for agg, aname in ((0, "max"), (1, "sum")):
            ss.ss_score_blocks_variant(qq, metas[kind], kind, agg, HL.nblk, Bq, qc.Hq, qc.Hkv, nq, D, sc)
            ss.ss_select_topk(sc, HL.nblk, Bq, qc.Hkv, nq, qc.k, sel)
            sh = sel.cpu().numpy()
            rec_planted = float(np.mean([len(planted[(b, g)] & set(sh[b, g].tolist())) / qc.n_plant
                                         for b in range(Bq) for g in range(qc.Hkv)]))
            mass_rec = [float(m[:, sh[b, g][sh[b, g] >= 0]].sum(axis=1).mean()) for b, g, m, _, _ in refs]
            top_rec = [len(t & set(sh[b, g].tolist())) / len(t) for b, g, _, t, _ in refs]
            res[f"{kname}-{aname}"].update({"planted_recall": round(rec_planted, 4),
                                            "attention_mass_in_selection": round(float(np.mean(mass_rec)), 4),
                                            "exact_topk_overlap": round(float(np.mean(top_rec)), 4)})
    res["exact_topk_attention_mass"] = round(float(np.mean([r[4] for r in refs])), 4)
    res["quality_workload"] = f"{qc.name}, seed {seed}; attention mass over {len(refs)} sampled units"
    del HL, mean, metas, sc, sel
    torch.cuda.empty_cache()
    log(f"score variants: {res}")
    return res


def working_set_study(cfg, L, q32, first_step, seed, ss, torch, steps=28, window=12):
    """Decoding working sets on the workload itself (Section 3.3), after the
    timed region: `steps` more decode steps with the query drift continuing.
    Each step's selection (its host copy) goes to a working-set tracker; the
    figures are the tracker's cost per layer-step and per estimate, the
    working sets (window 12), Algorithm 1 against the layer's HBM cache, and
    the mean overlap between each step's selection and the union of the
    preceding w steps' selections (the paper's Figure 7 measurement, on
    synthetic data), for steps after the first 16."""
    from synth import gen
    B, Hkv, k = cfg.B, cfg.Hkv, cfg.k
    ids = np.arange(B, dtype=np.int64)
    tr = ss.ss_ws_create(1, Hkv, window, cfg.record_bytes)
    hist = []
    obs_ms = []
    try:
        for i in range(steps):
            q32, q = gen.drift(q32, cfg.drift, seed, 0, first_step + i)
            L.step(first_step + i, q)
            torch.cuda.synchronize()
            sel = L.sel.cpu().numpy()  # the device copy: both resolve paths write it
            hist.append(sel)
            t0 = time.perf_counter()
            ss.ss_ws_observe(tr, 0, first_step + i, ids, sel)
            obs_ms.append((time.perf_counter() - t0) * 1e3)
        t0 = time.perf_counter()
        ws = ss.ss_ws_decode_bytes(tr, ids)
        est_ms = (time.perf_counter() - t0) * 1e3
        cache_bytes = int(L.capacity.astype(np.int64).sum()) * cfg.record_bytes
        admit, used = ss.ss_schedule_batch(ws, cache_bytes)
        # a tighter HBM budget: a quarter of the cache
        admit_q, used_q = ss.ss_schedule_batch(ws, cache_bytes // 4)
    finally:
        ss.ss_ws_destroy(tr)
    overlap = {}
    H = np.stack(hist)  # [steps][B][Hkv][k]
    for w in (1, 2, 4, 8, 12, 16):
        fr = []
        for t in range(16, steps):
            for b in range(B):
                for g in range(Hkv):
                    cur = H[t, b, g]
                    cur = cur[cur >= 0]
                    prev = np.unique(H[max(0, t - w):t, b, g])
                    fr.append(np.isin(cur, prev).mean() if cur.size else 1.0)
        overlap[str(w)] = round(float(np.mean(fr)), 4)
    blocks = ws / cfg.record_bytes / Hkv
    res = {"window": window, "observe_ms_per_layer_step": round(float(np.median(obs_ms[2:])), 4),
           "estimate_ms_for_batch": round(est_ms, 4),
           "ws_blocks_per_head": {"mean": round(float(blocks.mean()), 1), "min": int(blocks.min()),
                                  "max": int(blocks.max()), "k": k},
           "ws_bytes_total": int(ws.sum()), "hbm_cache_bytes": cache_bytes,
           "alg1_admitted_full_cache": int(admit.sum()), "alg1_admitted_quarter_cache": int(admit_q.sum()),
           "overlap_with_preceding_window": overlap, "steps": steps}
    log(f"working sets: {res}")
    return res


def batch_control_study(cfg, L, pool, ss, torch, H, seed, window=12, fill=16, timed=8, budget_frac=0.5):
    """Working-set-aware batch control (Section 3.3, Algorithm 1) with the
    decode step itself.  The batch's decoding working sets (window 12) are
    estimated from `window` steps of the whole batch on this layer; the HBM
    budget for the block caches is then set to `budget_frac` of their sum.
    Two runs share that budget, split evenly over the running requests'
    (sequence, KV head) units:
      no_control  every request runs; each unit gets budget / (B * Hkv)
                  slots, fewer than its working set
      alg1        the requests Algorithm 1 admits run; each unit gets
                  budget / (admitted * Hkv) slots
    Each run starts from an empty cache, fills it over `fill` steps and
    times `timed` more (the same drifting queries for both); misses come
    from the GPU resolve's own count.  The layer's DRAM records and
    metadata are shared, so the study allocates only the caches."""
    import dataclasses
    B, Hkv, k, rb = cfg.B, cfg.Hkv, cfg.k, cfg.record_bytes
    qs = H.query_stream(cfg, seed + 7, 0, window + fill + timed)
    ids = np.arange(B, dtype=np.int64)
    first = 1 << 20  # step numbers after any the layer's cache has seen
    tr = ss.ss_ws_create(1, Hkv, window, rb)
    try:
        for t in range(window):
            L.step(first + t, qs[t][1])
            torch.cuda.synchronize()
            ss.ss_ws_observe(tr, 0, t, ids, L.sel.cpu().numpy())
        ws = ss.ss_ws_decode_bytes(tr, ids)
    finally:
        ss.ss_ws_destroy(tr)
    budget = int(budget_frac * ws.sum())
    admit, used = ss.ss_schedule_batch(ws, budget)
    out = {"window": window, "ws_bytes_total": int(ws.sum()), "budget_bytes": budget,
           "admitted": int(admit.sum()), "fill_steps": fill, "timed_steps": timed}
    for name, idx in (("no_control", np.arange(B)), ("alg1", np.nonzero(admit)[0])):
        n = len(idx)
        if n == 0:
            out[name] = None
            continue
        nb = L.nblk_host[idx]
        slots = np.minimum(np.maximum(budget // (n * Hkv * rb), np.minimum(k, nb)), nb)
        units = (idx[:, None] * Hkv + np.arange(Hkv)).reshape(-1)
        meta = L.meta if n == B else L.meta[torch.from_numpy(idx).cuda()].contiguous()
        parts = H.ramp_parts(n) if n >= 40 else max(1, min(4, round(n / 5)))
        Ln = H.HierLayer(dataclasses.replace(cfg, B=n), nb, np.repeat(slots, Hkv).astype(np.int32), pool,
                         L.pool_off_host[units], meta, parts, dev_cache=True)
        qi = torch.from_numpy(idx).cuda()
        try:
            for t in range(fill):
                Ln.step(t, qs[window + t][1].index_select(0, qi))
            torch.cuda.synchronize()
            m0 = ss.ss_dev_cache_total_misses(Ln.dev)
            t0 = time.perf_counter()
            for t in range(fill, fill + timed):
                Ln.step(t, qs[window + t][1].index_select(0, qi))
            torch.cuda.synchronize()
            wall = time.perf_counter() - t0
            m = ss.ss_dev_cache_total_misses(Ln.dev) - m0
        finally:
            Ln.close()
        out[name] = {"requests": n, "slots_per_head": int(slots.min()), "cache_bytes": int(slots.sum()) * Hkv * rb,
                     "miss_rate": round(m / (timed * n * Hkv * k), 4),
                     "block_loads_per_step": round(m / timed, 1),
                     "ms_per_step": round(wall / timed * 1e3, 4), "tokens_per_s": round(n * timed / wall, 1)}
    log(f"batch control: {out}")
    return out


def prefill_study(ss, torch, H, T=131072, layers=8, Hkv=8, blk=16):
    """The saving side of a layer-segmented prefill (Section 3.4) of one
    128k-token prompt: per plan item, metadata of the completed blocks built
    from the layer's token-major KV in HBM and a FlashD2H save of its tokens
    (8 host threads); every layer takes the same KV so that only this side
    is timed.  One layer's KV (T x Hkv x 512 B) is in HBM at a time."""
    res = {"prompt_tokens": T, "layers": layers, "kv_heads": Hkv, "block": blk,
           "hbm_kv_bytes_one_layer": T * Hkv * 2 * D * 2, "hbm_kv_bytes_all_layers": T * Hkv * 2 * D * 2 * layers}
    for max_inject in (T, T // 4):
        ex = H.PrefillExecutor(T, layers, Hkv, blk, max_inject, seed=1, threads=8, same_kv=True)
        try:
            ex.run()  # warm-up (first touch of the staging memory)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            batches = ex.run()
            wall = time.perf_counter() - t0
        finally:
            ex.close()
        kv_bytes = res["hbm_kv_bytes_all_layers"]
        res[f"max_inject_{max_inject}"] = {"batches": batches, "ms": round(wall * 1e3, 2),
                                           "GBps_saved": round(kv_bytes / wall / 1e9, 2),
                                           "layer_tokens_per_s": round(T * layers / wall, 1)}
    log(f"prefill: {res}")
    return res


def load_comparison(cfg, L, pool, ss, torch, reps=3):
    """Loading one decode step's missed blocks into their HBM slots two ways
    (the comparison of Section 3.2.1): the last timed step's miss rows of
    this layer, each an 8 KiB (blk 16) record from the pinned DRAM pool.
      memcpy_per_block  one hipMemcpyAsync (host to device) per record, issued
                        from Python (~1 us of its overhead per call)
      flashh2d          the gather kernel over the same rows (ss_gather_blocks)
    Both rewrite the bytes the step already placed, so the cache is
    unchanged.  GB/s = record bytes / wall time from issue to completion
    (median of 3)."""
    import ctypes
    if L.dev is None:
        rows = L.miss_h.numpy()[:L.last_n_miss].copy()
    else:
        counts, per_unit, err = L.dev_miss_rows()
        rows = np.concatenate([per_unit[u, :counts[u]] for u in range(L.units)] + [np.zeros((0, 4), np.int32)])
    n = len(rows)
    if n == 0:
        return None
    rb = cfg.record_bytes
    u = rows[:, 0].astype(np.int64) * cfg.Hkv + rows[:, 1]
    src = [int(x) for x in pool.host + L.pool_off_host[u] + rows[:, 2].astype(np.int64) * rb]
    dst = [int(x) for x in L.cache.data_ptr() + L.cache_off_host[u] + rows[:, 3].astype(np.int64) * rb]
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipMemcpyAsync.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_void_p]
    hip.hipMemcpyAsync.restype = ctypes.c_int
    stream = torch.cuda.current_stream().cuda_stream
    nbytes = n * rb
    ts = []
    for _ in range(reps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for d_, s_ in zip(dst, src):
            if hip.hipMemcpyAsync(d_, s_, rb, 1, stream) != 0:
                raise RuntimeError("hipMemcpyAsync failed")
        torch.cuda.synchronize()
        ts.append(time.perf_counter() - t0)
    memcpy = nbytes / float(np.median(ts)) / 1e9
    miss = torch.from_numpy(rows).cuda()
    ts = []
    for _ in range(reps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ss.ss_gather_blocks(miss, n, pool.dev, L.pool_off, L.cache, L.cache_off, L.nblk, L.cap_dev, cfg.B, cfg.Hkv,
                            rb)
        torch.cuda.synchronize()
        ts.append(time.perf_counter() - t0)
    flash = nbytes / float(np.median(ts)) / 1e9
    res = {"records": n, "record_bytes": rb, "memcpy_per_block_GBps": round(memcpy, 2),
           "flashh2d_GBps": round(flash, 2), "speedup": round(flash / memcpy, 2)}
    log(f"loading {n} records: {res}")
    return res


def save_bandwidth(ss, torch, H, B=4, n=8192, Hkv=8, reps=3, comparisons=False):
    """Saving a prefill-sized batch of new KV (B sequences x n tokens x Hkv
    heads, 128 MiB) to a pinned DRAM pool as block records, for blocks of 8,
    16 and 32 tokens (Section 3.2.2):
      flashd2h   one device-to-host copy of the contiguous tensor, then the
                 library's host threads place the tokens (ss_kv_save)
    and, with `comparisons`, the paper's alternatives:
      per_block  one hipMemcpyAsync per block record from HBM (issued from
                 Python; ~1 us of its overhead per call)
      gpu_direct a kernel stores the records into mapped host memory (the
                 gather kernel with source and destination swapped)
    GB/s = new-KV bytes / wall time from issue to completion (median of 3)."""
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipMemcpyAsync.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_void_p]
    hip.hipMemcpyAsync.restype = ctypes.c_int
    nbytes = B * n * Hkv * 2 * D * 2
    kv = torch.randint(-16000, 16000, (B, n, Hkv, 2, D), dtype=torch.int16, device="cuda")
    rec_dev = torch.randint(-16000, 16000, (nbytes // 2,), dtype=torch.int16, device="cuda")
    pool = H.HostPool(nbytes)
    res = {"bytes": nbytes, "threads": 8}
    try:
        for blk in (8, 16, 32):
            rb = 2 * blk * D * 2
            nb = n // blk
            units = B * Hkv
            off = np.arange(units, dtype=np.int64) * nb * rb
            out = {}
            saver = ss.ss_kv_saver_create(B, Hkv, blk, D, pool.host, off, np.full(B, nb, np.int32), n, 1, 8)
            try:
                ts = []
                for r in range(reps + 1):  # the first, untimed, also lets idle worker threads settle
                    torch.cuda.synchronize()
                    t0 = time.perf_counter()
                    ss.ss_kv_save(saver, kv, n, np.zeros(B, np.int32))
                    ss.ss_kv_save_wait(saver)
                    if r:
                        ts.append(time.perf_counter() - t0)
                out["flashd2h"] = round(nbytes / float(np.median(ts)) / 1e9, 2)
            finally:
                ss.ss_kv_saver_destroy(saver)
            if not comparisons:
                res[f"blk{blk}"] = out
                log(f"saving {nbytes >> 20} MiB, blk {blk}: {out} GB/s")
                continue
            stream = torch.cuda.current_stream().cuda_stream
            src0 = rec_dev.data_ptr()
            ts = []
            for _ in range(reps):
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                for u in range(units):
                    for j in range(nb):
                        o = int(off[u]) + j * rb
                        if hip.hipMemcpyAsync(pool.host + o, src0 + o, rb, 2, stream) != 0:
                            raise RuntimeError("hipMemcpyAsync failed")
                torch.cuda.synchronize()
                ts.append(time.perf_counter() - t0)
            out["per_block"] = round(nbytes / float(np.median(ts)) / 1e9, 2)
            rows = torch.from_numpy(np.stack(np.meshgrid(np.arange(B), np.arange(Hkv), np.arange(nb), indexing="ij"),
                                             -1).reshape(-1, 3)).to(torch.int32)
            miss = torch.cat([rows, rows[:, 2:3]], 1).contiguous().cuda()  # (b, g, block, slot = block)
            off_dev = torch.from_numpy(off).cuda()
            nblk_dev = torch.full((B,), nb, dtype=torch.int32, device="cuda")
            cap_dev = torch.full((units,), nb, dtype=torch.int32, device="cuda")
            ts = []
            for _ in range(reps):
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                ss.ss_gather_blocks(miss, miss.shape[0], rec_dev, off_dev, pool.dev, off_dev, nblk_dev, cap_dev, B,
                                    Hkv, rb)
                torch.cuda.synchronize()
                ts.append(time.perf_counter() - t0)
            out["gpu_direct"] = round(nbytes / float(np.median(ts)) / 1e9, 2)
            res[f"blk{blk}"] = out
            log(f"saving {nbytes >> 20} MiB, blk {blk}: {out} GB/s")
    finally:
        pool.close()
    return res


def isolated_rates(cfg, L, q, ss, torch, reps=10):
    """Median duration of score, top-k and attention over the full batch,
    each launched alone after a cache flush, as a fraction of the HBM peak.
    The timing events are attached to the kernel dispatch itself
    (ss_time_next_kernel), so they bracket the kernel's execution without
    the queue's dispatch latency."""
    B, Hq, Hkv, k = cfg.B, cfg.Hq, cfg.Hkv, cfg.k
    nb = L.nblk_host
    blocks = int(nb.sum()) * Hkv
    valid = int((L.slots >= 0).sum().item())
    ws_bytes = ss.ss_sparse_attention_workspace(B, Hq, Hkv, D, cfg.blk, k)
    ws = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device="cuda")
    out = torch.empty(B, Hq, D, dtype=torch.float32, device="cuda")
    runs = {
        "score": (lambda: ss.ss_score_blocks(q, L.meta, L.nblk, B, Hq, Hkv, L.nblk_max, D, L.scores),
                  blocks * (2 * D * 2 + 4) + B * Hq * D * 2),
        "topk": (lambda: ss.ss_select_topk(L.scores, L.nblk, B, Hkv, L.nblk_max, k, L.sel),
                 blocks * 4 + B * Hkv * k * 4),
        "attention": (lambda: ss.ss_sparse_attention(q, L.cache, L.cache_off, L.slots, L.cap_dev, int(L.capacity.max()), B, Hq,
                                                     Hkv, D, cfg.blk, k, 1.0 / math.sqrt(D), out, ws, ws_bytes),
                      valid * cfg.record_bytes + B * Hq * D * (2 + 4)),
    }
    res = {}
    # a 1 GiB read before every timed launch evicts the 256 MB last-level
    # cache, so each launch streams its bytes from HBM
    flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    flush.fill_(1.0)
    for name, (fn, nbytes) in runs.items():
        ts = []
        for _ in range(reps):
            flush.sum()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()  # creates the events
            e1.record()
            ss.ss_time_next_kernel(e0, e1)
            fn()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        ms = float(np.median(ts))
        ach = nbytes / (ms * 1e-3) / 1e9
        res[name] = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(ach / HBM_PEAK_GBS, 4), "bytes_per_launch": int(nbytes), "ms_per_launch": round(ms, 4)}
    return res


def cpu_baseline(cfg, pool, L, qs, nblk, args):
    """The oracle on the first `cpu_seqs` sequences of layer 0: its own
    metadata (untimed), a cache-fill step (untimed), then `cpu_steps` timed
    steps of score, select, LRU resolve, gather and attention, one thread
    per sequence, on every CPU the process may run on."""
    import oracle
    from synth import gen
    O = oracle.Oracle()
    nseq = min(args.cpu_seqs, cfg.B)
    nsteps = min(args.cpu_steps, len(qs) - 1)
    allowed = len(os.sched_getaffinity(0))
    threads = min(allowed, nseq)
    rb, Hkv = cfg.record_bytes, cfg.Hkv
    qh = [gen.to_u16(qs[s][1]) for s in range(nsteps + 1)]
    log(f"cpu baseline: oracle on {nseq} sequences x {nsteps} steps, {threads} threads")

    def prepare(b):
        units = np.arange(b * Hkv, (b + 1) * Hkv)
        nb = nblk[b:b + 1]
        meta = O.build_metadata(pool.host, L.pool_off_host[units], nb, 1, Hkv, cfg.nblk_max, cfg.blk, D)
        cap = L.capacity[units]
        lru = O.lru(1, Hkv, nb, cap)
        img_off = np.concatenate([[0], np.cumsum(cap.astype(np.int64))[:-1]]) * rb
        img = np.zeros(int(cap.sum()) * rb + rb, np.uint8)
        state = dict(meta=meta, lru=lru, img=img, img_off=img_off, off=L.pool_off_host[units], nb=nb)
        step(b, state, 0)
        return state

    def step(b, st, s):
        q = qh[s][b:b + 1]
        S = O.score(q, st["meta"], st["nb"], cfg.Hq, Hkv, cfg.nblk_max, D)
        sel = O.select(S, st["nb"], cfg.k)
        slots, miss = st["lru"].step(s, sel)
        O.gather(miss, pool.host, st["off"], st["img"], st["img_off"], rb, Hkv)
        O.attention(q, st["img"], st["img_off"], slots, Hkv, cfg.blk)

    with ThreadPoolExecutor(threads) as ex:
        states = list(ex.map(prepare, range(nseq)))
        t0 = time.perf_counter()
        list(ex.map(lambda b: [step(b, states[b], s) for s in range(1, nsteps + 1)], range(nseq)))
        wall = time.perf_counter() - t0
    # the same steps on one thread, for a few fresh sequences
    n1 = min(4, nseq)
    states1 = [prepare(b) for b in range(n1)]
    t0 = time.perf_counter()
    for b in range(n1):
        for s in range(1, nsteps + 1):
            step(b, states1[b], s)
    wall1 = time.perf_counter() - t0
    hf = host_facts()
    return {"value": round(nseq * nsteps / wall, 3), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{nseq} of {cfg.B} sequences (all {Hkv} KV heads each) x {nsteps} decode steps of layer 0 "
                      f"after an untimed cache-fill step; score, select, LRU resolve, gather, attention; "
                      f"{wall:.2f} s wall, {threads} threads, one sequence per thread",
            "os_cpu_count": hf["os_cpu_count"], "affinity_cpus": allowed,
            "cgroup_cpus": hf.get("cgroup_cpus"), "cpu": hf["cpu"],
            "single_thread": {"value": round(n1 * nsteps / wall1, 3), "unit": "tokens/s", "cores": 1,
                              "sample": f"{n1} sequences x {nsteps} steps on one thread, {wall1:.2f} s"}}


if __name__ == "__main__":
    main()
