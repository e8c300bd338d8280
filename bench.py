#!/usr/bin/env python3
"""Throughput of the routed MoE FFN forward (EPS-MoE hot path) on one MI355X.

One step = one moe_ffn_forward over one batch of synthetic tokens: router,
dispatch, gather, expert GEMMs (GroupGemm or DenseGemm per stage), shared
experts when the workload has them, and the weighted combine.  Inputs are
resident in HBM before the timed region starts.

Default workload: Mixtral-8x7B-shaped tensor-parallel shard (16384 tokens,
hidden 4096, 8 experts, SwiGLU width 3584, top-2 renormalised), synthetic
Gaussian inputs.  Prints one JSON line; see --help for the other workloads
and the GroupGemm/DenseGemm load sweep.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "MoE FFN prefill tokens/sec on 1 MI355X; expert-GEMM % of bf16 MFMA peak"
PEAK_BF16_FLOPS = 2.5e15   # MI355X dense bf16 MFMA, published
PHASE_STEPS = 5            # steps with every phase timed, for the breakdown
PEAK_HBM_BYTES = 8.0e12    # MI355X HBM3E, published

WORKLOAD_TEXT = {
    "tiny": "tiny MoE FFN: T=512 H=256 E=8 I=512 top-2 renorm",
    "mixtral": "Mixtral-8x7B-shaped TP shard: T=16384 H=4096 E=8 I=3584 top-2 renorm",
    "dbrx": "DBRX-shaped TP shard: T=8192 H=6144 E=16 I=1344 top-4 renorm",
    "dsv2": "DeepSeekV2-shaped EP share: T=16384 H=5120 E=160 (20 local) I=1536 top-6 "
            "+ 2 shared experts I=1536",
    "zipf": "DeepSeekV2 local-expert shape, Zipf(1.2) expert popularity: H=5120 E=160 "
            "(20 local) I=1536 top-6",
    "mixtral_ep": "Mixtral-8x7B EP share (4 GPUs): T=16384 H=4096 E=8 (2 local) I=14336 "
                  "top-2 renorm",
    "dbrx_ep": "DBRX EP share (8 GPUs): T=8192 H=6144 E=16 (2 local) I=10752 top-4 renorm",
}


def parse_args(argv=None):
    p = argparse.ArgumentParser(description=__doc__,
                                formatter_class=argparse.RawDescriptionHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--config", default="mixtral", choices=sorted(WORKLOAD_TEXT))
    p.add_argument("--tokens", type=int, default=0, help="override T (zipf sweep point)")
    p.add_argument("--mode", default="auto", choices=["auto", "group", "dense"])
    p.add_argument("--pn", type=int, default=1,
                   help="pipeline number (divides the local experts for expert stages)")
    p.add_argument("--chunk-mode", default="experts", choices=["experts", "tokens"],
                   help="pipeline stages: expert groups (default) or token ranges")
    p.add_argument("--cu-budget", type=int, default=0)
    p.add_argument("--dense-min-rows", type=int, default=0)
    p.add_argument("--group-tile-rows", type=int, default=0,
                   help="force the GroupGemm tile height (128, 192, 256, 320; 0 = model)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="target CPU time of the oracle baseline sample")
    p.add_argument("--sweep", action="store_true",
                   help="GroupGemm vs DenseGemm vs AUTO over the zipf token counts")
    p.add_argument("--pn-sweep", action="store_true",
                   help="step time over pipeline numbers and both stage kinds for --config")
    p.add_argument("--pn-fit", action="store_true",
                   help="fit the paper's pipeline overhead model R(N) = kN + b from serial "
                        "stages of --config, choose PN with it and compare with the "
                        "measured best PN")
    p.add_argument("--cu-sweep", action="store_true",
                   help="step time of --config over grouped-GEMM CU budgets and PN")
    p.add_argument("--gemm-study", action="store_true",
                   help="GroupGemm throughput over group counts, rows per group and CU "
                        "budgets on the DeepSeekV2 expert shape")
    p.add_argument("--pn-enable", action="store_true",
                   help="the paper's pipeline enable condition over the zipf loads: eps0 and "
                        "eps1 per PN, measured (serial stages) and from the library's model")
    p.add_argument("--side-cus", type=int, default=0,
                   help="CUs of the CU-masked gather/combine streams (0: no masks)")
    p.add_argument("--trace-overlap", metavar="CSV", default="",
                   help="summarise a rocprofv3 kernel-trace CSV of pipelined forwards: when "
                        "each stage's combine ran against the next stage's GEMMs (no GPU)")
    p.add_argument("--trace-stats", metavar="CSV", default="",
                   help="per-kernel durations from a rocprofv3 kernel-trace CSV of a bench.py "
                        "run, over its timed forwards only (--warmup, --steps as in that "
                        "run; no GPU)")
    p.add_argument("--tile-study", action="store_true",
                   help="DenseGemm launch time of one expert for every tile height and "
                        "row count (the data of the launch-cost model)")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                   help="only run a plain device copy of BYTES (HBM counter calibration)")
    return p.parse_args(argv)


def gemm_flops(s, counts_total):
    """Algorithmic GEMM flops of one forward: gate+up 4*R*H*I, down 2*R*H*I,
    shared 6*T*H*Is."""
    R = counts_total
    routed_gateup = 4.0 * R * s.H * s.I
    routed_down = 2.0 * R * s.H * s.I
    shared = 6.0 * s.T * s.H * s.shared_inter
    return routed_gateup, routed_down, shared


def cpu_baseline(inp, target_s):
    """The oracle as it stands, on a bounded sample of the same workload:
    routing of the sampled tokens plus their full MoE FFN output."""
    import numpy as np

    import oracle

    s = inp.shape
    cores = len(os.sched_getaffinity(0))
    rng = np.random.default_rng(0)

    def run(n):
        tok = np.sort(rng.choice(s.T, size=n, replace=False))
        xs = inp.x[tok]
        t0 = time.perf_counter()
        _, ids, w = oracle.route(xs, inp.w_router, inp.bias, s.k, s.renorm)
        oracle.moe_tokens(xs, ids, w, np.arange(n), inp.w_gate, inp.w_up, inp.w_down, s.e0,
                          s.n_shared, inp.shared_gate, inp.shared_up, inp.shared_down)
        return time.perf_counter() - t0

    n = 16
    dt = run(n)
    if dt < target_s / 4:
        n = int(min(s.T, max(n, n * target_s / max(dt, 1e-3))))
        dt = run(n)
    return {"value": n / dt, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "cpu": cpu_model(),
            "sample": f"{n} of {s.T} tokens of the same workload (routing + MoE FFN output "
                      f"per token, fp64 expert rows), {dt:.1f} s wall"}


def cpu_model():
    """The host CPU's model name (first 'model name' line of /proc/cpuinfo)."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def copy_calibration(nbytes):
    import torch

    a = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1.0)
    torch.cuda.synchronize()
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": nbytes, "launches": 5}))


def run_workload(args, shape, inp, steps, warmup, timing=True, serial=False, dev_inputs=None):
    import torch

    from paper_2410_12247_amd import moe
    from paper_2410_12247_amd.workload import DeviceInputs

    mode = {"auto": moe.GEMM_AUTO, "group": moe.GEMM_GROUP, "dense": moe.GEMM_DENSE}[args.mode]
    chunk = {"experts": moe.CHUNK_EXPERTS, "tokens": moe.CHUNK_TOKENS}[args.chunk_mode]
    o = moe.opts(gemm_mode=mode, pipeline_n=args.pn, gemm_cu_budget=args.cu_budget,
                 dense_min_rows=args.dense_min_rows, timing=timing, chunk_mode=chunk,
                 serial=serial, side_cus=args.side_cus, group_tile_rows=args.group_tile_rows)
    g = dev_inputs if dev_inputs is not None else DeviceInputs(inp)
    buf = g.buffers(o)

    for _ in range(warmup):
        g.run(buf)
    torch.cuda.synchronize()
    if timing and warmup > 0:
        moe.last_timing()  # the record of the warm-up calls is dropped
    t0 = time.perf_counter()
    for _ in range(steps):
        g.run(buf)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # timed calls add up in the library until read: one read after the loop
    tms = [moe.last_timing()] if timing else []
    counts = buf.counts.cpu().numpy()
    return wall, tms, counts


def measured_traffic(workload, kernel_prefix):
    """HBM bytes per launch of a GEMM kernel from the committed rocprofv3
    counter summary (FETCH_SIZE / WRITE_SIZE scaled by the copy calibration),
    or None when the GEMM source changed since the counters were taken."""
    import hashlib

    path = os.path.join(ROOT, "profiles", f"{workload}_hbm_counters.json")
    if not os.path.exists(path):
        return None
    d = json.load(open(path))
    src = open(os.path.join(ROOT, "paper_2410_12247_amd", "csrc", "gemm.hip"), "rb").read()
    if d.get("gemm_source_sha256") != hashlib.sha256(src).hexdigest():
        return None
    # with shared experts the summary lists the routed launch separately
    keys = [k for k in d["kernels"] if k.startswith(kernel_prefix)]
    routed = [k for k in keys if k.endswith("(routed)")]
    for k in routed or keys:
        return d["kernels"][k]["bytes"]
    return None


def gateup_bytes(s, counts):
    """Algorithmic HBM bytes of the gate/up GEMMs of one forward: the gate
    and up weights of every local expert that has rows, read once, the token
    rows read once per routed row, the activation written once."""
    active = int((counts > 0).sum())
    R = int(counts.sum())
    return 2.0 * active * s.I * s.H * 2 + R * s.H * 2 + R * s.I * 2


def phase_bytes(s, R, accumulate):
    """Algorithmic HBM bytes of the memory-bound phases of one forward."""
    return {
        "route": s.T * s.H * 2 + s.E * s.H * 4 + s.T * s.k * 8,
        "permute": s.T * s.k * 12,
        "gather": 2 * R * s.H * 2,
        "combine": R * s.H * 4 + s.T * s.H * 4 * (2 if accumulate else 1) + s.T * s.k * 8,
    }


def summarize_timing(tms):
    """Per-call averages of moe_last_timing records (each may sum several
    timed calls)."""
    calls = sum(t["calls"] for t in tms)
    out = {k: sum(t[k] for t in tms) / calls for k in tms[0].keys()}
    out["pipeline_n"] = tms[-1]["pipeline_n"]
    out["calls"] = calls
    return out


def main(argv=None):
    args = parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the path is the "
              f"one-GPU share of an expert-parallel layer and has no multi-GPU mode.",
              file=sys.stderr)
        return 2
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return 0
    if args.trace_overlap:
        return trace_overlap(args.trace_overlap, args.warmup, args.steps)
    if args.trace_stats:
        return trace_stats(args.trace_stats, args.warmup, args.steps)

    import torch

    from paper_2410_12247_amd import synth

    torch.cuda.set_device(0)
    if args.sweep:
        return sweep(args)
    if args.pn_sweep:
        return pn_sweep(args)
    if args.pn_fit:
        return pn_fit(args)
    if args.cu_sweep:
        return cu_sweep(args)
    if args.gemm_study:
        return gemm_study(args)
    if args.tile_study:
        return tile_study(args)
    if args.pn_enable:
        return pn_enable(args)
    shape = synth.SHAPES[args.config]
    if args.tokens:
        shape = shape.with_tokens(args.tokens)
    inp = synth.make_inputs(shape)
    # timed steps: events around the GEMM launches only (an event between two
    # kernels delays the second); then a few steps with every phase timed
    # for the breakdown of the other phases
    wall, tms, counts = run_workload(args, shape, inp, args.steps, args.warmup, timing="gemm")
    tm = summarize_timing(tms)
    _, tms_all, _ = run_workload(args, shape, inp, PHASE_STEPS, 1, timing=True)
    tm_all = summarize_timing(tms_all)
    for k in ("route_ms", "permute_ms", "gather_ms", "combine_ms", "total_ms"):
        tm[k] = tm_all[k]
    R = int(counts.sum())
    fg, fd, fs = gemm_flops(shape, R)
    ms = wall / args.steps * 1e3
    gemm_ms = tm["gateup_ms"] + tm["down_ms"] + tm["shared_ms"]
    gemm_flops_total = fg + fd + fs
    # dominant kernel: the fused gate/up GEMM; per-launch average from HIP
    # events recorded on the GEMM stream around each launch
    per_launch_ms = tm["gateup_ms"] / max(tm["gateup_launches"], 1)
    per_launch_flops = fg / max(tm["gateup_launches"], 1)
    # bound by MFMA or by HBM: the gate/up GEMM's flops per algorithmic byte
    # against the machine balance (2.5e15 / 8e12 = 312 flop/B); few tokens
    # per expert (decode) leave it streaming weights
    per_launch_bytes = gateup_bytes(shape, counts) / max(tm["gateup_launches"], 1)
    hbm_bound = fg / max(gateup_bytes(shape, counts), 1.0) < PEAK_BF16_FLOPS / PEAK_HBM_BYTES
    if hbm_bound:
        achieved = per_launch_bytes / (per_launch_ms * 1e-3) / 1e9
        peak = PEAK_HBM_BYTES / 1e9
    else:
        achieved = per_launch_flops / (per_launch_ms * 1e-3) / 1e12
        peak = PEAK_BF16_FLOPS / 1e12
    pb = phase_bytes(shape, R, shape.shared_inter > 0)
    gbps = {k: round(v / (tm[f"{k}_ms"] * 1e-3) / 1e9, 1) for k, v in pb.items()
            if tm[f"{k}_ms"] > 0}
    routed_ms = tm["gateup_ms"] + tm["down_ms"]
    traffic = None
    if tm["group_stages"] and not tm["dense_stages"] and args.pn == 1 and not args.tokens:
        kname = "group_kernel<0"
        t = measured_traffic(f"{args.config}_group", kname)
        traffic = None if t is None else round(t)
    line = {
        "metric": METRIC,
        "value": round(shape.T / (ms * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": WORKLOAD_TEXT[args.config] +
                   (f" (T={shape.T})" if args.tokens else ""),
                   "tokens": shape.T, "hidden": shape.H, "inter": shape.I,
                   "experts": shape.E, "local_experts": shape.EL, "top_k": shape.k,
                   "renormalize": shape.renorm, "shared_inter": shape.shared_inter,
                   "gemm_mode": args.mode, "pipeline_n": args.pn,
                   "chunk_mode": args.chunk_mode,
                   "gemm_cu_budget": args.cu_budget, "side_cus": args.side_cus,
                   "group_tile_rows": args.group_tile_rows,
                   "parallelism": "single GPU"},
        "roofline": {"bound": "hbm" if hbm_bound else "mfma", "achieved": round(achieved, 1),
                     "peak": peak, "unit": "GB/s" if hbm_bound else "TFLOP/s",
                     "frac": round(achieved / peak, 4),
                     "traffic": traffic,
                     "kernel": "gate/up GEMM (fused SiLU*mul)",
                     "per_launch_ms": round(per_launch_ms, 4),
                     "per_launch_gflop": round(per_launch_flops / 1e9, 2),
                     "per_launch_mb": round(per_launch_bytes / 1e6, 1)},
        "gemm": {"tflops_per_s_wall": round(gemm_flops_total / (ms * 1e-3) / 1e12, 1),
                 "tflops_per_s_busy": round(gemm_flops_total / (gemm_ms * 1e-3) / 1e12, 1),
                 "mfma_frac_busy": round(gemm_flops_total / (gemm_ms * 1e-3) / PEAK_BF16_FLOPS, 4),
                 "routed_mfma_frac_busy": round((fg + fd) / (routed_ms * 1e-3) / PEAK_BF16_FLOPS,
                                                4) if routed_ms > 0 else None,
                 "shared_mfma_frac_busy": round(fs / (tm["shared_ms"] * 1e-3) / PEAK_BF16_FLOPS,
                                                4) if tm["shared_ms"] > 0 else None,
                 "gflop": round(gemm_flops_total / 1e9, 1), "routed_rows": R},
        "hbm_gbps": {**gbps, "peak": PEAK_HBM_BYTES / 1e9},
        "phases_ms": {k: round(v, 4) for k, v in tm.items() if k.endswith("_ms")},
        "stages": {k: tm[k] for k in ("dense_stages", "group_stages")},
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(inp, args.cpu_seconds)
    print(json.dumps(line), flush=True)
    return 0


def sweep(args):
    """GroupGemm-forced vs DenseGemm-forced vs AUTO over the zipf token counts
    on identical routing, with all 20 local experts in one stage (PN = 1) and
    with one expert per stage (PN = 20, where the paper's Sec. 4.3 has the
    grouped GEMM become a dense one); one JSON line per point."""
    from paper_2410_12247_amd import moe, synth

    base = synth.SHAPES["zipf"]
    for T in synth.ZIPF_TOKENS:
        shape = base.with_tokens(T)
        inp = synth.make_inputs(shape)
        for pn in (1, shape.EL):
            res = {}
            for mode in ("group", "dense", "auto"):
                a = argparse.Namespace(**{**vars(args), "mode": mode, "pn": pn})
                wall, tms, counts = run_workload(a, shape, inp, args.steps, args.warmup,
                                                 timing="gemm")
                tm = summarize_timing(tms)
                res[mode] = {"ms": round(wall / args.steps * 1e3, 4),
                             "gemm_ms": round(tm["gateup_ms"] + tm["down_ms"], 4),
                             "dense_stages": tm["dense_stages"]}
            fg, fd, _ = gemm_flops(shape, int(counts.sum()))
            best = min(res["group"]["gemm_ms"], res["dense"]["gemm_ms"])
            d = moe.dims(shape.T, shape.H, shape.I, shape.E, shape.k, shape.e0, shape.EL,
                         shape.renorm)
            per = shape.EL // pn
            tiles = []
            for st in range(pn):
                tiles += moe.gemm_plan(d, moe.opts(gemm_mode=moe.GEMM_DENSE),
                                       counts[st * per:(st + 1) * per])[1]
            print(json.dumps({"sweep": "zipf", "tokens": T, "pipeline_n": pn,
                              "routed_rows": int(counts.sum()),
                              "rows_per_expert": counts.tolist(),
                              "dense_tile_rows": tiles,
                              "gemm_gflop": round((fg + fd) / 1e9, 2), **res,
                              "auto_regret": round(res["auto"]["gemm_ms"] / best - 1, 4)}),
                  flush=True)
    return 0


def pn_sweep(args):
    """Step time of --config over pipeline numbers, with expert-group stages
    (PN dividing the local experts) and token-range stages; one JSON line per
    point, each with the per-phase device times summed over stages."""
    from paper_2410_12247_amd import synth

    shape = synth.SHAPES[args.config]
    if args.tokens:
        shape = shape.with_tokens(args.tokens)
    inp = synth.make_inputs(shape)
    for chunk in ("experts", "tokens"):
        for pn in (1, 2, 4, 5, 8, 10, 20):
            if chunk == "experts" and shape.EL % pn:
                continue
            if chunk == "tokens" and (pn == 1 or pn * shape.EL > 256):
                continue
            a = argparse.Namespace(**{**vars(args), "pn": pn, "chunk_mode": chunk})
            wall, tms, counts = run_workload(a, shape, inp, args.steps, args.warmup)
            tm = summarize_timing(tms)
            wall_u, _, _ = run_workload(a, shape, inp, args.steps, args.warmup, timing=False)
            print(json.dumps({"pn_sweep": args.config, "tokens": shape.T, "chunk_mode": chunk,
                              "pipeline_n": pn, "gemm_mode": args.mode,
                              "ms_per_step": round(wall_u / args.steps * 1e3, 4),
                              "phases_ms": {k: round(v, 4) for k, v in tm.items()
                                            if k.endswith("_ms")}}), flush=True)
    return 0


def _shape_of(args):
    from paper_2410_12247_amd import synth

    shape = synth.SHAPES[args.config]
    return shape.with_tokens(args.tokens) if args.tokens else shape


def pn_fit(args):
    """The paper's pipeline-number model (Sec. 5.2) fitted on one GPU.  The
    serial mode (every stage on one stream, nothing overlapped) gives the
    cost of cutting the work into N expert-group stages, R(N) = T_serial(N)
    - T_serial(1), fitted as kN + b by least squares; C = min(T_comm,
    T_comp) from the unsplit forward's phases, with T_comm the one-GPU
    stand-in for the dispatch and combine all2alls (gather + combine) and
    T_comp the expert GEMMs.  moe_choose_pipeline_n picks PN from (C, k, b);
    the measured best is the PN with the lowest pipelined step time."""
    import numpy as np

    from paper_2410_12247_amd import moe, synth
    from paper_2410_12247_amd.workload import DeviceInputs

    shape = _shape_of(args)
    inp = synth.make_inputs(shape)
    g = DeviceInputs(inp)
    pns = [n for n in range(1, min(shape.EL, 20) + 1) if shape.EL % n == 0]
    a1 = argparse.Namespace(**{**vars(args), "pn": 1, "chunk_mode": "experts"})
    _, tms, _ = run_workload(a1, shape, inp, args.steps, args.warmup, timing=True, dev_inputs=g)
    tm = summarize_timing(tms)
    t_comm = tm["gather_ms"] + tm["combine_ms"]
    t_comp = tm["gateup_ms"] + tm["down_ms"]
    ser, pipe = {}, {}
    for pn in pns:
        a = argparse.Namespace(**{**vars(args), "pn": pn, "chunk_mode": "experts"})
        w_s, _, _ = run_workload(a, shape, inp, args.steps, args.warmup, timing=False,
                                 serial=True, dev_inputs=g)
        w_p, _, _ = run_workload(a, shape, inp, args.steps, args.warmup, timing=False,
                                 dev_inputs=g)
        ser[pn] = w_s / args.steps * 1e3
        pipe[pn] = w_p / args.steps * 1e3
    n = np.array(pns, dtype=np.float64)
    r = np.array([ser[p] - ser[1] for p in pns])
    k, b = np.polyfit(n, r, 1) if len(pns) > 1 else (0.0, 0.0)
    C = min(t_comm, t_comp)
    chosen, gain = moe.choose_pipeline_n(C, max(k, 0.0), b, shape.EL)
    best = min(pipe, key=pipe.get)
    print(json.dumps({
        "pn_fit": args.config, "tokens": shape.T, "local_experts": shape.EL,
        "t_comm_ms": round(t_comm, 4), "t_comp_ms": round(t_comp, 4), "C_ms": round(C, 4),
        "k_ms": round(float(k), 4), "b_ms": round(float(b), 4),
        "serial_ms": {p: round(v, 4) for p, v in ser.items()},
        "pipelined_ms": {p: round(v, 4) for p, v in pipe.items()},
        "predicted_gain_ms": {p: round(C - b - (C / p + k * p), 4) for p in pns if p > 1},
        "measured_gain_ms": {p: round(pipe[1] - pipe[p], 4) for p in pns if p > 1},
        "chosen_pn": chosen, "chosen_gain_ms": round(gain, 4), "measured_best_pn": best,
        "agree": chosen == best}), flush=True)
    return 0


def cu_sweep(args):
    """Step time of --config over the grouped GEMM's persistent grid (its CU
    budget: CUs left to the gather and combine of the other stages, the
    paper's SM control, Sec. 5.2) and the pipeline number."""
    from paper_2410_12247_amd import synth
    from paper_2410_12247_amd.workload import DeviceInputs

    shape = _shape_of(args)
    inp = synth.make_inputs(shape)
    g = DeviceInputs(inp)
    for pn in [p for p in (1, 2, 4) if shape.EL % p == 0]:
        for budget in (256, 248, 240, 224, 192, 160, 128):
            a = argparse.Namespace(**{**vars(args), "pn": pn, "chunk_mode": "experts",
                                      "cu_budget": budget})
            w, _, _ = run_workload(a, shape, inp, args.steps, args.warmup, timing=False,
                                   dev_inputs=g)
            _, tms, _ = run_workload(a, shape, inp, PHASE_STEPS, 1, timing="gemm", dev_inputs=g)
            tm = summarize_timing(tms)
            print(json.dumps({"cu_sweep": args.config, "tokens": shape.T, "pipeline_n": pn,
                              "gemm_cu_budget": budget,
                              "ms_per_step": round(w / args.steps * 1e3, 4),
                              "gateup_ms": round(tm["gateup_ms"], 4),
                              "down_ms": round(tm["down_ms"], 4)}), flush=True)
    return 0


def gemm_study(args):
    """GroupGemm (moe_ffn_group: gate/up + SiLU + down) on the DeepSeekV2
    expert shape [1536, 5120], as in the paper's GEMM profiling (Sec. 3.2,
    Conclusions 2 and 3): throughput over the group count at several rows
    per group, relative to the best group count of the same rows (Fig. 4b),
    and over the CU budget at 6144 rows per group (Fig. 4c); then GroupGemm
    against one DenseGemm launch per expert at uniform load, 16 experts of m
    rows each (Fig. 4a) and a single expert of m rows (Sec. 4.3's E = N).
    Inputs are seeded Gaussian bf16 tensors; the rows of
    each group are contiguous."""
    import torch

    from paper_2410_12247_amd import moe

    H, I = 5120, 1536
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev)
    gen.manual_seed(2410)

    def normal(shape, sigma):
        return (torch.randn(shape, generator=gen, device=dev) * sigma).to(torch.bfloat16)

    GMAX, MMAX = 20, 6144
    x = normal((GMAX * MMAX, H), 1.0)
    wg, wu, wd = normal((GMAX, I, H), 0.02), normal((GMAX, I, H), 0.02), normal((GMAX, H, I), 0.02)
    act = torch.empty((GMAX * MMAX, I), dtype=torch.bfloat16, device=dev)
    y = torch.empty((GMAX * MMAX, H), dtype=torch.float32, device=dev)

    def time_group(G, m, budget):
        d = moe.dims(G * m, H, I, G, 1)
        off = torch.arange(0, G * m + 1, m, dtype=torch.int32, device=dev)
        run = lambda: moe.ffn_group(d, 0, G, off, x, wg, wu, wd, act, y, budget)  # noqa: E731
        for _ in range(args.warmup):
            run()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record()
        for _ in range(args.steps):
            run()
        ev[1].record()
        torch.cuda.synchronize()
        ms = ev[0].elapsed_time(ev[1]) / args.steps
        return ms, 6.0 * G * m * H * I / (ms * 1e-3) / 1e12

    for m in (128, 512, 2048, 6144):
        res = {G: time_group(G, m, 0) for G in (1, 2, 4, 8, 16, 20)}
        top = max(v[1] for v in res.values())
        print(json.dumps({"gemm_study": "groups", "rows_per_group": m,
                          "tflops": {G: round(v[1], 1) for G, v in res.items()},
                          "relative": {G: round(v[1] / top, 3) for G, v in res.items()}}),
              flush=True)
    for G in (1, 4, 16):
        res = {b: time_group(G, MMAX, b) for b in (256, 224, 192, 160, 128, 96, 64, 32)}
        print(json.dumps({"gemm_study": "cu_budget", "groups": G, "rows_per_group": MMAX,
                          "tflops": {b: round(v[1], 1) for b, v in res.items()}}), flush=True)

    # GroupGemm vs DenseGemm at uniform load (Fig. 4a): 16 experts of m rows
    # each as one grouped launch, or as one dense launch per expert
    def time_dense(G, m):
        def run():
            for e in range(G):
                r = slice(e * m, (e + 1) * m)
                moe.ffn_dense(m, H, I, x[r], wg[e], wu[e], wd[e], act[r], y[r])
        for _ in range(args.warmup):
            run()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record()
        for _ in range(args.steps):
            run()
        ev[1].record()
        torch.cuda.synchronize()
        ms = ev[0].elapsed_time(ev[1]) / args.steps
        return ms, 6.0 * G * m * H * I / (ms * 1e-3) / 1e12

    for G in (16, 1):
        for m in (128, 512, 1024, 2048, 4096, 6144):
            g_ms, g_tf = time_group(G, m, 0)
            d_ms, d_tf = time_dense(G, m)
            dd = moe.dims(G * m, H, I, G, 1)
            _, tiles, _, _ = moe.gemm_plan(dd, moe.opts(gemm_mode=moe.GEMM_DENSE,
                                                        exact_order=True), [m])
            print(json.dumps({"gemm_study": "group_vs_dense", "experts": G,
                              "rows_per_expert": m, "group_ms": round(g_ms, 4),
                              "dense_ms": round(d_ms, 4), "group_tflops": round(g_tf, 1),
                              "dense_tflops": round(d_tf, 1), "dense_tile_rows": tiles[0]}),
                  flush=True)
    return 0


def pn_enable(args):
    """Sec. 5.2 item 4 over the zipf loads: for each T and each PN dividing
    the 20 local experts, eps1 = N G(m/N, E/N) / G(m, E) - 1 (the stages'
    expert-GEMM time summed, over the unsplit one) and eps0 = N S(m/N) /
    S(m) - 1 (the same for the combine, the one-GPU stand-in for the
    all2alls), measured with every stage on one stream (nothing overlapped,
    every phase timed) and predicted by moe_pipeline_plan from the same row
    counts; then the PN the library would choose and the pipelined step
    time at each PN."""
    import numpy as np

    from paper_2410_12247_amd import moe, synth
    from paper_2410_12247_amd.workload import DeviceInputs

    base = synth.SHAPES["zipf"]
    for T in synth.ZIPF_TOKENS:
        shape = base.with_tokens(T)
        inp = synth.make_inputs(shape)
        g = DeviceInputs(inp)
        meas, model, step = {}, {}, {}
        counts = None
        for pn in (1, 2, 4, 5, 10, 20):
            a = argparse.Namespace(**{**vars(args), "pn": pn, "chunk_mode": "experts"})
            _, tms, counts = run_workload(a, shape, inp, args.steps, args.warmup, timing=True,
                                          serial=True, dev_inputs=g)
            tm = summarize_timing(tms)
            meas[pn] = (tm["gateup_ms"] + tm["down_ms"], tm["combine_ms"])
            w, _, _ = run_workload(a, shape, inp, args.steps, args.warmup, timing=False,
                                   dev_inputs=g)
            step[pn] = round(w / args.steps * 1e3, 4)
            model[pn] = moe.pipeline_plan(g.d, moe.opts(), counts, pn)
        g1, s1 = meas[1]
        chosen = moe.pipeline_plan(g.d, moe.opts(), counts, 0)["pipeline_n"]
        print(json.dumps({
            "pn_enable": "zipf", "tokens": T, "routed_rows": int(np.sum(counts)),
            "G_ms": round(g1, 4), "S_ms": round(s1, 4),
            "eps1_measured": {p: round(v[0] / g1 - 1, 4) for p, v in meas.items() if p > 1},
            "eps0_measured": {p: round(v[1] / s1 - 1, 4) for p, v in meas.items() if p > 1},
            "eps1_model": {p: round(m["eps1"], 4) for p, m in model.items() if p > 1},
            "eps0_model": {p: round(m["eps0"], 4) for p, m in model.items() if p > 1},
            "gain_model_ms": {p: round(m["gain_us"] / 1e3, 4) for p, m in model.items() if p > 1},
            "enabled_model": {p: m["enabled"] for p, m in model.items() if p > 1},
            "chosen_pn": chosen, "pipelined_ms": step}), flush=True)
        del g
    return 0


def _kernel_label(name):
    """Short kernel name: the function and its first template argument."""
    base = name[5:] if name.startswith("void ") else name
    base = base.replace("moe::(anonymous namespace)::", "").replace("moe::", "").split("(")[0]
    if "<" in base:
        head, rest = base.split("<", 1)
        first = rest.split(",")[0].split(">")[0].strip()
        tile = ""
        if "PingPong<" in rest:
            tile = " BM=" + rest.split("PingPong<", 1)[1].split(">")[0].split(",")[-1].strip()
        return f"{head}<{first}>{tile}"
    return base


def _trace_forwards(path):
    """Kernel dispatches of a kernel-trace CSV in the order they were
    enqueued (dispatch id; kernels on the forward's side streams overlap, and
    a kernel's start stamp can precede that of the one before it on its own
    stream), cut into forwards: each runs from the first kernel after the
    previous forward's last combine (the shared FFN's GEMMs, enqueued before
    the router, when the workload has shared experts) through its own."""
    import csv

    ev = []
    for r in csv.DictReader(open(path)):
        ev.append((int(r.get("Dispatch_Id") or 0), int(r["Start_Timestamp"]),
                   int(r["End_Timestamp"]), _kernel_label(r.get("Kernel_Name", ""))))
    ev.sort(key=lambda e: (e[0], e[1]))
    ev = [e[1:] for e in ev]
    routers = [i for i, e in enumerate(ev)
               if e[2].startswith("route") and "select" not in e[2]]
    starts = []
    for r in routers:
        i = r - 1
        while i >= 0 and not ev[i][2].startswith("combine"):
            i -= 1
        starts.append(i + 1)
    fwd = [ev[a:b] for a, b in zip(starts, starts[1:] + [len(ev)])]
    # shared experts: grouped GEMM launches ahead of a forward's router
    has_shared = any(e[2].startswith("group_kernel")
                     for a, r in zip(starts, routers) for e in ev[a:r])
    return fwd, has_shared


def trace_stats(path, warmup, steps):
    """Average duration of each kernel over the timed forwards [warmup,
    warmup + steps) of a kernel trace of one bench.py run (the GEMM-timed
    steps whose HIP events give the line's roofline), and over every
    forward in the trace for comparison.  With shared experts the first
    grouped gate/up and down launches of a forward are the shared FFN's."""
    fwd, has_shared = _trace_forwards(path)

    def stats(forwards):
        acc = {}
        for f in forwards:
            seen = {}
            for s_, e_, n in f:
                k = n
                if has_shared and n.startswith("group_kernel"):
                    seen[n] = seen.get(n, 0) + 1
                    k = n + (" (shared)" if seen[n] == 1 else " (routed)")
                acc.setdefault(k, []).append((e_ - s_) / 1e3)
        return acc

    timed = stats(fwd[warmup:warmup + steps])
    every = stats(fwd)
    print(f"forwards in trace: {len(fwd)}; timed: [{warmup}, {warmup + steps})\n")
    print("| kernel | calls (timed) | avg us (timed) | min | max | calls (all) | avg us (all) |")
    print("|---|---|---|---|---|---|---|")
    for k in sorted(timed, key=lambda k: -sum(timed[k])):
        t, a = timed[k], every[k]
        print(f"| {k} | {len(t)} | {sum(t) / len(t):.1f} | {min(t):.1f} | {max(t):.1f} | "
              f"{len(a)} | {sum(a) / len(a):.1f} |")
    return 0


def trace_overlap(path, warmup, steps):
    """Stage overlap in a rocprofv3 kernel trace (--kernel-trace, CSV) of a
    bench.py run with pipelined forwards: each forward starts at a router
    kernel; the timed forwards are numbers [warmup, warmup + steps) (the
    benchmark's GEMM-timed steps).  For the combine of each stage the line
    gives how long it ran, how long of that a GEMM kernel (group_kernel or a
    K-split fixup, necessarily of a later stage: a stage's combine waits for
    its own GEMMs) was running too, and whether it started inside such a
    GEMM's interval.  Prints a markdown table and totals."""
    fwd, _ = _trace_forwards(path)
    lines = ["| forward | combine | ran (us) | beside a later GEMM (us) | started inside a "
             "later GEMM |", "|---|---|---|---|---|"]
    tot_c, tot_o, n_inside, n_comb = 0.0, 0.0, 0, 0
    for fi, f in enumerate(fwd[warmup:warmup + steps]):
        gemms = [e for e in f if "group_kernel" in e[2] or "split_fixup" in e[2]]
        combs = [e for e in f if "combine_kernel" in e[2]]
        for ci, (cs, ce, _) in enumerate(combs):
            # combine i waits for stage i's GEMMs, so any GEMM kernel running
            # beside it belongs to a later stage
            ov = 0
            for gs, ge, _ in gemms:
                ov += max(0, min(ce, ge) - max(cs, gs))
            inside = any(gs <= cs < ge for gs, ge, _ in gemms)
            tot_c += (ce - cs) / 1e3
            tot_o += ov / 1e3
            n_inside += int(inside)
            n_comb += 1
            lines.append(f"| {fi} | {ci} | {(ce - cs) / 1e3:.1f} | {ov / 1e3:.1f} | "
                         f"{'yes' if inside else 'no'} |")
    print("\n".join(lines))
    print(f"\ncombines: {n_comb}, started inside a GEMM: {n_inside}, "
          f"combine time {tot_c:.1f} us, of it beside GEMMs {tot_o:.1f} us")
    return 0


def tile_study(args):
    """One expert's gate/up and down GEMMs as DenseGemm launches with each
    tile height (128, 192, 256, 320 token rows), over row counts, on the
    DeepSeekV2 and Mixtral expert shapes; the data the launch-cost model's
    per-tile step and epilogue costs are fitted to.  Every token is routed
    to the one expert (E = 1, k = 1), so the launch covers m rows; times are
    HIP events around each GEMM launch (MOE_FLAG_TIMING_GEMM), in exact order
    (no K split: a launch is whole rounds of tiles) and with the K split of
    a partial last round."""
    from paper_2410_12247_amd import moe, synth
    from paper_2410_12247_amd.workload import DeviceInputs

    for H, I, label in ((5120, 1536, "dsv2_expert"), (4096, 3584, "mixtral_expert")):
        for m in (512, 1024, 2048, 4096, 8192, 16384, 32768):
            shp = synth.custom_shape(name=f"tile{m}", index=230, T=m, H=H, I=I, E=1, EL=1,
                                     k=1, renorm=True)
            g = DeviceInputs(synth.make_inputs(shp))
            for exact in (True, False):
                res = {}
                for bm in (128, 192, 256, 320):
                    o = moe.opts(gemm_mode=moe.GEMM_DENSE, dense_tile_rows=bm, timing="gemm",
                                 exact_order=exact)
                    buf = g.buffers(o)
                    for _ in range(args.warmup):
                        g.run(buf)
                    tms = []
                    for _ in range(args.steps):
                        g.run(buf)
                        tms.append(moe.last_timing())
                    tm = summarize_timing(tms)
                    res[bm] = {"gateup_us": round(tm["gateup_ms"] * 1e3, 2),
                               "down_us": round(tm["down_ms"] * 1e3, 2)}
                    del buf
                _, tiles, gus, dus = moe.gemm_plan(g.d, moe.opts(exact_order=exact), [m])
                print(json.dumps({"tile_study": label, "hidden": H, "inter": I, "rows": m,
                                  "k_split": not exact, "by_tile_rows": res,
                                  "model_pick": tiles[0], "model_dense_us": round(dus, 1)}),
                      flush=True)
            del g
    return 0


if __name__ == "__main__":
    sys.exit(main())
