#!/usr/bin/env python3
"""Benchmark: best-found schedule of a contraction workload on one MI355X.

One step is one execution of the workload's operator in its tuned schedule
(every kernel of the operator: for attention the single fused kernel) over
inputs already resident in HBM.  W untimed warm-up steps, then exactly K
steps back to back, bracketed by torch.cuda.synchronize(); value = the
operator's algorithmic FLOPs x K / elapsed wall time.  The default workload
is the largest: the gated MLP 2048 x 4096 x 14336.  The steps cycle through
R copies of the inputs, R chosen so that R x the input bytes is at least
twice the 256 MB last-level cache: each step reads its operands from HBM.

roofline: HIP events recorded on the launch stream around every kernel of
every timed step give the dominant kernel's mean duration; achieved =
algorithmic bytes (HBM-bound operators) or FLOPs (MFMA-bound) of one launch
divided by that duration.  traffic: measured HBM bytes per launch from the
rocprofv3 FETCH_SIZE / WRITE_SIZE summaries in profiles/, when present for
the same kernel source and schedule, else null.

cpu_baseline: the CPU oracle (test infrastructure) on the same workload, or a
bounded sample of it, timed on the host cores.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "best-schedule TFLOP/s and % of MFMA peak per operator; samples to reach it"
DEFAULT_WORKLOAD = "gated_mlp_t2048_h4096_i14336"
MALL_BYTES = 256 << 20            # MI355X last-level cache (Infinity Cache)
HBM_PEAK_GBS = 8000.0

DTYPE = {"gemm_f32_128": "f32", "gemm_f32_m16_n2048_k7168": "f32"}   # the others: bf16 (fp32 accumulation)


def _oracle_baseline(name, op, host, budget_s):
    """Time the CPU oracle on the workload (whole, or a bounded row sample)."""
    import oracle
    kind = op.kind
    from paper_2506_01374_amd import rc
    flops_total = op.flops()
    t0 = time.perf_counter()
    reps = 0
    if kind == rc.RC_OP_ATTENTION:
        B, H, S, _ = op.dims
        causal = bool(op.flags & 1)
        rows = None
        frac = 1.0
        sample = "all query rows of all heads (whole workload)"
        if not causal and B * H * S > 16384:
            # without the mask every query row costs the same: time a prefix
            rows = np.arange(16384)
            frac = 16384 / (B * H * S)
            sample = f"first 16384 of {B * H * S} query rows"
        while True:
            oracle.attention_bf16(host["Q"], host["K"], host["V"], causal=causal, rows=rows)
            reps += 1
            if time.perf_counter() - t0 > budget_s:
                break
    elif kind == rc.RC_OP_GEMM_F32:
        sample = "whole workload"
        frac = 1.0
        while True:
            oracle.gemm_f32(host["A"], host["B"])
            reps += 1
            if time.perf_counter() - t0 > budget_s:
                break
    else:
        n = {rc.RC_OP_GATED_MLP: 32, rc.RC_OP_MOE: 32, rc.RC_OP_CONV2D: 512}[kind]
        rows = np.arange(n)
        total = op.dims[0] if kind != rc.RC_OP_CONV2D else op.dims[0] * op.dims[1] * op.dims[2]
        frac = n / total
        sample = f"first {n} of {total} independent output rows"
        while True:
            if kind == rc.RC_OP_GATED_MLP:
                oracle.gated_mlp_bf16(host["X"], host["Wg"], host["Wu"], host["Wd"], rows=rows)
            elif kind == rc.RC_OP_MOE:
                oracle.moe_bf16(host["X"], host["ids"], host["w"], host["Wg"], host["Wu"], host["Wd"],
                                rows=rows)
            else:
                oracle.conv2d_bf16(host["x"], host["w"], host["bias"], pad=op.dims[7], pixels=rows)
            reps += 1
            if time.perf_counter() - t0 > budget_s:
                break
    dt = time.perf_counter() - t0
    return {"value": flops_total * frac * reps / dt / 1e12, "unit": "TFLOP/s",
            "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"{sample}, {reps} repetition(s) in {dt:.2f} s"}


def _output_bytes(op):
    from paper_2506_01374_amd import workloads as W
    shape, dt = W.output_shape(op)
    return float(np.prod(shape)) * (4 if dt == "float32" else 2)


def _search_summary(name, op, sched):
    """Samples the search needed to reach the tuned schedule, from the
    committed campaign records of this workload (results/), if any: one
    entry per record (the policy comparison, the sequence-proposal
    comparison, the longer-budget run), each against its own reference."""
    import glob
    out = []
    for path in sorted(glob.glob(os.path.join(ROOT, "results", f"{name}.campaign*.json"))):
        try:
            rec = json.load(open(path))
        except (OSError, ValueError):
            continue
        summ = rec.get("summary")
        if not summ:
            continue
        try:       # records name the knobs of their day; unnamed knobs take their defaults
            same = str(op.from_string(rec.get("reference_schedule") or "")) == str(sched)
        except Exception:
            same = False
        pols = {}
        for name, p in summ.items():       # the record's summary, without per-seed detail
            curve = p.get("best_so_far_over_reference", {})
            pols[name] = {"best_so_far_over_reference": {n: round(v["mean"], 4) for n, v in curve.items()},
                          "best_over_reference": round(p.get("best_over_reference", 0.0), 4)}
            for key in ("samples_to_50pct", "samples_to_75pct", "samples_to_90pct", "samples_to_99pct"):
                if key in p:
                    pols[name][key] = {k: p[key].get(k) for k in ("reached", "of", "median")}
        out.append({"source": os.path.relpath(path, ROOT), "reference_is_tuned": same,
                    "budget": rec.get("budget"), "seeds": len(rec.get("seeds") or []), "policies": pols})
    return out or None


def _search_headline(records):
    """The policy with the best mean best-so-far after 200 samples among the
    campaign records taken against the present tuned schedule: its mean,
    and how many runs reached 90 % and 99 % of the tuned schedule (median
    samples to get there)."""
    best = None
    for rec in records or []:
        if not rec["reference_is_tuned"]:
            continue
        for name, p in rec["policies"].items():
            at = p["best_so_far_over_reference"].get("200")
            if at is not None and (best is None or at > best["mean_best_over_tuned_at_200"]):
                best = {"source": rec["source"], "policy": name, "mean_best_over_tuned_at_200": at,
                        "best_run_over_tuned": p["best_over_reference"],
                        "samples_to_90pct": p.get("samples_to_90pct"),
                        "samples_to_99pct": p.get("samples_to_99pct")}
    return best


def _p0_speedup(name, op, sched):
    """The tuned schedule's cold speedup over the untransformed program P0
    (results/<workload>.p0.json, written by `tune.py --p0`), only if that
    record was taken with this exact schedule; else null."""
    path = os.path.join(ROOT, "results", f"{name}.p0.json")
    try:
        rec = json.load(open(path))
        if str(op.from_string(rec["tuned_schedule"])) != str(sched):
            return None
        return {"source": os.path.relpath(path, ROOT), "value": round(rec["tuned_speedup_over_p0"], 3),
                "p0_us": rec["p0_us"], "tuned_us": rec["tuned_us"], "measurement": rec.get("measurement")}
    except Exception:      # no record, or one this version cannot read
        return None


def _kernel_source(name):
    from paper_2506_01374_amd import rc, workloads as W
    kind = W.workload_op(name).kind
    return {rc.RC_OP_ATTENTION: "attention.hip", rc.RC_OP_GEMM_F32: "gemm_f32.hip"}.get(kind, "gemm_bf16.hip")


def _load_traffic(name, op, sched):
    """Counter-measured HBM bytes per launch, only if recorded for this exact
    schedule and this exact kernel source (else null: the kernel changed)."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path)).get(name)
    except (OSError, ValueError):
        return None
    if not rec:
        return None
    try:       # the record names the knobs of its day; unnamed knobs take their defaults
        if str(op.from_string(rec.get("key") or "")) != str(sched):
            return None
    except Exception:
        return None
    src = os.path.join(ROOT, "paper_2506_01374_amd", "csrc", "kernels", _kernel_source(name))
    if hashlib.sha1(open(src, "rb").read()).hexdigest()[:16] != rec.get("kernel_source_sha1"):
        return None
    return rec.get("bytes_per_launch")


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--schedule", default=None, help="schedule string (default: tuned.json)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--eager", action="store_true",
                    help="launch each step from the host instead of replaying a captured HIP graph")
    ap.add_argument("--cpu-budget", type=float, default=10.0, help="seconds of oracle work")
    ap.add_argument("--rotate", type=int, default=0, metavar="R",
                    help="cycle the steps through R copies of the inputs; 0 (default) picks the "
                         "smallest R >= 2 with R x the input bytes >= 2 x the 256 MB MALL, so "
                         "every step reads its operands from HBM, not from the cache")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES, --steps times "
                         "(the reference reading for HBM traffic counters)")
    args = ap.parse_args()

    if args.calibrate_copy:
        import torch
        n = args.calibrate_copy // 2
        src = torch.ones(n, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": 2 * n, "steps": args.steps}), flush=True)
        return

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the library has no "
              "multi-GPU path.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2506_01374_amd import rc, workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    rc.set_cache_dir(os.path.join(ROOT, "paper_2506_01374_amd", "jit_cache"))
    torch.cuda.set_device(0)
    name = args.workload
    op = W.workload_op(name)
    tuned = json.load(open(os.path.join(ROOT, "paper_2506_01374_amd", "tuned.json")))
    sched = op.from_string(args.schedule if args.schedule else tuned[name])
    host = W.host_inputs(op, seed=0)
    in_bytes = op.bytes() - _output_bytes(op)
    R = args.rotate if args.rotate > 0 else int(min(64, max(2, -(-2 * MALL_BYTES // int(in_bytes)))))
    devs = [W.to_device(W.stored_inputs(op, sched, host)) for _ in range(R)]
    out = W.empty_output(op)
    plan = rc.Plan(op, sched)
    ws = plan.workspace()
    nk, dom = plan.nkernels, plan.dominant

    K = args.steps
    # Steps run on a side stream (default priority).  By default the K timed
    # steps are captured once as a HIP graph and replayed, so host launch
    # latency stays out of the timed region; HIP events recorded on that
    # stream immediately before and after the replay time the region.
    # Events recorded inside a graph do not bracket its kernels, so the
    # per-kernel split of a step (needed only for operators with several
    # kernels) comes from a short eager pass with events around each kernel.
    stream = torch.cuda.Stream()
    ev_region = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    with torch.cuda.stream(stream):
        preps = [plan.prepare(d, out, ws, stream) for d in devs]
        for i in range(args.warmup):
            preps[i % R].launch()
        # eager pass: per-kernel events (also the whole measurement with --eager)
        n_eager = K if args.eager else min(K, 20)
        eager_ev = [[torch.cuda.Event(enable_timing=True) for _ in range(nk + 1)] for _ in range(n_eager)]
        for row in eager_ev:        # torch creates an event on its first record
            for e in row:
                e.record(stream)
        ev_arrays = [preps[i % R].events(row) for i, row in enumerate(eager_ev)]
    torch.cuda.synchronize()
    graph = None
    if not args.eager:
        try:
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph, stream=stream):
                for i in range(K):
                    preps[i % R].launch()
            torch.cuda.synchronize()
            graph.replay()              # warm replay
            torch.cuda.synchronize()
        except Exception as e:          # capture unsupported: time the eager loop instead
            print(f"graph capture failed ({e}); timing eager launches", file=sys.stderr)
            graph = None
            torch.cuda.synchronize()
    t0 = time.perf_counter()
    with torch.cuda.stream(stream):
        ev_region[0].record(stream)
        if graph is not None:
            graph.replay()
        else:
            for i in range(K):
                preps[i % R].launch_timed(ev_arrays[i % len(ev_arrays)])
        ev_region[1].record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    region_ms = ev_region[0].elapsed_time(ev_region[1])
    if graph is not None:
        with torch.cuda.stream(stream):
            for i in range(len(ev_arrays)):
                preps[i % R].launch_timed(ev_arrays[i])
        torch.cuda.synchronize()
    ms_per_step = elapsed * 1e3 / K
    flops = op.flops()
    value = flops / (elapsed / K) / 1e12
    n_ev = len(eager_ev)
    eager_kern_ms = [float(np.mean([eager_ev[i][k].elapsed_time(eager_ev[i][k + 1]) for i in range(n_ev)]))
                     for k in range(nk)]
    step_ms = region_ms / K                     # event-timed step inside the timed region
    dshare = eager_kern_ms[dom] / sum(eager_kern_ms) if nk > 1 else 1.0
    dom_ms = step_ms * dshare
    kern_ms = [step_ms * x / sum(eager_kern_ms) for x in eager_kern_ms]
    # the roofline that binds: algorithmic intensity against the ridge point
    # (bf16 2516.6 TFLOP/s / 8 TB/s = 314.6 FLOP/B; fp32 19.7 FLOP/B)
    bound = op.bound()
    if bound == "hbm":
        achieved = op.bytes() / (dom_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS}
    else:
        # the dominant kernel's own algorithmic FLOPs
        achieved = plan.kernel_flops(dom) / (dom_ms * 1e-3) / 1e12
        peak = op.peak_flops() / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                "frac": achieved / peak}
    roof["traffic"] = _load_traffic(name, op, sched)
    roof["kernel"] = ["rc_attention"] if op.kind == rc.RC_OP_ATTENTION else None
    roof["dominant_kernel_ms"] = dom_ms
    roof["kernel_ms"] = kern_ms
    roof["timing"] = ("HIP events around the replayed graph of the timed steps; "
                      "kernel split from an eager per-kernel event pass" if graph is not None
                      else "HIP events around every kernel of every timed step")
    roof["mfma_frac"] = (flops / (sum(kern_ms) * 1e-3)) / op.peak_flops()
    # the whole operator (every kernel of the step) against the same roof
    op_s = step_ms * 1e-3
    if bound == "hbm":
        roof["operator"] = {"achieved": op.bytes() / op_s / 1e9, "frac": op.bytes() / op_s / 1e9 / HBM_PEAK_GBS,
                            "step_ms": step_ms}
    else:
        roof["operator"] = {"achieved": flops / op_s / 1e12, "frac": flops / op_s / op.peak_flops(),
                            "step_ms": step_ms}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = _oracle_baseline(name, op, host, args.cpu_budget)
    search = _search_summary(name, op, sched)

    rec = {
        "metric": METRIC, "value": value, "unit": "TFLOP/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": DTYPE.get(name, "bf16"),
        "data": "synthetic (seeded SplitMix64 inputs of the workload's shape and distribution)",
        "config": {"workload": name, "dims": list(op.dims), "flags": op.flags,
                   "schedule": str(sched), "parallelism": "single GPU",
                   "launch": "hip_graph" if graph is not None else "eager",
                   "input_copies": R, "input_bytes_per_copy": in_bytes,
                   "frac_of_mfma_peak": value * 1e12 / op.peak_flops()},
        "roofline": roof, "cpu_baseline": cpu,
        "search": search,
        "search_headline": _search_headline(search),
        "tuned_speedup_over_p0": _p0_speedup(name, op, sched),
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
