"""Schedule tuning: run the search of Sec. 3.2 over a workload's knob space
with the measured throughput on the GPU as the objective.

Each valid sample is one distinct legal schedule compiled and timed
(warm-ups, then repeated launches bracketed by HIP events, each after an
overwrite of a 512 MiB buffer so no operand is cache-resident).  Its reward
is the fraction of the operator's binding roofline reached: MFMA peak for
contraction-bound operators, HBM bandwidth for attention (arithmetic
intensity below the MI355X ridge point).

Usage (GPU):
  python -m paper_2506_01374_amd.tune --workload NAME --policy uct --budget 64 --seeds 0,1
  python -m paper_2506_01374_amd.tune --workload NAME --policy exhaustive --out results/
Usage (CPU, no GPU needed):
  python -m paper_2506_01374_amd.tune --workload NAME --enumerate --precompile
  python -m paper_2506_01374_amd.tune --workload NAME --replay table.jsonl --policy uct --seeds 0-19

--replay evaluates against a table of measured samples (a previous run's
JSONL); schedules missing from it count as invalid.  This reruns search
policies over many seeds without new GPU work.
"""
from __future__ import annotations

import argparse
import itertools
import json
import math
import os
import sys
import time
from typing import Dict, List, Optional

if __package__ in (None, ""):
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    __package__ = "paper_2506_01374_amd"

from . import rc
from . import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))
POLICIES = {"random": rc.RC_POLICY_RANDOM, "uct": rc.RC_POLICY_UCT, "exhaustive": rc.RC_POLICY_EXHAUSTIVE}


def reward_of(op: rc.Op, ms: float) -> float:
    """Fraction of the binding roofline reached (HBM or MFMA, by intensity)."""
    sec = ms * 1e-3
    if op.bound() == "hbm":
        return op.bytes() / sec / rc.lib().rc_peak_bytes_per_s()
    return op.flops() / sec / op.peak_flops()


def legal_space(op: rc.Op, limit: Optional[int] = None) -> List[rc.Schedule]:
    """Every legal schedule (cartesian product of knob values, filtered)."""
    names = op.knob_names()
    values = [op.knob_values(i) for i in range(len(names))]
    out = []
    base = op.default()
    for combo in itertools.product(*values):
        s = base.copy()
        for i, v in enumerate(combo):
            s.raw.knob[i] = v
        if s.validate() == "":
            out.append(s)
            if limit and len(out) >= limit:
                break
    return out


def random_walk_space(op: rc.Op, n: int, seed: int, horizon: int = 12) -> List[rc.Schedule]:
    """n distinct schedules from random legal transformation sequences."""
    import random
    rng = random.Random(seed)
    seen, out = set(), []
    tries = 0
    while len(out) < n and tries < 50 * n:
        tries += 1
        s = op.default()
        for _ in range(horizon):
            mv = s.moves()
            if not mv:
                break
            s = s.apply(rng.choice(mv))
        if s.hash() not in seen:
            seen.add(s.hash())
            out.append(s)
    return out


class GpuEvaluator:
    def __init__(self, op: rc.Op, repeat: int = 10, warmup: int = 2, log=None):
        import torch
        self.torch = torch
        self.op = op
        self.host = W.host_inputs(op, seed=0)
        self.repeat, self.warmup = repeat, warmup
        self.cache: Dict[str, dict] = {}
        self.log = log
        self._dev: Dict[str, list] = {}
        self.out = W.empty_output(op)

    def _inputs(self, sched: rc.Schedule):
        # inputs depend on the schedule only through the weight layout knobs
        key = ",".join(f"{k}={v}" for k, v in sched.as_dict().items() if k.endswith("layout"))
        if key not in self._dev:
            self._dev[key] = W.to_device(W.stored_inputs(self.op, sched, self.host))
        return self._dev[key]

    def measure(self, sched: rc.Schedule) -> dict:
        text = str(sched)
        if text in self.cache:
            return self.cache[text]
        t0 = time.time()
        rec = {"schedule": text}
        try:
            plan = rc.Plan(self.op, sched)
            ws = plan.workspace()
            t = plan.time(self._inputs(sched), self.out, ws, warmup=self.warmup, repeat=self.repeat,
                          flush=True)
            rec.update(valid=True, ms=t.median_ms, q1_ms=t.q1_ms, q3_ms=t.q3_ms, tflops=t.tflops,
                       gbps=t.gbps, reward=reward_of(self.op, t.median_ms),
                       kernel_ms=list(t.kernel_ms)[: t.nkernels])
            del plan, ws
        except rc.RCError as e:
            rec.update(valid=False, error=str(e)[:300])
        rec["eval_s"] = time.time() - t0
        self.cache[text] = rec
        if self.log:
            self.log.write(json.dumps({"kind": "measure", **rec}) + "\n")
            self.log.flush()
        return rec


def _compile_one(job):
    """Worker process: compile one schedule into the code-object cache."""
    kind, dims, flags, text, cache = job
    if cache:
        rc.set_cache_dir(cache)
    op = rc.Op(kind, dims, flags)
    return rc.precompile(op, [op.from_string(text)], nthreads=1)[0]


class ParallelGpuEvaluator:
    """GpuEvaluator shared by several searches running in threads: each
    schedule is compiled in a pool of worker processes (hipRTC serialises
    the compilations of one process), and the GPU measurements are
    serialised by a lock so that no two timings overlap.  A schedule
    requested by several searches is compiled and measured once.

    A schedule whose first timed launch takes longer than `slow_ms` is
    recorded from that launch alone (marked "coarse"): its reward is far
    below the best and more repeats would only spend GPU time."""

    def __init__(self, op: rc.Op, jobs: int = 8, repeat: int = 10, warmup: int = 2,
                 slow_ms: float = 50.0, cache_dir: Optional[str] = None, log=None,
                 time_fn=None, compile_fn=None, flush: bool = True, rotate: int = 0):
        import threading
        from concurrent.futures import ProcessPoolExecutor
        import multiprocessing as mp
        self.op, self.slow_ms, self.cache_dir, self.flush = op, slow_ms, cache_dir, flush
        # rotate > 0: the benchmark's condition - back-to-back steps cycling
        # through `rotate` copies of the inputs, no flush
        self.rotate = rotate
        self._copies: Dict[str, list] = {}
        # time_fn / compile_fn replace the GPU timing and the worker-process
        # compilation (CPU tests of the bookkeeping)
        self.inner = None if time_fn else GpuEvaluator(op, repeat=repeat, warmup=warmup, log=None)
        self._time_fn = time_fn or self._time
        self._compile_fn = compile_fn
        self.pool = None if compile_fn else ProcessPoolExecutor(max_workers=jobs,
                                                                mp_context=mp.get_context("spawn"))
        self.gpu = threading.Lock()
        self.mu = threading.Lock()
        self.pending: Dict[str, "threading.Event"] = {}
        self.cache: Dict[str, dict] = {}
        self.log = log
        self.order: List[str] = []     # distinct schedules in measurement order

    def _rotated(self, sched: rc.Schedule):
        """`rotate` device copies of the schedule's stored inputs."""
        inner = self.inner
        key = ",".join(f"{k}={v}" for k, v in sched.as_dict().items() if k.endswith("layout"))
        if key not in self._copies:
            first = inner._inputs(sched)
            self._copies[key] = [first] + [[t.clone() for t in first] for _ in range(self.rotate - 1)]
        return self._copies[key]

    def _time_rotated(self, plan, sched, ws, steps: int, warm: bool = True) -> float:
        """Milliseconds per step over `steps` back-to-back launches that cycle
        through the input copies (HIP events around the launches), after one
        warm-up pass over the copies when `warm`."""
        torch = self.inner.torch
        copies = self._rotated(sched)
        preps = [plan.prepare(c, self.inner.out, ws) for c in copies]
        for i in range(len(preps) if warm else 0):
            preps[i].launch()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for i in range(steps):
            preps[i % len(preps)].launch()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    def _time(self, sched: rc.Schedule) -> dict:
        inner = self.inner
        rec = {"schedule": str(sched)}
        if self.rotate > 0:
            try:
                plan = rc.Plan(self.op, sched)
                ws = plan.workspace()
                ms = self._time_rotated(plan, sched, ws, 1, warm=False)
                if ms > self.slow_ms:
                    rec.update(coarse=True)
                else:
                    ms = self._time_rotated(plan, sched, ws, max(inner.repeat, int(20.0 / max(ms, 1e-3))))
                rec.update(valid=True, ms=ms, q1_ms=ms, q3_ms=ms, tflops=self.op.flops() / ms / 1e9,
                           gbps=self.op.bytes() / ms / 1e6, reward=reward_of(self.op, ms))
                del plan, ws
            except rc.RCError as e:
                rec.update(valid=False, error=str(e)[:300])
            return rec
        try:
            plan = rc.Plan(self.op, sched)
            ws = plan.workspace()
            ins = inner._inputs(sched)
            t = plan.time(ins, inner.out, ws, warmup=0, repeat=1, flush=self.flush)
            if t.median_ms > self.slow_ms:
                rec.update(coarse=True)
            else:
                t = plan.time(ins, inner.out, ws, warmup=inner.warmup, repeat=inner.repeat, flush=self.flush)
            rec.update(valid=True, ms=t.median_ms, q1_ms=t.q1_ms, q3_ms=t.q3_ms, tflops=t.tflops,
                       gbps=t.gbps, reward=reward_of(self.op, t.median_ms),
                       kernel_ms=list(t.kernel_ms)[: t.nkernels])
            del plan, ws
        except rc.RCError as e:
            rec.update(valid=False, error=str(e)[:300])
        return rec

    def measure(self, sched: rc.Schedule) -> dict:
        import threading
        text = str(sched)
        with self.mu:
            if text in self.cache:
                return self.cache[text]
            ev = self.pending.get(text)
            owner = ev is None
            if owner:
                ev = self.pending[text] = threading.Event()
        if not owner:
            ev.wait()
            return self.cache[text]
        t0 = time.time()
        job = (self.op.kind, self.op.dims, self.op.flags, text, self.cache_dir)
        st = self._compile_fn(job) if self._compile_fn else self.pool.submit(_compile_one, job).result()
        t1 = time.time()
        if st != 0:
            why = "spill" if st == rc.RC_ERR_ILLEGAL_SCHEDULE else f"compile status {st}"
            rec = {"schedule": text, "valid": False, "error": why}
        else:
            with self.gpu:
                rec = self._time_fn(sched)
        rec["compile_s"], rec["eval_s"] = t1 - t0, time.time() - t0
        with self.mu:
            self.cache[text] = rec
            self.order.append(text)
            del self.pending[text]
            if self.log:
                self.log.write(json.dumps({"kind": "measure", **rec}) + "\n")
                self.log.flush()
        ev.set()
        return rec

    def close(self):
        if self.pool is not None:
            self.pool.shutdown()


def time_p0_and_tuned(op: rc.Op, name: str, tuned_text: str, repeat: int = 10, rounds: int = 2) -> dict:
    """Cold times of the untransformed program P0 and of the tuned schedule
    (cache flushed before each launch, median of `repeat` launches),
    alternating `rounds` times in one process, and the tuned schedule's
    speedup over P0: the factor that turns a search's best / tuned into its
    best speedup over the untransformed program, the quantity of the
    paper's best-speedup-against-samples table (Sec. 4.2, Table 3)."""
    import statistics
    ev = GpuEvaluator(op, repeat=repeat, warmup=1)
    pair = (("p0", op.default()), ("tuned", op.from_string(tuned_text)))
    times: Dict[str, List[float]] = {"p0": [], "tuned": []}
    for _ in range(rounds):
        for key, sched in pair:
            ev.cache.pop(str(sched), None)       # time again, not from the cache
            rec = ev.measure(sched)
            if not rec.get("valid"):
                raise RuntimeError(f"{key} schedule did not run: {rec.get('error')}")
            times[key].append(rec["ms"] * 1e3)
    p0_us, tuned_us = statistics.median(times["p0"]), statistics.median(times["tuned"])
    return {"workload": name, "p0_schedule": str(pair[0][1]), "tuned_schedule": str(pair[1][1]),
            "measurement": f"cold: a 512 MiB buffer overwritten before each timed launch; median of "
                           f"{repeat} launches; P0 and the tuned schedule alternating {rounds} times",
            "p0_us": times["p0"], "tuned_us": times["tuned"],
            "p0_reward": reward_of(op, p0_us * 1e-3), "tuned_reward": reward_of(op, tuned_us * 1e-3),
            "tuned_speedup_over_p0": p0_us / tuned_us}


PAPER_AXES = (18, 36, 72, 150, 200)   # sample counts of the paper's best-vs-samples table


def _policy_args(name: str):
    """'random', 'uct', 'uct+feedback', 'uct+sequence', 'uct+feedback+surrogate'
    (B = 4 with the surrogate, as in the replay study), ..."""
    parts = name.split("+")
    proposer = next((p for p in ("model", "sequence", "feedback") if p in parts), None)
    if proposer == "model" and "structural" in parts:
        proposer = "model_structural"
    elif proposer == "model" and "repair" in parts:
        proposer = "model_repair"
    return {"policy": parts[0], "proposer": proposer,
            "surrogate": "surrogate" in parts, "branching": 4 if "surrogate" in parts else 2}


def summarize_campaign(runs: List[dict], ref_reward: float, budget: int) -> Dict[str, dict]:
    """Per policy: mean best-so-far (as a fraction of the reference reward)
    at the paper's sample counts, and samples to reach 50 / 75 / 90 / 99 %
    of the reference per seed."""
    import statistics
    out: Dict[str, dict] = {}
    by: Dict[str, List[dict]] = {}
    for r in runs:
        by.setdefault(r["policy_name"], []).append(r)
    for name, rs in by.items():
        rs = sorted(rs, key=lambda r: r["seed"])
        at = {}
        for n in PAPER_AXES:
            if n > budget:
                continue
            vals = [(r["curve"][min(n, len(r["curve"])) - 1] if r["curve"] else 0.0) / ref_reward for r in rs]
            at[str(n)] = {"mean": statistics.fmean(vals),
                          "stderr": statistics.stdev(vals) / math.sqrt(len(vals)) if len(vals) > 1 else 0.0}

        def reach(frac):
            got = []
            for r in rs:
                k = next((i + 1 for i, v in enumerate(r["curve"]) if v >= frac * ref_reward), None)
                got.append(k)
            hit = [k for k in got if k is not None]
            return {"per_seed": got, "reached": len(hit), "of": len(got),
                    "median": statistics.median(hit) if hit else None}
        best = max(rs, key=lambda r: r["best_reward"])
        out[name] = {"best_so_far_over_reference": at, "samples_to_50pct": reach(0.50),
                     "samples_to_75pct": reach(0.75), "samples_to_90pct": reach(0.90),
                     "samples_to_99pct": reach(0.99),
                     "best_over_reference": best["best_reward"] / ref_reward,
                     "best_schedule": best["best"], "seeds": [r["seed"] for r in rs]}
    return out


def default_horizon(op: rc.Op) -> int:
    """Sequence length T: 12 transformations per GEMM block of knobs (the
    gated MLP and the MoE carry two blocks, gate/up and down, so their
    tuned schedules lie about twenty single-knob transformations from P0)."""
    return 24 if op.kind in (rc.RC_OP_GATED_MLP, rc.RC_OP_MOE) else 12


def run_campaign(op: rc.Op, name: str, policies: List[str], seeds: List[int], budget: int,
                 reference: str, jobs: int, out_path: str, cache_dir: Optional[str],
                 repeat: int = 10, slow_ms: float = 50.0, log=None, time_fn=None, compile_fn=None,
                 horizon: Optional[int] = None, flush: bool = True, rotate: int = 0) -> dict:
    """Every (policy, seed) search in its own thread against one shared
    ParallelGpuEvaluator; the reference (tuned) schedule is measured the
    same way before and after.  flush=False times warm: back-to-back
    launches on the same inputs, which a workload that fits the last-level
    cache then reads from it (no buffer is overwritten between launches).
    rotate > 0 times the benchmark's way: back-to-back steps cycling through
    that many copies of the inputs."""
    import threading
    T = horizon if horizon else default_horizon(op)
    ev = ParallelGpuEvaluator(op, jobs=jobs, repeat=repeat, slow_ms=slow_ms, cache_dir=cache_dir, log=log,
                              time_fn=time_fn, compile_fn=compile_fn, flush=flush, rotate=rotate)
    ref_sched = op.from_string(reference)
    ref0 = ev._time_fn(ref_sched)
    runs: List[dict] = []
    errors: List[str] = []
    t0 = time.time()

    def one(pname, seed):
        try:
            a = _policy_args(pname)
            r = run_search(op, ev, a["policy"], budget, seed, horizon=T, branching=a["branching"],
                           proposer=a["proposer"], surrogate=a["surrogate"])
            r["policy_name"] = pname
            r["wall_s"] = time.time() - t0
            runs.append(r)
            print(f"[campaign] {name} {pname} seed {seed}: best {r['best_reward']:.4f} "
                  f"after {r['valid']} samples ({time.time() - t0:.0f}s)", flush=True)
        except Exception as e:      # noqa: BLE001 - reported in the record
            errors.append(f"{pname} seed {seed}: {e!r}")
            print(f"[campaign] {name} {pname} seed {seed} failed: {e!r}", flush=True)

    threads = [threading.Thread(target=one, args=(p, s)) for p in policies for s in seeds]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    ref1 = ev._time_fn(ref_sched)
    ev.close()
    ref_reward = max(ref0.get("reward", 0.0), ref1.get("reward", 0.0))
    rec = {"workload": name, "dims": list(op.dims), "flags": op.flags, "budget": budget,
           "seeds": seeds, "policies": policies, "horizon": T,
           "measurement": (f"benchmark: back-to-back steps cycling through {rotate} input copies, "
                           f"mean over at least {repeat} steps and 20 ms" if rotate > 0 else
                           (f"cold: a 512 MiB buffer overwritten before each timed launch; median of "
                            if flush else "warm: back-to-back launches on the same inputs; median of ")
                           + f"{repeat} launches (one launch when it exceeds {slow_ms:g} ms)"),
           "reward": "fraction of the binding roofline (bf16 MFMA peak or HBM bandwidth) at the median",
           "reference_schedule": reference,
           "reference_reward": ref_reward, "reference_us": [ref0.get("ms", 0) * 1e3, ref1.get("ms", 0) * 1e3],
           "distinct_schedules": len(ev.order),
           "invalid": sum(1 for r in ev.cache.values() if not r.get("valid")),
           "wall_s": time.time() - t0, "errors": errors,
           "summary": summarize_campaign(runs, ref_reward, budget) if runs else {},
           "runs": [{k: v for k, v in r.items()} for r in sorted(runs, key=lambda r: (r["policy_name"], r["seed"]))]}
    with open(out_path, "w") as f:
        json.dump(rec, f, indent=1)
    return rec


class TableEvaluator:
    """Measured samples replayed from a table: a previous run's JSONL, or a
    TSV of one sub-space (comment lines, a '# fixed: knob=v,...' line, a
    header of the varying knobs and one or more timing columns named 'us' or
    '*_us', then one row per schedule with its median microseconds or the
    reason it was rejected).  `column` picks the timing column (default: the
    last)."""

    def __init__(self, path: str, op: Optional[rc.Op] = None, column: Optional[str] = None):
        self.table: Dict[str, dict] = {}
        if path.endswith(".tsv"):
            if op is None:
                raise ValueError("a TSV table needs the operator")
            fixed, header = "", None
            for line in open(path):
                line = line.rstrip("\n")
                if line.startswith("# fixed:"):
                    fixed = line.split(":", 1)[1].strip()
                elif line.startswith("#") or not line:
                    continue
                elif header is None:
                    header = line.split("\t")
                    nk = sum(1 for h in header if not (h == "us" or h.endswith("_us")))
                    col = header.index(column) if column else len(header) - 1
                else:
                    vals = line.split("\t")
                    text = ",".join([fixed] + [f"{k}={v}" for k, v in zip(header[:nk], vals[:nk])])
                    key = str(op.from_string(text))
                    if vals[col] in ("spill", "error"):
                        self.table[key] = {"schedule": key, "valid": False, "error": vals[col]}
                    else:
                        ms = float(vals[col]) * 1e-3
                        self.table[key] = {"schedule": key, "valid": True, "ms": ms,
                                           "reward": reward_of(op, ms)}
            return
        for line in open(path):
            r = json.loads(line)
            if "schedule" in r and "valid" in r:
                self.table[r["schedule"]] = r

    def contains(self, sched: rc.Schedule) -> bool:
        """Whether the schedule lies in the measured space (outside it the
        table plays the part of a compiler that rejects it)."""
        return str(sched) in self.table

    def measure(self, sched: rc.Schedule) -> dict:
        return self.table.get(str(sched), {"schedule": str(sched), "valid": False, "error": "not in table"})


class FeedbackProposer:
    """Expansion proposals from measured history (Sec. 3.1's proposal step,
    with the language model replaced by a plain rule): take the `top`
    best schedules measured so far, find each knob's most common value among
    them, and propose setting one knob (chosen at random among those where
    the node disagrees with that consensus) to its consensus value.  With
    `sequence`, the proposal is a sequence of such transformations applied
    together (Sec. 3.1 proposes sequences): every disagreeing knob set to its
    consensus value, then a random two or three of them, then each alone, as
    alternatives tried in that order.  Before `warm` valid samples exist, or
    when the node already agrees everywhere, it proposes nothing and the
    search expands with a random legal transformation."""

    def __init__(self, op: rc.Op, seed: int, top: int = 8, warm: int = 8, sequence: bool = False):
        import random
        self.op, self.top, self.warm, self.sequence = op, top, warm, sequence
        self.rng = random.Random(seed)
        self.names = op.knob_names()
        self.classes = [op.knob_class(i) for i in range(len(self.names))]
        self.seen: List[tuple] = []          # (reward, {knob: value})

    def record(self, sched: rc.Schedule, reward: Optional[float], measured: bool = True):
        if reward is not None:
            self.seen.append((reward, sched.as_dict()))

    def __call__(self, at: rc.Schedule, parent, grandparent) -> str:
        if len(self.seen) < self.warm:
            return ""
        best = sorted(self.seen, key=lambda t: -t[0])[: self.top]
        cur = at.as_dict()
        moves = []
        for i, name in enumerate(self.names):
            counts: Dict[int, int] = {}
            for _, d in best:
                counts[d[name]] = counts.get(d[name], 0) + 1
            value = max(counts, key=lambda v: (counts[v], -abs(v - cur[name])))
            if value != cur[name]:
                moves.append(f"{self.classes[i]}({name}={value})")
        if not moves:
            return ""
        if not self.sequence:
            return self.rng.choice(moves)
        self.rng.shuffle(moves)
        alts = []
        if len(moves) > 1:
            alts.append(" + ".join(moves))
        if len(moves) > 3:
            alts.append(" + ".join(moves[: self.rng.choice((2, 3))]))
        return "\n".join(alts + moves)


class ModelProposer:
    """Expansion proposals guided by a learned model of the measured rewards
    (Sec. 3.1's proposal step, with the language model's judgement of which
    program to try next replaced by the regression model of Sec. 3.2's
    f-hat).  A pool of candidates is drawn around the best measured
    schedules: each of the `top` best, changed in one to four randomly
    chosen knobs, kept if legal and not measured yet.  The model (the
    search's surrogate when it has one, else an ensemble of randomised
    regression trees fitted here on the measurements) scores the pool; each
    expansion is offered the `offer` best-scoring candidates, best first,
    each as the sequence of transformations that turns the expanded node
    into it (the search keeps the first that is legal and not in its tree);
    a candidate offered first is not offered again.  The pool is redrawn
    and rescored whenever the model is refitted.  Before `warm`
    measurements it proposes nothing (random expansion).  With `repair`,
    an illegal candidate is not dropped: up to `repair` times, the knob
    that the legality check's reason names is set to the value it asks
    for, or redrawn (`REPAIR_RULES`), until the candidate is legal, so the
    pool also holds the coupled multi-knob moves that legality forces (a
    staging path with the vector width and layout it needs, a tile with a
    matching wave split, a ring that fits the LDS).  With `structural`,
    each elite also yields the `STRUCTURAL` moves of every GEMM block
    (repaired the same way) besides its random mutations."""

    # reason text -> knobs of the block the reason names (its prefix before
    # ':'), each with the value the reason asks for or None (redraw)
    REPAIR_RULES = [
        ("(vec 8)", [("vec", 8)]),
        ("weights stored N x K", [("layout", 1)]),
        ("two waves per SIMD (occ 2)", [("occ", 2)]),
        ("fused SwiGLU", [("fuse", 1)]),
        ("tail split", [("tail", 0)]),
        ("do not combine", [("split", 1)]),
        ("K-split tail", [("tail", 1)]),
        ("tile_m/waves_m", [("waves_m", None)]),
        ("tile_n/waves_n", [("waves_n", None)]),
        ("needs 8 waves", [("waves_m", None), ("waves_n", None)]),
        ("wave-loads", [("waves_m", None), ("waves_n", None), ("tile_k", None)]),
        ("ring stages", [("tile_k", None), ("occ", None), ("tile_n", None)]),
        ("LDS", [("tile_k", None), ("occ", None), ("stages", None)]),
        ("registers", [("waves_m", None), ("waves_n", None), ("occ", None)]),
        ("accumulators", [("waves_m", None), ("waves_n", None), ("occ", None)]),
        ("vector-memory counter", [("tile_k", None), ("waves_m", None)]),
        ("unroll", [("unroll", 1)]),
        ("threads x", [("vec", None), ("waves_n", None)]),
        ("does not divide", [("tile_k", None), ("tile_n", None)]),
        ("padded im2col", [("stages", None)]),
    ]

    # structural moves tried on every elite with `structural`: staging on the
    # direct-to-LDS ring, the tail and K splits, the MoE row skip, the tile
    # orders (each completed by the repair)
    STRUCTURAL = [({"stages": 7, "vec": 8, "layout": 1},), ({"tail": 1},), ({"tail": 2},),
                  ({"split": 2},), ({"split": 4},), ({"skip": 1},), ({"grid": 1},), ({"grid": 2},)]

    def __init__(self, op: rc.Op, seed: int, surrogate=None, top: int = 8, warm: int = 16,
                 refit: int = 8, per_elite: int = 48, offer: int = 4, repair: int = 0,
                 structural: bool = False):
        import random
        self.op, self.sur, self.repair, self.structural = op, surrogate, repair, structural
        self.top, self.warm, self.refit, self.per_elite, self.offer = top, warm, refit, per_elite, offer
        self.rng = random.Random(seed)
        self.seed = seed
        self.names = op.knob_names()
        self.classes = [op.knob_class(i) for i in range(len(self.names))]
        self.values = [op.knob_values(i) for i in range(len(self.names))]
        self.measured: Dict[str, float] = {}      # schedule text -> measured reward (0 if invalid)
        self.X: List[List[float]] = []
        self.y: List[float] = []
        self.model = None
        self.fit_at = -1                           # measurements behind this proposer's own model
        self.rank_at = -1                          # measurements behind the model that ranked the pool
        self.ranked: List[tuple] = []             # (schedule text, knob values), best predicted first
        self.used: set = set()                     # candidates already offered first

    def record(self, sched: rc.Schedule, reward: Optional[float], measured: bool = True):
        if not measured:
            return
        text = str(sched)
        if text in self.measured:
            return
        self.measured[text] = reward if reward is not None else 0.0
        if self.sur is None:
            self.X.append(schedule_features(self.op, sched))
            self.y.append(reward if reward is not None else 0.0)

    def _predictor(self):
        """(model, number of measurements it was fitted on), or (None, 0)."""
        if self.sur is not None:
            return self.sur.model, self.sur.fitted_at
        n = len(self.y)
        if n >= self.warm and (self.model is None or n - self.fit_at >= self.refit):
            from sklearn.ensemble import ExtraTreesRegressor
            import numpy as np
            m = ExtraTreesRegressor(n_estimators=48, min_samples_leaf=2, random_state=self.seed)
            m.fit(np.array(self.X, dtype=np.float64), np.array(self.y, dtype=np.float64))
            self.model, self.fit_at = m, n
        return self.model, self.fit_at

    def _repair_step(self, d: Dict[str, int], why: str) -> None:
        """Change the knob(s) the legality reason `why` points at."""
        block = why.split(":", 1)[0] if ":" in why else ""
        prefix = block + "." if block in ("up", "down") else ""
        for key, fixes in self.REPAIR_RULES:
            if key in why:
                name, value = fixes[self.rng.randrange(len(fixes))]
                for full in (prefix + name, name):
                    if full in d:
                        i = self.names.index(full)
                        d[full] = value if value is not None and value in self.values[i] else \
                            self.rng.choice(self.values[i])
                        return
        i = self.rng.randrange(len(self.names))     # no rule: redraw any knob
        d[self.names[i]] = self.rng.choice(self.values[i])

    def _rank(self, model):
        import numpy as np
        elites = sorted(((r, t) for t, r in self.measured.items() if r > 0), reverse=True)[: self.top]
        pool: Dict[str, rc.Schedule] = {}
        blocks = sorted({n.split(".")[0] + "." for n in self.names if n.startswith(("up.", "down."))}) or [""]
        for _, text in elites:
            base = self.op.from_string(text).as_dict()
            moves = []
            if self.structural:
                for (move,) in self.STRUCTURAL:
                    for b in blocks:
                        m = {b + k: v for k, v in move.items() if b + k in base}
                        if m and any(base[k] != v for k, v in m.items()):
                            moves.append(m)
            for j in range(self.per_elite + len(moves)):
                d = dict(base)
                if j < len(moves):
                    d.update(moves[j])
                else:
                    for _ in range(self.rng.randint(1, 4)):
                        i = self.rng.randrange(len(self.names))
                        d[self.names[i]] = self.rng.choice(self.values[i])
                s = self.op.schedule(**d)
                for _ in range(self.repair):
                    why = s.validate()
                    if not why:
                        break
                    self._repair_step(d, why)
                    s = self.op.schedule(**d)
                t = str(s)
                if t in pool or t in self.measured or s.validate():
                    continue
                pool[t] = s
        if not pool:
            self.ranked = []
            return
        scheds = list(pool.values())
        feats = self.sur.features if self.sur is not None else (lambda s: schedule_features(self.op, s))
        pred = model.predict(np.array([feats(s) for s in scheds], dtype=np.float64))
        order = sorted(range(len(scheds)), key=lambda k: -pred[k])
        self.ranked = [(str(scheds[k]), scheds[k].as_dict()) for k in order]

    def __call__(self, at: rc.Schedule, parent, grandparent) -> str:
        if len(self.measured) < self.warm:
            return ""
        model, fitted = self._predictor()
        if model is None:
            return ""
        if fitted != self.rank_at or not self.ranked:
            self.rank_at = fitted
            self._rank(model)
        cur = at.as_dict()
        alts = []
        for text, d in self.ranked:
            if text in self.measured or text in self.used:
                continue
            moves = [f"{self.classes[i]}({n}={d[n]})" for i, n in enumerate(self.names) if d[n] != cur[n]]
            if moves:
                if not alts:
                    self.used.add(text)
                alts.append(" + ".join(moves))
            if len(alts) == self.offer:
                break
        return "\n".join(alts)


CUS, LDS_BYTES = 256, 163840          # MI355X compute units; LDS one workgroup may use


def _gemm_block_features(d: Dict[str, int], pre: str, M: int, N: int, K: int, nb: int) -> List[float]:
    """Resource and shape features of one bf16 GEMM stage (a cheap analytic
    description of what the knobs imply: the cost-model inputs of Sec. 3.2's
    f-hat)."""
    tm, tn, tk = d[pre + "tile_m"], d[pre + "tile_n"], d[pre + "tile_k"]
    waves = d[pre + "waves_m"] * d[pre + "waves_n"]
    wtm, wtn = tm / d[pre + "waves_m"], tn / d[pre + "waves_n"]
    st, occ = d[pre + "stages"], d[pre + "occ"]
    stage_bytes = (tm + nb * tn) * tk * 2
    nbuf = {1: 1, 2: 2, 3: 2, 4: 3, 5: 2, 6: 3}.get(st, 0)
    if st == 7:
        wgs = max(1, -(-occ * 4 // waves))
        nbuf = min(12, LDS_BYTES // (wgs * stage_bytes))
    lds = nbuf * stage_bytes
    acc = nb * tm * tn / (64 * waves)
    per_cu = max(1, min(LDS_BYTES // max(lds, 1), max(1, int(512 // max(acc + 64, 1)) * 4 // waves), 32 // waves))
    split = max(1, d.get(pre + "split", 1))      # K range cut over this many workgroups per tile
    K //= split
    n_wg = -(-M // tm) * (N // tn) * split
    slots = CUS * per_cu
    rounds = n_wg / slots
    tail = rounds / max(1, -(-n_wg // slots))
    return [math.log2(tm), math.log2(tn), math.log2(tk), waves, wtm, wtn, acc, lds / 1024.0, per_cu,
            rounds, tail, (wtm + nb * wtn) / (wtm * nb * wtn), (tm + nb * tn) / (tm * nb * tn),
            K / tk, st, d[pre + "mfma"], d[pre + "vec"], occ]


def schedule_features(op: rc.Op, sched: rc.Schedule) -> List[float]:
    """Surrogate input: the raw knob values plus analytic features derived
    from them and the operator's shape (tiles per compute unit, rounds of
    workgroups and the last round's fill, accumulator registers, LDS bytes,
    operand bytes per FLOP from LDS and from memory, dependent key tiles of
    the longest attention query tile)."""
    d = sched.as_dict()
    f = [float(v) for v in d.values()]
    D = op.dims
    if op.kind == rc.RC_OP_GATED_MLP:
        T, Hd, I = D
        f += _gemm_block_features(d, "up.", T, I, Hd, 2) + _gemm_block_features(d, "down.", T, Hd, I, 1)
    elif op.kind == rc.RC_OP_MOE:
        T, Hd, E, I, k = D
        rows = T * k + E * 64      # routed rows plus about half a tile of padding per expert
        f += _gemm_block_features(d, "up.", rows, I, Hd, 2) + _gemm_block_features(d, "down.", rows, Hd, I, 1)
    elif op.kind == rc.RC_OP_CONV2D:
        N, H, W, C, K, R, S, pad = D
        P, Q = H + 2 * pad - R + 1, W + 2 * pad - S + 1
        f += _gemm_block_features(d, "", N * P * Q, K, R * S * C, 1)
    elif op.kind == rc.RC_OP_ATTENTION:
        B, H, S, Dh = D
        bm, bn, w, sp, ch = d["block_m"], d["block_n"], d["waves"], d["splits"], d["chunk"]
        nkt = -(-S // bn)
        chain = (ch if ch > 0 else nkt) / sp          # dependent key tiles of the longest work item
        nq = -(-S // bm)
        items = B * H * nq * (1 if ch == 0 else -(-nkt // ch))
        f += [bm / w, w * sp, chain, items / CUS, bm * bn / (64.0 * w), d["stages"] * 1.0]
    return f


class SurrogateEvaluator:
    """Rollout rewards from a learned surrogate (Sec. 3.2: the terminal
    program of a rollout is scored by a cheap learned model f-hat rather
    than on hardware).  Wraps a real evaluator.  The first `warm` distinct
    schedules are measured; after that an ensemble of randomised regression
    trees, refitted every `refit` measurements on the measured knob vectors,
    predicts each new rollout terminal.  A terminal is measured only when
    its prediction is within `margin` of the best measured reward (or, with
    probability `explore`, at random); otherwise the prediction is the
    rollout reward and no sample is spent.  Only measurements are samples:
    `curve` is the best measured reward after each of them.  A schedule the
    inner evaluator places outside its space (a replayed table's `contains`)
    is invalid at no cost, as it is without the surrogate.  A schedule
    measured before (by an earlier tree of the same run) returns its
    measurement again at no cost."""

    def __init__(self, op: rc.Op, inner, seed: int, warm: int = 16, refit: int = 8,
                 margin: float = 0.9, explore: float = 0.05, feature_set: str = "analytic"):
        import random
        self.op, self.inner, self.seed = op, inner, seed
        self.warm, self.refit, self.margin, self.explore = warm, refit, margin, explore
        self.feature_set = feature_set          # "analytic" (schedule_features) or "raw" knob values
        self.rng = random.Random(seed)
        self.X: List[List[int]] = []
        self.y: List[float] = []
        self.model = None
        self.fitted_at = 0
        self.measured = 0
        self.predicted = 0
        self.calls = 0
        self.known: Dict[str, Optional[float]] = {}
        self.best = 0.0
        self.best_text: Optional[str] = None
        self.curve: List[float] = []

    def features(self, sched: rc.Schedule) -> List[float]:
        if self.feature_set == "raw":
            return [float(v) for v in sched.as_dict().values()]
        return schedule_features(self.op, sched)

    def _fit(self):
        from sklearn.ensemble import ExtraTreesRegressor
        import numpy as np
        m = ExtraTreesRegressor(n_estimators=48, min_samples_leaf=2, random_state=self.seed)
        m.fit(np.array(self.X, dtype=np.float64), np.array(self.y, dtype=np.float64))
        self.model, self.fitted_at = m, len(self.y)

    def _measure(self, sched: rc.Schedule) -> Optional[float]:
        r = self.inner.measure(sched)
        reward = r["reward"] if r.get("valid") else None
        self.known[str(sched)] = reward
        self.X.append(self.features(sched))
        self.y.append(reward if reward is not None else 0.0)   # invalid: learn it as worthless
        if reward is not None:
            self.measured += 1
            if reward > self.best:
                self.best, self.best_text = reward, str(sched)
            self.curve.append(self.best)
        return reward

    def __call__(self, sched: rc.Schedule) -> Optional[float]:
        self.calls += 1
        contains = getattr(self.inner, "contains", None)
        if contains is not None and not contains(sched):
            return None
        if str(sched) in self.known:
            return self.known[str(sched)]
        if len(self.y) < self.warm:
            return self._measure(sched)
        if self.model is None or len(self.y) - self.fitted_at >= self.refit:
            self._fit()
        import numpy as np
        pred = float(self.model.predict(np.array([self.features(sched)], dtype=np.float64))[0])
        if pred >= self.margin * self.best or self.rng.random() < self.explore:
            return self._measure(sched)
        self.predicted += 1
        return max(pred, 0.0)


def run_search(op, evaluator, policy: str, budget: int, seed: int, horizon=12, branching=2,
               c=math.sqrt(2.0), proposer: Optional[str] = None, surrogate: bool = False,
               surrogate_features: str = "analytic"):
    sur = SurrogateEvaluator(op, evaluator, seed, feature_set=surrogate_features) if surrogate else None
    if proposer in ("feedback", "sequence"):
        prop = FeedbackProposer(op, seed, sequence=proposer == "sequence")
    elif proposer == "model":
        prop = ModelProposer(op, seed, surrogate=sur)
    elif proposer == "model_repair":
        prop = ModelProposer(op, seed, surrogate=sur, repair=6)
    elif proposer == "model_structural":
        prop = ModelProposer(op, seed, surrogate=sur, repair=6, structural=True)
    else:
        prop = None

    def ev(s):
        if sur is not None:
            before = len(sur.y)                  # measurements, valid or not
            reward = sur(s)
            measured = len(sur.y) != before
        else:
            r = evaluator.measure(s)
            reward = r["reward"] if r.get("valid") else None
            measured = True
        if prop is not None:
            prop.record(s, reward, measured=measured)
        return reward

    # with a surrogate only measurements count, so the driver's own budget
    # (which counts every rollout reward) is a loose cap
    def new_tree(k):
        return rc.Search(op, ev, policy=POLICIES[policy], budget=budget * (40 if sur else 1), horizon=horizon,
                         branching=branching, c=c, seed=seed + 7919 * k, propose=prop)
    srch = new_tree(0)
    trees = 1
    if sur is None:
        srch.run()
    else:
        # With free rollouts a tree of at most B children per node and depth T
        # runs out of unscored schedules long before the measurements are
        # spent: when 20 x budget rollouts bring nothing new, a fresh tree
        # (another seed; the surrogate and the measurements carry over) takes
        # over, up to 16 trees.
        while sur.measured < budget and trees <= 16:
            last, idle = sur.calls, 0
            while sur.measured < budget and idle < 20 * budget and not srch.step():
                idle = 0 if sur.calls != last else idle + 1
                last = sur.calls
            if sur.measured < budget and trees < 16:
                srch = new_tree(trees)
            trees += 1
    hist = srch.history()
    if sur is None:
        try:
            best, reward, idx = srch.best()
            best_text = str(best)
        except rc.RCError:
            best_text, reward, idx = None, 0.0, -1
        curve = [h["best_so_far"] for h in hist if h["valid"]]
    else:
        best_text, reward, idx = sur.best_text, sur.best, len(sur.curve) - 1
        curve = sur.curve
    # samples to reach the run's best (within 1%)
    to_best = next((i + 1 for i, v in enumerate(curve) if v >= 0.99 * reward), None) if curve else None
    return {"policy": policy, "proposer": proposer, "surrogate": surrogate, "trees": min(trees, 16),
            "fallbacks": srch.fallbacks() if prop else None,
            "seed": seed, "budget": budget, "valid": len(curve) if sur else sum(h["valid"] for h in hist),
            "invalid": sum(not h["valid"] for h in hist), "predicted": sur.predicted if sur else 0,
            "best": best_text, "best_reward": reward,
            "best_index": idx, "samples_to_best": to_best, "curve": curve}


def _parse_seeds(text: str) -> List[int]:
    out = []
    for part in text.split(","):
        if "-" in part:
            a, b = part.split("-")
            out.extend(range(int(a), int(b) + 1))
        elif part:
            out.append(int(part))
    return out


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--workload", required=True, choices=list(W.WORKLOADS))
    ap.add_argument("--policy", default="uct", choices=list(POLICIES) + ["list"])
    ap.add_argument("--budget", type=int, default=64)
    ap.add_argument("--seeds", default="0")
    ap.add_argument("--horizon", type=int, default=0,
                    help="sequence length T (default: 12 per GEMM block of knobs, 24 for the MLP and MoE)")
    ap.add_argument("--branching", type=int, default=2)
    ap.add_argument("--c", type=float, default=math.sqrt(2.0))
    ap.add_argument("--proposer", default=None, choices=["feedback", "sequence", "model", "model_repair", "model_structural"],
                    help="expansion proposals from measured history (default: random legal)")
    ap.add_argument("--surrogate", action="store_true",
                    help="score rollouts with a learned surrogate; measure only promising ones")
    ap.add_argument("--surrogate-features", default="analytic", choices=["analytic", "raw"],
                    help="surrogate inputs: knob values plus analytic resource features, or knob values only")
    ap.add_argument("--repeat", type=int, default=10)
    ap.add_argument("--out", default="tune_out")
    ap.add_argument("--enumerate", action="store_true", help="list the whole legal space")
    ap.add_argument("--walks", type=int, default=0, help="list N random-walk schedules")
    ap.add_argument("--precompile", action="store_true", help="compile the listed schedules (CPU)")
    ap.add_argument("--list-file", default=None, help="measure the schedules in this file (policy list)")
    ap.add_argument("--replay", default=None, help="evaluate against a measured table (JSONL or TSV)")
    ap.add_argument("--column", default=None, help="timing column of a TSV table (default: the last)")
    ap.add_argument("--threads", type=int, default=os.cpu_count() or 8)
    ap.add_argument("--cache-dir", default=os.path.join(HERE, "jit_cache"))
    ap.add_argument("--campaign", default=None, metavar="POLICIES",
                    help="comma-separated policies (random, uct, uct+feedback, uct+sequence, uct+model, "
                         "each optionally +surrogate) searched concurrently over --seeds with parallel "
                         "compilation; writes <out>/<workload>.campaign.json")
    ap.add_argument("--bench-timing", type=int, default=0, metavar="R",
                    help="campaign timing as the benchmark's: back-to-back steps through R input copies")
    ap.add_argument("--warm", action="store_true",
                    help="campaign timing without the cache flush (back-to-back launches on the same inputs)")
    ap.add_argument("--jobs", type=int, default=12, help="compile worker processes (--campaign)")
    ap.add_argument("--p0", action="store_true",
                    help="time the untransformed program P0 and the tuned schedule cold in one process "
                         "(the tuned schedule's speedup over P0)")
    ap.add_argument("--slow-ms", type=float, default=50.0,
                    help="a schedule slower than this on its first launch is timed once (--campaign)")
    args = ap.parse_args(argv)

    rc.set_cache_dir(args.cache_dir)
    op = W.workload_op(args.workload)
    os.makedirs(args.out, exist_ok=True)

    if args.enumerate or args.walks:
        space = legal_space(op) if args.enumerate else random_walk_space(op, args.walks, 12345)
        path = os.path.join(args.out, f"{args.workload}.space.txt")
        with open(path, "w") as f:
            for s in space:
                f.write(str(s) + "\n")
        print(f"{len(space)} legal schedules -> {path}", flush=True)
        if args.precompile:
            t0 = time.time()
            chunk = 256
            bad = 0
            for i in range(0, len(space), chunk):
                st = rc.precompile_parallel(op, space[i:i + chunk], args.threads, args.cache_dir)
                bad += sum(1 for x in st if x != 0)
                print(f"compiled {min(i + chunk, len(space))}/{len(space)} ({bad} rejected) "
                      f"{time.time() - t0:.0f}s", flush=True)
        return

    if args.p0:
        tuned = json.load(open(os.path.join(HERE, "tuned.json")))
        rec = time_p0_and_tuned(op, args.workload, tuned[args.workload], repeat=args.repeat)
        with open(os.path.join(args.out, f"{args.workload}.p0.json"), "w") as f:
            json.dump(rec, f, indent=1)
        print(json.dumps({k: rec[k] for k in ("workload", "p0_us", "tuned_us", "tuned_speedup_over_p0")}),
              flush=True)
        return

    if args.campaign:
        tuned = json.load(open(os.path.join(HERE, "tuned.json")))
        pols = [p for p in args.campaign.split(",") if p]
        path = os.path.join(args.out, f"{args.workload}.campaign.json")
        log = open(os.path.join(args.out, f"{args.workload}.campaign.jsonl"), "a")
        rec = run_campaign(op, args.workload, pols, _parse_seeds(args.seeds), args.budget,
                           tuned[args.workload], args.jobs, path, args.cache_dir, repeat=args.repeat,
                           slow_ms=args.slow_ms, log=log, horizon=args.horizon, flush=not args.warm,
                           rotate=args.bench_timing)
        print(json.dumps({k: rec[k] for k in ("workload", "reference_reward", "distinct_schedules",
                                               "invalid", "wall_s", "errors")}), flush=True)
        for pname, sm in rec["summary"].items():
            print(pname, json.dumps({k: (sm[k] if k == "best_over_reference" else sm[k]["median"])
                                     for k in ("best_over_reference", "samples_to_50pct", "samples_to_75pct",
                                               "samples_to_90pct", "samples_to_99pct")}), flush=True)
        return

    tag = args.policy + (f"+{args.proposer}" if args.proposer else "") + ("+surrogate" if args.surrogate else "")
    if args.surrogate and args.surrogate_features != "analytic":
        tag += "-" + args.surrogate_features
    log = open(os.path.join(args.out, f"{args.workload}.{tag}.jsonl"), "a")
    if args.replay:
        evaluator = TableEvaluator(args.replay, op, args.column)
    else:
        evaluator = GpuEvaluator(op, repeat=args.repeat, log=log)

    if args.policy == "list":
        scheds = [op.from_string(line.strip()) for line in open(args.list_file) if line.strip()]
        t0 = time.time()
        for i, s in enumerate(scheds):
            r = evaluator.measure(s)
            if (i + 1) % 25 == 0 or i + 1 == len(scheds):
                print(f"measured {i + 1}/{len(scheds)} {time.time() - t0:.0f}s", flush=True)
        best = max((r for r in evaluator.cache.values() if r.get("valid")), key=lambda r: r["reward"],
                   default=None)
        print(json.dumps({"kind": "list_best", "workload": args.workload, **(best or {})}), flush=True)
        log.write(json.dumps({"kind": "list_best", "workload": args.workload, **(best or {})}) + "\n")
        return

    horizon = args.horizon if args.horizon else default_horizon(op)
    for seed in _parse_seeds(args.seeds):
        t0 = time.time()
        res = run_search(op, evaluator, args.policy, args.budget, seed, horizon, args.branching, args.c,
                         args.proposer, args.surrogate, args.surrogate_features)
        res.update(workload=args.workload, kind="search", wall_s=time.time() - t0)
        log.write(json.dumps(res) + "\n")
        log.flush()
        print(json.dumps({k: v for k, v in res.items() if k != "curve"}), flush=True)


if __name__ == "__main__":
    main()
