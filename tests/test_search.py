"""CPU tests of the search driver (Sec. 3.2) against fake evaluators, and of
the report metrics against Table 1."""
import csv
import math
import random
import os

import pytest

from paper_2506_01374_amd import rc, report

HERE = os.path.dirname(os.path.abspath(__file__))
C = math.sqrt(2.0)


def tiny_op():
    # fp32 GEMM 16x16x4: only stages {1,2} x layout {0,1} are legal.
    return rc.Op(rc.RC_OP_GEMM_F32, (16, 16, 4))


def test_tiny_space_has_four_points():
    op = tiny_op()
    from paper_2506_01374_amd.tune import legal_space
    pts = {(s["stages"], s["layout"]) for s in legal_space(op)}
    assert pts == {(1, 0), (2, 0), (1, 1), (2, 1)}


def test_uct_selection_and_backprop_match_hand_computation():
    op = tiny_op()
    rewards = {(2, 0): 0.3, (1, 1): 0.5, (2, 1): 0.9, (1, 0): 0.1}
    evals = []

    def ev(s):
        evals.append((s["stages"], s["layout"]))
        return rewards[(s["stages"], s["layout"])]

    # The proposer fixes expansion order: child A = stages 2, child B = layout 1.
    prop = lambda at, par, gpar: "ComputeLocation(stages=2);Layout(layout=1)"
    s = rc.Search(op, ev, policy=rc.RC_POLICY_UCT, budget=3, horizon=1, branching=2, c=C, seed=0,
                  propose=prop)
    A = [op.parse("ComputeLocation(stages=2)")]
    B = [op.parse("Layout(layout=1)")]
    s.step()
    s.step()
    assert evals == [(2, 0), (1, 1)]
    assert s.node_stats(A) == (1, pytest.approx(0.3))
    assert s.node_stats(B) == (1, pytest.approx(0.5))
    assert s.node_stats([]) == (2, pytest.approx(0.8))
    # Iteration 3: both children visited once; UCT = W/N + c sqrt(ln 2 / 1) -> B.
    s.step()
    assert s.node_stats(B) == (2, pytest.approx(1.0))
    # Iteration 4: UCT_A = 0.3 + c sqrt(ln 3 / 1) = 1.782 > UCT_B = 0.5 + c sqrt(ln 3 / 2) = 1.548.
    ua = 0.3 + C * math.sqrt(math.log(3) / 1)
    ub = 0.5 + C * math.sqrt(math.log(3) / 2)
    assert ua > ub
    s.step()
    assert s.node_stats(A) == (2, pytest.approx(0.6))
    # Iteration 5: UCT_A = 0.3 + c sqrt(ln 4 / 2) < UCT_B = 0.5 + c sqrt(ln 4 / 2) -> B.
    s.step()
    assert s.node_stats(B) == (3, pytest.approx(1.5))
    assert s.node_stats([]) == (5, pytest.approx(0.3 + 0.5 + 0.5 + 0.3 + 0.5))
    # Re-selected leaves are not measured again (dedupe): two evaluations only.
    assert evals == [(2, 0), (1, 1)]
    assert s.fallbacks() == 0


def test_fallback_when_no_proposal_is_valid():
    op = tiny_op()
    calls = []
    prop = lambda at, par, gpar: "Make it faster please;TileSize(tile_m=48);Unroll(layout=1)"
    s = rc.Search(op, lambda x: calls.append(1) or 0.5, policy=rc.RC_POLICY_UCT, budget=3,
                  horizon=2, branching=2, seed=1, propose=prop)
    s.run()
    assert s.fallbacks() >= 2          # every expansion fell back to a random legal move
    best, r, _ = s.best()
    assert r == 0.5


def test_sequence_proposals_apply_their_steps_together():
    # An alternative chaining transformations with '+' is applied as one
    # expansion (Sec. 3.1 proposes sequences): unparsable steps are
    # discarded, intermediate schedules need not be legal, an illegal result
    # gives way to the next alternative.
    op = tiny_op()
    evals = []
    prop = lambda at, par, gpar: "ComputeLocation(stages=2) + no such step + Layout(layout=1)"
    s = rc.Search(op, lambda x: evals.append((x["stages"], x["layout"])) or 0.5, policy=rc.RC_POLICY_UCT,
                  budget=1, horizon=1, branching=2, seed=0, propose=prop)
    s.step()
    assert evals == [(2, 1)] and s.fallbacks() == 0
    g = rc.Op(rc.RC_OP_GEMM_F32, (128, 128, 128))
    with pytest.raises(rc.RCError, match="multiple of 16"):
        g.default().apply(g.parse("Parallel(waves_m=2)"))            # alone it is illegal
    seen = []
    prop = lambda at, par, gpar: ("Parallel(waves_m=2) + TileSize(tile_m=32)\n"       # illegal result
                                  "Parallel(waves_m=2) + TileSize(tile_m=32) + TileSize(tile_k=16)")
    s = rc.Search(g, lambda x: seen.append((x["tile_m"], x["waves_m"], x["tile_k"])) or 0.5,
                  policy=rc.RC_POLICY_UCT, budget=1, horizon=1, branching=2, seed=0, propose=prop)
    s.step()
    assert seen == [(32, 2, 16)] and s.fallbacks() == 0


def test_sequence_feedback_proposer_offers_the_consensus_jump_first():
    from paper_2506_01374_amd.tune import FeedbackProposer, legal_space
    op = rc.Op(rc.RC_OP_GEMM_F32, (128, 128, 128))
    space = legal_space(op)
    prop = FeedbackProposer(op, seed=0, top=4, warm=4, sequence=True)
    good = [s for s in space if s["tile_m"] == 64 and s["tile_n"] == 64 and s["vec"] == 4][:4]
    for s in good:
        prop.record(s, 1.0)
    at = op.default()
    lines = prop(at, None, None).split("\n")
    first = [t.strip() for t in lines[0].split("+")]
    assert len(first) >= 3 and all(op.parse(t) for t in first)
    assert any("tile_m=64" in t for t in first) and any("vec=4" in t for t in first)
    singles = [l for l in lines if "+" not in l]
    assert set(singles) == set(first)             # then every step alone
    d = at.as_dict()
    for t in first:                               # each step moves toward the consensus
        name, value = t[t.index("(") + 1:-1].split("=")
        assert d[name] != int(value)


def test_model_proposer_offers_the_best_predicted_unmeasured_schedules():
    from paper_2506_01374_amd.tune import ModelProposer, legal_space
    op = rc.Op(rc.RC_OP_GEMM_F32, (128, 128, 128))
    space = legal_space(op)
    prop = ModelProposer(op, seed=0, top=4, warm=16, offer=3)
    at = op.default()
    assert prop(at, None, None) == ""             # nothing before the warm-up
    rng = random.Random(1)
    for s in rng.sample(space, 60):
        prop.record(s, synthetic_reward(s))
    lines = prop(at, None, None).split("\n")
    assert 1 <= len(lines) <= 3
    d0 = at.as_dict()
    targets = []
    for line in lines:
        steps = [t.strip() for t in line.split("+")]
        sched = at.copy()
        for t in steps:
            name, value = t[t.index("(") + 1:-1].split("=")
            assert d0[name] != int(value)         # every step changes the node
            sched = sched.apply(op.parse(t))
        assert sched.validate() == "" and str(sched) not in prop.measured
        targets.append(sched)
    # the candidates come from around the best measured schedules and are
    # ranked by the model: the first scores at least the median measured reward
    import numpy as np
    from paper_2506_01374_amd.tune import schedule_features
    pred = prop.model.predict(np.array([schedule_features(op, s) for s in targets]))
    assert list(pred) == sorted(pred, reverse=True)
    assert pred[0] >= np.median(prop.y)
    # the candidate offered first is not offered first again
    again = prop(at, None, None).split("\n")[0]
    assert again != lines[0]
    # measurements behind a surrogate's predictions are not recorded
    n = len(prop.measured)
    prop.record(space[0], 0.5, measured=False)
    assert len(prop.measured) == n
    # a refit (every 8 new measurements) redraws and reranks the pool
    first_model = prop.model
    for s in rng.sample(space, 40):
        prop.record(s, synthetic_reward(s))
    prop(at, None, None)
    assert prop.model is not first_model and prop.rank_at == len(prop.y)


def test_model_proposer_repairs_candidates_by_the_legality_reason():
    # a candidate put on the direct-to-LDS ring with a narrow vector and
    # K x N weights is illegal for two stated reasons; the repair sets the
    # values those reasons ask for and the candidate becomes legal
    from paper_2506_01374_amd.tune import ModelProposer
    from paper_2506_01374_amd import workloads as W
    op = W.workload_op("gated_mlp_t2048_h4096_i14336")
    d = op.default().as_dict()
    d.update({"up.tile_m": 128, "up.tile_n": 128, "up.tile_k": 32, "up.waves_m": 2, "up.waves_n": 2,
              "up.stages": 7, "up.vec": 2, "up.layout": 0})
    why = op.schedule(**d).validate()
    assert why.startswith("up:") and ("N x K" in why or "vec 8" in why)
    prop = ModelProposer(op, seed=0, repair=6)
    for _ in range(6):
        why = op.schedule(**d).validate()
        if not why:
            break
        prop._repair_step(d, why)
    assert op.schedule(**d).validate() == ""
    assert d["up.vec"] == 8 and d["up.layout"] == 1 and d["up.stages"] == 7


def test_model_proposer_structural_moves_reach_the_ring_from_a_register_staged_elite():
    from paper_2506_01374_amd.tune import ModelProposer
    from paper_2506_01374_amd import workloads as W
    import numpy as np

    class Zero:
        def predict(self, X):
            return np.zeros(len(X))

    op = W.workload_op("gated_mlp_t2048_h4096_i14336")
    d = op.default().as_dict()
    d.update({"up.tile_m": 128, "up.tile_n": 128, "up.tile_k": 32, "up.waves_m": 2, "up.waves_n": 2,
              "up.stages": 2, "up.vec": 2, "up.layout": 0})
    elite = op.schedule(**d)
    assert elite.validate() == ""
    for structural, expect in ((False, False), (True, True)):
        prop = ModelProposer(op, seed=0, repair=6, structural=structural, per_elite=0)
        prop.measured[str(elite)] = 0.5
        prop._rank(Zero())
        ring = [t for t, k in prop.ranked if k["up.stages"] == 7]
        assert bool(ring) == expect
        for t, k in prop.ranked:
            assert op.from_string(t).validate() == ""


def synthetic_reward(s):
    # a smooth, single-peaked function of the knobs of the fp32 GEMM
    d = s.as_dict()
    return (1.0 / (1 + abs(math.log2(d["tile_m"]) - 5)) * 1.0 / (1 + abs(math.log2(d["tile_n"]) - 6))
            * (1.2 if d["stages"] == 2 else 1.0) * (1.1 if d["vec"] == 4 else 1.0)
            * (1.0 + 0.05 * math.log2(d["tile_k"])) / (1 + 0.1 * d["unroll"]))


def test_exhaustive_finds_global_best_and_uct_random_approach_it():
    op = rc.Op(rc.RC_OP_GEMM_F32, (128, 128, 128))
    ex = rc.Search(op, synthetic_reward, policy=rc.RC_POLICY_EXHAUSTIVE, budget=100000).run()
    hist = ex.history()
    assert len(hist) == 1716                      # the whole legal space, once each
    best, r_ex, _ = ex.best()
    assert r_ex == pytest.approx(max(h["reward"] for h in hist))
    for pol in (rc.RC_POLICY_UCT, rc.RC_POLICY_RANDOM):
        bests = []
        for seed in range(3):
            s = rc.Search(op, synthetic_reward, policy=pol, budget=300, seed=seed).run()
            _, r, _ = s.best()
            assert r <= r_ex + 1e-12
            bests.append(r)
        assert max(bests) >= 0.9 * r_ex


def test_uct_reaches_the_optimum_of_a_tiny_space():
    op = tiny_op()
    rewards = {(2, 0): 0.3, (1, 1): 0.5, (2, 1): 0.9, (1, 0): 0.1}
    for seed in range(5):
        s = rc.Search(op, lambda x: rewards[(x["stages"], x["layout"])], policy=rc.RC_POLICY_UCT,
                      budget=4, horizon=2, seed=seed).run()
        _, r, _ = s.best()
        assert r == 0.9


def test_dedupe_monotone_best_and_determinism():
    op = rc.Op(rc.RC_OP_GEMM_F32, (128, 128, 128))
    runs = []
    for seed in (7, 7, 8):
        s = rc.Search(op, synthetic_reward, policy=rc.RC_POLICY_UCT, budget=60, seed=seed).run()
        h = s.history()
        valid = [x for x in h if x["valid"]]
        assert len(valid) == 60
        assert len({str(x["schedule"]) for x in valid}) == 60          # no schedule measured twice
        curve = [x["best_so_far"] for x in valid]
        assert curve == report.best_so_far([x["reward"] for x in valid])
        runs.append([str(x["schedule"]) for x in valid])
    assert runs[0] == runs[1] and runs[0] != runs[2]


def test_invalid_samples_cost_no_budget_and_keep_the_tree_consistent():
    op = rc.Op(rc.RC_OP_GEMM_F32, (128, 128, 128))

    def flaky(s):
        if s["vec"] == 4:
            raise RuntimeError("simulated compile failure")
        if s["layout"] == 1:
            return None
        return synthetic_reward(s)

    s = rc.Search(op, flaky, policy=rc.RC_POLICY_UCT, budget=40, seed=3).run()
    h = s.history()
    assert sum(x["valid"] for x in h) == 40
    assert all(x["schedule"]["vec"] != 4 and x["schedule"]["layout"] != 1 for x in h if x["valid"])
    assert any(not x["valid"] for x in h)
    assert s.node_stats([])[0] == len([x for x in h]) or s.node_stats([])[0] >= 40


def test_all_invalid_space_ends_cleanly():
    op = rc.Op(rc.RC_OP_GEMM_F32, (128, 128, 128))
    s = rc.Search(op, lambda x: None, policy=rc.RC_POLICY_RANDOM, budget=10, max_invalid=25).run()
    h = s.history()
    assert all(not x["valid"] for x in h) and len(h) == 26
    with pytest.raises(rc.RCError):
        s.best()


def test_report_metrics_reproduce_table1():
    rows = []
    with open(os.path.join(HERE, "golden", "table1_layerwise.csv")) as f:
        lines = [l for l in f if not l.startswith("#")]
    for r in csv.DictReader(lines):
        rows.append(r)
    body, gm = rows[:-1], rows[-1]
    assert len(body) == 25
    off = 0
    for r in body:
        red = report.sample_reduction(float(r["tvm_n"]), float(r["rc_n"]))
        gain = report.efficiency_gain(float(r["rc_s"]), float(r["rc_n"]), float(r["tvm_s"]),
                                      float(r["tvm_n"]))
        # printed speedups carry one decimal, so derived columns agree to rounding
        assert abs(red - float(r["red"])) <= 0.051
        if abs(gain - float(r["gain"])) > 0.051:
            off += 1
            assert abs(gain - float(r["gain"])) <= 0.25
    assert off <= 4
    assert round(report.geomean(float(r["tvm_s"]) for r in body), 1) == float(gm["tvm_s"])
    assert round(report.geomean(float(r["rc_s"]) for r in body), 1) == float(gm["rc_s"])
    assert round(report.geomean(float(r["red"]) for r in body), 1) == float(gm["red"])
    assert round(report.geomean(float(r["gain"]) for r in body), 1) == float(gm["gain"])


def test_report_helpers():
    assert report.speedup(10.0, 2.0) == 5.0
    assert report.sample_efficiency(12.1, 200) == pytest.approx(0.0605)
    assert report.best_so_far([1, 3, 2, 5, 4]) == [1, 3, 3, 5, 5]
    assert report.samples_to_reach([1, 3, 3, 5, 5], 4) == 4
    assert report.samples_to_reach([1, 2], 4) is None
    assert report.mean_curve([[1, 2, 3], [3, 4]]) == [2, 3]


def test_feedback_proposer_moves_toward_the_best_measured_schedules():
    # Before `warm` samples it proposes nothing (the search falls back to a
    # random legal transformation); afterwards it proposes one knob set to
    # the value most common among the best measured schedules, as text that
    # the proposal parser accepts.
    from paper_2506_01374_amd.tune import FeedbackProposer, legal_space
    op = rc.Op(rc.RC_OP_GEMM_F32, (128, 128, 128))
    space = legal_space(op)
    prop = FeedbackProposer(op, seed=0, top=4, warm=4)
    at = op.default()
    assert prop(at, None, None) == ""
    good = [s for s in space if s["tile_m"] == 64 and s["vec"] == 4][:4]
    bad = [s for s in space if s["tile_m"] == 16][:4]
    for s in good:
        prop.record(s, 1.0)
    for s in bad:
        prop.record(s, 0.1)
    prop.record(space[0], None)                   # invalid samples are ignored
    seen = set()
    for _ in range(50):
        text = prop(at, None, None)
        assert text
        op.parse(text)                            # a valid proposal for this operator
        seen.add(text)
    assert any("tile_m=64" in t for t in seen) and any("vec=4" in t for t in seen)
    # with a single best schedule, that schedule is the consensus: a node
    # equal to it gets no proposal
    solo = FeedbackProposer(op, seed=0, top=1, warm=1)
    solo.record(good[0], 1.0)
    assert solo(good[0], None, None) == ""


def test_uct_with_feedback_proposer_runs_and_uses_proposals():
    from paper_2506_01374_amd.tune import FeedbackProposer
    op = rc.Op(rc.RC_OP_GEMM_F32, (128, 128, 128))
    prop = FeedbackProposer(op, seed=1)

    def ev(s):
        r = synthetic_reward(s)
        prop.record(s, r)
        return r

    s = rc.Search(op, ev, policy=rc.RC_POLICY_UCT, budget=200, seed=1, propose=prop).run()
    hist = s.history()
    assert sum(h["valid"] for h in hist) == 200
    # some expansions came from proposals (not every one fell back)
    assert s.fallbacks() < 200
    _, r, _ = s.best()
    assert r > 0


@pytest.mark.parametrize("B", [2, 4])
def test_branching_factor_bounds_children_per_node(B):
    # B is the most children a node gets (Sec. 3.2; the branching ablation
    # compares B = 2 and B = 4): the root is expanded until it has B
    # children, after which iterations only select among them.
    op = rc.Op(rc.RC_OP_GEMM_F32, (128, 128, 128))
    moves = ["TileSize(tile_m=32)", "TileSize(tile_n=32)", "Unroll(unroll=2)", "Layout(layout=1)"]
    evals = []

    def ev(s):
        evals.append(str(s))
        return 0.5

    s = rc.Search(op, ev, policy=rc.RC_POLICY_UCT, budget=100, horizon=1, branching=B, seed=0,
                  propose=lambda at, par, gpar: ";".join(moves))
    for _ in range(8):
        s.step()
    visits = [s.node_stats([op.parse(m)])[0] for m in moves]
    assert all(v > 0 for v in visits[:B]) and all(v == 0 for v in visits[B:])
    assert sum(visits) == 8 and s.node_stats([])[0] == 8
    assert len(evals) == B and len(set(evals)) == B     # each leaf measured once
    assert s.fallbacks() == 0


class _SyntheticTable:
    """A measured-table stand-in: the synthetic reward of every schedule."""

    def __init__(self):
        self.calls = 0

    def measure(self, s):
        self.calls += 1
        return {"schedule": str(s), "valid": True, "reward": synthetic_reward(s)}


def test_surrogate_scores_rollouts_and_counts_only_measurements():
    # Rollout terminals are predicted by the learned surrogate and measured
    # only when promising (Sec. 3.2): the GPU budget counts measurements, not
    # rollouts; the curve is the best measured reward per measurement.
    from paper_2506_01374_amd.tune import run_search
    op = rc.Op(rc.RC_OP_GEMM_F32, (128, 128, 128))
    ex = rc.Search(op, synthetic_reward, policy=rc.RC_POLICY_EXHAUSTIVE, budget=100000).run()
    _, r_ex, _ = ex.best()
    table = _SyntheticTable()
    res = run_search(op, table, "uct", budget=64, seed=3, surrogate=True)
    # (the driver may run out of new schedules in this small space first)
    assert res["valid"] == len(res["curve"]) == table.calls and 32 <= table.calls <= 64
    assert res["predicted"] > table.calls
    assert res["curve"] == sorted(res["curve"]) and res["best_reward"] == res["curve"][-1]
    assert res["best_reward"] <= r_ex + 1e-12 and res["best_reward"] >= 0.8 * r_ex
    # deterministic for a seed
    again = run_search(op, _SyntheticTable(), "uct", budget=64, seed=3, surrogate=True)
    assert again["curve"] == res["curve"] and again["best"] == res["best"]


def test_measured_attention_tables_parse_and_hold_the_tuned_schedule():
    # The committed tables of measured schedules (one sub-space of causal
    # attention, cold; its direct-to-LDS part, warm) replay through the same
    # evaluator interface as a live GPU run; every row is a legal schedule of
    # the workload.  The benchmark runs warm, and its tuned schedule is the
    # warm table's fastest (within the 1 % the table's ties span).
    import json
    from paper_2506_01374_amd import workloads as W
    from paper_2506_01374_amd.tune import TableEvaluator
    name = "attention_causal_b1_h32_s1024_d128"
    op = W.workload_op(name)
    tuned = str(op.from_string(json.load(open(os.path.join(HERE, "..", "paper_2506_01374_amd", "tuned.json")))[name]))
    cold = TableEvaluator(os.path.join(HERE, "..", "results", f"{name}.space.tsv"), op)
    assert len(cold.table) == 3174
    assert all(op.from_string(k).validate() == "" for k in cold.table)
    valid = [r for r in cold.table.values() if r["valid"]]
    assert len(valid) == 2916
    assert cold.table[tuned]["valid"]
    warm = TableEvaluator(os.path.join(HERE, "..", "results", f"{name}.direct_lds.warm.tsv"), op)
    assert len(warm.table) == 166 and all(r["valid"] for r in warm.table.values())
    assert set(warm.table) <= set(cold.table)
    fastest = min(r["ms"] for r in warm.table.values())
    assert warm.table[tuned]["ms"] <= 1.01 * fastest


def test_surrogate_replay_spends_nothing_outside_the_measured_space():
    # Replayed against a table, a schedule the table does not hold is
    # invalid at no cost: it is neither measured nor predicted, exactly as
    # it is for the search without a surrogate.
    from paper_2506_01374_amd import workloads as W
    from paper_2506_01374_amd.tune import SurrogateEvaluator, TableEvaluator
    name = "attention_causal_b1_h32_s1024_d128"
    op = W.workload_op(name)
    tab = TableEvaluator(os.path.join(HERE, "..", "results", f"{name}.space.tsv"), op)
    looked = []

    class Spy:
        contains = staticmethod(tab.contains)

        def measure(self, s):
            looked.append(str(s))
            return tab.measure(s)

    sur = SurrogateEvaluator(op, Spy(), seed=1)
    srch = rc.Search(op, sur, policy=rc.RC_POLICY_UCT, budget=2000, seed=1)
    while sur.measured < 24 and not srch.step():
        pass
    assert sur.measured >= 24 and sur.predicted > 0
    assert all(k in tab.table for k in looked)
    spills = sum(1 for k in looked if not tab.table[k]["valid"])
    invalid = sum(1 for h in srch.history() if not h["valid"])
    assert len(looked) == sur.measured + spills
    assert sur.calls == sur.measured + sur.predicted + invalid and invalid > spills


def test_measured_gemm_table_is_the_whole_space_and_its_optimum_is_tuned():
    # The committed fp32 GEMM 128^3 table holds every legal schedule once (the
    # enumeration of the space), and its cold optimum is the tuned schedule.
    import json
    from paper_2506_01374_amd import workloads as W
    from paper_2506_01374_amd.tune import TableEvaluator, legal_space
    op = W.workload_op("gemm_f32_128")
    tab = TableEvaluator(os.path.join(HERE, "..", "results", "gemm_f32_128.space.tsv"), op)
    assert set(tab.table) == {str(s) for s in legal_space(op)}
    valid = [r for r in tab.table.values() if r["valid"]]
    assert len(valid) == 1714
    tuned = json.load(open(os.path.join(HERE, "..", "paper_2506_01374_amd", "tuned.json")))["gemm_f32_128"]
    assert max(valid, key=lambda r: r["reward"])["schedule"] == str(op.from_string(tuned))


def test_flux_table_columns_and_the_warm_optimum_is_tuned():
    # The bidirectional-attention table carries a warm and a cold timing per
    # schedule; the benchmark runs warm and its tuned schedule is the warm
    # optimum.
    import json
    from paper_2506_01374_amd import workloads as W
    from paper_2506_01374_amd.tune import TableEvaluator
    name = "attention_noncausal_b1_h24_s4096_d128"
    op = W.workload_op(name)
    path = os.path.join(HERE, "..", "results", f"{name}.vec8.tsv")
    warm = TableEvaluator(path, op, column="warm_us")
    cold = TableEvaluator(path, op)
    assert len(warm.table) == len(cold.table) == 2808
    assert sum(r["valid"] for r in warm.table.values()) == 2343
    assert all(op.from_string(k).validate() == "" for k in warm.table)
    tuned = json.load(open(os.path.join(HERE, "..", "paper_2506_01374_amd", "tuned.json")))[name]
    best = max((r for r in warm.table.values() if r["valid"]), key=lambda r: r["reward"])
    assert best["schedule"] == str(op.from_string(tuned))
    k = str(op.from_string(tuned))
    assert cold.table[k]["ms"] > warm.table[k]["ms"]


def test_causal_vec8_table_warm_optimum_is_tuned():
    # Every 16-byte-vector, unchunked causal schedule timed warm and cold: the
    # tuned schedule is the warm optimum; the cold optimum is a one-split
    # pipelined schedule (one tile in flight per split costs more from HBM).
    import json
    from paper_2506_01374_amd import workloads as W
    from paper_2506_01374_amd.tune import TableEvaluator
    name = "attention_causal_b1_h32_s1024_d128"
    op = W.workload_op(name)
    path = os.path.join(HERE, "..", "results", f"{name}.vec8.tsv")
    warm = TableEvaluator(path, op, column="warm_us")
    cold = TableEvaluator(path, op, column="cold_us")
    assert len(warm.table) == 2808 and sum(r["valid"] for r in warm.table.values()) == 2366
    tuned = json.load(open(os.path.join(HERE, "..", "paper_2506_01374_amd", "tuned.json")))[name]
    bw = max((r for r in warm.table.values() if r["valid"]), key=lambda r: r["reward"])
    bc = max((r for r in cold.table.values() if r["valid"]), key=lambda r: r["reward"])
    assert bw["schedule"] == str(op.from_string(tuned))
    assert op.from_string(bc["schedule"]).as_dict()["splits"] == 1


def test_campaign_threads_share_measurements_and_summarise(tmp_path):
    # Several searches in threads against one evaluator: each distinct
    # schedule is measured once, the record holds one run per (policy,
    # seed), and samples-to-reach counts follow the curves.
    import json
    import threading
    from paper_2506_01374_amd import tune
    op = rc.Op(rc.RC_OP_GEMM_F32, (128, 128, 128))
    calls = {}
    lock = threading.Lock()

    def fake_time(sched):
        d = sched.as_dict()
        with lock:
            calls[str(sched)] = calls.get(str(sched), 0) + 1
        score = (d["tile_m"] + d["tile_n"]) / 128.0 + 0.1 * d["vec"] + 0.05 * d["waves_m"]
        return {"schedule": str(sched), "valid": True, "ms": 1.0 / score, "reward": score / 2.0}

    ref = "tile_m=64,tile_n=64,tile_k=16,waves_m=2,waves_n=1,vec=4,stages=2,unroll=1,layout=0"
    out = tmp_path / "c.json"
    rec = tune.run_campaign(op, "gemm_f32_128", ["random", "uct"], [0, 1, 2], 24, ref, 1, str(out), None,
                            time_fn=fake_time, compile_fn=lambda job: 0)
    assert not rec["errors"], rec["errors"]
    assert len(rec["runs"]) == 6
    assert all(n == 1 for s, n in calls.items() if s != str(op.from_string(ref))), calls
    saved = json.load(open(out))
    for pname in ("random", "uct"):
        sm = saved["summary"][pname]
        assert set(sm["best_so_far_over_reference"]) == {"18"}
        for r in (r for r in saved["runs"] if r["policy_name"] == pname):
            k = next((i + 1 for i, v in enumerate(r["curve"]) if v >= 0.9 * saved["reference_reward"]), None)
            assert k == sm["samples_to_90pct"]["per_seed"][sm["seeds"].index(r["seed"])]
            assert all(b >= a for a, b in zip(r["curve"], r["curve"][1:]))
    assert saved["measurement"].startswith("cold")
    warm = tune.run_campaign(op, "gemm_f32_128", ["random"], [0], 8, ref, 1, str(tmp_path / "w.json"), None,
                             time_fn=fake_time, compile_fn=lambda job: 0, flush=False)
    assert warm["measurement"].startswith("warm")


def test_campaign_benchmark_timing_cycles_the_input_copies():
    # rotate > 0: steps launched back to back through that many input
    # copies, no flush; the record says so
    from paper_2506_01374_amd import tune
    op = rc.Op(rc.RC_OP_GEMM_F32, (128, 128, 128))
    launched = []

    class FakeEvent:
        def __init__(self, enable_timing=True):
            pass

        def record(self):
            pass

        def elapsed_time(self, other):
            return 2.0 * max(1, len(launched))

    class FakeTorch:
        class cuda:
            Event = FakeEvent

            @staticmethod
            def synchronize():
                pass

    class FakePrepared:
        def __init__(self, copy):
            self.copy = copy

        def launch(self):
            launched.append(self.copy)

    class FakePlan:
        def __init__(self, op, sched):
            pass

        def workspace(self):
            return None

        def prepare(self, inputs, out, ws):
            return FakePrepared(inputs[0])

    class FakeTensor:
        def __init__(self, tag):
            self.tag = tag

        def clone(self):
            return FakeTensor(self.tag + "'")

    class FakeInner:
        warmup, repeat, out, torch = 1, 4, None, FakeTorch

        def _inputs(self, sched):
            return [FakeTensor("a")]

    ev = tune.ParallelGpuEvaluator(op, time_fn=lambda s: {}, compile_fn=lambda job: 0, rotate=2)
    ev.inner = FakeInner()
    orig = tune.rc.Plan
    tune.rc.Plan = FakePlan
    try:
        rec = ev._time(op.default())
    finally:
        tune.rc.Plan = orig
    assert rec["valid"] and rec["ms"] > 0
    tags = [t.tag for t in launched]
    assert set(tags) == {"a", "a'"}                  # both copies were used
    assert all(x != y for x, y in zip(tags[1:], tags[2:]))   # alternating within a timed run


def test_campaign_timing_passes_the_flush_choice_to_the_timer():
    # the evaluator's own timer asks for the cache flush only in cold mode
    from paper_2506_01374_amd import tune
    op = rc.Op(rc.RC_OP_GEMM_F32, (128, 128, 128))
    seen = []

    class FakePlan:
        def __init__(self, op, sched):
            pass

        def workspace(self):
            return None

        def time(self, ins, out, ws, warmup, repeat, flush):
            seen.append(flush)

            class T:
                median_ms, q1_ms, q3_ms, tflops, gbps, nkernels, kernel_ms = 1.0, 1.0, 1.0, 1.0, 1.0, 0, []
            return T()

    class FakeInner:
        warmup, repeat, out = 1, 2, None

        def _inputs(self, sched):
            return []

    for flush in (True, False):
        ev = tune.ParallelGpuEvaluator(op, time_fn=lambda s: {}, compile_fn=lambda job: 0, flush=flush)
        ev.inner = FakeInner()
        orig = tune.rc.Plan
        tune.rc.Plan = FakePlan
        try:
            ev._time(op.default())
        finally:
            tune.rc.Plan = orig
        assert seen and all(f is flush for f in seen)
        seen.clear()


def test_p0_timing_alternates_and_reports_the_tuned_speedup(monkeypatch):
    # P0 and the tuned schedule are timed alternately, each again rather
    # than from the evaluator's cache; the speedup is the ratio of medians
    from paper_2506_01374_amd import tune
    op = rc.Op(rc.RC_OP_GEMM_F32, (128, 128, 128))
    tuned_text = "tile_m=32,tile_n=32,tile_k=32,waves_m=1,waves_n=2,vec=4,stages=2,unroll=1,layout=0"
    assert op.from_string(tuned_text).validate() == ""
    order = []

    class FakeEvaluator:
        def __init__(self, op, repeat=10, warmup=2, log=None):
            self.cache = {}

        def measure(self, sched):
            text = str(sched)
            assert text not in self.cache
            order.append(text)
            ms = 0.9 if text == str(op.default()) else 0.3
            self.cache[text] = {"valid": True, "ms": ms + 0.01 * len(order)}
            return self.cache[text]

    monkeypatch.setattr(tune, "GpuEvaluator", FakeEvaluator)
    rec = tune.time_p0_and_tuned(op, "gemm_f32_128", tuned_text, repeat=3, rounds=2)
    p0, tuned = str(op.default()), str(op.from_string(tuned_text))
    assert order == [p0, tuned, p0, tuned]
    assert all(math.isclose(a, b) for a, b in zip(rec["p0_us"] + rec["tuned_us"], [910.0, 930.0, 320.0, 340.0]))
    assert abs(rec["tuned_speedup_over_p0"] - 920.0 / 330.0) < 1e-9
    assert rec["p0_reward"] < rec["tuned_reward"]
