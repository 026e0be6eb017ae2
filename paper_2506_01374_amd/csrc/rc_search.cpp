// Schedule search over transformation sequences (Sec. 2 MDP; Sec. 3.2 MCTS).
//
// State = schedule (program variant), action = one transformation,
// transitions are deterministic (Sec. 2).  The UCT policy runs the four MCTS
// phases of Sec. 3.2:
//   selection     descend from the root by UCT(P_i) = W_i / N_i +
//                 c sqrt(ln N_parent / N_i), unvisited children first, ties to
//                 the earliest-inserted child;
//   expansion     a node with fewer than B children (B = branching) gets a new
//                 child from a proposed transformation, or a proposed
//                 sequence of them applied together; proposals are
//                 validated and, when none is valid, a random legal
//                 transformation is used (Sec. 3.1); a child whose program
//                 already exists in the tree is not added, keeping the tree
//                 acyclic;
//   rollout       q = T - depth random legal transformations give P_sim,
//                 whose measured reward (the objective f, not a learned
//                 surrogate) scores the new node;
//   backprop      W_A += R and N_A += 1 for the new node and every ancestor.
// One sample is one distinct legal schedule evaluated; a schedule already
// evaluated is not evaluated again (its stored reward is reused and no
// budget is spent).  Evaluations that fail cost no budget, back-propagate a
// reward of 0 and are counted.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <limits>
#include <memory>
#include <random>
#include <string>
#include <unordered_map>
#include <vector>

#include "rc_internal.h"

using namespace rc;

namespace {

struct Node {
    rc_schedule sched;
    int parent;
    rc_transform via;     // transformation applied at the parent
    int depth;
    std::vector<int> children;
    bool exhausted = false;   // no further distinct legal child exists
    int visits = 0;
    double W = 0.0;
};

}  // namespace

struct rc_search {
    rc_op_desc desc;
    rc_search_opts opts;
    rc_eval_fn eval;
    void *eval_user;
    rc_propose_fn propose = nullptr;
    void *propose_user = nullptr;
    std::mt19937_64 rng;
    std::vector<Node> tree;
    std::unordered_map<uint64_t, int> in_tree;         // schedule hash -> node
    std::unordered_map<uint64_t, double> measured;     // schedule hash -> reward (valid only)
    std::unordered_map<uint64_t, int> failed;          // schedule hash -> 1
    std::vector<rc_sample> history;
    int valid = 0, invalid = 0, fallbacks = 0, iterations = 0;
    double best = -1.0;
    rc_schedule best_sched;
    int best_index = -1;
    bool done = false;
    // exhaustive enumeration cursor
    std::vector<int32_t> cursor;
    bool cursor_end = false;
};

namespace {

std::vector<rc_transform> legal_moves(rc_search *s, const rc_schedule &at) {
    size_t n = 0;
    rc_enumerate(&s->desc, &at, nullptr, 0, &n);
    std::vector<rc_transform> v(n);
    if (n) rc_enumerate(&s->desc, &at, v.data(), n, &n);
    return v;
}

rc_schedule rollout(rc_search *s, rc_schedule at, int steps) {
    for (int i = 0; i < steps; ++i) {
        auto mv = legal_moves(s, at);
        if (mv.empty()) break;
        rc_transform t = mv[std::uniform_int_distribution<size_t>(0, mv.size() - 1)(s->rng)];
        rc_schedule nx;
        if (rc_apply(&s->desc, &at, &t, &nx) == RC_OK) at = nx;
    }
    return at;
}

// Evaluate with dedupe.  Returns reward (0 for invalid); *spent = a valid
// new sample was measured.
double evaluate(rc_search *s, const rc_schedule &sc, bool *spent, bool *ok) {
    uint64_t h = rc_schedule_hash(&sc);
    *spent = false;
    auto it = s->measured.find(h);
    if (it != s->measured.end()) {
        *ok = true;
        return it->second;
    }
    if (s->failed.count(h)) {
        *ok = false;
        return 0.0;
    }
    double r = 0.0;
    int32_t st = s->eval(s->eval_user, &sc, &r);
    rc_sample smp;
    std::memset(&smp, 0, sizeof smp);
    smp.schedule = sc;
    if (st == 0 && std::isfinite(r) && r >= 0.0) {
        s->measured[h] = r;
        smp.valid = 1;
        smp.reward = r;
        smp.index = s->valid++;
        if (r > s->best) {
            s->best = r;
            s->best_sched = sc;
            s->best_index = smp.index;
        }
        *spent = true;
        *ok = true;
    } else {
        s->failed[h] = 1;
        smp.valid = 0;
        smp.index = -1;
        ++s->invalid;
        r = 0.0;
        *ok = false;
    }
    smp.best_so_far = s->best;
    s->history.push_back(smp);
    return r;
}

int add_child(rc_search *s, int parent, const rc_transform &t, const rc_schedule &sc) {
    Node n;
    n.sched = sc;
    n.parent = parent;
    n.via = t;
    n.depth = s->tree[parent].depth + 1;
    s->tree.push_back(n);
    int id = (int)s->tree.size() - 1;
    s->tree[parent].children.push_back(id);
    s->in_tree[rc_schedule_hash(&sc)] = id;
    return id;
}

// Expansion of node `at`: a proposal first, then a random legal move.
int expand(rc_search *s, int at) {
    const Node &nd = s->tree[at];
    rc_schedule cur = nd.sched;
    if (s->propose) {
        const rc_schedule *par = nd.parent >= 0 ? &s->tree[nd.parent].sched : nullptr;
        const rc_schedule *gpar =
            (nd.parent >= 0 && s->tree[nd.parent].parent >= 0) ? &s->tree[s->tree[nd.parent].parent].sched : nullptr;
        char buf[4096];
        buf[0] = 0;
        s->propose(s->propose_user, &cur, par, gpar, buf, sizeof buf);
        buf[sizeof buf - 1] = 0;
        // Alternatives are separated by ';' or newlines and tried in order;
        // an alternative may chain transformations with '+' (a proposed
        // sequence, Sec. 3.1): its steps are applied in order, steps that do
        // not parse are discarded, intermediate schedules need not be legal,
        // and the resulting schedule must be legal and new to the tree.
        std::string text(buf);
        size_t pos = 0;
        while (pos <= text.size()) {
            size_t e = text.find_first_of(";\n", pos);
            if (e == std::string::npos) e = text.size();
            std::string item = text.substr(pos, e - pos);
            pos = e + 1;
            rc_schedule nx = cur;
            rc_transform first{-1, 0};
            size_t q = 0;
            while (q <= item.size()) {
                size_t f = item.find('+', q);
                if (f == std::string::npos) f = item.size();
                std::string step = item.substr(q, f - q);
                q = f + 1;
                rc_transform t;
                if (step.find_first_not_of(" \t\r") == std::string::npos ||
                    rc_parse_transform(&s->desc, step.c_str(), &t) != RC_OK)
                    continue;
                if (nx.knob[t.knob] == t.value) continue;
                nx.knob[t.knob] = t.value;
                if (first.knob < 0) first = t;
            }
            if (first.knob < 0) continue;
            if (!check_schedule(&s->desc, &nx).empty()) continue;
            if (s->in_tree.count(rc_schedule_hash(&nx))) continue;
            return add_child(s, at, first, nx);
        }
        ++s->fallbacks;
    }
    auto mv = legal_moves(s, cur);
    std::shuffle(mv.begin(), mv.end(), s->rng);
    for (auto &t : mv) {
        rc_schedule nx;
        if (rc_apply(&s->desc, &cur, &t, &nx) != RC_OK) continue;
        if (s->in_tree.count(rc_schedule_hash(&nx))) continue;
        return add_child(s, at, t, nx);
    }
    s->tree[at].exhausted = true;
    return -1;
}

double uct(const rc_search *s, const Node &child, int parent_visits) {
    if (child.visits == 0) return std::numeric_limits<double>::infinity();
    return child.W / child.visits +
           s->opts.c * std::sqrt(std::log((double)std::max(parent_visits, 1)) / child.visits);
}

void backprop(rc_search *s, int node, double r) {
    for (int n = node; n >= 0; n = s->tree[n].parent) {
        s->tree[n].W += r;
        s->tree[n].visits += 1;
    }
}

bool next_point(rc_search *s, rc_schedule &out) {
    const auto &kt = knobs_for(s->desc.kind);
    while (!s->cursor_end) {
        rc_schedule sc;
        std::memset(&sc, 0, sizeof sc);
        sc.struct_size = sizeof sc;
        sc.nknobs = (int32_t)kt.size();
        for (size_t i = 0; i < kt.size(); ++i) sc.knob[i] = kt[i].values[s->cursor[i]];
        // advance the odometer (last knob fastest)
        int i = (int)kt.size() - 1;
        for (; i >= 0; --i) {
            if (++s->cursor[i] < (int)kt[i].values.size()) break;
            s->cursor[i] = 0;
        }
        if (i < 0) s->cursor_end = true;
        if (check_schedule(&s->desc, &sc).empty()) {
            out = sc;
            return true;
        }
    }
    return false;
}

}  // namespace

extern "C" {

void rc_search_opts_init(rc_search_opts *o) {
    if (!o) return;
    std::memset(o, 0, sizeof *o);
    o->struct_size = sizeof *o;
    o->policy = RC_POLICY_UCT;
    o->budget = 64;
    o->horizon = 12;
    o->branching = 2;
    o->c = std::sqrt(2.0);
    o->seed = 0;
    o->max_invalid = -1;
}

rc_status rc_search_create(const rc_op_desc *d, const rc_search_opts *o, rc_eval_fn eval,
                           void *eval_user, rc_search **out) {
    if (!desc_ok(d) || !o || !eval || !out || o->struct_size < sizeof(rc_search_opts))
        return fail(RC_ERR_INVALID_ARGUMENT, "bad arguments");
    if (o->budget < 1 || o->horizon < 0 || o->branching < 1 || !(o->c >= 0))
        return fail(RC_ERR_INVALID_ARGUMENT, "budget >= 1, horizon >= 0, branching >= 1, c >= 0");
    if (o->policy < RC_POLICY_RANDOM || o->policy > RC_POLICY_EXHAUSTIVE)
        return fail(RC_ERR_INVALID_ARGUMENT, "unknown policy");
    std::unique_ptr<rc_search> s(new rc_search());
    s->desc = *d;
    s->opts = *o;
    if (s->opts.max_invalid < 0) s->opts.max_invalid = 10 * o->budget;
    s->eval = eval;
    s->eval_user = eval_user;
    s->rng.seed(o->seed);
    Node root;
    rc_status r = rc_default_schedule(d, &root.sched);
    if (r != RC_OK) return r;
    root.parent = -1;
    root.via = rc_transform{-1, 0};
    root.depth = 0;
    s->tree.push_back(root);
    s->in_tree[rc_schedule_hash(&root.sched)] = 0;
    s->best_sched = root.sched;
    s->cursor.assign(knobs_for(d->kind).size(), 0);
    *out = s.release();
    return RC_OK;
}

rc_status rc_search_set_proposer(rc_search *s, rc_propose_fn fn, void *user) {
    if (!s) return fail(RC_ERR_INVALID_ARGUMENT, "null search");
    s->propose = fn;
    s->propose_user = user;
    return RC_OK;
}

rc_status rc_search_step(rc_search *s, int32_t *done) {
    if (!s) return fail(RC_ERR_INVALID_ARGUMENT, "null search");
    auto finish = [&]() {
        s->done = true;
        if (done) *done = 1;
        return RC_OK;
    };
    if (s->done || s->valid >= s->opts.budget || s->invalid > s->opts.max_invalid) return finish();
    ++s->iterations;
    bool spent = false, ok = false;
    switch (s->opts.policy) {
        case RC_POLICY_RANDOM: {
            rc_schedule sim = rollout(s, s->tree[0].sched, s->opts.horizon);
            evaluate(s, sim, &spent, &ok);
            break;
        }
        case RC_POLICY_EXHAUSTIVE: {
            rc_schedule pt;
            if (!next_point(s, pt)) return finish();
            evaluate(s, pt, &spent, &ok);
            break;
        }
        case RC_POLICY_UCT: {
            int node = 0;
            for (;;) {
                Node &nd = s->tree[node];
                bool can_expand = nd.depth < s->opts.horizon && !nd.exhausted &&
                                  (int)nd.children.size() < s->opts.branching;
                if (can_expand) {
                    int c = expand(s, node);
                    if (c >= 0) {
                        node = c;
                        break;
                    }
                    continue;   // node became exhausted; re-check
                }
                if (nd.children.empty()) break;   // terminal leaf: roll out from here
                int pick = -1;
                double bestv = -std::numeric_limits<double>::infinity();
                for (int ch : nd.children) {
                    double v = uct(s, s->tree[ch], nd.visits);
                    if (v > bestv) {   // strict: ties keep the earliest child
                        bestv = v;
                        pick = ch;
                    }
                }
                node = pick;
            }
            int steps = std::max(0, s->opts.horizon - s->tree[node].depth);
            rc_schedule sim = rollout(s, s->tree[node].sched, steps);
            double r = evaluate(s, sim, &spent, &ok);
            backprop(s, node, r);
            break;
        }
    }
    // Guard against spinning on an exhausted space: every iteration that
    // neither spends budget nor fails counts toward a generous cap.
    if (s->iterations > 200 * s->opts.budget + 1000) return finish();
    if (s->valid >= s->opts.budget || s->invalid > s->opts.max_invalid) return finish();
    if (done) *done = 0;
    return RC_OK;
}

rc_status rc_search_run(rc_search *s) {
    if (!s) return fail(RC_ERR_INVALID_ARGUMENT, "null search");
    int32_t done = 0;
    while (!done) {
        rc_status r = rc_search_step(s, &done);
        if (r != RC_OK) return r;
    }
    return RC_OK;
}

rc_status rc_search_best(const rc_search *s, rc_schedule *best, double *reward, int32_t *idx) {
    if (!s) return fail(RC_ERR_INVALID_ARGUMENT, "null search");
    if (s->best_index < 0) return fail(RC_ERR_BUDGET, "no valid sample");
    if (best) *best = s->best_sched;
    if (reward) *reward = s->best;
    if (idx) *idx = s->best_index;
    return RC_OK;
}

rc_status rc_search_history(const rc_search *s, rc_sample *buf, int32_t cap, int32_t *n) {
    if (!s || !n) return fail(RC_ERR_INVALID_ARGUMENT, "null argument");
    *n = (int32_t)s->history.size();
    for (int32_t i = 0; i < *n && i < cap && buf; ++i) buf[i] = s->history[i];
    return RC_OK;
}

rc_status rc_search_node_stats(const rc_search *s, const rc_transform *path, int32_t len,
                               int32_t *visits, double *W) {
    if (!s || (len > 0 && !path)) return fail(RC_ERR_INVALID_ARGUMENT, "null argument");
    int node = 0;
    for (int32_t i = 0; i < len && node >= 0; ++i) {
        int next = -1;
        for (int ch : s->tree[node].children)
            if (s->tree[ch].via.knob == path[i].knob && s->tree[ch].via.value == path[i].value) next = ch;
        node = next;
    }
    if (visits) *visits = node >= 0 ? s->tree[node].visits : 0;
    if (W) *W = node >= 0 ? s->tree[node].W : 0.0;
    return RC_OK;
}

rc_status rc_search_fallbacks(const rc_search *s, int32_t *n) {
    if (!s || !n) return fail(RC_ERR_INVALID_ARGUMENT, "null argument");
    *n = s->fallbacks;
    return RC_OK;
}

void rc_search_destroy(rc_search *s) { delete s; }

}  // extern "C"
