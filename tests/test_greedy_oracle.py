"""Pins of the dual-queue interleaving oracle (oracle/dip_greedy.c) to things
other than itself: hand traces worked out from the rules of Sec. 5.2
(tests/golden/greedy_hand_traces.txt), a decision-by-decision verifier that
re-derives every choice from the finished timeline, the independent simulator
oracle on the emitted orders, and invariants of the memory rule."""
import os

import numpy as np
import pytest

import oracle as O
import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))


# ---------------------------------------------------------------- hand traces

def _cases():
    cases, cur = [], None
    with open(os.path.join(HERE, "golden", "greedy_hand_traces.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            k, *v = line.split()
            if k == "case":
                cur = {"name": v[0], "order": {}}
                cases.append(cur)
            elif k == "order":
                cur["order"][int(v[0])] = [int(x) for x in v[1:]]
            else:
                cur[k] = [int(x) for x in v]
    return cases


def _pipeline_problem(P, M, fcost, comm, act, cap):
    f = np.asarray(fcost, np.int64)
    inst = W.pipeline_instance(P, M, f if f.size > 1 else int(f[0]), comm=comm, act=act,
                               mem_cap=cap)
    return W.compile_instance(inst)


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c["name"])
def test_hand_traces(case):
    P, M = case["P"][0], case["M"][0]
    prob = _pipeline_problem(P, M, case["fcost"], case["comm"][0], case["act"][0], case["cap"][0])
    g, G, _ = W.priority_groups(prob)
    prio = np.zeros(G, np.int32)
    for op in range(prob.n_total):
        m = int(prob.op_mb[op])
        prio[g[op]] = case["prio_b"][m] if prob.op_kind[op] else case["prio_f"][m]
    order, res, start, end = O.greedy_timeline(prob, g, G, prio)
    for r, want in case["order"].items():
        got = order[prob.rank_off[r]:prob.rank_off[r + 1]].tolist()
        assert got == want, f"rank {r}"
    assert res.makespan[0] == case["makespan"][0]
    assert res.bubble[0].tolist() == case["bubble"]
    assert res.peak[0].tolist() == case["peak"]
    assert int(res.flags[0]) == case["flags"][0]


# ---------------------------------------------------------------- verifier

def _t_start(prob, end):
    ts = np.zeros(prob.n_total, np.int64)
    for o in range(prob.n_total):
        b, e = prob.pred_ptr[o], prob.pred_ptr[o + 1]
        if e > b:
            ts[o] = max(int(end[prob.pred_op[k]]) + int(prob.edge_comm[k]) for k in range(b, e))
    return ts


def verify_decisions(prob, g, prio, order, start, end):
    """Re-derive every decision from the finished timeline.  Valid without
    caps when every edge carries cost(pred) + comm >= 1: then a stage whose
    t_start is at most a rank's decision time had all its predecessors
    decided earlier, so it was queued for that decision."""
    ts = _t_start(prob, end)
    kind = prob.op_kind

    def key(o):
        return (-int(prio[g[o]]), int(g[o]), o)

    for r in range(prob.n_ranks):
        base = int(prob.rank_off[r])
        seq = [base + int(x) for x in order[base:int(prob.rank_off[r + 1])]]
        t_last, last = 0, None
        for k, o in enumerate(seq):
            rest = seq[k:]
            s = int(start[o])
            assert s == max(t_last, ts[o]), "start is max(t_last, t_start)"
            assert int(end[o]) == s + int(prob.op_cost[o])
            if s > t_last:           # idle only while nothing was queued
                assert min(ts[x] for x in rest) == s
            eF = any(kind[x] == 0 and ts[x] < t_last for x in rest)
            eB = any(kind[x] == 1 and ts[x] < t_last for x in rest)
            avail = [x for x in rest if ts[x] <= s]
            if eF and eB:
                assert kind[o] != last, "1F1B alternation"
                avail = [x for x in avail if kind[x] == kind[o]]
            assert o == min(avail, key=key), "highest priority"
            t_last, last = int(end[o]), kind[o]


def _positive(cid):
    inst = W.make_instance(cid)
    inst.fcost = inst.fcost + 1
    inst.bcost = 2 * inst.fcost
    return W.compile_instance(inst)


def _random_pipeline(rng, v):
    P = int(rng.integers(1, 6))
    M = int(rng.integers(1, 9))
    f = rng.integers(1, 30, size=(P * v, M))
    inst = W.pipeline_instance(P, M, f, comm=int(rng.integers(0, 15)), v=v)
    return W.compile_instance(inst)


@pytest.mark.parametrize("which", ["c1", "c2_positive", "c3_positive", "pipelines"])
def test_every_decision_follows_the_rules(which):
    rng = np.random.default_rng(4)
    if which == "pipelines":
        probs = [_random_pipeline(rng, v) for v in (1, 1, 2, 2, 3) for _ in range(4)]
    elif which == "c1":
        probs = [W.make_problem(1)]
    else:
        probs = [_positive(2 if which == "c2_positive" else 3)]
    for prob in probs:
        prob.mem_cap[:] = -1
        g, G, cls = W.priority_groups(prob)
        rows = W.rollout_priorities(cls, 4, seed=9)
        rows[0] = 0                                   # every priority equal
        for prio in rows:
            order, res, start, end = O.greedy_timeline(prob, g, G, prio)
            verify_decisions(prob, g, prio, order, start, end)


def test_verifier_catches_a_planted_mistake():
    """Swapping two adjacent stages of a rank's order (re-timed by the
    simulator oracle) breaks some rule whenever the swap leaves a valid
    schedule."""
    prob = W.make_problem(1)
    g, G, cls = W.priority_groups(prob)
    prio = W.rollout_priorities(cls, 1, seed=1)[0]
    order, _, _, _ = O.greedy_timeline(prob, g, G, prio)
    checked = 0
    for r in range(prob.n_ranks):
        for i in range(int(prob.rank_off[r]), int(prob.rank_off[r + 1]) - 1):
            bad = order.copy()
            bad[i], bad[i + 1] = bad[i + 1], bad[i]
            res, start, end = O.timeline(prob, bad)
            if res.flags[0]:
                continue             # the swap deadlocks: rejected anyway
            with pytest.raises(AssertionError):
                verify_decisions(prob, g, prio, bad, start, end)
            checked += 1
    assert checked >= 10


# ---------------------------------------------------------------- consistency

@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_own_timeline_equals_simulator(cid):
    """The greedy's makespan, bubbles, peaks and flags equal the simulator
    oracle's on the emitted orders, which are permutations that never
    deadlock."""
    prob = W.make_problem(cid)
    g, G, cls = W.priority_groups(prob)
    n = {1: 64, 2: 32, 3: 6, 4: 3, 5: 1}[cid]
    prio = W.rollout_priorities(cls, n, seed=cid)
    orders, res = O.greedy(prob, g, G, prio, stride=prob.stride, threads=8)
    sim = O.evaluate(prob, orders, threads=8)
    assert not (sim.flags & (O.FLAG_DEADLOCK | O.FLAG_INVALID)).any()
    np.testing.assert_array_equal(sim.makespan, res.makespan)
    np.testing.assert_array_equal(sim.bubble, res.bubble)
    np.testing.assert_array_equal(sim.peak, res.peak)
    np.testing.assert_array_equal(sim.flags, res.flags)


@pytest.mark.parametrize("cap", [0, 1, 2, 3])
def test_caps_consistency(cap):
    rng = np.random.default_rng(cap)
    for v in (1, 2):
        inst = W.pipeline_instance(4, 7, rng.integers(1, 9, size=(4 * v, 7)), comm=2, v=v,
                                   mem_cap=cap)
        prob = W.compile_instance(inst)
        g, G, cls = W.priority_groups(prob)
        prio = W.rollout_priorities(cls, 16, seed=cap)
        orders, res = O.greedy(prob, g, G, prio)
        sim = O.evaluate(prob, orders)
        np.testing.assert_array_equal(sim.makespan, res.makespan)
        np.testing.assert_array_equal(sim.peak, res.peak)
        np.testing.assert_array_equal(sim.flags, res.flags)
        # a forward is taken past the cap only when no rank could move: the
        # flag is set exactly when some peak exceeds the cap
        np.testing.assert_array_equal(res.flags == O.FLAG_CAP, (res.peak > cap).any(axis=1))


def test_cap_that_never_binds_changes_nothing():
    prob = W.make_problem(2)
    g, G, cls = W.priority_groups(prob)
    prio = W.rollout_priorities(cls, 8, seed=5)
    prob.mem_cap[:] = -1
    free_orders, free = O.greedy(prob, g, G, prio)
    prob.mem_cap[:] = int(free.peak.max())
    capped_orders, capped = O.greedy(prob, g, G, prio)
    np.testing.assert_array_equal(capped_orders, free_orders)
    np.testing.assert_array_equal(capped.makespan, free.makespan)
    assert not capped.flags.any()


def test_tight_cap_lowers_the_peak():
    """Halving the free peak as a cap: the disabled forward queue keeps most
    ranks at or under it."""
    prob = W.make_problem(2)
    g, G, cls = W.priority_groups(prob)
    prio = W.rollout_priorities(cls, 8, seed=6)
    prob.mem_cap[:] = -1
    _, free = O.greedy(prob, g, G, prio)
    cap = int(free.peak.max()) // 2
    prob.mem_cap[:] = cap
    _, capped = O.greedy(prob, g, G, prio)
    assert capped.peak.max() < free.peak.max()


def test_single_rank_never_idles():
    """One rank and no transfers: the makespan is the sum of the costs."""
    rng = np.random.default_rng(2)
    for M in (1, 2, 5, 9):
        inst = W.pipeline_instance(1, M, rng.integers(1, 20, size=(1, M)), comm=0)
        prob = W.compile_instance(inst)
        g, G, cls = W.priority_groups(prob)
        _, res = O.greedy(prob, g, G, W.rollout_priorities(cls, 5, seed=M))
        assert (res.makespan == prob.op_cost.sum()).all()
        assert (res.bubble == 0).all()


def test_uniform_pipeline_lower_bound():
    """Uniform f, b and no transfers: no order beats (M + S - 1)(f + b), the
    last rank's start, its own work and the backward chain back to rank 0."""
    for S, M in ((2, 3), (3, 5), (4, 4), (4, 9)):
        prob = _pipeline_problem(S, M, [3], 0, 1, -1)
        g, G, cls = W.priority_groups(prob)
        _, res = O.greedy(prob, g, G, W.rollout_priorities(cls, 8, seed=S * M))
        assert (res.makespan >= (M + S - 1) * 9).all()


def test_cyclic_data_graph_is_an_error():
    prob = _pipeline_problem(2, 2, [3], 1, 1, -1)
    # add an edge B(0) on rank 0 -> F(0) on rank 0: a cycle through the chain
    pp, po, ec = list(prob.pred_ptr), list(prob.pred_op), list(prob.edge_comm)
    f0 = int(prob.rank_off[0])
    b0 = f0 + 1
    po.insert(pp[f0], b0)
    ec.insert(pp[f0], 0)
    for i in range(f0 + 1, len(pp)):
        pp[i] += 1
    prob.pred_ptr = np.array(pp, np.int32)
    prob.pred_op = np.array(po, np.int32)
    prob.edge_comm = np.array(ec, np.int32)
    g, G, cls = W.priority_groups(prob)
    with pytest.raises(RuntimeError):
        O.greedy(prob, g, G, np.zeros((1, G), np.int32))
