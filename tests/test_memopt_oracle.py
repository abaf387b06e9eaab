"""Pins of the memory-optimisation oracle (oracle/memopt.py, Sec. 5.3):
Pareto fronts and knapsack candidates against brute force over every
per-layer choice, the liveness against the simulator oracle's peak memory,
a selection worked by hand, the solver's gap to the exact optimum (by
enumeration, and by an independent MILP solver on the workloads' ranks), and
the costs of a re-timed schedule."""
import itertools

import numpy as np
import pytest

import oracle as O
import oracle.memopt as MO
import workloads as W
from workloads.strategies import strategy_table


def _brute_points(layers):
    return [(sum(c[0] for c in combo), sum(c[1] for c in combo))
            for combo in itertools.product(*layers)]


def test_pareto_front_and_candidates_by_brute_force():
    rng = np.random.default_rng(1)
    for _ in range(40):
        L = int(rng.integers(1, 6))
        layers = [[(int(t), int(m)) for t, m in zip(rng.integers(1, 20, 3), rng.integers(0, 30, 3))]
                  for _ in range(L)]
        pts = _brute_points(layers)
        front = MO.pareto(layers)
        # every front point is achievable and undominated; every point is dominated by one
        assert all(p in pts for p in front)
        for t, m in pts:
            assert any(ft <= t and fm <= m for ft, fm in front)
        for a in front:
            assert not any((b[0] <= a[0] and b[1] <= a[1] and b != a) for b in pts)
        S = int(rng.integers(2, 8))
        cand = MO.candidates(front, S)
        fastest = min(pts, key=lambda p: (p[0], p[1]))
        leanest = min(pts, key=lambda p: (p[1], p[0]))
        assert cand[0] == fastest and cand[-1] == leanest
        assert len(cand) <= S
        lo, hi = leanest[1], fastest[1]
        if S > 2:
            edges = [lo + ((hi - lo) * k) // (S - 2) for k in range(S - 1)]
            for k in range(1, S - 1):
                fit = [p for p in pts if p[1] <= edges[k]]
                assert min(fit) in cand            # knapsack at the bucket's upper edge
        ts = [c[0] for c in cand]
        ms = [c[1] for c in cand]
        assert ts == sorted(ts) and ms == sorted(ms, reverse=True) and len(set(ts)) == len(ts)


def test_liveness_matches_simulator_peak():
    """With every pair keeping all activations, the most loaded checkpoint
    of each rank equals the simulator oracle's peak memory."""
    prob = W.make_problem(2)
    tab = strategy_table(prob)
    keep = [[(1, int(prob.slot_act[s]))] for s in range(prob.n_slots)]
    rows = W.generator_for(prob, 2).generate(0, 12)
    sim = O.evaluate(prob, rows)
    for c, row in enumerate(rows):
        for r in range(prob.n_ranks):
            _, cands, live = MO.rank_problem(prob, tab, keep, row, r)
            load = [sum(cands[i][0][1] for i in live[k]) for k in range(len(cands))]
            assert max(load) == sim.peak[c, r]


def test_selection_by_hand():
    # pairs 0, 1, 2 all live at checkpoint 2, cap 10:
    # fastest loads 6 + 5 + 4 = 15; steps: pair 0 (5->3 time, 6->2 mem: 1 us per
    # 2 units), pair 1 (4->8, 5->1: 1 per 1), pair 2 (1->2, 4->3: 1 per 1)
    cands = [[(3, 6), (4, 2)], [(4, 5), (8, 1)], [(1, 4), (2, 3)]]
    pf, pb = [0, 1, 2], [5, 4, 3]
    live = MO.live_sets(pf, pb)
    assert live == [[0], [0, 1], [0, 1, 2]]
    cur, total, ok, peak = MO.greedy_select(cands, live, 10)
    # first move pair 0 (ratio 1/4): load 11; next best at checkpoint 2: pair 2
    # (1/1) ties pair 1 (4/4)? pair 1 is 4 per 4 = 1, pair 2 is 1 per 1 = 1:
    # tie -> lower index, pair 1: load 7 <= 10
    assert cur == [1, 1, 0] and total == 4 + 8 + 1 and ok and peak == 7
    assert MO.exact(cands, live, 10) == 4 + 4 + 2     # the greedy is 13, the optimum 10
    assert MO.greedy_select(cands, live, 1)[2] is False
    # the improvement pass cannot undo a single move here (pair 1 back to its
    # fastest needs 4 more units at checkpoint 2, which has 3 to spare); the
    # branch and bound from 13: pair 0 fast (6) + pair 1 fast (5) = 11 over
    # the cap at checkpoint 1?  no, checkpoint 1 holds pairs 0 and 1 only: 11
    # > 10, so pair 1 goes lean there; pair 0 lean (2) + pair 1 fast (5) +
    # pair 2 lean (3) = 10 reaches the optimum 4 + 4 + 2
    assert MO.tighten(cands, live, 10, cur) == [1, 1, 0]
    sel, tot, status, pk = MO.select(cands, live, pf, pb, 10)
    assert sel == [1, 0, 1] and tot == 10 and status == 1 and pk == 10
    assert MO.exact_bb(cands, live, pf, pb, 10) == 10
    assert MO.select(cands, live, pf, pb, 1)[2] == 0


def _random_case(rng):
    n = int(rng.integers(1, 7))
    cands = []
    for _ in range(n):
        k = int(rng.integers(1, 5))
        t = np.cumsum(rng.integers(1, 10, k))
        m = np.cumsum(rng.integers(1, 10, k))[::-1]
        cands.append(list(zip(t.tolist(), m.tolist())))
    pf = rng.permutation(n).tolist()
    pb = [int(pf[i]) + int(rng.integers(0, n)) for i in range(n)]
    cap = int(rng.integers(0, sum(c[0][1] for c in cands) + 2))
    return cands, pf, pb, cap


def test_selection_within_gap_on_random_small_instances():
    """The solver against exhaustive search on every seeded case: never below
    the optimum, proven within 5 % of it (Sec. 5.3's allowance); the
    exhaustive branch and bound reaches the optimum itself."""
    rng = np.random.default_rng(7)
    gaps = []
    for _ in range(1200):
        cands, pf, pb, cap = _random_case(rng)
        live = MO.live_sets(pf, pb)
        best = MO.exact(cands, live, cap)
        sel, total, status, peak = MO.select(cands, live, pf, pb, cap)
        assert MO.exact_bb(cands, live, pf, pb, cap) == best
        if best is None:
            assert status == 0
            continue
        assert status == 1
        assert total >= best and 100 * total <= 105 * best
        assert peak <= cap and total == sum(cands[i][sel[i]][0] for i in range(len(cands)))
        gaps.append(total / best - 1)
    print(f"selection gap: mean {np.mean(gaps):.3%}, max {np.max(gaps):.3%} over {len(gaps)} cases")


def _milp_optimum(cands, live, cap):
    """The optimum by an independent solver (HiGHS through scipy), exact for
    these integer data: one binary per (pair, candidate)."""
    from scipy.optimize import Bounds, LinearConstraint, milp
    n = len(cands)
    idx = [(i, j) for i, c in enumerate(cands) for j in range(len(c))]
    cost = np.array([cands[i][j][0] for i, j in idx], float)
    one = np.zeros((n, len(idx)))
    mem = np.zeros((n, len(idx)))
    for v, (i, j) in enumerate(idx):
        one[i, v] = 1
        for k in range(n):
            if i in live[k]:
                mem[k, v] = cands[i][j][1]
    res = milp(cost, constraints=[LinearConstraint(one, 1, 1), LinearConstraint(mem, -np.inf, cap)],
               integrality=np.ones(len(idx)), bounds=Bounds(0, 1),
               options={"mip_rel_gap": 0.0})
    return None if res.status != 0 else int(round(res.fun))


def test_lagrangian_bound_is_sound_and_certifies():
    """Step 4's bound never exceeds the optimum exhaustive search finds (so a
    certificate is never wrong), and with the branch and bound cut short
    (one placement) every selection the certificate proves is within 5 % of
    the optimum.  (On these tiny random cases the relaxation is often more
    than 5 % below the optimum, so it proves only some.)"""
    rng = np.random.default_rng(11)
    proved = tried = 0
    for _ in range(600):
        cands, pf, pb, cap = _random_case(rng)
        live = MO.live_sets(pf, pb)
        best = MO.exact(cands, live, cap)
        if best is None:
            continue
        for val, F in MO.lagrangian_values(cands, live, cap):
            assert val <= best << F, (val, F, best)
        cur, _, ok, _ = MO.greedy_select(cands, live, cap)
        cur = MO.tighten(cands, live, cap, cur)
        cur, proven, _ = MO.branch_and_bound(cands, pf, pb, cap, cur, 1)
        if proven:
            continue
        total = sum(cands[i][cur[i]][0] for i in range(len(cands)))
        tried += 1
        if MO.lagrangian_proof(cands, live, cap, total):
            proved += 1
            assert 100 * total <= 105 * best
    print(f"certificate: {proved} of {tried} selections the cut-short search left unproven")
    assert tried > 100 and proved > 0


def test_lagrangian_step_by_hand():
    """Two pairs live at both checkpoints, cap 10: pair 0 takes (t, m) = (1, 8)
    or (3, 2), pair 1 (1, 8) or (2, 4).  Within the cap: (3, 2) + (1, 8),
    time 4 (the optimum), and (3, 2) + (2, 4), time 5.  With both pairs live
    at both checkpoints the relaxation depends on the sum p of the two
    multipliers only:  L(p) = min(1 + 8p, 3 + 2p) + min(1 + 8p, 2 + 4p) - 10p,
    at most 11/3 (at p = 1/3).  Its first step (no multipliers) is 2; the
    steps climb towards 11/3 and never pass it; 1.05 * 11/3 < 4, so the
    certificate proves an incumbent of 3 but never the optimum 4."""
    cands = [[(1, 8), (3, 2)], [(1, 8), (2, 4)]]
    live = [[0, 1], [0, 1]]
    vals = [v / (1 << F) for v, F in MO.lagrangian_values(cands, live, 10)]
    assert vals[0] == 2
    assert 3.5 <= max(vals) <= 11 / 3
    assert MO.exact(cands, live, 10) == 4
    assert MO.lagrangian_proof(cands, live, 10, 3)
    assert not MO.lagrangian_proof(cands, live, 10, 4)


@pytest.mark.parametrize("frac,S", [(0.6, 6), (0.3, 6), (0.15, 4)])
def test_selection_on_workload_ranks_against_milp(frac, S):
    """The 8-rank VLM workload's ranks (32 and 68 stage pairs) under caps
    that bind: the solver never beats and stays within 5 % of the optimum
    an independent MILP solver finds, and proves it under the two looser
    caps."""
    pytest.importorskip("scipy")
    prob = W.make_problem(2)
    tab = strategy_table(prob)
    rows = W.generator_for(prob, 2).generate(0, 3)
    cap = int(np.median(O.evaluate(prob, rows).peak) * frac)
    cands = MO.pair_candidates(tab, S)
    n = 0
    for row in rows:
        for r in range(prob.n_ranks):
            _, c, live = MO.rank_problem(prob, tab, cands, row, r)
            pf, pb = MO.rank_positions(prob, tab, row, r)
            sel, total, status, peak = MO.select(c, live, pf, pb, cap)
            opt = _milp_optimum(c, live, cap)
            if opt is None:
                assert status == 0
                continue
            # proven within 5 % (by the search or the certificate), except
            # under the tightest cap with 4 candidates, where the relaxation
            # falls 5.5-7.5 % below the optimum on some ranks: there the
            # selection is within 5 % but stays unproven (status 3)
            assert (status == 1 if frac > 0.2 else status in (1, 3)) and peak <= cap
            assert total >= opt and 100 * total <= 105 * opt, (r, total, opt)
            n += 1
    assert n > 0


def test_retimed_costs():
    """Keeping every activation leaves every op's cost; a pair moved to full
    recomputation runs its forward again inside its backward."""
    prob = W.make_problem(2)
    tab = strategy_table(prob)
    cands = MO.pair_candidates(tab, 6)
    rows = W.generator_for(prob, 2).generate(0, 1)
    per = MO.optimise(prob, tab, cands, rows, caps=[-1] * prob.n_ranks)[0]
    np.testing.assert_array_equal(MO.retimed_costs(prob, tab, cands, per), prob.op_cost)
    s = 0
    r = int(tab.slot_rank[s])
    per = [list(x) for x in per]
    i = [q for q in range(prob.n_slots) if tab.slot_rank[q] == r].index(s)
    per[r][3] = list(per[r][3])
    per[r][3][i] = len(cands[s]) - 1                 # the leanest candidate
    cost = MO.retimed_costs(prob, tab, cands, per)
    f, b = int(tab.slot_f[s]), int(tab.slot_b[s])
    layers = range(tab.slot_layers[s], tab.slot_layers[s + 1])
    # this pair's leanest candidate recomputes every layer in full (its
    # activation is large enough that the three strategies' memory differs)
    assert cands[s][-1][0] == sum(int(tab.time[l][2]) for l in layers)
    assert cost[f] == prob.op_cost[f]
    assert cost[b] == cands[s][-1][0] - prob.op_cost[f] == prob.op_cost[b] + prob.op_cost[f]


def test_no_cap_keeps_the_fastest():
    prob = W.make_problem(2)
    tab = strategy_table(prob)
    cands = MO.pair_candidates(tab, 6)
    rows = W.generator_for(prob, 2).generate(0, 2)
    res = MO.optimise(prob, tab, cands, rows, caps=[-1] * prob.n_ranks)
    for r in range(prob.n_ranks):
        slots = [s for s in range(prob.n_slots) if tab.slot_rank[s] == r]
        assert res[0][r][0] == sum(cands[s][0][0] for s in slots) and res[0][r][1] == 1
