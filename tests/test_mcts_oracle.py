"""Pins of the MCTS oracle (oracle/mcts.py, Sec. 5.1): SplitMix64's published
outputs, uniformity of the rollout shuffles, a UCB selection worked out by
hand, brute force over every class sequence of a tiny instance, and the
backpropagation invariants of the finished tree."""
import itertools
import math

import numpy as np
import pytest

import oracle as O
import oracle.mcts as M
import workloads as W


def test_splitmix64_reference_outputs():
    # the reference generator's first outputs from state 0
    assert M.splitmix64(0, 3) == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_shuffle_is_uniform():
    counts = {}
    n = 24000
    for i in range(n):
        p = tuple(M.shuffled([0, 1, 2, 3], seed=5, draw=1, index=i))
        counts[p] = counts.get(p, 0) + 1
    assert len(counts) == 24
    exp = n / 24
    chi2 = sum((c - exp) ** 2 / exp for c in counts.values())
    assert chi2 < 49.7          # 23 degrees of freedom, p = 0.001


def test_priorities_follow_positions():
    seq = [2, 0, 3, 1]
    group_class = [0, 0, 1, 2, 3, 3]
    assert M.priorities_of(seq, group_class, 4).tolist() == [3, 3, 1, 4, 2, 2]


def test_ucb_choice_by_hand():
    """root N=10, s=100; children a (s=100, N=5), b (s=120, N=2), c (no score,
    N=1); alpha 1, beta 0.5:
      a: 1       + 0.5*sqrt(ln 10 / 5) = 1.3393
      b: 100/120 + 0.5*sqrt(ln 10 / 2) = 1.3698
      c: 0       + 0.5*sqrt(ln 10 / 1) = 0.7587   -> b."""
    root = M.Node(None, None, 3)
    root.untried = []
    root.N, root.s = 10, 100.0
    for cls, (s, n) in zip((0, 1, 2), ((100.0, 5), (120.0, 2), (M.INF, 1))):
        v = M.Node(cls, root, 3)
        v.s, v.N = s, n
        root.children[cls] = v
    assert abs(M.ucb(root.s, root.N, root.children[0], 1.0, 0.5) - 1.3393) < 1e-4
    assert abs(M.ucb(root.s, root.N, root.children[1], 1.0, 0.5) - 1.3698) < 1e-4
    assert abs(M.ucb(root.s, root.N, root.children[2], 1.0, 0.5) - 0.7587) < 1e-4
    assert M.select(root, 1.0, 0.5).cls == 1


def _tiny():
    inst = W.pipeline_instance(2, 2, np.array([[3, 7], [5, 2]]), comm=1)
    prob = W.compile_instance(inst)
    g, G, cls = W.priority_groups(prob)
    return prob, g, G, cls


def test_exhaustive_search_finds_the_brute_force_optimum():
    prob, g, G, cls = _tiny()
    n = int(cls.max()) + 1
    assert n == 4
    all_seq = list(itertools.permutations(range(n)))
    prio = np.stack([M.priorities_of(q, cls, n) for q in all_seq])
    _, res = O.greedy(prob, g, G, prio)
    brute = min(res.makespan)
    traj, best, root = M.search(prob, g, G, cls, iterations=500, rollouts=3, seed=1)
    assert len(traj) == 4 + 12 + 24 + 24       # every tree node expanded once, then stop
    assert root.done
    assert best[0] == brute
    # the best sequence reproduces its score
    _, r1 = O.greedy(prob, g, G, M.priorities_of(best[1], cls, n)[None, :])
    assert r1.makespan[0] == brute


def test_backpropagation_invariants():
    prob = W.make_problem(1)
    g, G, cls = W.priority_groups(prob)
    traj, best, root = M.search(prob, g, G, cls, iterations=40, rollouts=8, seed=2)
    # s and N of every node equal the min and the count over the iterations
    # whose rolled-out node lies in its subtree
    def walk(v):
        pre = tuple(v.prefix())
        hits = [sc for (p, sc, _) in traj if p[:len(pre)] == pre]
        assert v.N == len(hits)
        assert v.s == min(hits)
        assert v.N == (1 if v.cls is not None else 0) + sum(c.N for c in v.children.values())
        for c in v.children.values():
            walk(c)
    walk(root)
    assert best[0] == min(sc for (_, sc, _) in traj)
    assert root.s == best[0]


def test_caps_make_rollouts_infeasible():
    inst = W.pipeline_instance(2, 3, 4, comm=1, mem_cap=0)
    prob = W.compile_instance(inst)
    g, G, cls = W.priority_groups(prob)
    traj, best, root = M.search(prob, g, G, cls, iterations=5, rollouts=4, seed=3)
    assert all(sc == M.INF for (_, sc, _) in traj)
    assert best[1] is None and root.s == M.INF


def _dfs_prefixes(n):
    """Depth-first visiting order of the tree of class sequences, children in
    ascending class order: every proper and complete prefix, parents first."""
    out = []

    def walk(prefix):
        for c in range(n):
            if c not in prefix:
                out.append(tuple(prefix + [c]))
                walk(prefix + [c])
    walk([])
    return out


def test_dfs_policy_walks_the_tree_depth_first():
    """Depth-first search expands every node of the 4-class tree in DFS order
    (64 nodes), then stops, and its best is the brute-force optimum."""
    prob, g, G, cls = _tiny()
    n = int(cls.max()) + 1
    traj, best, root = M.search(prob, g, G, cls, iterations=500, rollouts=2, seed=4, policy="dfs")
    assert [p for (p, _, _) in traj] == _dfs_prefixes(n)
    assert len(traj) == 64 and root.done
    all_seq = list(itertools.permutations(range(n)))
    _, res = O.greedy(prob, g, G, np.stack([M.priorities_of(q, cls, n) for q in all_seq]))
    assert best[0] == min(res.makespan)
    # each complete prefix is scored exactly (every rollout is that sequence)
    by_seq = dict(zip(all_seq, res.makespan))
    for p, sc, _ in traj:
        if len(p) == n:
            assert sc == by_seq[p]


def test_random_policy_rolls_out_from_the_root():
    """Random exploration: every iteration R uniform sequences of all classes,
    the same shuffles as the rollouts of an empty prefix; the tree never grows."""
    prob = W.make_problem(1)
    g, G, cls = W.priority_groups(prob)
    n = int(cls.max()) + 1
    R = 6
    traj, best, root = M.search(prob, g, G, cls, iterations=5, rollouts=R, seed=9, policy="random")
    assert all(p == () for (p, _, _) in traj) and not root.children and root.N == 5
    for t, (_, sc, idx) in enumerate(traj):
        seqs = [M.shuffled(range(n), 9, t, i) for i in range(R)]
        _, res = O.greedy(prob, g, G, np.stack([M.priorities_of(q, cls, n) for q in seqs]))
        scores = [m if f == 0 else M.INF for m, f in zip(res.makespan, res.flags)]
        assert sc == min(scores) and idx == scores.index(min(scores))
    assert best[0] == min(sc for (_, sc, _) in traj)
    with pytest.raises(ValueError):
        M.search(prob, g, G, cls, iterations=1, rollouts=1, seed=0, policy="bfs")


def test_parallel_workers_explore_the_whole_tree():
    """Five workers per round on the 4-class tree: every node is expanded once
    (64 leaves), the search stops, and it finds the brute-force optimum."""
    prob, g, G, cls = _tiny()
    n = int(cls.max()) + 1
    traj, best, root = M.search(prob, g, G, cls, iterations=100, rollouts=2, seed=6, workers=5)
    assert root.done
    assert sorted(p for (p, _, _) in traj) == sorted(_dfs_prefixes(n))
    all_seq = list(itertools.permutations(range(n)))
    _, res = O.greedy(prob, g, G, np.stack([M.priorities_of(q, cls, n) for q in all_seq]))
    assert best[0] == min(res.makespan)


def test_parallel_workers_invariants():
    """W = 8 on config 1: the first round's leaves are 8 distinct children of
    the root (virtual visits never send two workers to one untried slot); in
    the finished tree N counts the leaves of each subtree and s is their best
    score; the best is the least leaf score."""
    prob = W.make_problem(1)
    g, G, cls = W.priority_groups(prob)
    n = int(cls.max()) + 1
    traj, best, root = M.search(prob, g, G, cls, iterations=6, rollouts=4, seed=8, workers=8)
    assert len(traj) == 48
    first = [p for (p, _, _) in traj[:8]]
    assert all(len(p) == 1 for p in first) and len(set(first)) == 8

    def walk(v):
        pre = tuple(v.prefix())
        hits = [sc for (p, sc, _) in traj if p[:len(pre)] == pre]
        assert v.N == len(hits)
        assert v.s == min(hits)
        for c in v.children.values():
            walk(c)
    walk(root)
    assert best[0] == min(sc for (_, sc, _) in traj)
    # one worker is the sequential search
    t1, b1, _ = M.search(prob, g, G, cls, iterations=12, rollouts=4, seed=8, workers=1)
    t2, b2, _ = M.search(prob, g, G, cls, iterations=12, rollouts=4, seed=8)
    assert t1 == t2 and b1[0] == b2[0]


def _capped_tiny(cap):
    inst = W.pipeline_instance(2, 3, np.array([[3, 7, 4], [5, 2, 6]]), comm=1, act=8, mem_cap=cap)
    prob = W.compile_instance(inst)
    g, G, cls = W.priority_groups(prob)
    return prob, g, G, cls


def test_memory_aware_scores():
    """Sec. 5.1's rollout score with the memory optimisation: equal to the
    makespan when nothing is capped; under a binding cap finite where the
    selection meets it, never below the same orders' makespan without
    recomputation, and +inf exactly where some rank's cap is out of reach."""
    from workloads.strategies import strategy_table
    import oracle.memopt as MO
    prob, g, G, cls = _capped_tiny(-1)
    tab = strategy_table(prob)
    mem = (tab, MO.pair_candidates(tab, 4))
    n = int(cls.max()) + 1
    seqs = list(itertools.permutations(range(n)))
    prio = np.stack([M.priorities_of(q, cls, n) for q in seqs])
    free = M.score_rollouts(prob, g, G, prio)
    assert M.score_rollouts(prob, g, G, prio, memory=mem) == free
    for cap in (20, 12, 8, 4, 1):
        pc, _, _, _ = _capped_tiny(cap)
        plain = M.score_rollouts(pc, g, G, prio)
        aware = M.score_rollouts(pc, g, G, prio, memory=mem)
        orders, _ = O.greedy(pc, g, G, prio)       # (the interleaving sees the cap)
        base = O.evaluate(pc, orders).makespan       # the same orders, nothing recomputed
        per = MO.optimise(pc, tab, mem[1], orders)
        for k in range(len(seqs)):
            reach = all(x[1] in (1, 3) for x in per[k])
            assert (aware[k] < M.INF) == reach, (cap, k)
            if reach:
                assert aware[k] >= base[k]
            if plain[k] < M.INF:              # within the cap as interleaved: kept as is
                assert aware[k] == plain[k]
        if cap == 4:   # below what the interleaving alone can meet: recomputation repairs it
            assert all(p == M.INF and a < M.INF for p, a in zip(plain, aware))


def test_exhaustive_memory_aware_search_finds_the_brute_force_optimum():
    from workloads.strategies import strategy_table
    import oracle.memopt as MO
    prob, g, G, cls = _capped_tiny(4)
    tab = strategy_table(prob)
    mem = (tab, MO.pair_candidates(tab, 4))
    n = int(cls.max()) + 1
    seqs = list(itertools.permutations(range(n)))
    prio = np.stack([M.priorities_of(q, cls, n) for q in seqs])
    brute = min(M.score_rollouts(prob, g, G, prio, memory=mem))
    traj, best, root = M.search(prob, g, G, cls, iterations=2000, rollouts=3, seed=1, memory=mem)
    assert root.done and best[0] == brute < M.INF
