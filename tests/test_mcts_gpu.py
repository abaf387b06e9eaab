"""GPU parity of the MCTS rollouts (dip_sim_rollouts) and of the GPU-batched
search (paper_2504_14145_amd.mcts) against the CPU oracle: rollout
priorities, scores and argmin bit-exact; whole search trajectories equal."""
import numpy as np
import pytest

import oracle as O
import oracle.mcts as OM
import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2504_14145_amd as dip
    from paper_2504_14145_amd.mcts import Search

DEV = "cuda:0"


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _sim(prob):
    g, G, cls = W.priority_groups(prob)
    sim = dip.Sim(prob)
    assert sim.configure_greedy(G, g) == dip.OK
    # upload the costs once (a zero-candidate call records nothing)
    sim.greedy(torch.zeros((1, G), dtype=torch.int32, device=DEV))
    return sim, g, G, cls


@pytest.mark.parametrize("cid,depth,R", [(1, 0, 300), (1, 5, 257), (2, 17, 300), (1, 16, 9),
                                         (4, 40, 33), (5, 100, 17)])
def test_rollouts_match_oracle(cid, depth, R):
    need_gpu()
    prob = W.make_problem(cid)
    sim, g, G, cls = _sim(prob)
    n = int(cls.max()) + 1
    depth = min(depth, n)
    rng = np.random.default_rng(depth)
    prefix = [int(c) for c in rng.permutation(n)[:depth]]
    assert dip.configure_rollouts(sim.h, n, cls) == dip.OK
    prio = torch.empty((R, G), dtype=torch.int32, device=DEV)
    ms = torch.empty(R, dtype=torch.int32, device=DEV)
    fl = torch.empty(R, dtype=torch.uint8, device=DEV)
    key = torch.full((1,), -1, dtype=torch.int64, device=DEV)
    print(f"config {cid} depth {depth} rollouts {R}", flush=True)
    dip.rollouts(sim.h, prefix, R, 12345, 7, prio, ms, fl, key)
    torch.cuda.synchronize()
    rest = [c for c in range(n) if c not in set(prefix)]
    want = np.stack([OM.priorities_of(prefix + OM.shuffled(rest, 12345, 7, i), cls, n)
                     for i in range(R)])
    np.testing.assert_array_equal(prio.cpu().numpy(), want)
    _, res = O.greedy(prob, g, G, want, threads=16)
    np.testing.assert_array_equal(ms.cpu().numpy(), res.makespan)
    np.testing.assert_array_equal(fl.cpu().numpy(), res.flags)
    assert dip.decode_key(int(key.item())) == O.argmin(res.makespan, res.flags)[::1]
    sim.close()


def test_rollouts_reject_bad_prefixes_and_report_infeasible():
    need_gpu()
    inst = W.pipeline_instance(2, 3, 4, comm=1, mem_cap=0)
    prob = W.compile_instance(inst)
    sim, g, G, cls = _sim(prob)
    n = int(cls.max()) + 1
    assert dip.configure_rollouts(sim.h, n, cls) == dip.OK
    prio = torch.empty((8, G), dtype=torch.int32, device=DEV)
    ms = torch.empty(8, dtype=torch.int32, device=DEV)
    fl = torch.empty(8, dtype=torch.uint8, device=DEV)
    key = torch.full((1,), -1, dtype=torch.int64, device=DEV)
    with pytest.raises(dip.DipSimError):
        dip.rollouts(sim.h, [0, 0], 8, 1, 0, prio, ms, fl, key)      # repeated class
    with pytest.raises(dip.DipSimError):
        dip.rollouts(sim.h, [n], 8, 1, 0, prio, ms, fl, key)         # out of range
    dip.rollouts(sim.h, [], 8, 1, 0, prio, ms, fl, key)
    torch.cuda.synchronize()
    assert (fl.cpu().numpy() == dip.FLAG_CAP).all()
    assert dip.decode_key(int(key.item())) == (-1, -1)
    sim.close()


def _tiny():
    inst = W.pipeline_instance(2, 2, np.array([[3, 7], [5, 2]]), comm=1)
    return W.compile_instance(inst)


@pytest.mark.parametrize("case", ["tiny", "c1", "c2", "c3", "c4", "c5"])
def test_search_trajectory_matches_oracle(case):
    need_gpu()
    prob = _tiny() if case == "tiny" else W.make_problem(int(case[1]))
    iters, R = {"tiny": (200, 3), "c1": (40, 64), "c2": (12, 128), "c3": (4, 12), "c4": (3, 8),
                "c5": (2, 5)}[case]
    sim, g, G, cls = _sim(prob)
    print(f"{case}: {iters} iterations x {R} rollouts", flush=True)
    srch = Search(sim, cls, R, seed=21)
    traj, best = srch.run(iters)
    want_traj, want_best, root = OM.search(prob, g, G, cls, iters, R, seed=21, threads=16)
    assert traj == want_traj
    assert best[0] == want_best[0] and best[2:] == want_best[2:]
    assert best[1] == list(want_best[1])
    if case == "tiny":
        assert root.done and srch.done[0] and len(traj) == 64
    sim.close()


@pytest.mark.parametrize("policy", ["dfs", "random"])
@pytest.mark.parametrize("case", ["tiny", "c2", "c3"])
def test_other_policies_match_oracle(case, policy):
    """Depth-first and random exploration (the strategies the paper compares
    its search with) drive the same rollouts: trajectories equal the oracle's."""
    need_gpu()
    prob = _tiny() if case == "tiny" else W.make_problem(int(case[1]))
    iters, R = {"tiny": (80, 3), "c2": (10, 64), "c3": (4, 12)}[case]
    sim, g, G, cls = _sim(prob)
    print(f"{case} {policy}: {iters} iterations x {R} rollouts", flush=True)
    srch = Search(sim, cls, R, seed=5, policy=policy)
    traj, best = srch.run(iters)
    want_traj, want_best, root = OM.search(prob, g, G, cls, iters, R, seed=5, threads=16,
                                           policy=policy)
    assert traj == want_traj
    assert best[0] == want_best[0] and best[2:] == want_best[2:]
    assert best[1] == list(want_best[1])
    if case == "tiny" and policy == "dfs":
        assert len(traj) == 64 and srch.done[0]
    sim.close()


def test_rollouts_batch_equals_one_call_per_leaf():
    """dip_sim_rollouts_batch: leaf l's rows and key are those of
    dip_sim_rollouts on its prefix with draw_base + l; ragged prefixes
    (empty, partial, complete), and the oracle's shuffles."""
    need_gpu()
    prob = W.make_problem(2)
    sim, g, G, cls = _sim(prob)
    n = int(cls.max()) + 1
    assert dip.configure_rollouts(sim.h, n, cls) == dip.OK
    rng = np.random.default_rng(3)
    perm = [int(c) for c in rng.permutation(n)]
    prefixes = [[], perm[:5], perm[:n], [perm[7]], perm[:n - 1]]
    L, R = len(prefixes), 37
    prio = torch.empty((L * R, G), dtype=torch.int32, device=DEV)
    ms = torch.empty(L * R, dtype=torch.int32, device=DEV)
    fl = torch.empty(L * R, dtype=torch.uint8, device=DEV)
    keys = torch.full((L,), -1, dtype=torch.int64, device=DEV)
    print(f"batch of {L} leaves x {R}", flush=True)
    dip.rollouts_batch(sim.h, prefixes, R, 99, 40, prio, ms, fl, keys)
    torch.cuda.synchronize()
    want = []
    for l, p in enumerate(prefixes):
        rest = [c for c in range(n) if c not in set(p)]
        want += [OM.priorities_of(p + OM.shuffled(rest, 99, 40 + l, i), cls, n) for i in range(R)]
    want = np.stack(want)
    np.testing.assert_array_equal(prio.cpu().numpy(), want)
    _, res = O.greedy(prob, g, G, want, threads=16)
    np.testing.assert_array_equal(ms.cpu().numpy(), res.makespan)
    np.testing.assert_array_equal(fl.cpu().numpy(), res.flags)
    for l in range(L):
        seg = slice(l * R, (l + 1) * R)
        assert dip.decode_key(int(keys[l].item())) == O.argmin(res.makespan[seg], res.flags[seg])
        one = torch.full((1,), -1, dtype=torch.int64, device=DEV)
        dip.rollouts(sim.h, prefixes[l], R, 99, 40 + l, prio[:R], ms[:R], fl[:R], one)
        torch.cuda.synchronize()
        assert int(one.item()) == int(keys[l].item())
    with pytest.raises(dip.DipSimError):
        dip.rollouts_batch(sim.h, [[0], [1, 1]], R, 1, 0, prio, ms, fl, keys)   # repeated class
    sim.close()


@pytest.mark.parametrize("case,workers,policy", [("tiny", 5, "ucb"), ("c1", 8, "ucb"),
                                                 ("c2", 16, "ucb"), ("c3", 4, "ucb"),
                                                 ("c2", 6, "dfs"), ("c2", 3, "random")])
def test_parallel_search_matches_oracle(case, workers, policy):
    """W workers per round with virtual visits: trajectories equal the oracle's."""
    need_gpu()
    prob = _tiny() if case == "tiny" else W.make_problem(int(case[1]))
    rounds, R = {"tiny": (30, 3), "c1": (8, 16), "c2": (5, 64), "c3": (2, 8)}[case]
    sim, g, G, cls = _sim(prob)
    print(f"{case} {policy} x{workers}: {rounds} rounds x {R} rollouts", flush=True)
    srch = Search(sim, cls, R, seed=13, policy=policy, workers=workers)
    traj, best = srch.run(rounds)
    want_traj, want_best, root = OM.search(prob, g, G, cls, rounds, R, seed=13, threads=16,
                                           policy=policy, workers=workers)
    assert traj == want_traj
    assert best[0] == want_best[0] and best[2:] == want_best[2:]
    if want_best[1] is not None:
        assert best[1] == list(want_best[1])
    if case == "tiny":
        assert srch.done[0] and len(traj) == 64
    sim.close()


def _sim_memory(prob, S):
    """A handle with the greedy, the rollouts' classes and the memory
    selection configured: rollouts are then scored after the selection."""
    from workloads.strategies import strategy_table
    import oracle.memopt as MO
    sim, g, G, cls = _sim(prob)
    tab = strategy_table(prob)
    assert dip.configure_memopt(sim.h, tab.slot_layers, tab.time, tab.mem, S) == dip.OK
    return sim, g, G, cls, (tab, MO.pair_candidates(tab, S))


def _capped_tiny(cap):
    inst = W.pipeline_instance(2, 3, np.array([[3, 7, 4], [5, 2, 6]]), comm=1, act=8, mem_cap=cap)
    return W.compile_instance(inst)


def _capped_vlm(frac):
    """The 8-rank VLM workload with caps below what its interleavings reach."""
    prob = W.make_problem(2)
    g, G, cls = W.priority_groups(prob)
    n = int(cls.max()) + 1
    prio = np.stack([OM.priorities_of(list(np.random.default_rng(i).permutation(n)), cls, n)
                     for i in range(16)])
    _, res = O.greedy(prob, g, G, prio, threads=16)
    prob.mem_cap[:] = int(np.median(res.peak) * frac)
    return prob


@pytest.mark.parametrize("case,R", [("tiny", 60), ("c2", 48)])
def test_rollouts_scored_after_memory_selection(case, R):
    """Sec. 5.1's score: every rollout interleaved, memory-optimised and
    re-timed; makespans, flags and the best key against the oracle."""
    need_gpu()
    prob = _capped_tiny(4) if case == "tiny" else _capped_vlm(0.3)
    sim, g, G, cls, mem = _sim_memory(prob, 4 if case == "tiny" else 6)
    n = int(cls.max()) + 1
    assert dip.configure_rollouts(sim.h, n, cls) == dip.OK
    prefix = [int(c) for c in np.random.default_rng(5).permutation(n)[:n // 3]]
    prio = torch.empty((R, G), dtype=torch.int32, device=DEV)
    ms = torch.empty(R, dtype=torch.int32, device=DEV)
    fl = torch.empty(R, dtype=torch.uint8, device=DEV)
    key = torch.full((1,), -1, dtype=torch.int64, device=DEV)
    print(f"{case}: caps {prob.mem_cap.tolist()}, {R} rollouts", flush=True)
    dip.rollouts(sim.h, prefix, R, 777, 3, prio, ms, fl, key)
    torch.cuda.synchronize()
    rest = [c for c in range(n) if c not in set(prefix)]
    want_prio = np.stack([OM.priorities_of(prefix + OM.shuffled(rest, 777, 3, i), cls, n)
                          for i in range(R)])
    np.testing.assert_array_equal(prio.cpu().numpy(), want_prio)
    scores = OM.score_rollouts(prob, g, G, want_prio, threads=16, memory=mem)
    got_ms, got_fl = ms.cpu().numpy(), fl.cpu().numpy()
    for i in range(R):
        assert (got_fl[i] == 0) == (scores[i] < OM.INF), i
        if scores[i] < OM.INF:
            assert got_ms[i] == scores[i], i
    plain = OM.score_rollouts(prob, g, G, want_prio, threads=16)
    finite = [i for i in range(R) if scores[i] < OM.INF]
    assert finite and any(plain[i] == OM.INF for i in finite)   # the selection repaired some
    b = min(finite, key=lambda i: (scores[i], i))
    assert dip.decode_key(int(key.item())) == (b, int(scores[b]))
    sim.close()


@pytest.mark.parametrize("case", ["tiny", "c2"])
def test_memory_aware_search_matches_oracle(case):
    need_gpu()
    prob = _capped_tiny(4) if case == "tiny" else _capped_vlm(0.3)
    iters, R = {"tiny": (120, 3), "c2": (4, 16)}[case]
    sim, g, G, cls, mem = _sim_memory(prob, 4 if case == "tiny" else 6)
    print(f"{case}: {iters} iterations x {R} rollouts, memory-aware", flush=True)
    srch = Search(sim, cls, R, seed=17)
    traj, best = srch.run(iters)
    want_traj, want_best, root = OM.search(prob, g, G, cls, iters, R, seed=17, threads=16,
                                           memory=mem)
    assert traj == want_traj
    assert best[0] == want_best[0] and best[2:] == want_best[2:]
    if want_best[1] is not None:
        assert best[1] == list(want_best[1])
    assert want_best[0] < OM.INF
    sim.close()
