"""GPU parity of the next rows at the sizes and in the launch configuration
bench.py times (the 8-rank VLM workload): every output row of a sample --
the first, the last and random ones -- against the CPU oracle, element by
element; the rollout batch's best key against the oracle's over all of it."""
import numpy as np
import pytest

import oracle as O
import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2504_14145_amd as dip

DEV = "cuda:0"


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _sample(n, k, seed):
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([[0, n - 1], rng.integers(0, n, size=k)]))


def test_greedy_full_batch_sampled():
    need_gpu()
    cfg = W.get(2)
    prob = W.make_problem(cfg)
    g, G, cls = W.priority_groups(prob)
    n = cfg.n_cand
    prio = W.rollout_priorities(cls, n, seed=cfg.seed)
    print(f"greedy: {n} priority vectors", flush=True)
    sim = dip.Sim(prob)
    assert sim.configure_greedy(G, g) == dip.OK
    ords, (ms, bub, pk, fl) = sim.greedy(torch.from_numpy(prio).to(DEV))
    torch.cuda.synchronize()
    idx = _sample(n, 62, 1)
    want_o, want = O.greedy(prob, g, G, prio[idx], stride=prob.stride, threads=16)
    N = prob.n_total
    np.testing.assert_array_equal(ords.cpu().numpy()[idx, :N], want_o[:, :N])
    np.testing.assert_array_equal(ms.cpu().numpy()[idx], want.makespan)
    np.testing.assert_array_equal(bub.cpu().numpy()[idx], want.bubble)
    np.testing.assert_array_equal(pk.cpu().numpy()[idx], want.peak)
    np.testing.assert_array_equal(fl.cpu().numpy()[idx], want.flags)
    sim.close()


def test_memopt_full_batch_sampled():
    need_gpu()
    import oracle.memopt as MO
    from workloads.strategies import strategy_table
    cfg = W.get(2)
    prob = W.make_problem(cfg)
    tab = strategy_table(prob)
    n, S = cfg.n_cand, 6
    rows = W.generator_for(prob, cfg).generate(0, n)
    peak = O.evaluate(prob, rows[:2048], threads=16).peak
    prob.mem_cap[:] = int(np.median(peak) * 0.6)          # the bench's binding cap
    print(f"memopt: {n} schedules, cap {prob.mem_cap[0]}", flush=True)
    sim = dip.Sim(prob)
    assert dip.configure_memopt(sim.h, tab.slot_layers, tab.time, tab.mem, S) == dip.OK
    P = prob.n_ranks
    t = torch.empty((n, P), dtype=torch.int64, device=DEV)
    p = torch.empty((n, P), dtype=torch.int32, device=DEV)
    s = torch.empty((n, P), dtype=torch.uint8, device=DEV)
    dip.memopt(sim.h, torch.from_numpy(rows).to(DEV), n, t, p, s)
    torch.cuda.synchronize()
    idx = _sample(n, 22, 2)
    want = MO.optimise(prob, tab, MO.pair_candidates(tab, S), rows[idx])
    np.testing.assert_array_equal(t.cpu().numpy()[idx], [[x[0] for x in per] for per in want])
    np.testing.assert_array_equal(p.cpu().numpy()[idx], [[x[2] for x in per] for per in want])
    np.testing.assert_array_equal(s.cpu().numpy()[idx], [[x[1] for x in per] for per in want])
    sim.close()


def test_cost_tables_full_batch_sampled():
    need_gpu()
    import oracle.costmodel as OC
    from workloads.operators import N_KINDS, coefficient_sweep, operator_table
    cfg = W.get(2)
    prob = W.make_problem(cfg)
    tab = operator_table(prob)
    n = 16384
    coef = coefficient_sweep(n, seed=cfg.seed)
    print(f"cost tables: {n} configurations x {len(tab.item_ptr) - 1} items", flush=True)
    dt = dip.DeviceOpTable(tab, N_KINDS, DEV)
    out = torch.empty((n, len(tab.item_ptr) - 1), dtype=torch.int32, device=DEV)
    dip.cost_tables(dt, torch.from_numpy(coef).to(DEV), out)
    torch.cuda.synchronize()
    idx = _sample(n, 6, 3)
    np.testing.assert_array_equal(out.cpu().numpy()[idx], OC.cost_tables(tab, coef[idx]))


def test_rollout_batch_full_size():
    need_gpu()
    import oracle.mcts as OM
    cfg = W.get(2)
    prob = W.make_problem(cfg)
    g, G, cls = W.priority_groups(prob)
    ncls = int(cls.max()) + 1
    R = 16384
    sim = dip.Sim(prob)
    assert sim.configure_greedy(G, g) == dip.OK
    sim.greedy(torch.zeros((1, G), dtype=torch.int32, device=DEV))     # uploads the costs
    assert dip.configure_rollouts(sim.h, ncls, cls) == dip.OK
    prio = torch.empty((R, G), dtype=torch.int32, device=DEV)
    ms = torch.empty(R, dtype=torch.int32, device=DEV)
    fl = torch.empty(R, dtype=torch.uint8, device=DEV)
    key = torch.full((1,), -1, dtype=torch.int64, device=DEV)
    print(f"rollouts: {R} from the root", flush=True)
    dip.rollouts(sim.h, [], R, cfg.seed, 3, prio, ms, fl, key)
    torch.cuda.synchronize()
    want = np.stack([OM.priorities_of(OM.shuffled(range(ncls), cfg.seed, 3, i), cls, ncls)
                     for i in range(R)])
    got = prio.cpu().numpy()
    idx = _sample(R, 62, 4)
    np.testing.assert_array_equal(got[idx], want[idx])
    _, res = O.greedy(prob, g, G, want, threads=16)
    np.testing.assert_array_equal(ms.cpu().numpy(), res.makespan)
    np.testing.assert_array_equal(fl.cpu().numpy(), res.flags)
    assert dip.decode_key(int(key.item())) == O.argmin(res.makespan, res.flags)
    sim.close()
