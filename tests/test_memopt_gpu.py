"""GPU parity of the per-layer memory optimisation (dip_sim_memopt) against
the CPU oracle: per candidate schedule and rank, total time, peak and status,
bit-exact."""
import numpy as np
import pytest

import oracle as O
import oracle.memopt as MO
import workloads as W
from workloads.strategies import strategy_table

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2504_14145_amd as dip

DEV = "cuda:0"


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def run(prob, tab, rows, S):
    sim = dip.Sim(prob)
    assert dip.configure_memopt(sim.h, tab.slot_layers, tab.time, tab.mem, S) == dip.OK
    n = rows.shape[0]
    t = torch.empty((n, prob.n_ranks), dtype=torch.int64, device=DEV)
    pk = torch.empty((n, prob.n_ranks), dtype=torch.int32, device=DEV)
    st = torch.empty((n, prob.n_ranks), dtype=torch.uint8, device=DEV)
    dip.memopt(sim.h, torch.from_numpy(np.ascontiguousarray(rows)).to(DEV), n, t, pk, st)
    torch.cuda.synchronize()
    sim.close()
    return t.cpu().numpy(), pk.cpu().numpy(), st.cpu().numpy()


@pytest.mark.parametrize("cid,n,frac,S", [(2, 131, 0.6, 6), (2, 67, 0.15, 4), (3, 9, 0.5, 6),
                                          (3, 5, 0.1, 8), (2, 40, -1, 6)])
def test_memopt_matches_oracle(cid, n, frac, S):
    need_gpu()
    prob = W.make_problem(cid)
    tab = strategy_table(prob)
    rows = W.generator_for(prob, cid).generate(0, n)
    if frac < 0:
        prob.mem_cap[:] = -1
    else:
        peak = O.evaluate(prob, rows).peak
        prob.mem_cap[:] = int(np.median(peak) * frac)
    print(f"config {cid}: {n} schedules, cap {prob.mem_cap[0]}, S {S}", flush=True)
    got_t, got_p, got_s = run(prob, tab, rows, S)
    cands = MO.pair_candidates(tab, S)
    want = MO.optimise(prob, tab, cands, rows)
    wt = np.array([[x[0] for x in per] for per in want])
    wp = np.array([[x[2] for x in per] for per in want])
    ws = np.array([[1 if x[1] else 0 for x in per] for per in want])
    np.testing.assert_array_equal(got_s, ws)
    np.testing.assert_array_equal(got_t, wt)
    np.testing.assert_array_equal(got_p, wp)
    if frac == 0.1:
        assert (ws == 0).any()            # a cap tight enough to be out of reach somewhere


def test_memopt_flags_invalid_orders():
    need_gpu()
    prob = W.make_problem(2)
    tab = strategy_table(prob)
    rows = W.generator_for(prob, 2).generate(0, 4)
    rows[1, 3] = rows[1, 4]                               # a repeated id on rank 0
    rows[2, int(prob.rank_off[5])] = 999                  # out of range on rank 5
    t, pk, st = run(prob, tab, rows, 6)
    assert st[1, 0] == 2 and t[1, 0] == -1 and pk[1, 0] == -1
    assert st[2, 5] == 2
    assert (st[0] != 2).all() and (st[3] != 2).all()


@pytest.mark.parametrize("frac", [0.5, 0.85])
def test_memopt_ranks_with_many_pairs(frac):
    """Ranks of more than 512 stage pairs take the one-thread-per-rank kernel;
    a rank of fewer takes the wave kernel in the same problem family."""
    need_gpu()
    for M in (520, 200):
        inst = W.pipeline_instance(2, M, np.arange(2 * M).reshape(2, M) % 9 + 2, comm=3, act=2)
        prob = W.compile_instance(inst)
        g, G, cls = W.priority_groups(prob)
        rows, res = O.greedy(prob, g, G, W.rollout_priorities(cls, 3, seed=4), stride=prob.stride)
        tab = strategy_table(prob)
        prob.mem_cap[:] = (np.median(res.peak, axis=0) * frac).astype(prob.mem_cap.dtype)
        print(f"pipeline M {M}: caps {prob.mem_cap.tolist()}", flush=True)
        got_t, got_p, got_s = run(prob, tab, rows, 6)
        want = MO.optimise(prob, tab, MO.pair_candidates(tab, 6), rows)
        np.testing.assert_array_equal(got_s, [[1 if x[1] else 0 for x in per] for per in want])
        np.testing.assert_array_equal(got_t, [[x[0] for x in per] for per in want])
        np.testing.assert_array_equal(got_p, [[x[2] for x in per] for per in want])
