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


def run(prob, tab, rows, S, choices=False):
    sim = dip.Sim(prob)
    assert dip.configure_memopt(sim.h, tab.slot_layers, tab.time, tab.mem, S) == dip.OK
    n = rows.shape[0]
    t = torch.empty((n, prob.n_ranks), dtype=torch.int64, device=DEV)
    pk = torch.empty((n, prob.n_ranks), dtype=torch.int32, device=DEV)
    st = torch.empty((n, prob.n_ranks), dtype=torch.uint8, device=DEV)
    ch = torch.empty((n, prob.n_slots), dtype=torch.uint8, device=DEV)
    dip.memopt(sim.h, torch.from_numpy(np.ascontiguousarray(rows)).to(DEV), n, t, pk, st, ch)
    torch.cuda.synchronize()
    sim.close()
    out = t.cpu().numpy(), pk.cpu().numpy(), st.cpu().numpy()
    return out + (ch.cpu().numpy(),) if choices else out


def compare(want, got_t, got_p, got_s, got_c=None, tab=None):
    np.testing.assert_array_equal(got_s, [[x[1] for x in per] for per in want])
    np.testing.assert_array_equal(got_t, [[x[0] for x in per] for per in want])
    np.testing.assert_array_equal(got_p, [[x[2] for x in per] for per in want])
    if got_c is not None:
        for c, per in enumerate(want):
            np.testing.assert_array_equal(got_c[c], MO.choice_row(tab, per))


@pytest.mark.parametrize("cid,n,frac,S", [(2, 131, 0.6, 6), (2, 67, 0.15, 4), (3, 9, 0.5, 6),
                                          (3, 5, 0.1, 8), (2, 40, -1, 6), (2, 64, 0.3, 6)])
def test_memopt_matches_oracle(cid, n, frac, S):
    """Statuses, totals, peaks and every pair's choice (warm start,
    improvement pass and branch and bound) bit-exact."""
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
    got = run(prob, tab, rows, S, choices=True)
    cands = MO.pair_candidates(tab, S)
    want = MO.optimise(prob, tab, cands, rows)
    compare(want, *got, tab=tab)
    ws = got[2]
    if frac == 0.1:
        assert (ws == 0).any()            # a cap tight enough to be out of reach somewhere
    if 0.3 <= frac < 1:
        assert (ws == 1).any()            # searches that ended proven
    print(f"statuses: {np.bincount(ws.ravel(), minlength=4).tolist()}", flush=True)


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
    """Ranks of more than 512 stage pairs take the one-thread-per-rank kernel
    (no search: status 3 under a cap it meets); a rank of fewer takes the
    wave kernel in the same problem family."""
    need_gpu()
    for M in (520, 200):
        inst = W.pipeline_instance(2, M, np.arange(2 * M).reshape(2, M) % 9 + 2, comm=3, act=2)
        prob = W.compile_instance(inst)
        g, G, cls = W.priority_groups(prob)
        rows, res = O.greedy(prob, g, G, W.rollout_priorities(cls, 3, seed=4), stride=prob.stride)
        tab = strategy_table(prob)
        prob.mem_cap[:] = (np.median(res.peak, axis=0) * frac).astype(prob.mem_cap.dtype)
        print(f"pipeline M {M}: caps {prob.mem_cap.tolist()}", flush=True)
        got = run(prob, tab, rows, 6, choices=True)
        want = MO.optimise(prob, tab, MO.pair_candidates(tab, 6), rows)
        compare(want, *got, tab=tab)


@pytest.mark.parametrize("cid,n,frac", [(2, 70, 0.4), (3, 6, 0.5)])
def test_evaluate_selected_matches_oracle(cid, n, frac):
    """Schedules re-timed with the GPU's selection: makespan, bubbles, peaks
    (chosen memories) and flags against the simulator oracle run on the
    re-timed problem."""
    need_gpu()
    prob = W.make_problem(cid)
    tab = strategy_table(prob)
    rows = W.generator_for(prob, cid).generate(0, n)
    prob.mem_cap[:] = int(np.median(O.evaluate(prob, rows).peak) * frac)
    S = 6
    cands = MO.pair_candidates(tab, S)
    want = MO.optimise(prob, tab, cands, rows)
    sim = dip.Sim(prob)
    assert dip.configure_memopt(sim.h, tab.slot_layers, tab.time, tab.mem, S) == dip.OK
    orders = torch.from_numpy(np.ascontiguousarray(rows)).to(DEV)
    sim.evaluate(orders)                                  # sends the costs
    t = torch.empty((n, prob.n_ranks), dtype=torch.int64, device=DEV)
    pk = torch.empty((n, prob.n_ranks), dtype=torch.int32, device=DEV)
    st = torch.empty((n, prob.n_ranks), dtype=torch.uint8, device=DEV)
    ch = torch.empty((n, prob.n_slots), dtype=torch.uint8, device=DEV)
    dip.memopt(sim.h, orders, n, t, pk, st, ch)
    ms, bub, peak, fl = sim.outputs(n, DEV)
    dip.evaluate_selected(sim.h, orders, ch, n, ms, bub, peak, fl)
    torch.cuda.synchronize()
    ms, bub, peak, fl = (x.cpu().numpy() for x in (ms, bub, peak, fl))
    sim.close()
    for c in range(n):
        sp = MO.selected_problem(prob, tab, cands, want[c])
        w = O.evaluate(sp, rows[c:c + 1])
        assert fl[c] == w.flags[0] and ms[c] == w.makespan[0], c
        np.testing.assert_array_equal(bub[c], w.bubble[0])
        np.testing.assert_array_equal(peak[c], w.peak[0])
        # the chosen memory at every forward start stays where the selection put it
        ok = [x[1] in (1, 3) for x in want[c]]
        if all(ok):
            assert (peak[c] == [x[2] for x in want[c]]).all()
