"""GPU parity of the operator-level cost tables (dip_cost_tables) against the
CPU oracle, bit-exact, and a table fed to the simulator as its costs."""
import numpy as np
import pytest

import oracle as O
import oracle.costmodel as OC
import workloads as W
from workloads.operators import (K_ELEM, K_GEMM, N_KINDS, OperatorTable, coefficient_sweep,
                                 operator_table)

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2504_14145_amd as dip

DEV = "cuda:0"


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def run(table, coef):
    dt = dip.DeviceOpTable(table, N_KINDS, DEV)
    c = torch.from_numpy(np.ascontiguousarray(coef)).to(DEV)
    out = torch.empty((coef.shape[0], dt.n_items), dtype=torch.int32, device=DEV)
    dip.cost_tables(dt, c, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("cid,n", [(2, 37), (3, 3), (4, 2)])
def test_tables_match_oracle(cid, n):
    need_gpu()
    prob = W.make_problem(cid)
    tab = operator_table(prob)
    coef = coefficient_sweep(n, seed=cid)
    print(f"config {cid}: {len(tab.item_ptr) - 1} items, {len(tab.kind)} rows, {n} configurations",
          flush=True)
    np.testing.assert_array_equal(run(tab, coef), OC.cost_tables(tab, coef))


def test_edge_cases_and_many_configurations():
    need_gpu()
    rows = [(K_GEMM, 3.5e9, 3e6, 0.0), (K_ELEM, 1e9, 12.75e6, 0.0),   # item 0
            (9, 1.0, 1.0, 1.0),                                          # item 1: bad kind
            (K_ELEM, 0.0, 3e12 * 30000.0, 0.0)]                          # item 3: overflow
    ptr = np.array([0, 2, 3, 3, 4], np.int32)                            # item 2 empty
    a = np.array(rows, np.float64)
    tab = OperatorTable(ptr, a[:, 1].copy(), a[:, 2].copy(), a[:, 3].copy(),
                        a[:, 0].astype(np.uint8), 4, 0)
    coef = coefficient_sweep(70001, seed=3)          # many blocks of configurations
    got = run(tab, coef)
    assert (got[:, 1] == -1).all() and (got[:, 2] == 0).all() and (got[:, 3] == -1).all()
    # items 0 and 3 against the oracle (it has no notion of a bad kind)
    keep = OperatorTable(np.array([0, 2, 3], np.int32), tab.n_fop[[0, 1, 3]],
                         tab.n_mem[[0, 1, 3]], tab.n_net[[0, 1, 3]], tab.kind[[0, 1, 3]], 2, 0)
    np.testing.assert_array_equal(got[:, [0, 3]], OC.cost_tables(keep, coef))


def test_table_feeds_the_simulator():
    """Config 2's stage and edge costs from one configuration, handed to
    dip_sim_evaluate as its costs: the GPU simulation equals the simulator
    oracle's with the same costs."""
    need_gpu()
    prob = W.make_problem(2)
    tab = operator_table(prob)
    cost = run(tab, coefficient_sweep(1, seed=9))[0]
    assert (cost >= 0).all()
    prob.op_cost = cost[:prob.n_total].astype(np.int32)
    prob.edge_comm = cost[prob.n_total:].astype(np.int32)
    rows = W.generator_for(prob, 2).generate(0, 300)
    want = O.evaluate(prob, rows, threads=16)
    sim = dip.Sim(prob)
    ms, bub, pk, fl = sim.evaluate(torch.from_numpy(rows).to(DEV))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(ms.cpu().numpy(), want.makespan)
    np.testing.assert_array_equal(bub.cpu().numpy(), want.bubble)
    np.testing.assert_array_equal(fl.cpu().numpy(), want.flags)
    sim.close()
