"""Input generators: shapes, determinism, permutation property, int32 bounds."""
import numpy as np
import pytest

import workloads as W
from workloads.instance import comm_from_tokens, op_cost_from_tokens

from kahn import data_edges, ops_of_rank


def test_cost_and_comm_formulas():
    # a*tok + c*tok^2/1e4 with (a, c) = (0.5, 0.5) at 8192 tokens: 4096 + 3355.4
    assert op_cost_from_tokens(8192, 50, 50) == 7451
    assert op_cost_from_tokens(0, 100, 25) == 0
    assert op_cost_from_tokens(65536, 10, 5) == 28028   # floor(6553.6 + 21474.8)
    # 8192 B per token at 400 GB/s: 0.02048 us per token, rounded up
    assert comm_from_tokens(8192) == 168
    assert comm_from_tokens(1) == 1 and comm_from_tokens(0) == 0


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_instance_shapes(cid):
    cfg = W.get(cid)
    prob = W.make_problem(cid)
    assert prob.n_ranks == cfg.P
    assert int(prob.n_ops.max()) < (1 << 15)
    assert prob.stride % 8 == 0 and prob.stride >= prob.n_total
    assert prob.n_total == 2 * prob.n_slots
    # every microbatch crosses every segment
    inst = prob.inst
    for s in range(inst.n_seg):
        assert set(inst.unit_mb[inst.unit_seg == s]) == set(range(cfg.samples))
    # the simulator's int32 bound: sum of all costs and latencies
    assert int(prob.op_cost.astype(np.int64).sum() + prob.edge_comm.astype(np.int64).sum()) < 2**31 - 1
    for r in range(prob.n_ranks):
        sl = prob.op_slot[prob.rank_off[r]:prob.rank_off[r + 1]]
        assert int(prob.slot_act[np.unique(sl)].astype(np.int64).sum()) < 2**31 - 1
    if cid == 1:
        assert prob.n_total == 64
        # 10 us on every cross-rank edge, 0 on the same-rank loss turnaround
        src_rank = np.searchsorted(prob.rank_off, prob.pred_op, side="right") - 1
        dst = np.repeat(np.arange(prob.n_total), np.diff(prob.pred_ptr))
        dst_rank = np.searchsorted(prob.rank_off, dst, side="right") - 1
        np.testing.assert_array_equal(prob.edge_comm, np.where(src_rank != dst_rank, 10, 0))


def test_compiled_edges_match_high_level_description():
    """The CSR built by the instance compiler holds exactly the edges the
    independent checker derives from lanes, segments and units."""
    inst = W.make_instance(2)
    prob = W.compile_instance(inst)
    ids = {}
    for r in range(inst.P):
        for i, op in enumerate(ops_of_rank(inst, r)):
            ids[op] = int(prob.rank_off[r]) + i
    want = sorted((ids[a], ids[b], w) for (a, b, w) in data_edges(inst))
    got = sorted((int(prob.pred_op[e]), g, int(prob.edge_comm[e]))
                 for g in range(prob.n_total)
                 for e in range(prob.pred_ptr[g], prob.pred_ptr[g + 1]))
    assert got == want


@pytest.mark.parametrize("cid,n", [(1, 1024), (2, 512), (3, 64), (4, 64), (5, 16)])
def test_candidates_are_permutations(cid, n):
    prob = W.make_problem(cid)
    rows = W.generator_for(prob, cid).generate(0, n)
    for r in range(prob.n_ranks):
        sec = np.sort(rows[:, prob.rank_off[r]:prob.rank_off[r + 1]], axis=1)
        assert (sec == np.arange(prob.n_ops[r])[None, :]).all()
    assert (rows[:, prob.n_total:] == 0).all()


@pytest.mark.parametrize("cid", [1, 2, 4])
def test_candidates_deterministic_and_chunk_independent(cid):
    prob = W.make_problem(cid)
    g = W.generator_for(prob, cid)
    full = g.generate(0, 300, threads=1)
    part = g.generate(120, 100, threads=4)
    np.testing.assert_array_equal(full[120:220], part)
    g2 = W.generator_for(W.make_problem(cid), cid)
    np.testing.assert_array_equal(g2.generate(0, 300, threads=3), full)


def test_instances_deterministic():
    a = W.make_problem(3)
    b = W.make_problem(3)
    for k in ("op_cost", "edge_comm", "slot_act", "pred_op", "pred_ptr"):
        np.testing.assert_array_equal(getattr(a, k), getattr(b, k))
    c = W.make_problem(3, seed=1)
    assert not np.array_equal(a.op_cost, c.op_cost)


def test_rng_stream_is_counter_based():
    x = [W.orders.draw(0, 2, 2, 7, k) for k in range(4)]
    assert len(set(x)) == 4
    assert W.orders.draw(0, 2, 2, 7, 2) == x[2]
    assert W.orders.draw(0, 2, 2, 8, 0) != x[0]
