"""Values at the limits the library accepts: op costs and latencies whose sum
is exactly INT32_MAX (makespans above 2**30, past the simulation kernel's
record fields, so evaluate runs the pool kernel), costs and latencies at the
largest values the records hold and one past them, and per-rank activations
that sum to exactly INT32_MAX under caps one below and at that peak.  Every
output must equal the oracle's on valid, deadlocked and invalid orders."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from test_gpu_random_instances import permuted, topo_orders

torch = pytest.importorskip("torch")
if torch.cuda.is_available():
    import paper_2504_14145_amd as dip

DEV = "cuda:0"
I32 = 2**31 - 1
REC_COST_MAX = 2**20 - 1     # the simulation kernel's cost field
REC_COMM_MAX = 2047          # and its latency field


def instance(seed, P=4, v=2, M=6):
    rng = np.random.default_rng(seed)
    fcost = rng.integers(1, 400, size=(P * v, M))
    return W.compile_instance(W.pipeline_instance(P, M, fcost, comm=3, v=v)), rng


def forward_first(prob):
    """Each rank's ops in the order of one topological order of the whole
    graph that takes a ready forward op before any backward one: every rank
    holds all of its activations at once, so its peak is the sum of them."""
    N, P = prob.n_total, prob.n_ranks
    rank = np.repeat(np.arange(P), prob.n_ops)
    succ = [[] for _ in range(N)]
    for g in range(N):
        for e in range(prob.pred_ptr[g], prob.pred_ptr[g + 1]):
            succ[prob.pred_op[e]].append(g)
    left = np.diff(prob.pred_ptr).astype(np.int64)
    ready = {g for g in range(N) if left[g] == 0}
    row = np.zeros(prob.stride, np.int16)
    fill = prob.rank_off[:-1].astype(np.int64).copy()
    while ready:
        g = min(ready, key=lambda x: (int(prob.op_kind[x]), x))
        ready.remove(g)
        r = rank[g]
        row[fill[r]] = g - prob.rank_off[r]
        fill[r] += 1
        for s in succ[g]:
            left[s] -= 1
            if left[s] == 0:
                ready.add(s)
    assert (fill == prob.rank_off[1:]).all()
    return row


def batch(prob, rng):
    rows = np.concatenate([forward_first(prob)[None], topo_orders(prob, rng, 40),
                           permuted(prob, 40, rng)])
    rows[-1, prob.rank_off[1]] = rows[-1, prob.rank_off[1] + 1]     # a repeated id
    return rows


def compare(prob, rows, want_variant):
    want = O.evaluate(prob, rows)
    sim = dip.Sim(prob)
    try:
        ms, bub, pk, fl = sim.evaluate(torch.from_numpy(rows).to(DEV))
        torch.cuda.synchronize()
        info = sim.info
        print(f"  variant {info['variant']}, max makespan {want.makespan.max()}, "
              f"max peak {want.peak.max()}, flags {np.bincount(want.flags, minlength=8)[:8]}",
              flush=True)
        assert info["variant"] == want_variant
        np.testing.assert_array_equal(fl.cpu().numpy(), want.flags)
        np.testing.assert_array_equal(ms.cpu().numpy(), want.makespan)
        np.testing.assert_array_equal(bub.cpu().numpy(), want.bubble)
        np.testing.assert_array_equal(pk.cpu().numpy(), want.peak)
    finally:
        sim.close()
    return want


@pytest.mark.gpu
@pytest.mark.parametrize("seed", [0, 1])
def test_costs_summing_to_int32_max(seed):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    prob, rng = instance(50 + seed)
    prob.edge_comm[:] = rng.integers(0, 10**6, prob.n_edges)
    w = rng.integers(1, 1000, prob.n_total).astype(np.int64)
    budget = I32 - int(prob.edge_comm.astype(np.int64).sum())
    cost = w * budget // int(w.sum())
    cost[int(rng.integers(prob.n_total))] += budget - int(cost.sum())
    prob.op_cost[:] = cost
    assert int(prob.op_cost.astype(np.int64).sum() + prob.edge_comm.astype(np.int64).sum()) == I32
    print(f"seed {seed}: costs up to {prob.op_cost.max()}", flush=True)
    want = compare(prob, batch(prob, rng), 8)
    assert want.makespan.max() > 2**30


@pytest.mark.gpu
@pytest.mark.parametrize("over", [None, "cost", "comm"])
def test_record_field_limits(over):
    """Costs and latencies at the records' largest values keep the
    simulation kernel; one value past either field sends the call to the
    pool kernel, with the same outputs."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    prob, rng = instance(60, P=8, v=1, M=8)
    prob.op_cost[:] = REC_COST_MAX - rng.integers(0, 3, prob.n_total)
    prob.edge_comm[:] = REC_COMM_MAX - rng.integers(0, 3, prob.n_edges)
    if over == "cost":
        prob.op_cost[int(rng.integers(prob.n_total))] = REC_COST_MAX + 1
    elif over == "comm":
        prob.edge_comm[int(rng.integers(prob.n_edges))] = REC_COMM_MAX + 1
    print(f"over {over}", flush=True)
    compare(prob, batch(prob, rng), 9 if over is None else 8)


@pytest.mark.gpu
def test_activations_summing_to_int32_max():
    """Each rank's activations sum to INT32_MAX; the forward-first order
    peaks there on every rank, so a cap one below flags it and a cap equal
    to it does not."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    prob, rng = instance(70)
    for r in range(prob.n_ranks):
        sl = np.unique(prob.op_slot[prob.rank_off[r]:prob.rank_off[r + 1]])
        w = rng.integers(1, 1000, len(sl)).astype(np.int64)
        a = w * I32 // int(w.sum())
        a[0] += I32 - int(a.sum())
        prob.slot_act[sl] = a
    prob.mem_cap[:] = -1
    prob.mem_cap[1] = I32
    prob.mem_cap[2] = I32 - 1
    rows = batch(prob, rng)
    want = compare(prob, rows, 9)
    assert (want.peak[0] == I32).all()
    assert want.flags[0] == 2


def test_limits_helpers_on_cpu():
    """The forward-first order is a schedule without deadlock whose peak is
    every rank's whole activation sum (oracle only)."""
    prob, _ = instance(80)
    row = forward_first(prob)[None]
    res = O.evaluate(prob, row)
    assert res.flags[0] == 0
    for r in range(prob.n_ranks):
        sl = np.unique(prob.op_slot[prob.rank_off[r]:prob.rank_off[r + 1]])
        assert res.peak[0, r] == int(prob.slot_act[sl].sum())

