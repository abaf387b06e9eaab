"""Seeded random pipeline instances -- 1 to 64 ranks (powers of two and not),
one to three model chunks per rank, uneven forward costs, latencies between
ranks, caps that bind -- with three kinds of candidate orders: each rank's
ops in a random topological order of the whole graph (never deadlocks), the
same after random adjacent swaps (some deadlock, some break an own-rank
order), and random permutations of each rank's ops (mostly deadlocks, many
with full pools).  Every variant the library picks, at pool sizes 4, 8 and
16, must give the oracle's outputs on every candidate."""
import numpy as np
import pytest

import oracle as O
import workloads as W

torch = pytest.importorskip("torch")
if torch.cuda.is_available():
    import paper_2504_14145_amd as dip

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def random_instance(rng):
    P = int(rng.choice([1, 2, 3, 4, 6, 8, 16, 32, 64]))
    v = int(rng.integers(1, 4))
    M = int(rng.integers(1, 13))
    L = P * v
    fcost = rng.integers(1, 400, size=(L, M))
    comm = int(rng.integers(0, 60))
    return W.compile_instance(W.pipeline_instance(P, M, fcost, comm=comm, v=v))


def topo_orders(prob, rng, n):
    """n rows, each rank's ops in the order of one random topological order
    of the whole dependence graph."""
    N, P = prob.n_total, prob.n_ranks
    rank = np.repeat(np.arange(P), prob.n_ops)
    succ = [[] for _ in range(N)]
    for g in range(N):
        for e in range(prob.pred_ptr[g], prob.pred_ptr[g + 1]):
            succ[prob.pred_op[e]].append(g)
    rows = np.zeros((n, prob.stride), np.int16)
    for c in range(n):
        left = np.diff(prob.pred_ptr).astype(np.int64)
        ready = [g for g in range(N) if left[g] == 0]
        fill = prob.rank_off[:-1].astype(np.int64).copy()
        while ready:
            g = ready.pop(int(rng.integers(len(ready))))
            r = rank[g]
            rows[c, fill[r]] = g - prob.rank_off[r]
            fill[r] += 1
            for s in succ[g]:
                left[s] -= 1
                if left[s] == 0:
                    ready.append(s)
        assert (fill == prob.rank_off[1:]).all()
    return rows


def swapped(prob, rows, rng):
    out = rows.copy()
    for c in range(len(out)):
        for _ in range(int(rng.integers(1, 6))):
            r = int(rng.integers(prob.n_ranks))
            lo, hi = int(prob.rank_off[r]), int(prob.rank_off[r + 1])
            if hi - lo >= 2:
                p = int(rng.integers(lo, hi - 1))
                out[c, p], out[c, p + 1] = out[c, p + 1], out[c, p]
    return out


def permuted(prob, n, rng):
    rows = np.zeros((n, prob.stride), np.int16)
    for c in range(n):
        for r in range(prob.n_ranks):
            lo, hi = int(prob.rank_off[r]), int(prob.rank_off[r + 1])
            rows[c, lo:hi] = rng.permutation(hi - lo)
    return rows


@pytest.mark.parametrize("seed", range(40))
def test_random_instances_match_oracle(seed):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rng = np.random.default_rng(1000 + seed)
    prob = random_instance(rng)
    base = topo_orders(prob, rng, 48)
    rows = np.concatenate([base, swapped(prob, base, rng), permuted(prob, 96, rng)])
    # a cap between the smallest and the largest peak of the valid orders
    peak = O.evaluate(prob, base).peak
    prob.mem_cap[:] = int(rng.integers(peak.min(), peak.max() + 1))
    want = O.evaluate(prob, rows)
    print(f"seed {seed}: P {prob.n_ranks}, {prob.n_total} ops, {len(rows)} candidates, "
          f"deadlock {np.mean(want.flags & 1):.2f}, cap {np.mean((want.flags & 2) > 0):.2f}",
          flush=True)
    sim = dip.Sim(prob)
    orders = torch.from_numpy(rows).to(DEV)
    for slots in (4, 8, 16):
        assert sim.configure_pool(slots) == dip.OK
        ms, bub, pk, fl = sim.evaluate(orders)
        torch.cuda.synchronize()
        got = [t.cpu().numpy() for t in (ms, bub, pk, fl)]
        np.testing.assert_array_equal(got[3], want.flags)
        np.testing.assert_array_equal(got[0], want.makespan)
        np.testing.assert_array_equal(got[1], want.bubble)
        np.testing.assert_array_equal(got[2], want.peak)
    sim.close()


@pytest.mark.parametrize("seed", range(20))
def test_random_instances_greedy_matches_oracle(seed):
    """The dual-queue interleaving on the same random instances (caps that
    bind the forward queue), random rollout priorities: the emitted orders
    and their scores equal the oracle's."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rng = np.random.default_rng(1000 + seed)
    prob = random_instance(rng)
    base = topo_orders(prob, rng, 16)
    peak = O.evaluate(prob, base).peak
    prob.mem_cap[:] = int(rng.integers(peak.min(), peak.max() + 1))
    g, G, cls = W.priority_groups(prob)
    prio = W.rollout_priorities(cls, 96, seed=seed)
    want_o, want = O.greedy(prob, g, G, prio, stride=prob.stride, threads=16)
    print(f"seed {seed}: P {prob.n_ranks}, {prob.n_total} ops, {G} groups", flush=True)
    sim = dip.Sim(prob)
    assert sim.configure_greedy(G, g) == dip.OK
    ords, (ms, bub, pk, fl) = sim.greedy(torch.from_numpy(np.ascontiguousarray(prio, np.int32)).to(DEV))
    torch.cuda.synchronize()
    N = prob.n_total
    np.testing.assert_array_equal(ords.cpu().numpy()[:, :N], want_o[:, :N])
    np.testing.assert_array_equal(fl.cpu().numpy(), want.flags)
    np.testing.assert_array_equal(ms.cpu().numpy(), want.makespan)
    np.testing.assert_array_equal(bub.cpu().numpy(), want.bubble)
    np.testing.assert_array_equal(pk.cpu().numpy(), want.peak)
    sim.close()
