"""Pins for the CPU oracle: closed forms, brute force, an independent
longest-path checker, hand-built deadlocks, invariants and the paper's own
worked example.  CPU only."""
import itertools
import os

import numpy as np
import pytest

import oracle as O
import workloads as W
from workloads import KIND_B, KIND_F, gpipe_rank, one_f_one_b_rank, op_id, pack

from kahn import data_edges, longest_path, ops_of_rank

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def pipe(S, M, f, b=None, comm=0, act=1, mem_cap=-1, v=1):
    return W.compile_instance(W.pipeline_instance(S, M, f, b, comm=comm, act=act,
                                                  mem_cap=mem_cap, v=v))


# ---------------------------------------------------------------- closed forms

@pytest.mark.parametrize("S,M,f,b,c", [
    (1, 1, 3, 6, 0), (2, 1, 1, 2, 10), (2, 2, 1, 2, 10), (3, 5, 2, 3, 4),
    (4, 8, 50, 100, 10), (5, 3, 7, 7, 0), (8, 16, 11, 29, 13), (6, 1, 4, 9, 2)])
def test_gpipe_makespan_closed_form(S, M, f, b, c):
    """Uniform GPipe: T = (M+S-1)(f+b) + 2(S-1)c (forward wave of M+S-1
    steps, backward wave likewise, one hop of latency per stage boundary in
    each direction)."""
    prob = pipe(S, M, f, b, comm=c)
    r = O.evaluate(prob, pack(prob, [gpipe_rank(M)] * S))
    assert r.flags[0] == 0
    assert r.makespan[0] == (M + S - 1) * (f + b) + 2 * (S - 1) * c


@pytest.mark.parametrize("S,M,f,b", [(1, 4, 5, 9), (2, 2, 1, 2), (4, 8, 50, 100),
                                     (4, 3, 5, 5), (8, 32, 3, 7), (16, 64, 2, 4)])
def test_1f1b_makespan_closed_form_zero_comm(S, M, f, b):
    """Uniform 1F1B with zero latency also reaches (M+S-1)(f+b)."""
    prob = pipe(S, M, f, b)
    r = O.evaluate(prob, pack(prob, [one_f_one_b_rank(S, s, M) for s in range(S)]))
    assert r.flags[0] == 0
    assert r.makespan[0] == (M + S - 1) * (f + b)


@pytest.mark.parametrize("S,M", [(2, 2), (4, 8), (4, 3), (8, 5), (16, 64)])
def test_activation_peak_closed_form(S, M):
    """act = 1 per (stage, microbatch): 1F1B holds min(S-s, M) activations on
    stage s at its peak, GPipe holds all M."""
    prob = pipe(S, M, 3, 6)
    rows = np.stack([pack(prob, [one_f_one_b_rank(S, s, M) for s in range(S)]),
                     pack(prob, [gpipe_rank(M)] * S)])
    r = O.evaluate(prob, rows)
    assert list(r.peak[0]) == [min(S - s, M) for s in range(S)]
    assert list(r.peak[1]) == [M] * S


def test_bubble_identity_and_definition():
    """bubble_r = T - busy_r, so sum_r bubble_r = P*T - sum(costs)."""
    prob = W.make_problem(2)
    g = W.generator_for(prob, 2)
    r = O.evaluate(prob, g.generate(0, 64))
    busy = np.array([prob.op_cost[prob.rank_off[k]:prob.rank_off[k + 1]].sum()
                     for k in range(prob.n_ranks)])
    ok = r.flags & O.FLAG_DEADLOCK == 0
    assert ok.any()
    np.testing.assert_array_equal(r.bubble[ok], r.makespan[ok, None] - busy[None, :])
    assert (r.bubble[ok] >= 0).all()


# ---------------------------------------------------------------- brute force

def _all_combos(S, M):
    perms = list(itertools.permutations(range(2 * M)))
    return [list(c) for c in itertools.product(perms, repeat=S)]


@pytest.mark.parametrize("S,M", [(2, 2), (3, 2)])
def test_brute_force_against_kahn(S, M):
    """Every combination of per-rank orders: the oracle's deadlock set is the
    set of cyclic schedule graphs, and its makespan is the longest path."""
    rng = np.random.default_rng(7)
    f = rng.integers(1, 9, size=(S, M))
    inst = W.pipeline_instance(S, M, f, 2 * f, comm=3)
    prob = W.compile_instance(inst)
    combos = _all_combos(S, M)
    rows = np.stack([pack(prob, c) for c in combos])
    r = O.evaluate(prob, rows, threads=4)
    for i, c in enumerate(combos):
        k = longest_path(inst, c)
        assert bool(r.flags[i] & O.FLAG_DEADLOCK) == k["deadlock"], c
        if not k["deadlock"]:
            assert r.makespan[i] == k["makespan"], c


@pytest.mark.parametrize("S,M", [(2, 2), (3, 2)])
def test_brute_force_minimum_is_closed_form(S, M):
    """Uniform f, b and zero latency: no order beats (M+S-1)(f+b), because
    stage s idles at least s*f before its first op and s*b after its last."""
    f, b = 2, 5
    prob = pipe(S, M, f, b)
    rows = np.stack([pack(prob, c) for c in _all_combos(S, M)])
    r = O.evaluate(prob, rows, threads=4)
    ok = r.flags == 0
    assert r.makespan[ok].min() == (M + S - 1) * (f + b)
    # and the count of deadlock-free combinations matches Kahn's acyclic count
    inst = W.pipeline_instance(S, M, f, b)
    n_acyclic = sum(not longest_path(inst, c)["deadlock"] for c in _all_combos(S, M))
    assert ok.sum() == n_acyclic


# ---------------------------------------------------------------- deadlocks

def test_deadlock_backward_before_own_forward():
    S, M = 1, 2
    prob = pipe(S, M, 1, 2)
    r = O.evaluate(prob, pack(prob, [[op_id(0, KIND_B), op_id(0, KIND_F),
                                      op_id(1, KIND_F), op_id(1, KIND_B)]]))
    assert r.flags[0] == O.FLAG_DEADLOCK and r.makespan[0] == -1
    assert (r.bubble[0] == -1).all()


def test_deadlock_cross_rank_cycle():
    """rank 0 [F0 B0 F1 B1], rank 1 [F1 B1 F0 B0]: rank 0 needs B0 from rank 1,
    which sits behind F1 on rank 1, which needs F1 from rank 0, which sits
    behind B0 on rank 0."""
    prob = pipe(2, 2, 1, 2)
    r0 = [op_id(0, 0), op_id(0, 1), op_id(1, 0), op_id(1, 1)]
    r1 = [op_id(1, 0), op_id(1, 1), op_id(0, 0), op_id(0, 1)]
    r = O.evaluate(prob, pack(prob, [r0, r1]))
    assert r.flags[0] == O.FLAG_DEADLOCK
    # peaks still come from the order scan
    assert list(r.peak[0]) == [1, 1]


def test_deadlock_three_rank_ring():
    """A cycle through all three ranks: rank 0 waits for B0 (from rank 1)
    before it sends F1; rank 1 waits for F1 before it runs F0; rank 2 needs F0
    from rank 1 before its turnaround produces B0 for rank 1."""
    S, M = 3, 3
    F = lambda m: op_id(m, KIND_F)
    B = lambda m: op_id(m, KIND_B)
    o0 = [F(0), B(0), F(1), B(1), F(2), B(2)]
    o1 = [F(1), F(0), B(0), B(1), F(2), B(2)]
    o2 = [F(0), B(0), F(1), B(1), F(2), B(2)]
    inst = W.pipeline_instance(S, M, 1, 1)
    assert longest_path(inst, [o0, o1, o2])["deadlock"]
    prob = W.compile_instance(inst)
    r = O.evaluate(prob, pack(prob, [o0, o1, o2]))
    assert r.flags[0] == O.FLAG_DEADLOCK


def test_invalid_sections():
    prob = pipe(2, 2, 1, 2)
    good = [[0, 2, 1, 3], [0, 1, 2, 3]]
    rows = [pack(prob, good)]
    bad_range = [list(good[0]), list(good[1])]
    bad_range[1][3] = 4                      # id out of range
    rows.append(pack(prob, bad_range))
    dup = [list(good[0]), list(good[1])]
    dup[0][3] = 0                            # duplicate id
    rows.append(pack(prob, dup))
    neg = [list(good[0]), list(good[1])]
    neg[0][0] = -1
    rows.append(pack(prob, neg))
    r = O.evaluate(prob, np.stack(rows))
    assert r.flags[0] == 0
    for i in (1, 2, 3):
        assert r.flags[i] == O.FLAG_INVALID
        assert r.makespan[i] == -1 and (r.bubble[i] == -1).all() and (r.peak[i] == -1).all()


def test_int32_overflow_is_an_error():
    prob = pipe(2, 2, 1 << 29, 1 << 29)
    with pytest.raises(RuntimeError):
        O.evaluate(prob, pack(prob, [gpipe_rank(2)] * 2))


# ---------------------------------------------------------------- memory cap

def test_cap_flips_exactly_at_peak():
    S, M = 4, 6
    base = pipe(S, M, 2, 4)
    rows = pack(base, [one_f_one_b_rank(S, s, M) for s in range(S)])
    peak0 = O.evaluate(base, rows).peak[0, 0]
    flags = []
    for cap in (peak0 - 1, peak0, peak0 + 1):
        prob = pipe(S, M, 2, 4, mem_cap=int(cap))
        flags.append(int(O.evaluate(prob, rows).flags[0]))
    assert flags == [O.FLAG_CAP, 0, 0]


# ---------------------------------------------------------------- random DAGs

def random_instance(rng, P, v, nseg, M, zero_costs=True):
    L = P * v
    cuts = sorted(rng.choice(np.arange(1, L), size=nseg - 1, replace=False)) if nseg > 1 else []
    bounds = [0] + [int(c) for c in cuts] + [L]
    seg_lo = bounds[:-1]
    seg_hi = [b - 1 for b in bounds[1:]]
    useg, umb, upc = [], [], []
    split_seg = rng.integers(0, nseg, size=M)
    for s in range(nseg):
        for j in range(M):
            k = int(rng.integers(1, 4)) if split_seg[j] == s else 1
            for p in range(k):
                useg.append(s); umb.append(j); upc.append(p)
    U = len(useg)
    lo = 0 if zero_costs else 1
    f = rng.integers(lo, 12, size=(L, U))
    b = rng.integers(lo, 20, size=(L, U))
    return W.Instance(P=P, v=v, seg_lo=seg_lo, seg_hi=seg_hi,
                      unit_seg=np.array(useg), unit_mb=np.array(umb),
                      unit_piece=np.array(upc), unit_tok=np.zeros(U, np.int64),
                      fcost=f, bcost=b, act=rng.integers(0, 7, size=(L, U)),
                      unit_comm=rng.integers(0, 6, size=U), mem_cap=-1)


@pytest.mark.parametrize("seed", range(12))
def test_random_multisegment_against_kahn(seed):
    """Joins, interleaved lanes, zero costs and latencies, valid and
    deadlocked orders: the oracle equals the Kahn longest path."""
    rng = np.random.default_rng(100 + seed)
    P = int(rng.integers(1, 4))
    v = int(rng.integers(1, 3))
    nseg = int(rng.integers(1, min(3, P * v) + 1))
    inst = random_instance(rng, P, v, nseg, M=int(rng.integers(1, 4)))
    prob = W.compile_instance(inst)
    gen = W.OrderGenerator(prob, W.MODE_LIST, max_swaps=3, seed=seed, cid=99)
    rows = gen.generate(0, 24)
    # plus a few uniformly random permutations (mostly deadlocked)
    extra = []
    for _ in range(8):
        extra.append(pack(prob, [list(rng.permutation(int(n))) for n in prob.n_ops]))
    rows = np.concatenate([rows, np.stack(extra)])
    r = O.evaluate(prob, rows)
    busy = None
    for i, row in enumerate(rows):
        orders = W.unpack(prob, row)
        k = longest_path(inst, orders)
        assert bool(r.flags[i] & O.FLAG_DEADLOCK) == k["deadlock"]
        if busy is None:
            busy = k["busy"]
        if not k["deadlock"]:
            assert r.makespan[i] == k["makespan"]
            assert list(r.bubble[i]) == [k["makespan"] - x for x in busy]


def test_list_orders_without_swaps_never_deadlock():
    rng = np.random.default_rng(5)
    for trial in range(6):
        inst = random_instance(rng, P=3, v=2, nseg=3, M=3)
        prob = W.compile_instance(inst)
        rows = W.OrderGenerator(prob, W.MODE_LIST, max_swaps=0, seed=trial, cid=98).generate(0, 16)
        assert (O.evaluate(prob, rows).flags & O.FLAG_DEADLOCK == 0).all()


def test_peak_second_definition_from_times():
    """With positive costs, the order-scan peak equals the largest live
    activation over [start F, end B) intervals, sampled at each F start."""
    rng = np.random.default_rng(11)
    inst = random_instance(rng, P=3, v=2, nseg=2, M=3, zero_costs=False)
    prob = W.compile_instance(inst)
    rows = W.OrderGenerator(prob, W.MODE_LIST, max_swaps=0, seed=3, cid=97).generate(0, 8)
    for row in rows:
        res, st, en = O.timeline(prob, row)
        assert res.flags[0] == 0
        for r in range(prob.n_ranks):
            a, b = int(prob.rank_off[r]), int(prob.rank_off[r + 1])
            slots = {}
            for g in range(a, b):
                slots.setdefault(int(prob.op_slot[g]), {})[int(prob.op_kind[g])] = g
            best = 0
            for g in range(a, b):
                if prob.op_kind[g] != KIND_F:
                    continue
                t = st[g]
                live = sum(int(prob.slot_act[s]) for s, fb in slots.items()
                           if st[fb[KIND_F]] <= t < en[fb[KIND_B]])
                best = max(best, live)
            assert res.peak[0, r] == best


# ---------------------------------------------------------------- invariants

@pytest.mark.parametrize("cid,n", [(1, 64), (2, 12), (3, 3)])
def test_invariants_on_workloads(cid, n):
    prob = W.make_problem(cid)
    inst = prob.inst
    rows = W.generator_for(prob, cid).generate(0, n)
    crit = longest_path(inst, None)["makespan"]   # data-DAG critical path
    busy = [int(prob.op_cost[prob.rank_off[k]:prob.rank_off[k + 1]].sum())
            for k in range(prob.n_ranks)]
    for row in rows:
        res, st, en = O.timeline(prob, row)
        if res.flags[0] & O.FLAG_DEADLOCK:
            continue
        T = int(res.makespan[0])
        assert T >= max(busy) and T >= crit
        assert T == en.max()
        for g in range(prob.n_total):
            for e in range(prob.pred_ptr[g], prob.pred_ptr[g + 1]):
                assert st[g] >= en[prob.pred_op[e]] + prob.edge_comm[e]
        for r, order in enumerate(W.unpack(prob, row)):
            gs = [int(prob.rank_off[r]) + o for o in order]
            for x, y in zip(gs, gs[1:]):
                assert st[y] >= en[x]          # one op at a time per rank


def test_scaling_and_monotonicity():
    prob = W.make_problem(2)
    rows = W.generator_for(prob, 2).generate(0, 32)
    r1 = O.evaluate(prob, rows)
    k = 3
    scaled = O.OracleInstance(prob.n_ranks, prob.rank_off, prob.pred_ptr, prob.pred_op,
                              prob.op_kind, prob.op_slot, prob.n_slots, prob.mem_cap,
                              prob.op_cost * k, prob.edge_comm * k, prob.slot_act)
    r3 = O.evaluate(scaled, rows)
    ok = r1.flags & O.FLAG_DEADLOCK == 0
    np.testing.assert_array_equal(r3.makespan[ok], k * r1.makespan[ok])
    cost = prob.op_cost.copy()
    cost[np.argmax(cost)] += 1000
    bumped = O.OracleInstance(prob.n_ranks, prob.rank_off, prob.pred_ptr, prob.pred_op,
                              prob.op_kind, prob.op_slot, prob.n_slots, prob.mem_cap,
                              cost, prob.edge_comm, prob.slot_act)
    rb = O.evaluate(bumped, rows)
    assert (rb.makespan[ok] >= r1.makespan[ok]).all()


# ---------------------------------------------------------------- argmin

def test_argmin_against_lexsort_with_planted_ties():
    rng = np.random.default_rng(3)
    for trial in range(20):
        n = int(rng.integers(1, 400))
        ms = rng.integers(0, 50, size=n).astype(np.int32)
        fl = (rng.random(n) < 0.3).astype(np.uint8) * rng.integers(1, 8, size=n).astype(np.uint8)
        base = int(rng.integers(0, 1 << 20))
        idx, best = O.argmin(ms, fl, base)
        ok = np.nonzero(fl == 0)[0]
        if ok.size == 0:
            assert (idx, best) == (-1, -1)
            continue
        order = np.lexsort((ok, ms[ok]))
        assert idx == base + ok[order[0]] and best == ms[ok[order[0]]]
    assert O.argmin(np.array([5, 5], np.int32), np.array([0, 0], np.uint8)) == (0, 5)
    assert O.argmin(np.zeros(0, np.int32), np.zeros(0, np.uint8)) == (-1, -1)


# ---------------------------------------------------------------- paper example

def _read_golden(name):
    vals = {}
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.strip()
            if line and not line.startswith("#"):
                k, v = line.split()
                vals[k] = float(v)
    return vals


def _contiguous_partitions(layer_lat, stages, lo, hi):
    n = len(layer_lat)
    prefix = np.concatenate([[0], np.cumsum(layer_lat)])
    out = []

    def rec(start, k, cuts):
        if k == stages:
            if start == n:
                out.append(list(cuts))
            return
        for end in range(start + 1, n + 1):
            lat = prefix[end] - prefix[start]
            if lat > hi:
                break
            if lat >= lo:
                cuts.append(end)
                rec(end, k + 1, cuts)
                cuts.pop()

    rec(0, 0, [])
    return out


def test_paper_37b_vlm_bubble():
    """Replay of the 16-stage, 64-microbatch 1F1B example with 63-73.5 ms
    stages: the idle fraction sum_r bubble_r / (P*T) of every admissible
    partition lies within 0.3 points of the printed figure, and the printed
    figure lies inside the replayed range."""
    g = _read_golden("e2_vlm37b_1f1b.txt")
    nv, nl = int(g["vit_layers"]), int(g["lm_layers"])
    vit_us = int(round(g["vit_ms_per_layer_fwd_bwd"] * 1000))
    lm_us = int(round(g["lm_ms_per_layer_fwd_bwd"] * 1000))
    S, M = int(g["stages"]), int(g["microbatches"])
    lat = np.array([vit_us] * nv + [lm_us] * nl)
    parts = _contiguous_partitions(lat, S, int(g["stage_latency_min_ms"] * 1000),
                                   int(g["stage_latency_max_ms"] * 1000))
    assert len(parts) > 0
    ratios = []
    for cuts in parts:
        bounds = [0] + cuts
        stage_fb = np.array([lat[bounds[i]:bounds[i + 1]].sum() for i in range(S)])
        f = stage_fb // 3                    # forward : backward = 1 : 2
        b = stage_fb - f
        prob = pipe(S, M, f, b)
        r = O.evaluate(prob, pack(prob, [one_f_one_b_rank(S, s, M) for s in range(S)]))
        assert r.flags[0] == 0
        ratios.append(r.bubble[0].sum() / (S * r.makespan[0]) * 100)
    printed = g["extra_bubble_percent"]
    assert min(ratios) - 0.05 <= printed <= max(ratios) + 0.05
    assert all(abs(x - printed) <= 0.3 for x in ratios)
