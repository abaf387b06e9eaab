"""GPU parity: the HIP path through the C ABI against the CPU oracle,
element by element and bit-exact (all quantities are integers)."""
import dataclasses

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


def run_gpu(sim, rows_np):
    orders = torch.from_numpy(np.ascontiguousarray(rows_np)).to(DEV)
    ms, bub, pk, fl = sim.evaluate(orders)
    torch.cuda.synchronize()
    return ms.cpu().numpy(), bub.cpu().numpy(), pk.cpu().numpy(), fl.cpu().numpy()


def assert_same(got, want, idx=None):
    ms, bub, pk, fl = got
    if idx is not None:
        ms, bub, pk, fl = ms[idx], bub[idx], pk[idx], fl[idx]
    np.testing.assert_array_equal(fl, want.flags)
    np.testing.assert_array_equal(ms, want.makespan)
    np.testing.assert_array_equal(bub, want.bubble)
    np.testing.assert_array_equal(pk, want.peak)


SMALL = {1: 1024, 2: 4099, 3: 515, 4: 259, 5: 67}


def own_rank_swap(prob, row, r, rng):
    """Swap, in rank r's section of row, an op that has a predecessor on its
    own rank with that predecessor's position, if the predecessor comes first
    (the op then comes first: the two wait for each other)."""
    b, e = int(prob.rank_off[r]), int(prob.rank_off[r + 1])
    sec = row[b:e]
    where = {int(x): q for q, x in enumerate(sec)}
    swaps = []
    for q, lid in enumerate(sec):
        if not 0 <= int(lid) < e - b:
            continue
        g = b + int(lid)
        for k in range(prob.pred_ptr[g], prob.pred_ptr[g + 1]):
            p = int(prob.pred_op[k])
            if b <= p < e and where.get(p - b, e) < q:
                swaps.append((q, where[p - b]))
    if swaps:
        q, pq = swaps[int(rng.integers(len(swaps)))]
        sec[q], sec[pq] = sec[pq], sec[q]


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_parity_small_all_variants(cid):
    """Every config at an oracle-friendly size with a ragged tail, under every
    kernel variant that fits the device."""
    need_gpu()
    prob = W.make_problem(cid)
    rows = W.generator_for(prob, cid).generate(0, SMALL[cid])
    want = O.evaluate(prob, rows, threads=16)
    sim = dip.Sim(prob)
    print(f"config {cid} auto variant: {sim.info}", flush=True)
    tried = 0
    for variant in (0, 1, 2, 3, 4, 8, 9):
        for wpb in (0, 1, 4):
            if sim.configure(variant, wpb) != dip.OK:
                continue
            tried += 1
            print(f"  variant {variant} wpb {wpb}: {sim.info['variant']}", flush=True)
            assert_same(run_gpu(sim, rows), want)
    assert tried >= 2
    sim.close()


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_parity_pool_kernel_slots(cid):
    """The pool kernel and the simulation kernel (each after the check kernel,
    with the list-mode fallback) at every pool size and block shape; the
    smallest pools send many candidates through the fallback, the results
    must not change."""
    need_gpu()
    prob = W.make_problem(cid)
    rows = W.generator_for(prob, cid).generate(0, SMALL[cid])
    want = O.evaluate(prob, rows, threads=16)
    sim = dip.Sim(prob)
    for slots in (4, 8, 16):
        assert sim.configure(0, 0) == dip.OK      # drop the last forced shape first
        assert sim.configure_pool(slots) == dip.OK
        for variant, wpb in ((8, 0), (8, 1), (8, 4), (9, 0), (9, 1), (9, 4), (9, 16)):
            rc = sim.configure(variant, wpb)
            if variant == 9 and wpb == 16 and rc == dip.E_UNSUPPORTED:
                continue
            assert rc == dip.OK
            run_gpu(sim, rows[:1])            # costs uploaded, the shape is known
            info = sim.info
            assert info["variant"] == variant and info["pool_slots"] == slots
            print(f"  slots {slots} variant {variant} wpb {wpb}: {info}", flush=True)
            assert_same(run_gpu(sim, rows), want)
    sim.close()


def test_pool_fallback_when_pools_fill():
    """Two ranks, five microbatches: rank 0 runs F0..F4 then B0..B4 and the
    last rank runs F4 B4 F3 B3 ... F0 B0, so rank 0 must hold five end times
    before rank 1 reads any.  With four slots per pool the pool kernel stalls
    on it without a deadlock; the candidate goes to the general kernel and the
    outputs (pre-filled with a sentinel) must still be the oracle's."""
    need_gpu()
    M = 5
    prob = W.compile_instance(W.pipeline_instance(2, M, [[5, 7, 11, 13, 2], [13, 17, 19, 3, 4]],
                                                  comm=3))
    row = np.zeros(prob.stride, np.int16)
    row[:2 * M] = [2 * u for u in range(M)] + [2 * u + 1 for u in range(M)]
    row[2 * M:4 * M] = [x for u in reversed(range(M)) for x in (2 * u, 2 * u + 1)]
    gpipe = row.copy()
    gpipe[2 * M:4 * M] = row[:2 * M]
    rows = np.stack([row, gpipe, row])
    want = O.evaluate(prob, rows)
    assert (want.flags == 0).all()
    sim = dip.Sim(prob)
    for slots, variant in ((4, 8), (8, 8), (4, 9), (8, 9)):
        assert sim.configure_pool(slots) == dip.OK
        assert sim.configure(variant, 0) == dip.OK
        orders = torch.from_numpy(rows).to(DEV)
        out = sim.outputs(len(rows))
        for t in out:
            t.fill_(-5 if t.dtype != torch.uint8 else 0x55)
        dip.evaluate(sim.h, sim.costs, orders, len(rows), *out)
        torch.cuda.synchronize()
        assert_same(tuple(t.cpu().numpy() for t in out), want)
        if (slots, variant) == (4, 9):
            assert dip.last_retries(sim.h)[0] > 0   # a stall of live orders retries
    sim.close()


def test_deadlock_with_full_pools_settled_in_first_pass():
    """Four ranks, six microbatches: rank 0 runs all forwards first, rank 1
    alternates F and B, rank 2 runs F0 F1 before B0, so rank 1 waits at B0 on
    rank 2 and rank 2 waits at F1 on rank 1 (a cycle), and rank 3 waits on
    rank 2.  Rank 0's forwards pile up for rank 1: with four slots per pool
    rank 0 is held at F5.  The waiting ranks wait on one another in a cycle,
    so the simulation kernel gives the deadlock verdict in its first pass (no
    retry) and every output equals the oracle's."""
    need_gpu()
    M = 6
    prob = W.compile_instance(W.pipeline_instance(4, M, 5, comm=2))
    ro = prob.rank_off
    row = np.zeros(prob.stride, np.int16)
    alt = [x for j in range(M) for x in (2 * j, 2 * j + 1)]   # F0 B0 F1 B1 ...
    row[ro[0]:ro[1]] = [2 * j for j in range(M)] + [2 * j + 1 for j in range(M)]
    row[ro[1]:ro[2]] = alt
    row[ro[2]:ro[3]] = [0, 2, 1, 3] + alt[4:]
    row[ro[3]:ro[4]] = alt
    rows = np.stack([row, row, row])
    want = O.evaluate(prob, rows)
    assert (want.flags == dip.FLAG_DEADLOCK).all()
    sim = dip.Sim(prob)
    for slots in (4, 8):
        assert sim.configure_pool(slots) == dip.OK
        assert sim.configure(9, 0) == dip.OK
        assert_same(run_gpu(sim, rows), want)
        assert dip.last_retries(sim.h) == (0, 0)
    sim.close()


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_check_kernels_caps_and_invalid_ids(cid):
    """Both kernels of the order-only verdict (one wave per candidate; tiles
    of 64 candidates with the ranks split between the waves of a block, then
    the own-rank order kernel) against
    the oracle, with per-rank caps at the median peak (so some candidates are
    capped and some are not) and ids out of range (n_r itself, the overflow
    bit of the tile kernel), negative or repeated, planted on random ranks and
    on the last rank."""
    need_gpu()
    prob = W.make_problem(cid)
    n = SMALL[cid]
    rows = W.generator_for(prob, cid).generate(1, n).copy()
    peaks = O.evaluate(prob, rows[:64], threads=16).peak
    cap = np.median(peaks, axis=0).astype(np.int32)
    prob = dataclasses.replace(prob, mem_cap=cap)
    rng = np.random.default_rng(cid)
    P, ro = prob.n_ranks, prob.rank_off
    planted = rng.choice(n, size=max(3, n // 16), replace=False)
    for i in planted:
        r = int(rng.integers(P)) if i % 2 else P - 1
        b, e = int(ro[r]), int(ro[r + 1])
        p = int(rng.integers(b, e))
        if i % 3 == 0:
            rows[i, p] = e - b
        elif i % 3 == 1:
            rows[i, p] = -1 - int(rng.integers(100))
        else:
            rows[i, p] = rows[i, b if p != b else e - 1]
    # ops moved before their own-rank predecessor on the last rank (the loss
    # turnaround), on rows that hold no planted id
    planted = set(int(i) for i in planted)
    for i in range(n):
        if i % 4 == 3 and i not in planted:
            own_rank_swap(prob, rows[i], P - 1, rng)
    want = O.evaluate(prob, rows, threads=16)
    assert (want.flags & O.FLAG_INVALID).any() and (want.flags & O.FLAG_CAP).any()
    sim = dip.Sim(prob)
    tried = 0
    for mode in (1, 2):
        rc = sim.configure_check(mode)
        if rc == dip.E_UNSUPPORTED:
            continue
        assert rc == dip.OK
        assert sim.info["check_kernel"] == mode
        print(f"config {cid} check kernel {mode}", flush=True)
        assert_same(run_gpu(sim, rows), want)
        tried += 1
    assert tried >= 1
    sim.close()


def test_check_kernels_empty_rank():
    """A rank with no ops between two that have some: its peak is 0, it never
    flags a candidate, and the other ranks keep their sections."""
    need_gpu()
    M = 4
    base = W.compile_instance(W.pipeline_instance(3, M, [[4, 6, 5, 7], [5, 5, 6, 6], [7, 3, 4, 5]],
                                                  comm=2))
    ro = np.asarray(base.rank_off)
    prob = dataclasses.replace(
        base, n_ranks=4, n_ops=np.array([base.n_ops[0], base.n_ops[1], 0, base.n_ops[2]], np.int32),
        rank_off=np.array([ro[0], ro[1], ro[2], ro[2], ro[3]], ro.dtype),
        mem_cap=np.array([-1, 0, 0, -1], np.int32))
    one = np.zeros(prob.stride, np.int16)
    for r in range(3):
        k = int(base.n_ops[r])
        one[ro[r]:ro[r] + k] = np.arange(k)
    rows = np.stack([one] * 130)
    rows[7, int(ro[2])] = int(base.n_ops[2])          # out of range on the rank after the empty one
    want = O.evaluate(prob, rows)
    assert want.flags[7] == O.FLAG_INVALID and (want.flags[:7] == O.FLAG_CAP).all()
    assert (want.peak[:, 2] <= 0).all()
    sim = dip.Sim(prob)
    for mode in (1, 2):
        if sim.configure_check(mode) == dip.E_UNSUPPORTED:
            continue
        assert_same(run_gpu(sim, rows), want)
    sim.close()


def with_microbatch_order(base, comm):
    """The pipeline instance `base` (one unit per lane and microbatch, v = 1)
    with an extra edge F(u, r) -> F(u + 1, r) on every rank r (latency
    `comm`): every rank then has ops that wait on an op of their own rank."""
    P, ro = base.n_ranks, np.asarray(base.rank_off)
    preds = [list(base.pred_op[base.pred_ptr[g]:base.pred_ptr[g + 1]]) for g in range(int(ro[-1]))]
    comms = [list(base.edge_comm[base.pred_ptr[g]:base.pred_ptr[g + 1]]) for g in range(int(ro[-1]))]
    for r in range(P):
        for lid in range(2, int(base.n_ops[r]), 2):   # F(u) at 2u, B(u) at 2u + 1
            preds[ro[r] + lid].append(int(ro[r]) + lid - 2)
            comms[ro[r] + lid].append(comm)
    ptr = np.zeros(len(preds) + 1, base.pred_ptr.dtype)
    ptr[1:] = np.cumsum([len(x) for x in preds])
    return dataclasses.replace(base, pred_ptr=ptr,
                               pred_op=np.array([q for x in preds for q in x], base.pred_op.dtype),
                               edge_comm=np.array([c for x in comms for c in x], base.edge_comm.dtype))


@pytest.mark.parametrize("comm", [0, 2])
def test_own_rank_order_on_every_rank(comm):
    """Every rank has ops that wait on an op of their own rank (the extra
    microbatch-order edges, plus the loss turnaround on the last rank), so the
    order kernel runs on all four ranks at once: orders that keep each F(u)
    before F(u + 1) and orders that swap them, against the oracle, under both
    check kernels and every variant that fits (with latency 0 the simulation
    kernel drops these edges and relies on the order check; with latency 2 it
    keeps them)."""
    need_gpu()
    rng = np.random.default_rng(40 + comm)
    M = 12
    base = W.compile_instance(W.pipeline_instance(4, M, rng.integers(5, 40, size=(4, M)), comm=3))
    prob = with_microbatch_order(base, comm)
    ro = np.asarray(prob.rank_off)
    n = 700
    rows = np.zeros((n, prob.stride), np.int16)
    def one_f_one_b(d):
        # d forwards first, then each backward followed by the next forward
        ids = [2 * u for u in range(d)]
        for k in range(M):
            ids.append(2 * k + 1)
            if k + d < M:
                ids.append(2 * (k + d))
        return np.array(ids, np.int16)
    for i in range(n):
        # warm-up depths that do not grow along the pipeline are deadlock free;
        # on some rows one rank's depth exceeds its predecessor's (a cycle
        # across ranks the simulation finds)
        d = np.sort(rng.integers(1, M + 1, size=prob.n_ranks))[::-1].copy()
        if i % 5 == 1:
            r = int(rng.integers(1, prob.n_ranks))
            d[r] = min(M, d[r - 1] + 1)
        for r in range(prob.n_ranks):
            rows[i, ro[r]:ro[r + 1]] = one_f_one_b(int(d[r]))
        if i % 3 == 0:   # F(u + 1) moved before F(u) on one rank: an own-rank order violation
            r = int(rng.integers(prob.n_ranks))
            sec = rows[i, ro[r]:ro[r + 1]]
            pairs = [q for q in range(len(sec) - 1) if sec[q] % 2 == 0 and sec[q + 1] == sec[q] + 2]
            if pairs:
                q = pairs[int(rng.integers(len(pairs)))]
                sec[q], sec[q + 1] = sec[q + 1], sec[q]
    want = O.evaluate(prob, rows, threads=16)
    dead = np.mean(want.flags & O.FLAG_DEADLOCK > 0)
    print(f"comm {comm}: deadlocked {dead:.2f}", flush=True)
    assert 0.1 < dead < 0.9
    sim = dip.Sim(prob)
    tried = 0
    for variant in (0, 3, 8, 9):
        for mode in (1, 2):
            if sim.configure(variant, 0) != dip.OK or sim.configure_check(mode) != dip.OK:
                continue
            print(f"variant {variant} check {mode}: {sim.info['variant']}", flush=True)
            assert_same(run_gpu(sim, rows), want)
            tried += 1
    assert tried >= 4
    sim.close()


def test_retry_passes_16_and_32_slots():
    """Candidates whose pools fill go through the passes with 16 and then 32
    slots per pool before the general kernel; with 4 and 8 slots in the first
    pass on the 32-rank diffusion workload (a third of its orders deadlock,
    and deadlocked orders fill small pools), every output still equals the
    oracle's and the passes leave next to nothing to the general kernel.
    With 4 slots some live orders stall on full pools and must retry; with 8
    the stalls are deadlocks whose waiting lanes wait on one another in a
    cycle, which the first pass settles itself (no retry)."""
    need_gpu()
    prob = W.make_problem(4)
    n = 3000
    rows = W.generator_for(prob, 4).generate(11, n)
    want = O.evaluate(prob, rows, threads=16)
    sim = dip.Sim(prob)
    dip.profile(sim.h, True)
    for slots in (4, 8):
        assert sim.configure_pool(slots) == dip.OK
        got = run_gpu(sim, rows)
        first, left = dip.last_retries(sim.h)
        times = dip.last_profile(sim.h)
        print(f"slots {slots}: first-pass retries {first}, left to the general kernel {left}, "
              f"kernel ms {[round(t, 3) for t in times]}", flush=True)
        assert_same(got, want)
        if slots == 4:
            assert first > 0 and left <= first // 20
        else:
            assert first <= n // 100 and left == 0
        if sim.info["variant"] == 9:
            assert len(times) == 5
    dip.profile(sim.h, False)
    sim.close()


def test_parity_full_bench_workload():
    """The 8-stage VLM workload at its full 65,536 candidates, in the launch
    configuration the benchmark times, compared on every candidate, plus the
    argmin."""
    need_gpu()
    prob = W.make_problem(2)
    cfg = W.get(2)
    rows = W.generator_for(prob, 2).generate(0, cfg.n_cand)
    want = O.evaluate(prob, rows, threads=16)
    sim = dip.Sim(prob)
    got = run_gpu(sim, rows)
    assert_same(got, want)
    key = sim.argmin(torch.from_numpy(got[0]).to(DEV), torch.from_numpy(got[3]).to(DEV))
    torch.cuda.synchronize()
    assert dip.decode_key(int(key.item())) == O.argmin(want.makespan, want.flags)
    sim.close()


def test_edge_cases_invalid_deadlock_single():
    need_gpu()
    prob = W.make_problem(1)
    base = W.generator_for(prob, 1).generate(0, 8)
    rows = [base[i].copy() for i in range(8)]
    rows[1][3] = 99                     # id out of range on rank 0
    rows[2][16 + 2] = rows[2][16 + 5]   # duplicate on rank 1
    i0, i1 = int(np.nonzero(rows[3][:16] == 0)[0][0]), int(np.nonzero(rows[3][:16] == 1)[0][0])
    rows[3][i0], rows[3][i1] = 1, 0     # B0 before F0 on rank 0: deadlock
    rows[4][-1] = -7                    # negative id on the last rank
    rows = np.stack(rows)
    want = O.evaluate(prob, rows)
    assert want.flags[1] == O.FLAG_INVALID and want.flags[3] & O.FLAG_DEADLOCK
    sim = dip.Sim(prob)
    for n in (1, 2, 5, 8):
        got = run_gpu(sim, rows[:n])
        assert_same(got, O.evaluate(prob, rows[:n]))
    sim.close()


def test_zero_candidates_is_noop():
    need_gpu()
    prob = W.make_problem(1)
    sim = dip.Sim(prob)
    out = sim.outputs(1)
    dip.evaluate(sim.h, sim.costs, torch.empty((0, prob.stride), dtype=torch.int16, device=DEV),
                 0, *out)
    torch.cuda.synchronize()
    sim.close()


def test_errors_through_abi():
    need_gpu()
    prob = W.make_problem(1)
    sim = dip.Sim(prob)
    rows = torch.zeros((4, prob.stride), dtype=torch.int16, device=DEV)
    out = sim.outputs(4)
    with pytest.raises(dip.DipSimError) as e:
        dip.evaluate(sim.h, None, rows, 4, *out)        # no costs yet
    assert e.value.code == dip.E_STATE
    dip.evaluate(sim.h, sim.costs, rows, 4, *out)
    flat = torch.zeros(4 * prob.stride + 8, dtype=torch.int16, device=DEV)
    with pytest.raises(dip.DipSimError) as e:
        dip.evaluate(sim.h, None, flat[1:], 4, *out)     # misaligned rows
    assert e.value.code == dip.E_INVAL
    key = torch.full((1,), -1, dtype=torch.int64, device=DEV)
    with pytest.raises(dip.DipSimError) as e:
        dip.argmin(sim.h, out[0], out[3], 4, 2**32 - 2, key)
    assert e.value.code == dip.E_RANGE
    torch.cuda.synchronize()
    sim.close()


def test_argmin_ties_chunks_and_empty():
    need_gpu()
    prob = W.make_problem(2)
    rows = W.generator_for(prob, 2).generate(0, 3000)
    rows = np.concatenate([rows, rows[:1000]])          # planted duplicates: ties
    want = O.evaluate(prob, rows, threads=16)
    sim = dip.Sim(prob)
    ms, bub, pk, fl = sim.evaluate(torch.from_numpy(rows).to(DEV))
    key = torch.full((1,), -1, dtype=torch.int64, device=DEV)
    # fold in uneven chunks; index_base keeps global indices
    cuts = [0, 1, 700, 2999, 3001, 4000]
    for a, b in zip(cuts, cuts[1:]):
        dip.argmin(sim.h, ms[a:b], fl[a:b], b - a, a, key)
    torch.cuda.synchronize()
    assert dip.decode_key(int(key.item())) == O.argmin(want.makespan, want.flags)
    # all candidates flagged: the key stays "none"
    bad = torch.ones_like(fl)
    key2 = sim.argmin(ms, bad)
    torch.cuda.synchronize()
    assert dip.decode_key(int(key2.item())) == (-1, -1)
    sim.close()


def test_deterministic_repeat_and_reused_costs():
    need_gpu()
    prob = W.make_problem(3)
    rows = W.generator_for(prob, 3).generate(0, 300)
    sim = dip.Sim(prob)
    a = run_gpu(sim, rows)
    b = run_gpu(sim, rows)           # costs not resent: reused
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
    sim.close()


def test_streamed_chunks_two_streams():
    """The 16 x 4 large configuration streamed in chunks through the
    double-buffered copy/compute streams: every chunk's outputs against the
    oracle, and the argmin folded over all chunks against the oracle's."""
    need_gpu()
    from paper_2504_14145_amd.stream import ChunkStream
    prob = W.make_problem(5)
    chunk, n_chunks = 96, 5
    rows = W.generator_for(prob, 5).generate(0, chunk * n_chunks - 17)   # ragged last chunk
    want = O.evaluate(prob, rows, threads=16)
    sim = dip.Sim(prob)
    cs = ChunkStream(sim, chunk, keep_outputs=True)
    for k in range(n_chunks):
        lo, hi = k * chunk, min((k + 1) * chunk, len(rows))
        host = torch.from_numpy(np.ascontiguousarray(rows[lo:hi])).pin_memory()
        cs.submit(host, lo)
    key = cs.finish()
    for base, outs in cs.host_outs:
        idx = np.arange(base, base + outs[0].shape[0])
        ms, bub, pk, fl = (t.numpy() for t in outs)
        np.testing.assert_array_equal(fl, want.flags[idx])
        np.testing.assert_array_equal(ms, want.makespan[idx])
        np.testing.assert_array_equal(bub, want.bubble[idx])
        np.testing.assert_array_equal(pk, want.peak[idx])
    assert dip.decode_key(int(key.item())) == O.argmin(want.makespan, want.flags)
    sim.close()
