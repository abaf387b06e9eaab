"""GPU parity of the dual-queue interleaving (dip_sim_greedy) against the CPU
oracle: emitted orders and scores element by element, bit-exact."""
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


def run_greedy(sim, prio_np):
    prio = torch.from_numpy(np.ascontiguousarray(prio_np, np.int32)).to(DEV)
    ords, (ms, bub, pk, fl) = sim.greedy(prio)
    torch.cuda.synchronize()
    return (ords.cpu().numpy(), ms.cpu().numpy(), bub.cpu().numpy(), pk.cpu().numpy(),
            fl.cpu().numpy())


def check_against_oracle(prob, groups, prio, sim=None, tag=""):
    g, G = groups[0], groups[1]
    want_o, want = O.greedy(prob, g, G, prio, stride=prob.stride, threads=16)
    own = sim is None
    if own:
        sim = dip.Sim(prob)
        assert sim.configure_greedy(G, g) == dip.OK
    print(f"{tag}: n={len(prio)} N={prob.n_total} G={G}", flush=True)
    ords, ms, bub, pk, fl = run_greedy(sim, prio)
    N = prob.n_total
    np.testing.assert_array_equal(ords[:, :N], want_o[:, :N])
    np.testing.assert_array_equal(fl, want.flags)
    np.testing.assert_array_equal(ms, want.makespan)
    np.testing.assert_array_equal(bub, want.bubble)
    np.testing.assert_array_equal(pk, want.peak)
    if own:
        sim.close()
    return ords, ms, bub, pk, fl


SMALL = {1: 300, 2: 203, 3: 37, 4: 67, 5: 21}


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_greedy_parity_rollouts(cid):
    """Random rollout priorities (ragged counts) on the workload shapes."""
    need_gpu()
    prob = W.make_problem(cid)
    g, G, cls = W.priority_groups(prob)
    prio = W.rollout_priorities(cls, SMALL[cid], seed=11)
    check_against_oracle(prob, (g, G), prio, tag=f"config {cid}")


@pytest.mark.parametrize("cid", [1, 2, 3])
def test_greedy_emitted_orders_simulate_to_same_scores(cid):
    """The greedy's own timeline equals the simulator's on its emitted orders
    (dip_sim_evaluate on the GPU, same handle)."""
    need_gpu()
    prob = W.make_problem(cid)
    g, G, cls = W.priority_groups(prob)
    prio = W.rollout_priorities(cls, 64, seed=3)
    sim = dip.Sim(prob)
    assert sim.configure_greedy(G, g) == dip.OK
    ords, ms, bub, pk, fl = run_greedy(sim, prio)
    ev = sim.evaluate(torch.from_numpy(ords).to(DEV))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(ev[0].cpu().numpy(), ms)
    np.testing.assert_array_equal(ev[1].cpu().numpy(), bub)
    np.testing.assert_array_equal(ev[2].cpu().numpy(), pk)
    np.testing.assert_array_equal(ev[3].cpu().numpy(), fl)
    sim.close()


def test_greedy_fifo_equal_and_reversed_priorities():
    """Base priorities: first-in first-out, all equal (ties go by group index)
    and reversed."""
    need_gpu()
    prob = W.make_problem(2)
    g, G, cls = W.priority_groups(prob)
    fifo = W.fifo_priorities(prob, cls, g)
    prio = np.stack([fifo, np.zeros(G, np.int32), -fifo, np.arange(G, dtype=np.int32)])
    check_against_oracle(prob, (g, G), prio, tag="fifo/equal/reversed")


def _pipeline(P, M, f, comm, cap=-1, act=1, v=1):
    inst = W.pipeline_instance(P, M, f, comm=comm, act=act, mem_cap=cap, v=v)
    prob = W.compile_instance(inst)
    g, G, cls = W.priority_groups(prob)
    return prob, g, G, cls


@pytest.mark.parametrize("cap", [-1, 1, 2, 0])
def test_greedy_memory_caps(cap):
    """Tight caps: the forward queue is disabled, and at cap 0 every forward is
    a forced decision (flagged)."""
    need_gpu()
    prob, g, G, cls = _pipeline(4, 9, np.arange(4 * 9).reshape(4, 9) % 7 + 3, comm=2, cap=cap)
    prio = W.rollout_priorities(cls, 70, seed=cap + 5)
    _, _, _, _, fl = check_against_oracle(prob, (g, G), prio, tag=f"cap {cap}")
    if cap == 0:
        assert (fl == dip.FLAG_CAP).all()


def test_greedy_inbox_overflow_goes_through_retry():
    """A long transfer latency piles many future arrivals into one rank's
    inbox: those candidates are finished by the second launch, and later
    calls get larger inboxes."""
    need_gpu()
    prob, g, G, cls = _pipeline(2, 40, 10, comm=1000)
    prio = W.rollout_priorities(cls, 19, seed=2)
    sim = dip.Sim(prob)
    assert sim.configure_greedy(G, g) == dip.OK
    k0 = sim.info["greedy_inbox"]
    for call in range(3):
        check_against_oracle(prob, (g, G), prio, sim=sim, tag=f"overflow call {call}")
    assert sim.info["greedy_inbox"] > k0
    sim.close()


def test_greedy_skips_first_launch_when_most_overflow():
    """On the large 16 x 64-lane workload most candidates overflow even the
    largest inboxes that fit in LDS: after a few calls the inboxes stop
    growing and later calls give every candidate to the second launch
    (greedy_inbox -1), with results equal to the oracle's on every call."""
    need_gpu()
    prob = W.make_problem(5)
    g, G, cls = W.priority_groups(prob)
    prio = W.rollout_priorities(cls, SMALL[5], seed=13)
    sim = dip.Sim(prob)
    assert sim.configure_greedy(G, g) == dip.OK
    seen = []
    for call in range(8):
        check_against_oracle(prob, (g, G), prio, sim=sim, tag=f"large call {call}")
        seen.append(sim.info["greedy_inbox"])
    print(f"inbox after each call: {seen}", flush=True)
    assert seen[-1] == -1
    assert sim.set_greedy_inbox(0) == dip.OK and sim.info["greedy_inbox"] == 8
    sim.close()


@pytest.mark.parametrize("cid", [2, 3, 4, 5])
def test_greedy_second_launch_for_every_candidate(cid):
    """Inboxes of one stage in the first launch: nearly every candidate
    overflows and is simulated by the second launch, whose inboxes hold a
    whole rank -- in LDS on configs 2 and 3, in device memory on configs 4
    and 5 (594 and 1,413 groups per kind)."""
    need_gpu()
    prob = W.make_problem(cid)
    g, G, cls = W.priority_groups(prob)
    sim = dip.Sim(prob)
    assert sim.configure_greedy(G, g) == dip.OK
    assert sim.set_greedy_inbox(1) == dip.OK
    assert sim.set_greedy_inbox(3) == dip.E_INVAL
    assert sim.info["greedy_inbox"] == 1
    ring = sim.info["greedy_retry_ring_bytes"]
    assert (ring > 0) == (cid >= 4), ring
    prio = W.rollout_priorities(cls, {2: 70, 3: 19, 4: 9, 5: 5}[cid], seed=31)
    for call in range(2):                    # fixed size: no growth between calls
        check_against_oracle(prob, (g, G), prio, sim=sim, tag=f"config {cid} inbox 1 call {call}")
    assert sim.info["greedy_inbox"] == 1
    assert sim.set_greedy_inbox(0) == dip.OK and sim.info["greedy_inbox"] == 8
    sim.close()


def test_greedy_interleaved_and_single_rank():
    """Virtual stages (v = 3) and a single rank (P = 1)."""
    need_gpu()
    prob, g, G, cls = _pipeline(3, 7, np.arange(9 * 7).reshape(9, 7) % 5 + 1, comm=3, v=3)
    check_against_oracle(prob, (g, G), W.rollout_priorities(cls, 33, seed=7), tag="v3")
    prob, g, G, cls = _pipeline(1, 6, 4, comm=0)
    check_against_oracle(prob, (g, G), W.rollout_priorities(cls, 9, seed=8), tag="P1")


def test_greedy_rejects_bad_groups():
    need_gpu()
    prob = W.make_problem(1)
    g, G, cls = W.priority_groups(prob)
    sim = dip.Sim(prob)
    bad = g.copy()
    bad[0] = G
    assert sim.configure_greedy(G, bad) == dip.E_TOPO
    mixed = np.zeros_like(g)          # one group holding both kinds
    assert sim.configure_greedy(G, mixed) == dip.E_TOPO
    prio = torch.zeros((4, G), dtype=torch.int32, device=DEV)
    with pytest.raises(dip.DipSimError):
        sim.greedy(prio)              # not configured
    sim.close()
