"""dip_sim_evaluate_static (working memory in a static device array, no
allocation during the call) against dip_sim_evaluate: bit-exact outputs on
two calls in a row, the second with a smaller batch, under the kernel
variants that use retry lists and one that does not."""
import numpy as np
import pytest

import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2504_14145_amd as dip

DEV = "cuda:0"


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def host(out):
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in out]


def assert_same(got, want):
    for g, w in zip(got, want):
        np.testing.assert_array_equal(g, w)


# (workload, variant, pool slots, first batch, second batch); pools of 4
# slots on the 8x2 workload make candidates retry, so the retry lists and
# counters in the static array carry data from one call into the next
CASES = [
    (2, 0, 0, 5000, 1234),
    (2, 9, 4, 4099, 515),
    (2, 8, 4, 4099, 515),
    (2, 3, 0, 1029, 67),
    (3, 0, 0, 3000, 700),
    (5, 0, 0, 2500, 333),
]


@pytest.mark.parametrize("cid,variant,slots,n1,n2", CASES)
def test_static_matches_evaluate_twice(cid, variant, slots, n1, n2):
    need_gpu()
    print(f"no-alloc: workload {cid} variant {variant} slots {slots} n {n1},{n2}", flush=True)
    prob = W.make_problem(cid)
    gen = W.generator_for(prob, cid)
    sim = dip.Sim(prob)
    if sim.configure(variant, 0) != dip.OK:
        pytest.skip(f"variant {variant} does not fit")
    if slots and sim.configure_pool(slots) != dip.OK:
        pytest.skip(f"{slots} pool slots do not fit")
    info = sim.info
    for seed, n in ((11, n1), (12, n2)):
        orders = torch.from_numpy(np.ascontiguousarray(gen.generate(seed, n))).to(DEV)
        want = host(sim.evaluate(orders))
        want_retries = dip.last_retries(sim.h)
        rc, out = sim.evaluate_static(orders)
        assert rc == dip.OK, dip.strerror(rc)
        got = host(out)
        assert_same(got, want)
        assert dip.last_retries(sim.h) == want_retries
        if variant in (8, 9) and seed == 11 and info["variant"] in (8, 9):
            # the forced small pools do make candidates retry here
            assert want_retries[0] > 0
    assert sim.info["variant"] == info["variant"]


def test_static_state_and_capacity_errors():
    """Checked on the host before anything is launched."""
    need_gpu()
    prob = W.make_problem(2)
    sim = dip.Sim(prob)
    orders = torch.zeros((4, prob.stride), dtype=torch.int16, device=DEV)
    rc, _ = sim.evaluate_static(orders)
    assert rc == dip.E_STATE  # no costs were sent yet
    sim.evaluate(orders)
    torch.cuda.synchronize()
    out = sim.outputs(4, DEV)
    rc = dip.evaluate_static(sim.h, orders, dip.STATIC_MAX_CAND + 1, *out)
    assert rc == dip.E_CAPACITY
    rc = dip.evaluate_static(sim.h, orders, 0, *out)
    assert rc == dip.OK
