"""Candidate hand-out of the pool kernel on batches larger than its resident
slots: with short candidates most of the batch goes to fixed successors and
the rest on demand.  Every tile of a tiled batch must give the literal
batch's outputs, and sampled candidates the oracle's."""
import numpy as np
import pytest

import oracle as O
import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2504_14145_amd as dip

DEV = "cuda:0"


@pytest.mark.parametrize("variant", [8, 9])
@pytest.mark.parametrize("cid,n", [(2, 65536), (1, 4096)])
def test_tiled_batch_past_the_slots(cid, n, variant):
    """The pool kernel (variant 8) and the compact-record simulation kernel
    (variant 9, the default here) alike."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cfg = W.get(cid)
    prob = W.make_problem(cfg)
    rows = W.generator_for(prob, cfg).generate(0, n)
    sim = dip.Sim(prob)
    assert sim.configure(variant, 0) == dip.OK
    orders = torch.from_numpy(rows).to(DEV)
    ms, bub, pk, fl = sim.evaluate(orders)       # (variant 9's shape follows the costs)
    info = sim.info
    assert info["variant"] == variant
    slots = info["max_blocks"] * info["waves_per_block"] * info["groups_per_wave"]
    assert slots > 0
    reps = int(np.ceil(2.5 * slots / n)) + 1          # well past twice the slots
    print(f"config {cid} variant {variant}: {n} x {reps} candidates, {slots} slots", flush=True)
    big = orders.repeat(reps, 1)
    bms, bbub, bpk, bfl = sim.evaluate(big)
    torch.cuda.synchronize()
    for t in range(reps):
        seg = slice(t * n, (t + 1) * n)
        torch.testing.assert_close(bms[seg], ms, rtol=0, atol=0)
        torch.testing.assert_close(bbub[seg], bub, rtol=0, atol=0)
        torch.testing.assert_close(bpk[seg], pk, rtol=0, atol=0)
        torch.testing.assert_close(bfl[seg], fl, rtol=0, atol=0)
    idx = np.unique(np.random.default_rng(5).integers(0, n * reps, size=48))
    want = O.evaluate(prob, rows[idx % n], threads=16)
    np.testing.assert_array_equal(bms.cpu().numpy()[idx], want.makespan)
    np.testing.assert_array_equal(bfl.cpu().numpy()[idx], want.flags)
    sim.close()
