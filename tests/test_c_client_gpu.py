"""The C ABI from plain C: tests/c_client/dip_client (built by
__graft_entry__.build(), no Python or torch inside) reads an instance and a
batch of orders from a file, runs dip_sim_create / dip_sim_evaluate /
dip_sim_argmin on device buffers it allocates itself, and writes the outputs
back; every output and the argmin must equal the oracle's."""
import os
import subprocess

import numpy as np
import pytest

import oracle as O
import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))
CLIENT = os.path.join(HERE, "c_client", "dip_client")

pytestmark = pytest.mark.gpu


def write_input(path, prob, rows):
    P, N, E = prob.n_ranks, prob.n_total, prob.n_edges
    with open(path, "wb") as f:
        np.array([P, N, E, prob.n_slots], np.int32).tofile(f)
        np.array([prob.stride, len(rows)], np.int64).tofile(f)
        for a, t in ((prob.n_ops, np.int32), (prob.pred_ptr, np.int32), (prob.pred_op, np.int32),
                     (prob.op_kind, np.uint8), (prob.op_slot, np.int32), (prob.mem_cap, np.int32),
                     (prob.op_cost, np.int32), (prob.edge_comm, np.int32),
                     (prob.slot_act, np.int32)):
            np.ascontiguousarray(a, dtype=t).tofile(f)
        np.ascontiguousarray(rows, dtype=np.int16).tofile(f)


def read_output(path, n, P):
    raw = open(path, "rb").read()
    off = 0

    def take(dtype, count):
        nonlocal off
        a = np.frombuffer(raw, dtype, count, off)
        off += a.nbytes
        return a

    ms = take(np.int32, n)
    bub = take(np.int32, n * P).reshape(n, P)
    pk = take(np.int32, n * P).reshape(n, P)
    fl = take(np.uint8, n)
    key = int(take(np.uint64, 1)[0])
    assert off == len(raw)
    return ms, bub, pk, fl, key


@pytest.mark.parametrize("cid,n", [(2, 3000), (5, 300), (1, 0)])
def test_c_client_matches_oracle(tmp_path, cid, n):
    if not os.path.exists(CLIENT):
        pytest.fail(f"{CLIENT} is not built; run __graft_entry__.build()")
    print(f"c client: workload {cid}, {n} candidates", flush=True)
    prob = W.make_problem(cid)
    rows = W.generator_for(prob, cid).generate(21, n)
    if n:
        # one row with a repeated id, which makes that candidate invalid
        ro = prob.rank_off
        rows[0, ro[0] + 1] = rows[0, ro[0]]
    want = O.evaluate(prob, rows, threads=16)
    write_input(tmp_path / "in.bin", prob, rows)
    run = subprocess.run([CLIENT, str(tmp_path / "in.bin"), str(tmp_path / "out.bin")],
                         capture_output=True, text=True, timeout=300)
    assert run.returncode == 0, run.stderr
    ms, bub, pk, fl, key = read_output(tmp_path / "out.bin", n, prob.n_ranks)
    np.testing.assert_array_equal(ms, want.makespan)
    np.testing.assert_array_equal(bub, want.bubble)
    np.testing.assert_array_equal(pk, want.peak)
    np.testing.assert_array_equal(fl, want.flags)
    best = O.argmin(want.makespan, want.flags)
    if best[0] < 0:
        assert key == (1 << 64) - 1
    else:
        assert (key & 0xFFFFFFFF, key >> 32) == best
    if n:
        assert fl[0] == 4
