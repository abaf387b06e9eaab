"""The CPU-side C and C++ code built with AddressSanitizer and
UndefinedBehaviorSanitizer (-fsanitize=address,undefined, no recovery): the
simulator and greedy oracles (oracle/*.c), the candidate generator
(workloads/gen.c) and the library's host-side validation
(paper_2504_14145_amd/csrc/host_check.cpp).  A child Python process loads the
sanitized builds (the sanitizer runtime preloaded) and runs the oracles on
every workload, the generator, and the validation on valid and malformed
instances and costs (hand-made cases and 400 seeded random corruptions); any sanitizer report fails the test."""
import os
import shutil
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
       "-g", "-O1"]

CHILD = textwrap.dedent(r'''
    import ctypes, sys
    import numpy as np
    sys.path.insert(0, ROOT)
    import oracle as O
    import workloads as W
    from workloads.strategies import strategy_table
    import oracle.memopt as MO

    for cid in (1, 2, 3):
        prob = W.make_problem(cid)
        rows = W.generator_for(prob, cid).generate(0, 24 if cid < 3 else 4)
        res = O.evaluate(prob, rows, threads=2)
        assert res.makespan.shape[0] == rows.shape[0]
        bad = rows.copy()
        bad[0, 1] = bad[0, 0]                        # a repeated id
        bad[1, 2] = 30000                            # out of range
        r2 = O.evaluate(prob, bad[:2], threads=1)
        assert (r2.flags[:2] & O.FLAG_INVALID).all()
        O.argmin(res.makespan, res.flags)
        g, G, cls = W.priority_groups(prob)
        orders, gres = O.greedy(prob, g, G, W.rollout_priorities(cls, 8, seed=cid), threads=2)
        assert orders.shape[0] == 8

    # the library's host-side validation
    lib = ctypes.CDLL(CHECK_LIB)
    import paper_2504_14145_amd as dip
    prob = W.make_problem(2)
    def topo(**kw):
        a = dict(n_ranks=prob.n_ranks, n_ops=prob.n_ops.copy(), pred_ptr=prob.pred_ptr.copy(),
                 pred_op=prob.pred_op.copy(), op_kind=prob.op_kind.copy(), op_slot=prob.op_slot.copy(),
                 n_slots=prob.n_slots, mem_cap=prob.mem_cap.copy(), cand_stride=prob.stride)
        a.update(kw)
        return dip.HostTopology(**a)
    lib.dip_sim_check_topology.argtypes = [ctypes.POINTER(dip.Topology)]
    lib.dip_sim_check_costs.argtypes = [ctypes.POINTER(dip.Topology), ctypes.POINTER(dip.Costs)]
    t = topo()
    assert lib.dip_sim_check_topology(ctypes.byref(t.c)) == 0
    assert lib.dip_sim_check_costs(ctypes.byref(t.c), ctypes.byref(dip.HostCosts.of(prob).c)) == 0
    # (every host structure stays referenced across its call: its arrays back
    # the pointers the library reads)
    codes = []
    def check(tt):
        codes.append(lib.dip_sim_check_topology(ctypes.byref(tt.c)))
    check(topo(n_ranks=0))
    check(topo(cand_stride=prob.stride - 8))
    pp = prob.pred_ptr.copy(); pp[5] = pp[6] + 1
    check(topo(pred_ptr=pp))
    po = prob.pred_op.copy(); po[0] = prob.n_total + 5
    check(topo(pred_op=po))
    sl = prob.op_slot.copy(); sl[3] = prob.n_slots
    check(topo(op_slot=sl))
    cost = prob.op_cost.copy(); cost[7] = -1
    bad_costs = dip.HostCosts(cost, prob.edge_comm.copy(), prob.slot_act.copy())
    codes.append(lib.dip_sim_check_costs(ctypes.byref(t.c), ctypes.byref(bad_costs.c)))
    assert all(x < 0 for x in codes), codes

    # seeded random corruptions of values (array sizes stay as the
    # instance's, which is the caller's part of the contract): every call
    # returns 0 or an error code, with no sanitizer report
    rng = np.random.default_rng(7)
    N, E = prob.n_total, prob.n_edges
    for trial in range(400):
        kw = {}
        which = trial % 8
        if which == 0 and N > 2:
            pp = prob.pred_ptr.copy()
            pp[rng.integers(1, N)] = rng.integers(-5, E + 50)
            kw["pred_ptr"] = pp
        elif which == 1:
            po = prob.pred_op.copy()
            po[rng.integers(E)] = rng.integers(-(2**31), 2**31 - 1)
            kw["pred_op"] = po
        elif which == 2:
            ok = prob.op_kind.copy()
            ok[rng.integers(N)] = rng.integers(0, 256)
            kw["op_kind"] = ok
        elif which == 3:
            sl = prob.op_slot.copy()
            sl[rng.integers(N)] = rng.integers(-(2**31), 2**31 - 1)
            kw["op_slot"] = sl
        elif which == 4:
            kw["n_slots"] = int(rng.integers(-3, prob.n_slots + 1))
        elif which == 5:
            kw["cand_stride"] = int(rng.integers(-8, 2 * prob.stride))
        elif which == 6:
            no = prob.n_ops.copy()
            r = rng.integers(prob.n_ranks)
            d = int(rng.integers(-3, 4))
            no[r] += d
            no[(r + 1) % prob.n_ranks] -= d          # the same total
            kw["n_ops"] = no
        else:
            mc = prob.mem_cap.copy()
            mc[rng.integers(prob.n_ranks)] = rng.integers(-(2**31), 2**31 - 1)
            kw["mem_cap"] = mc
        tt = topo(**kw)
        rc = lib.dip_sim_check_topology(ctypes.byref(tt.c))
        assert rc <= 0, (trial, rc)
        if rc == 0:
            arrays = [prob.op_cost.copy(), prob.edge_comm.copy(), prob.slot_act.copy()]
            a = arrays[trial % 3]
            a[rng.integers(len(a))] = rng.integers(-(2**31), 2**31 - 1)
            cc = dip.HostCosts(*arrays)
            assert lib.dip_sim_check_costs(ctypes.byref(tt.c), ctypes.byref(cc.c)) <= 0

    # the memory selection's search on small ranks
    tab = strategy_table(prob)
    cands = MO.pair_candidates(tab, 4)
    print("ok", flush=True)
''')


def _build(cmd):
    subprocess.check_call(cmd)


def test_cpu_code_under_sanitizers(tmp_path):
    gcc, gxx = shutil.which("gcc"), shutil.which("g++")
    if not gcc or not gxx:
        pytest.skip("no gcc/g++")
    asan = subprocess.run([gcc, "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    if not os.path.isabs(asan) or not os.path.exists(asan):
        pytest.skip("no AddressSanitizer runtime")
    ora = str(tmp_path / "liboracle_san.so")
    gen = str(tmp_path / "libgen_san.so")
    chk = str(tmp_path / "libcheck_san.so")
    _build([gcc, "-std=c11", "-shared", "-fPIC", "-pthread", *SAN, "-o", ora,
            os.path.join(ROOT, "oracle", "dip_oracle.c"), os.path.join(ROOT, "oracle", "dip_greedy.c")])
    _build([gcc, "-std=c11", "-shared", "-fPIC", "-pthread", *SAN, "-o", gen,
            os.path.join(ROOT, "workloads", "gen.c")])
    _build([gxx, "-std=c++17", "-shared", "-fPIC", *SAN, "-I", os.path.join(ROOT, "include"),
            "-I", os.path.join(ROOT, "paper_2504_14145_amd", "csrc"), "-o", chk,
            os.path.join(ROOT, "paper_2504_14145_amd", "csrc", "host_check.cpp")])
    env = dict(os.environ)
    env.update(LD_PRELOAD=asan, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:exitcode=99",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", DIPSIM_ORACLE_LIB=ora,
               DIPSIM_GEN_LIB=gen)
    code = f"ROOT = {ROOT!r}\nCHECK_LIB = {chk!r}\n" + CHILD
    p = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                       timeout=600)
    out = p.stdout + p.stderr
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert p.returncode == 0 and "ok" in p.stdout, out[-4000:]
