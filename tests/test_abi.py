"""C ABI contract on the CPU: the library loads, exports every declared
symbol, and host-side validation returns the documented codes without
touching a device."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2504_14145_amd as dip
import workloads as W

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "dip_sim.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dip_\w+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = dip.load()
    names = declared_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(dip.EXPORTS)
    assert lib.dip_sim_abi_version() == 8


def test_binding_constants_match_header():
    text = open(HEADER).read()
    assert int(re.search(r"#define DIP_SIM_PROFILE_MAX (\d+)", text).group(1)) == dip.PROFILE_MAX
    assert int(re.search(r"#define DIP_SIM_ABI_VERSION (\d+)", text).group(1)) == 8


def test_strerror_strings():
    for code in (0, -1, -2, -3, -4, -5, -7, -8):
        assert len(dip.strerror(code)) >= 2
    assert dip.strerror(12345) == "unknown error"


def topo_arrays(prob):
    return dict(n_ranks=prob.n_ranks, n_ops=prob.n_ops.copy(), pred_ptr=prob.pred_ptr.copy(),
                pred_op=prob.pred_op.copy(), op_kind=prob.op_kind.copy(),
                op_slot=prob.op_slot.copy(), n_slots=prob.n_slots, mem_cap=prob.mem_cap.copy(),
                cand_stride=prob.stride)


@pytest.fixture(scope="module")
def prob():
    return W.make_problem(2)


def test_valid_topology_and_costs(prob):
    t = dip.HostTopology(**topo_arrays(prob))
    assert dip.check_topology(t) == dip.OK
    assert dip.check_costs(t, dip.HostCosts.of(prob)) == dip.OK


@pytest.mark.parametrize("mutate,code", [
    (lambda a: a.update(n_ranks=0), dip.E_INVAL),
    (lambda a: a.update(n_ranks=65, n_ops=np.ones(65, np.int32),
                        mem_cap=-np.ones(65, np.int32)), dip.E_UNSUPPORTED),
    (lambda a: a["n_ops"].__setitem__(0, 40000), dip.E_TOPO),
    (lambda a: a["n_ops"].__setitem__(0, -1), dip.E_TOPO),
    (lambda a: a.update(cand_stride=a["cand_stride"] - 8), dip.E_INVAL),
    (lambda a: a.update(cand_stride=a["cand_stride"] + 4), dip.E_INVAL),
    (lambda a: a["pred_ptr"].__setitem__(0, 1), dip.E_TOPO),
    (lambda a: a["pred_ptr"].__setitem__(5, a["pred_ptr"][6] + 1), dip.E_TOPO),
    (lambda a: a["pred_op"].__setitem__(0, 10**6), dip.E_TOPO),
    (lambda a: a["pred_op"].__setitem__(0, -3), dip.E_TOPO),
    (lambda a: a["op_kind"].__setitem__(3, 2), dip.E_TOPO),
    (lambda a: a["op_slot"].__setitem__(3, a["n_slots"]), dip.E_TOPO),
])
def test_topology_errors(prob, mutate, code):
    a = topo_arrays(prob)
    mutate(a)
    t = dip.HostTopology(**a)
    assert dip.check_topology(t) == code
    # create validates before any device call, so it reports the same code
    h = ctypes.c_void_p()
    assert dip.load().dip_sim_create(ctypes.byref(t.c), ctypes.byref(h)) == code
    assert not h.value


def test_self_edge_rejected(prob):
    a = topo_arrays(prob)
    g = int(np.nonzero(np.diff(a["pred_ptr"]) > 0)[0][0])
    a["pred_op"][a["pred_ptr"][g]] = g
    assert dip.check_topology(dip.HostTopology(**a)) == dip.E_TOPO


def test_null_pointers_rejected():
    lib = dip.load()
    assert lib.dip_sim_check_topology(None) == dip.E_INVAL
    h = ctypes.c_void_p()
    assert lib.dip_sim_create(None, ctypes.byref(h)) == dip.E_INVAL
    assert lib.dip_sim_evaluate(None, None, None, 0, None, None, None, None, None) == dip.E_INVAL
    assert lib.dip_sim_argmin(None, None, None, 0, 0, None, None) == dip.E_INVAL
    assert lib.dip_sim_set_greedy_inbox(None, 8) == dip.E_INVAL
    assert lib.dip_sim_rollouts_batch(None, 1, None, None, 4, 0, 0, None, None, None, None,
                                      None) == dip.E_INVAL
    lib.dip_sim_destroy(None)     # no-op


@pytest.mark.parametrize("which,code", [
    ("neg_cost", dip.E_RANGE), ("neg_comm", dip.E_RANGE), ("neg_act", dip.E_RANGE),
    ("big_total", dip.E_RANGE), ("big_act", dip.E_RANGE)])
def test_cost_range_errors(prob, which, code):
    t = dip.HostTopology(**topo_arrays(prob))
    cost, comm, act = prob.op_cost.copy(), prob.edge_comm.copy(), prob.slot_act.copy()
    if which == "neg_cost":
        cost[7] = -1
    elif which == "neg_comm":
        comm[3] = -5
    elif which == "neg_act":
        act[2] = -1
    elif which == "big_total":
        cost[:] = 2**31 // len(cost) + 10
    elif which == "big_act":
        act[:] = 2**30
    assert dip.check_costs(t, dip.HostCosts(cost, comm, act)) == code
