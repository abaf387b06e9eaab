"""CPU oracle for batched pipeline-schedule simulation (ctypes front end).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are the only callers.  The GPU library never loads it, and it
shares no code with the GPU library.  The simulator itself is ``dip_oracle.c``
(a single-threaded discrete-event simulation per candidate) and the dual-queue
stage interleaving is ``dip_greedy.c``; each header states what it computes
and which passages of the paper each step follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRCS = [os.path.join(_HERE, "dip_oracle.c"), os.path.join(_HERE, "dip_greedy.c")]
# DIPSIM_ORACLE_LIB names another build of the same sources (the sanitizer test loads
# one built with -fsanitize=address,undefined); it is then used as it is
_LIB = os.environ.get("DIPSIM_ORACLE_LIB") or os.path.join(_HERE, "libdip_oracle.so")

FLAG_DEADLOCK = 1
FLAG_CAP = 2
FLAG_INVALID = 4


def build(force: bool = True) -> str:
    if os.environ.get("DIPSIM_ORACLE_LIB"):
        return _LIB
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared",
                               "-fPIC", "-pthread", "-o", tmp] + _SRCS)
        os.replace(tmp, _LIB)
    return _LIB


class _Inst(ctypes.Structure):
    _fields_ = [("n_ranks", ctypes.c_int32), ("rank_off", ctypes.c_void_p),
                ("pred_ptr", ctypes.c_void_p), ("pred_op", ctypes.c_void_p),
                ("op_kind", ctypes.c_void_p), ("op_slot", ctypes.c_void_p),
                ("n_slots", ctypes.c_int32), ("mem_cap", ctypes.c_void_p),
                ("op_cost", ctypes.c_void_p), ("edge_comm", ctypes.c_void_p),
                ("slot_act", ctypes.c_void_p)]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        vp = ctypes.c_void_p
        lib.dor_eval.restype = ctypes.c_int
        lib.dor_eval.argtypes = [ctypes.POINTER(_Inst), vp, ctypes.c_int64, ctypes.c_int64,
                                 vp, vp, vp, vp, ctypes.c_int32]
        lib.dor_timeline.restype = ctypes.c_int
        lib.dor_timeline.argtypes = [ctypes.POINTER(_Inst), vp, vp, vp, vp, vp, vp, vp]
        lib.dor_argmin.restype = ctypes.c_int64
        lib.dor_argmin.argtypes = [vp, vp, ctypes.c_int64, ctypes.c_int64, vp]
        lib.dgr_greedy.restype = ctypes.c_int
        lib.dgr_greedy.argtypes = [ctypes.POINTER(_Inst), vp, ctypes.c_int32, vp, ctypes.c_int64,
                                   ctypes.c_int64, vp, vp, vp, vp, vp, ctypes.c_int32]
        lib.dgr_greedy_timeline.restype = ctypes.c_int
        lib.dgr_greedy_timeline.argtypes = [ctypes.POINTER(_Inst), vp, vp, vp, vp, vp, vp, vp,
                                            vp, vp]
        _lib = lib
    return _lib


def _i32(a):
    return np.ascontiguousarray(a, np.int32)


class OracleInstance:
    """Keeps the instance arrays alive for the C structure that points at them."""

    def __init__(self, n_ranks, rank_off, pred_ptr, pred_op, op_kind, op_slot, n_slots,
                 mem_cap, op_cost, edge_comm, slot_act):
        self.P = int(n_ranks)
        self.rank_off = np.ascontiguousarray(rank_off, np.int64)
        self.arr = dict(pred_ptr=_i32(pred_ptr), pred_op=_i32(pred_op) if len(pred_op) else np.zeros(1, np.int32),
                        op_kind=np.ascontiguousarray(op_kind, np.uint8), op_slot=_i32(op_slot),
                        mem_cap=_i32(mem_cap), op_cost=_i32(op_cost),
                        edge_comm=_i32(edge_comm) if len(edge_comm) else np.zeros(1, np.int32),
                        slot_act=_i32(slot_act) if len(slot_act) else np.zeros(1, np.int32))
        a = self.arr
        self.c = _Inst(self.P, self.rank_off.ctypes.data, a["pred_ptr"].ctypes.data,
                       a["pred_op"].ctypes.data, a["op_kind"].ctypes.data,
                       a["op_slot"].ctypes.data, int(n_slots), a["mem_cap"].ctypes.data,
                       a["op_cost"].ctypes.data, a["edge_comm"].ctypes.data,
                       a["slot_act"].ctypes.data)

    @property
    def n_total(self):
        return int(self.rank_off[-1])

    @classmethod
    def from_problem(cls, prob):
        return cls(prob.n_ranks, prob.rank_off, prob.pred_ptr, prob.pred_op, prob.op_kind,
                   prob.op_slot, prob.n_slots, prob.mem_cap, prob.op_cost, prob.edge_comm,
                   prob.slot_act)


@dataclass
class Result:
    makespan: np.ndarray   # int32 [n]
    bubble: np.ndarray     # int32 [n, P]
    peak: np.ndarray       # int32 [n, P]
    flags: np.ndarray      # uint8 [n]


def _inst(x):
    return x if isinstance(x, OracleInstance) else OracleInstance.from_problem(x)


def evaluate(prob, orders: np.ndarray, threads: int = 1) -> Result:
    """Simulate every candidate row of ``orders`` (int16 [n, stride])."""
    inst = _inst(prob)
    orders = np.ascontiguousarray(orders, np.int16)
    if orders.ndim == 1:
        orders = orders[None, :]
    n, stride = orders.shape
    if stride < inst.n_total:
        raise ValueError("stride shorter than the op count")
    P = inst.P
    res = Result(np.zeros(n, np.int32), np.zeros((n, P), np.int32),
                 np.zeros((n, P), np.int32), np.zeros(n, np.uint8))
    rc = _load().dor_eval(ctypes.byref(inst.c), orders.ctypes.data, n, stride,
                          res.makespan.ctypes.data, res.bubble.ctypes.data,
                          res.peak.ctypes.data, res.flags.ctypes.data, int(threads))
    if rc != 0:
        raise RuntimeError(f"oracle failed with code {rc}")
    return res


def timeline(prob, order: np.ndarray):
    """One candidate: (Result of size 1, start[N], end[N]); -1 for ops never run."""
    inst = _inst(prob)
    order = np.ascontiguousarray(order, np.int16).reshape(-1)
    N, P = inst.n_total, inst.P
    ms = np.zeros(1, np.int32)
    bub = np.zeros((1, P), np.int32)
    pk = np.zeros((1, P), np.int32)
    fl = np.zeros(1, np.uint8)
    st = np.zeros(max(N, 1), np.int32)
    en = np.zeros(max(N, 1), np.int32)
    rc = _load().dor_timeline(ctypes.byref(inst.c), order.ctypes.data, ms.ctypes.data,
                              bub.ctypes.data, pk.ctypes.data, fl.ctypes.data,
                              st.ctypes.data, en.ctypes.data)
    if rc != 0:
        raise RuntimeError(f"oracle failed with code {rc}")
    return Result(ms, bub, pk, fl), st[:N], en[:N]


def argmin(makespan: np.ndarray, flags: np.ndarray, index_base: int = 0):
    """(global index, makespan) of the lexicographic minimum; (-1, -1) if none."""
    ms = np.ascontiguousarray(makespan, np.int32)
    fl = np.ascontiguousarray(flags, np.uint8)
    best = np.zeros(1, np.int32)
    idx = _load().dor_argmin(ms.ctypes.data, fl.ctypes.data, ms.size, int(index_base),
                             best.ctypes.data)
    return int(idx), int(best[0])


def _groups(inst, op_group, n_groups):
    g = np.ascontiguousarray(op_group, np.int32).reshape(-1)
    if g.size != inst.n_total:
        raise ValueError("op_group needs one entry per op")
    if g.size and (g.min() < 0 or g.max() >= n_groups):
        raise ValueError("op_group entries must lie in [0, n_groups)")
    return g


def greedy(prob, op_group, n_groups: int, prio: np.ndarray, stride: int | None = None,
           threads: int = 1):
    """Dual-queue interleaving (Sec. 5.2) of every candidate priority row.

    ``prio`` is int32 [n, n_groups] (larger first).  Returns (orders int16
    [n, stride], Result) where Result is the greedy's own timeline summary."""
    inst = _inst(prob)
    g = _groups(inst, op_group, n_groups)
    prio = np.ascontiguousarray(prio, np.int32)
    if prio.ndim == 1:
        prio = prio[None, :]
    n = prio.shape[0]
    if prio.shape[1] != n_groups:
        raise ValueError("prio needs one column per group")
    stride = inst.n_total if stride is None else int(stride)
    P = inst.P
    orders = np.zeros((n, max(stride, 1)), np.int16)
    res = Result(np.zeros(n, np.int32), np.zeros((n, P), np.int32),
                 np.zeros((n, P), np.int32), np.zeros(n, np.uint8))
    rc = _load().dgr_greedy(ctypes.byref(inst.c), g.ctypes.data, int(n_groups),
                            prio.ctypes.data, n, orders.shape[1], orders.ctypes.data,
                            res.makespan.ctypes.data, res.bubble.ctypes.data,
                            res.peak.ctypes.data, res.flags.ctypes.data, int(threads))
    if rc != 0:
        raise RuntimeError(f"greedy oracle failed with code {rc}")
    return orders[:, :stride], res


def greedy_timeline(prob, op_group, n_groups: int, prio: np.ndarray):
    """One candidate: (order int16 [N], Result of size 1, start[N], end[N])."""
    inst = _inst(prob)
    g = _groups(inst, op_group, n_groups)
    prio = np.ascontiguousarray(prio, np.int32).reshape(-1)
    if prio.size != n_groups:
        raise ValueError("prio needs one entry per group")
    N, P = inst.n_total, inst.P
    order = np.zeros(max(N, 1), np.int16)
    ms = np.zeros(1, np.int32)
    bub = np.zeros((1, P), np.int32)
    pk = np.zeros((1, P), np.int32)
    fl = np.zeros(1, np.uint8)
    st = np.zeros(max(N, 1), np.int32)
    en = np.zeros(max(N, 1), np.int32)
    rc = _load().dgr_greedy_timeline(ctypes.byref(inst.c), g.ctypes.data, prio.ctypes.data,
                                     order.ctypes.data, ms.ctypes.data, bub.ctypes.data,
                                     pk.ctypes.data, fl.ctypes.data, st.ctypes.data,
                                     en.ctypes.data)
    if rc != 0:
        raise RuntimeError(f"greedy oracle failed with code {rc}")
    return order[:N], Result(ms, bub, pk, fl), st[:N], en[:N]
