"""Python binding of the dip_sim C ABI (include/dip_sim.h).

Argument marshalling only: every step of the simulation and of the argmin
runs in the HIP kernels of ``libdip_sim.so``.  The functions keep the ABI's
names (create, evaluate, argmin, destroy, ...) and take host numpy arrays for
the instance and torch device tensors for candidates and outputs; PyTorch
provides device memory and the stream, nothing else.  Importing works without
a GPU; loading the library fails loudly if it has not been built.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import _build

LIB_PATH = _build.LIB

OK = 0
E_INVAL, E_TOPO, E_RANGE, E_UNSUPPORTED, E_NOMEM, E_HIP, E_STATE, E_CAPACITY = (
    -1, -2, -3, -4, -5, -6, -7, -8)
STATIC_MAX_CAND = 1 << 22
PROFILE_MAX = 8   # DIP_SIM_PROFILE_MAX: entries dip_sim_last_profile may write
FLAG_DEADLOCK, FLAG_CAP, FLAG_INVALID = 1, 2, 4
NO_KEY = (1 << 64) - 1

EXPORTS = ("dip_sim_abi_version", "dip_sim_check_topology", "dip_sim_check_costs",
           "dip_sim_create", "dip_sim_configure", "dip_sim_configure_pool",
           "dip_sim_configure_check", "dip_sim_get_info", "dip_sim_evaluate",
           "dip_sim_evaluate_static", "dip_sim_profile", "dip_sim_last_profile",
           "dip_sim_last_retries", "dip_sim_argmin", "dip_sim_configure_greedy", "dip_sim_set_greedy_inbox", "dip_sim_greedy",
           "dip_sim_configure_rollouts", "dip_sim_rollouts", "dip_sim_rollouts_batch",
           "dip_cost_tables",
           "dip_sim_configure_memopt", "dip_sim_memopt", "dip_sim_evaluate_selected",
           "dip_sim_destroy", "dip_sim_strerror")


class DipSimError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {strerror(code)} ({code})")


class Topology(ctypes.Structure):
    _fields_ = [("n_ranks", ctypes.c_int32), ("n_ops", ctypes.c_void_p),
                ("pred_ptr", ctypes.c_void_p), ("pred_op", ctypes.c_void_p),
                ("op_kind", ctypes.c_void_p), ("op_slot", ctypes.c_void_p),
                ("n_slots", ctypes.c_int32), ("mem_cap", ctypes.c_void_p),
                ("cand_stride", ctypes.c_int64)]


class Costs(ctypes.Structure):
    _fields_ = [("op_cost", ctypes.c_void_p), ("edge_comm", ctypes.c_void_p),
                ("slot_act", ctypes.c_void_p)]


class OpTable(ctypes.Structure):
    _fields_ = [("n_items", ctypes.c_int32), ("n_rows", ctypes.c_int32),
                ("n_kinds", ctypes.c_int32), ("item_ptr", ctypes.c_void_p),
                ("n_fop", ctypes.c_void_p), ("n_mem", ctypes.c_void_p),
                ("n_net", ctypes.c_void_p), ("kind", ctypes.c_void_p)]


class Info(ctypes.Structure):
    _fields_ = [("n_ranks", ctypes.c_int32), ("n_ops_total", ctypes.c_int32),
                ("n_edges", ctypes.c_int32), ("variant", ctypes.c_int32),
                ("cand_stride", ctypes.c_int64), ("lanes_per_group", ctypes.c_int32),
                ("groups_per_wave", ctypes.c_int32), ("waves_per_block", ctypes.c_int32),
                ("lds_bytes", ctypes.c_int32), ("max_blocks", ctypes.c_int32),
                ("scratch_bytes", ctypes.c_int64), ("pool_slots", ctypes.c_int32),
                ("check_kernel", ctypes.c_int32), ("greedy_inbox", ctypes.c_int32),
                ("greedy_lds_bytes", ctypes.c_int32), ("greedy_retry_ring_bytes", ctypes.c_int64)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


_lib = None


def load():
    """The built library; raises if it is missing (no silent fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(LIB_PATH)
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        lib.dip_sim_abi_version.restype = ctypes.c_int
        lib.dip_sim_check_topology.argtypes = [ctypes.POINTER(Topology)]
        lib.dip_sim_check_costs.argtypes = [ctypes.POINTER(Topology), ctypes.POINTER(Costs)]
        lib.dip_sim_create.argtypes = [ctypes.POINTER(Topology), ctypes.POINTER(vp)]
        lib.dip_sim_configure.argtypes = [vp, i32, i32]
        lib.dip_sim_configure_pool.argtypes = [vp, i32]
        lib.dip_sim_configure_check.argtypes = [vp, i32]
        lib.dip_sim_profile.argtypes = [vp, i32]
        lib.dip_sim_last_profile.argtypes = [vp, vp, vp]
        lib.dip_sim_last_retries.argtypes = [vp, vp, vp]
        lib.dip_sim_get_info.argtypes = [vp, ctypes.POINTER(Info)]
        lib.dip_sim_evaluate.argtypes = [vp, ctypes.POINTER(Costs), vp, i64, vp, vp, vp, vp, vp]
        lib.dip_sim_evaluate_static.argtypes = [vp, vp, i64, vp, vp, vp, vp, vp]
        lib.dip_sim_argmin.argtypes = [vp, vp, vp, i64, i64, vp, vp]
        lib.dip_sim_configure_greedy.argtypes = [vp, i32, vp]
        lib.dip_sim_set_greedy_inbox.argtypes = [vp, i32]
        lib.dip_sim_greedy.argtypes = [vp, ctypes.POINTER(Costs), vp, i64, vp, vp, vp, vp, vp, vp]
        lib.dip_sim_configure_rollouts.argtypes = [vp, i32, vp]
        lib.dip_cost_tables.argtypes = [ctypes.POINTER(OpTable), i64, vp, vp, vp]
        lib.dip_sim_configure_memopt.argtypes = [vp, vp, vp, vp, i32, i32, i32]
        lib.dip_sim_memopt.argtypes = [vp, vp, i64, vp, vp, vp, vp, vp]
        lib.dip_sim_evaluate_selected.argtypes = [vp, vp, vp, i64, vp, vp, vp, vp, vp]
        lib.dip_sim_rollouts.argtypes = [vp, vp, i32, i64, ctypes.c_uint64, ctypes.c_uint64,
                                         vp, vp, vp, vp, vp]
        lib.dip_sim_rollouts_batch.argtypes = [vp, i32, vp, vp, i64, ctypes.c_uint64,
                                               ctypes.c_uint64, vp, vp, vp, vp, vp]
        lib.dip_sim_destroy.argtypes = [vp]
        lib.dip_sim_destroy.restype = None
        lib.dip_sim_strerror.argtypes = [ctypes.c_int]
        lib.dip_sim_strerror.restype = ctypes.c_char_p
        for name in ("dip_sim_check_topology", "dip_sim_check_costs", "dip_sim_create",
                     "dip_sim_configure", "dip_sim_configure_pool", "dip_sim_configure_check",
                     "dip_sim_get_info",
                     "dip_sim_evaluate", "dip_sim_evaluate_static",
                     "dip_sim_profile", "dip_sim_last_profile",
                     "dip_sim_last_retries",
                     "dip_sim_argmin", "dip_sim_configure_greedy", "dip_sim_set_greedy_inbox", "dip_sim_greedy",
                     "dip_sim_configure_rollouts", "dip_sim_rollouts", "dip_sim_rollouts_batch",
           "dip_cost_tables",
                     "dip_sim_configure_memopt", "dip_sim_memopt", "dip_sim_evaluate_selected"):
            getattr(lib, name).restype = ctypes.c_int
        _lib = lib
    return _lib


def strerror(code: int) -> str:
    return load().dip_sim_strerror(int(code)).decode()


def _check(code: int, where: str):
    if code != OK:
        raise DipSimError(code, where)


# ------------------------------------------------------------ host marshalling

class HostTopology:
    """Contiguous host copies of an instance's topology plus the ctypes view."""

    def __init__(self, n_ranks, n_ops, pred_ptr, pred_op, op_kind, op_slot, n_slots,
                 mem_cap, cand_stride):
        self.keep = dict(
            n_ops=np.ascontiguousarray(n_ops, np.int32),
            pred_ptr=np.ascontiguousarray(pred_ptr, np.int32),
            pred_op=np.ascontiguousarray(pred_op, np.int32) if len(pred_op) else np.zeros(1, np.int32),
            op_kind=np.ascontiguousarray(op_kind, np.uint8),
            op_slot=np.ascontiguousarray(op_slot, np.int32),
            mem_cap=np.ascontiguousarray(mem_cap, np.int32))
        k = self.keep
        self.c = Topology(int(n_ranks), k["n_ops"].ctypes.data, k["pred_ptr"].ctypes.data,
                          k["pred_op"].ctypes.data, k["op_kind"].ctypes.data,
                          k["op_slot"].ctypes.data, int(n_slots), k["mem_cap"].ctypes.data,
                          int(cand_stride))

    @classmethod
    def of(cls, prob):
        return cls(prob.n_ranks, prob.n_ops, prob.pred_ptr, prob.pred_op, prob.op_kind,
                   prob.op_slot, prob.n_slots, prob.mem_cap, prob.stride)


class HostCosts:
    def __init__(self, op_cost, edge_comm, slot_act):
        self.keep = [np.ascontiguousarray(op_cost, np.int32),
                     np.ascontiguousarray(edge_comm, np.int32) if len(edge_comm) else np.zeros(1, np.int32),
                     np.ascontiguousarray(slot_act, np.int32) if len(slot_act) else np.zeros(1, np.int32)]
        self.c = Costs(*(a.ctypes.data for a in self.keep))

    @classmethod
    def of(cls, prob):
        return cls(prob.op_cost, prob.edge_comm, prob.slot_act)


# ------------------------------------------------------------ ABI, same names

def check_topology(topo: HostTopology) -> int:
    return load().dip_sim_check_topology(ctypes.byref(topo.c))


def check_costs(topo: HostTopology, costs: HostCosts) -> int:
    return load().dip_sim_check_costs(ctypes.byref(topo.c), ctypes.byref(costs.c))


def create(topo: HostTopology) -> ctypes.c_void_p:
    h = ctypes.c_void_p()
    _check(load().dip_sim_create(ctypes.byref(topo.c), ctypes.byref(h)), "dip_sim_create")
    return h


def configure(h, variant: int = 0, waves_per_block: int = 0) -> int:
    return load().dip_sim_configure(h, int(variant), int(waves_per_block))


def configure_pool(h, slots_per_rank: int = 0) -> int:
    return load().dip_sim_configure_pool(h, int(slots_per_rank))


def configure_check(h, mode: int = 0) -> int:
    return load().dip_sim_configure_check(h, int(mode))


def profile(h, enable: bool = True) -> int:
    return load().dip_sim_profile(h, int(bool(enable)))


def last_profile(h) -> list:
    """Kernel times (ms) of the last evaluate, in launch order."""
    buf = (ctypes.c_float * PROFILE_MAX)()
    n = ctypes.c_int32(0)
    _check(load().dip_sim_last_profile(h, buf, ctypes.byref(n)), "dip_sim_last_profile")
    return [float(buf[i]) for i in range(n.value)]


def last_retries(h) -> tuple:
    """(candidates whose pools filled in the first simulation pass, those left
    to the general kernel) of the last evaluate; waits for its stream."""
    a, b = ctypes.c_int64(0), ctypes.c_int64(0)
    _check(load().dip_sim_last_retries(h, ctypes.byref(a), ctypes.byref(b)), "dip_sim_last_retries")
    return int(a.value), int(b.value)


def get_info(h) -> dict:
    info = Info()
    _check(load().dip_sim_get_info(h, ctypes.byref(info)), "dip_sim_get_info")
    return info.as_dict()


def _stream_ptr(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def evaluate(h, costs, orders, n_cand, out_makespan, out_bubble, out_peakmem, out_flags,
             stream=None) -> None:
    """Device tensors in, device tensors out; enqueued on ``stream`` (torch's
    current stream by default)."""
    rc = load().dip_sim_evaluate(
        h, ctypes.byref(costs.c) if costs is not None else None, orders.data_ptr(),
        int(n_cand), out_makespan.data_ptr(), out_bubble.data_ptr(),
        out_peakmem.data_ptr(), out_flags.data_ptr(), _stream_ptr(stream))
    _check(rc, "dip_sim_evaluate")


def evaluate_static(h, orders, n_cand, out_makespan, out_bubble, out_peakmem, out_flags,
                    stream=None) -> int:
    """The allocation-free evaluate (costs of an earlier evaluate call);
    returns the ABI code, so that callers can see DIP_E_CAPACITY."""
    return load().dip_sim_evaluate_static(
        h, orders.data_ptr(), int(n_cand), out_makespan.data_ptr(), out_bubble.data_ptr(),
        out_peakmem.data_ptr(), out_flags.data_ptr(), _stream_ptr(stream))


def argmin(h, makespan, flags, n_cand, index_base, inout_best_key, stream=None) -> None:
    rc = load().dip_sim_argmin(h, makespan.data_ptr(), flags.data_ptr(), int(n_cand),
                               int(index_base), inout_best_key.data_ptr(),
                               _stream_ptr(stream))
    _check(rc, "dip_sim_argmin")


def configure_greedy(h, n_groups: int, op_group) -> int:
    """``op_group``: host int32 [N]; returns the ABI code."""
    g = np.ascontiguousarray(op_group, np.int32)
    return load().dip_sim_configure_greedy(h, int(n_groups), g.ctypes.data)


def set_greedy_inbox(h, k: int) -> int:
    """Fix the first launch's inbox size (power of two, 1..256); 0: adaptive."""
    return load().dip_sim_set_greedy_inbox(h, int(k))


def greedy(h, costs, prio, n_cand, out_orders, out_makespan, out_bubble, out_peakmem,
           out_flags, stream=None) -> None:
    """Priorities (device int32 [n, G]) in, orders and scores out (device);
    ``out_orders`` may be None."""
    rc = load().dip_sim_greedy(
        h, ctypes.byref(costs.c) if costs is not None else None, prio.data_ptr(), int(n_cand),
        out_orders.data_ptr() if out_orders is not None else None, out_makespan.data_ptr(),
        out_bubble.data_ptr(), out_peakmem.data_ptr(), out_flags.data_ptr(),
        _stream_ptr(stream))
    _check(rc, "dip_sim_greedy")


def configure_rollouts(h, n_classes: int, group_class) -> int:
    c = np.ascontiguousarray(group_class, np.int32)
    return load().dip_sim_configure_rollouts(h, int(n_classes), c.ctypes.data)


def rollouts(h, prefix, n_rollouts, seed, draw, out_prio, out_makespan, out_flags,
             inout_best_key, stream=None) -> None:
    """``prefix``: host sequence of classes; outputs are device tensors."""
    pre = np.ascontiguousarray(prefix, np.int32)
    rc = load().dip_sim_rollouts(h, pre.ctypes.data if pre.size else None, int(pre.size),
                                 int(n_rollouts), int(seed) & ((1 << 64) - 1),
                                 int(draw) & ((1 << 64) - 1), out_prio.data_ptr(),
                                 out_makespan.data_ptr(), out_flags.data_ptr(),
                                 inout_best_key.data_ptr(), _stream_ptr(stream))
    _check(rc, "dip_sim_rollouts")


def rollouts_batch(h, prefixes, per_leaf, seed, draw_base, out_prio, out_makespan, out_flags,
                   inout_keys, stream=None) -> None:
    """``prefixes``: host list of class sequences, one per leaf; leaf l's
    rollouts are rows l*per_leaf.. of the device outputs, drawn with
    draw_base + l; inout_keys: device int64 [len(prefixes)]."""
    depths = np.ascontiguousarray([len(p) for p in prefixes], np.int32)
    flat = np.ascontiguousarray([c for p in prefixes for c in p], np.int32)
    rc = load().dip_sim_rollouts_batch(
        h, int(depths.size), depths.ctypes.data, flat.ctypes.data if flat.size else None,
        int(per_leaf), int(seed) & ((1 << 64) - 1), int(draw_base) & ((1 << 64) - 1),
        out_prio.data_ptr(), out_makespan.data_ptr(), out_flags.data_ptr(), inout_keys.data_ptr(),
        _stream_ptr(stream))
    _check(rc, "dip_sim_rollouts_batch")


class DeviceOpTable:
    """Device copies of an operator table (workloads.operators.OperatorTable
    or any object with item_ptr, n_fop, n_mem, n_net, kind)."""

    def __init__(self, table, n_kinds: int, device="cuda"):
        import torch
        self.t = dict(
            item_ptr=torch.from_numpy(np.ascontiguousarray(table.item_ptr, np.int32)).to(device),
            n_fop=torch.from_numpy(np.ascontiguousarray(table.n_fop, np.float64)).to(device),
            n_mem=torch.from_numpy(np.ascontiguousarray(table.n_mem, np.float64)).to(device),
            n_net=torch.from_numpy(np.ascontiguousarray(table.n_net, np.float64)).to(device),
            kind=torch.from_numpy(np.ascontiguousarray(table.kind, np.uint8)).to(device))
        d = self.t
        self.n_items = int(d["item_ptr"].numel()) - 1
        self.c = OpTable(self.n_items, int(d["kind"].numel()), int(n_kinds),
                         d["item_ptr"].data_ptr(), d["n_fop"].data_ptr(), d["n_mem"].data_ptr(),
                         d["n_net"].data_ptr(), d["kind"].data_ptr())


def cost_tables(table: DeviceOpTable, coef, out, stream=None) -> None:
    """coef: device float64 [n_configs][n_kinds][3]; out: device int32 [n_configs][n_items]."""
    rc = load().dip_cost_tables(ctypes.byref(table.c), int(coef.shape[0]), coef.data_ptr(),
                                out.data_ptr(), _stream_ptr(stream))
    _check(rc, "dip_cost_tables")


def configure_memopt(h, slot_layers, layer_time, layer_mem, n_candidates: int,
                     bb_nodes: int = 0) -> int:
    """Host arrays: slot_layers int32 [n_slots+1], layer_time / layer_mem int64
    [layers][n_strategies]; bb_nodes 0: the library's default."""
    sl = np.ascontiguousarray(slot_layers, np.int32)
    lt = np.ascontiguousarray(layer_time, np.int64)
    lm = np.ascontiguousarray(layer_mem, np.int64)
    ns = lt.shape[1] if lt.ndim == 2 else 1
    return load().dip_sim_configure_memopt(h, sl.ctypes.data, lt.ctypes.data, lm.ctypes.data,
                                           int(ns), int(n_candidates), int(bb_nodes))


def memopt(h, orders, n_cand, out_time, out_peak, out_status, out_choice=None,
           stream=None) -> None:
    rc = load().dip_sim_memopt(h, orders.data_ptr(), int(n_cand), out_time.data_ptr(),
                               out_peak.data_ptr(), out_status.data_ptr(),
                               out_choice.data_ptr() if out_choice is not None else None,
                               _stream_ptr(stream))
    _check(rc, "dip_sim_memopt")


def evaluate_selected(h, orders, choice, n_cand, out_makespan, out_bubble, out_peakmem,
                      out_flags, stream=None) -> None:
    rc = load().dip_sim_evaluate_selected(h, orders.data_ptr(), choice.data_ptr(), int(n_cand),
                                          out_makespan.data_ptr(), out_bubble.data_ptr(),
                                          out_peakmem.data_ptr(), out_flags.data_ptr(),
                                          _stream_ptr(stream))
    _check(rc, "dip_sim_evaluate_selected")


def destroy(h) -> None:
    if h:
        load().dip_sim_destroy(h)


def decode_key(key: int):
    """(best global index, best makespan), or (-1, -1) when nothing was valid."""
    key = int(key) & NO_KEY
    if key == NO_KEY:
        return -1, -1
    return key & 0xFFFFFFFF, key >> 32


# ------------------------------------------------------------ convenience

class Sim:
    """Owns one handle; tensors are torch CUDA tensors."""

    def __init__(self, prob, costs=True):
        self.topo = HostTopology.of(prob)
        self.P = int(prob.n_ranks)
        self.stride = int(prob.stride)
        self.h = create(self.topo)
        self.costs = HostCosts.of(prob) if costs is True else costs
        self._costs_sent = False

    def close(self):
        if self.h:
            destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def configure(self, variant=0, waves_per_block=0) -> int:
        return configure(self.h, variant, waves_per_block)

    def configure_pool(self, slots_per_rank=0) -> int:
        return configure_pool(self.h, slots_per_rank)

    def configure_check(self, mode=0) -> int:
        return configure_check(self.h, mode)

    @property
    def info(self) -> dict:
        return get_info(self.h)

    def outputs(self, n, device="cuda"):
        import torch
        return (torch.empty(n, dtype=torch.int32, device=device),
                torch.empty((n, self.P), dtype=torch.int32, device=device),
                torch.empty((n, self.P), dtype=torch.int32, device=device),
                torch.empty(n, dtype=torch.uint8, device=device))

    def evaluate(self, orders, out=None, stream=None, resend_costs=False):
        n = int(orders.shape[0])
        assert orders.dtype.itemsize == 2 and orders.is_contiguous()
        assert orders.shape[1] == self.stride
        out = self.outputs(n, orders.device) if out is None else out
        send = self.costs if (resend_costs or not self._costs_sent) else None
        evaluate(self.h, send, orders, n, *out, stream=stream)
        self._costs_sent = True
        return out

    def evaluate_static(self, orders, out=None, stream=None) -> int:
        """The allocation-free evaluate; the costs must have gone with an
        earlier evaluate.  Returns the ABI code."""
        n = int(orders.shape[0])
        assert orders.dtype.itemsize == 2 and orders.is_contiguous()
        assert orders.shape[1] == self.stride
        out = self.outputs(n, orders.device) if out is None else out
        return evaluate_static(self.h, orders, n, *out, stream=stream), out

    def configure_greedy(self, n_groups, op_group) -> int:
        rc = configure_greedy(self.h, n_groups, op_group)
        if rc == OK:
            self._greedy_costs = False
        return rc

    def set_greedy_inbox(self, k) -> int:
        return set_greedy_inbox(self.h, k)

    def greedy(self, prio, out=None, orders=True, stream=None):
        """Interleave every priority row; returns (orders or None, outputs)."""
        import torch
        n = int(prio.shape[0])
        assert prio.dtype == torch.int32 and prio.is_contiguous()
        out = self.outputs(n, prio.device) if out is None else out
        ords = torch.empty((n, self.stride), dtype=torch.int16, device=prio.device) if orders else None
        send = self.costs if not getattr(self, "_greedy_costs", False) else None
        greedy(self.h, send, prio, n, ords, *out, stream=stream)
        self._greedy_costs = True
        self._costs_sent = True
        return ords, out

    def argmin(self, makespan, flags, index_base=0, key=None, stream=None):
        import torch
        if key is None:
            key = torch.full((1,), -1, dtype=torch.int64, device=makespan.device)
        argmin(self.h, makespan, flags, int(makespan.shape[0]), index_base, key, stream=stream)
        return key
