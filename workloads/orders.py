"""Candidate orders: ctypes front end of ``gen.c`` and small order helpers.

Orders are int16 arrays ``[n_cand, stride]``; inside a candidate, rank 0's
section comes first, then rank 1's, with no gaps, and entries past the last
rank are padding.  Each section is a permutation of the rank-local op ids.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from .configs import WorkloadConfig, get
from .instance import KIND_B, KIND_F, Problem

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gen.c")
# DIPSIM_GEN_LIB names another build of the same sources (the sanitizer test loads
# one built with -fsanitize=address,undefined); it is then used as it is
_LIB = os.environ.get("DIPSIM_GEN_LIB") or os.path.join(_HERE, "libdipgen.so")

MODE_1F1B = 0
MODE_LIST = 1
PURPOSE_CAND = 2
PURPOSE_POOL = 3


def build(force: bool = True) -> str:
    if os.environ.get("DIPSIM_GEN_LIB"):
        return _LIB
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-shared", "-fPIC",
                               "-pthread", "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


class _Topo(ctypes.Structure):
    _fields_ = [("n_ranks", ctypes.c_int32), ("n_mb", ctypes.c_int32),
                ("n_lanes", ctypes.c_int32),
                ("rank_off", ctypes.c_void_p), ("pred_ptr", ctypes.c_void_p),
                ("succ_ptr", ctypes.c_void_p), ("succ_op", ctypes.c_void_p),
                ("op_kind", ctypes.c_void_p), ("op_mb", ctypes.c_void_p),
                ("op_rank", ctypes.c_void_p), ("rank_first_lane", ctypes.c_void_p)]


class _Recipe(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("max_swaps", ctypes.c_int32),
                ("pool", ctypes.c_int32), ("limit_jitter", ctypes.c_int32),
                ("seed", ctypes.c_uint64), ("cid", ctypes.c_uint64),
                ("pool_orders", ctypes.c_void_p), ("stride", ctypes.c_int64)]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        lib.dipgen_orders.restype = ctypes.c_int
        lib.dipgen_orders.argtypes = [ctypes.POINTER(_Topo), ctypes.POINTER(_Recipe),
                                      ctypes.c_int32, ctypes.c_int64, ctypes.c_int64,
                                      ctypes.c_void_p, ctypes.c_int32]
        lib.dipgen_draw.restype = ctypes.c_uint64
        lib.dipgen_draw.argtypes = [ctypes.c_uint64] * 4 + [ctypes.c_int64]
        _lib = lib
    return _lib


def draw(seed, cid, purpose, index, k) -> int:
    return int(_load().dipgen_draw(seed, cid, purpose, index, k))


def default_threads() -> int:
    n = os.cpu_count() or 1
    return max(1, min(n, 16))


class OrderGenerator:
    """Deterministic candidate orders for one compiled instance."""

    def __init__(self, prob: Problem, mode: int, max_swaps: int = 0, pool: int = 0,
                 seed: int = 0, cid: int = 0, limit_jitter: int = 2):
        self.prob = prob
        P = prob.n_ranks
        N = prob.n_total
        pred_ptr = prob.pred_ptr.astype(np.int32)
        counts = np.zeros(N, np.int64)
        np.add.at(counts, prob.pred_op, 1)
        succ_ptr = np.zeros(N + 1, np.int32)
        succ_ptr[1:] = np.cumsum(counts)
        succ_op = np.zeros(max(1, prob.n_edges), np.int32)
        fill = succ_ptr[:-1].copy()
        for g in range(N):
            for e in range(pred_ptr[g], pred_ptr[g + 1]):
                p = prob.pred_op[e]
                succ_op[fill[p]] = g
                fill[p] += 1
        op_rank = np.repeat(np.arange(P, dtype=np.int32),
                            np.diff(prob.rank_off).astype(np.int64))
        rank_first_lane = np.arange(P, dtype=np.int32)
        n_mb = int(prob.op_mb.max()) + 1 if N else 1
        self._arrays = dict(
            rank_off=np.ascontiguousarray(prob.rank_off, np.int64),
            pred_ptr=np.ascontiguousarray(pred_ptr), succ_ptr=succ_ptr, succ_op=succ_op,
            op_kind=np.ascontiguousarray(prob.op_kind, np.uint8),
            op_mb=np.ascontiguousarray(prob.op_mb, np.int32), op_rank=op_rank,
            rank_first_lane=rank_first_lane)
        a = self._arrays
        self._topo = _Topo(P, n_mb, int(prob.op_lane.max()) + 1 if N else P,
                           *(a[k].ctypes.data for k in
                             ("rank_off", "pred_ptr", "succ_ptr", "succ_op",
                              "op_kind", "op_mb", "op_rank", "rank_first_lane")))
        self.mode, self.max_swaps, self.pool = mode, max_swaps, pool
        self.seed, self.cid, self.jitter = seed, cid, limit_jitter
        self._pool_orders = None
        if pool > 0:
            self._pool_orders = self._run(PURPOSE_POOL, 0, pool, None)

    def _recipe(self):
        po = self._pool_orders
        return _Recipe(self.mode, self.max_swaps, self.pool, self.jitter,
                       self.seed, self.cid, po.ctypes.data if po is not None else None,
                       self.prob.stride)

    def _run(self, purpose, first, n, threads):
        out = np.zeros((n, self.prob.stride), np.int16)
        rc = _load().dipgen_orders(ctypes.byref(self._topo), ctypes.byref(self._recipe()),
                                   purpose, first, n, out.ctypes.data,
                                   threads or default_threads())
        if rc != 0:
            raise RuntimeError(f"order generation failed ({rc})")
        return out

    def generate(self, first: int, n: int, threads: int | None = None,
                 out: np.ndarray | None = None) -> np.ndarray:
        """Candidates ``first .. first+n-1`` as int16 ``[n, stride]``."""
        if out is not None:
            assert out.shape == (n, self.prob.stride) and out.dtype == np.int16
            assert out.flags.c_contiguous
            rc = _load().dipgen_orders(ctypes.byref(self._topo), ctypes.byref(self._recipe()),
                                       PURPOSE_CAND, first, n, out.ctypes.data,
                                       threads or default_threads())
            if rc != 0:
                raise RuntimeError(f"order generation failed ({rc})")
            return out
        return self._run(PURPOSE_CAND, first, n, threads)


def generator_for(prob: Problem, cfg: WorkloadConfig | int) -> OrderGenerator:
    if not isinstance(cfg, WorkloadConfig):
        cfg = get(cfg)
    mode = MODE_1F1B if cfg.order_mode == "1f1b" else MODE_LIST
    return OrderGenerator(prob, mode, cfg.max_swaps, cfg.pool, cfg.seed, cfg.cid)


# --------------------------------------------------------------------------
# Plain order constructors for hand-built cases (single segment, v = 1).
# --------------------------------------------------------------------------

def op_id(m: int, kind: int) -> int:
    """Rank-local id of microbatch m's F or B on a one-lane-per-rank pipeline."""
    return 2 * m + kind


def gpipe_rank(M: int) -> list:
    return [op_id(m, KIND_F) for m in range(M)] + [op_id(m, KIND_B) for m in range(M)]


def one_f_one_b_rank(S: int, s: int, M: int) -> list:
    w = min(S - s - 1, M)
    o = [op_id(m, KIND_F) for m in range(w)]
    for i in range(M - w):
        o += [op_id(w + i, KIND_F), op_id(i, KIND_B)]
    o += [op_id(m, KIND_B) for m in range(M - w, M)]
    return o


def pack(prob: Problem, per_rank_orders: list) -> np.ndarray:
    """One candidate from per-rank lists of rank-local ids."""
    row = np.zeros(prob.stride, np.int16)
    for r, o in enumerate(per_rank_orders):
        a, b = int(prob.rank_off[r]), int(prob.rank_off[r + 1])
        assert len(o) == b - a, (r, len(o), b - a)
        row[a:b] = np.asarray(o, np.int16)
    return row


def unpack(prob: Problem, row: np.ndarray) -> list:
    return [list(map(int, row[int(prob.rank_off[r]):int(prob.rank_off[r + 1])]))
            for r in range(prob.n_ranks)]
