"""Per-layer memory strategies of the stage pairs, for Sec. 5.3's memory
optimisation (DIP, arXiv 2504.14145).

A stage pair is a forward and its backward (one activation slot).  It covers
its lane's L layers of the module; each layer can keep its activations,
recompute the attention part in the backward (selective), or recompute the
whole layer (full).  Per layer, with f, b, a the pair's forward time,
backward time and activation split evenly over the layers (remainders to the
first layers):
    keep        time f + b              memory a
    selective   time f + b + ceil(f/3)  memory ceil(a/2)
    full        time 2 f + b            memory ceil(a/8)
Integers throughout (microseconds, memory units).  This module only builds
the tables; choosing among them is the method's.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .instance import KIND_B, Problem

N_STRATEGIES = 3


@dataclass
class StrategyTable:
    slot_layers: np.ndarray   # int32 [n_slots + 1] CSR offsets of each pair's layers
    time: np.ndarray          # int64 [layers, 3]
    mem: np.ndarray           # int64 [layers, 3]
    slot_rank: np.ndarray     # int32 [n_slots]
    slot_f: np.ndarray        # int32 [n_slots] global op index of the forward
    slot_b: np.ndarray        # int32 [n_slots] global op index of the backward


def _split(x: int, L: int):
    q, r = divmod(int(x), L)
    return [q + (1 if i < r else 0) for i in range(L)]


def strategy_table(prob: Problem) -> StrategyTable:
    inst = prob.inst
    from .configs import CONFIGS
    from .operators import SEGMENT_MODELS, LLAMA3_8B
    names = None
    if inst is not None:
        for cfg in CONFIGS.values():
            if cfg.name == inst.name:
                names = [s.name for s in cfg.segments]
    n = prob.n_slots
    f_of = np.full(n, -1, np.int64)
    b_of = np.full(n, -1, np.int64)
    for o in range(prob.n_total):
        if prob.op_kind[o] == KIND_B:
            b_of[prob.op_slot[o]] = o
        else:
            f_of[prob.op_slot[o]] = o
    rank = np.repeat(np.arange(prob.n_ranks), np.diff(prob.rank_off))
    ptr, t_rows, m_rows = [0], [], []
    for s in range(n):
        f, b = int(f_of[s]), int(b_of[s])
        L = 1
        if inst is not None and names is not None:
            seg = int(inst.unit_seg[prob.op_unit[f]])
            spec = SEGMENT_MODELS.get(names[seg], LLAMA3_8B)
            lanes = inst.seg_hi[seg] - inst.seg_lo[seg] + 1
            L = -(-spec.layers // lanes)
        fs = _split(prob.op_cost[f], L)
        bs = _split(prob.op_cost[b], L)
        acts = _split(prob.slot_act[s], L)
        for fl, bl, al in zip(fs, bs, acts):
            t_rows.append([fl + bl, fl + bl + -(-fl // 3), 2 * fl + bl])
            m_rows.append([al, -(-al // 2), -(-al // 8)])
        ptr.append(len(t_rows))
    return StrategyTable(np.array(ptr, np.int32), np.array(t_rows, np.int64).reshape(-1, 3),
                         np.array(m_rows, np.int64).reshape(-1, 3),
                         rank[f_of].astype(np.int32), f_of.astype(np.int32),
                         b_of.astype(np.int32))
