"""Priority groups and seeded priority vectors for the stage interleaving.

A priority group is a pipeline segment in the sense of DIP's schedule search
(Sec. 5.1): the forward or the backward of one sub-microbatch through a run of
at most P consecutive lanes of one modality module, i.e. one pass around the
physical ranks, so a group holds at most one stage per rank.  A candidate
gives one int32 priority per group (larger first).

The vectors drawn here stand in for MCTS rollouts (Sec. 5.1): each rollout
completes a segment sequence at random and gives the segment at position i of
n the priority n - i.  Segments of one modality module within one microbatch
(its pieces) share a priority, the search-space reduction of Sec. 5.1; the
interleaving orders such ties by group index.  This module draws inputs only;
it schedules nothing.
"""
from __future__ import annotations

import numpy as np

from .instance import Problem


def priority_groups(prob: Problem):
    """(op_group int32 [N], n_groups, group_class int32 [n_groups]).

    Groups are numbered by (unit, kind, pass) ascending; a group's class is
    (microbatch, segment, kind, pass), shared by the pieces of one module."""
    inst = prob.inst
    if inst is None:
        raise ValueError("priority groups need the high-level instance")
    P = inst.P
    seg = inst.unit_seg[prob.op_unit]
    lo = np.asarray(inst.seg_lo, np.int64)[seg]
    pas = (prob.op_lane.astype(np.int64) - lo) // P
    kind = prob.op_kind.astype(np.int64)
    n_pass = int(pas.max()) + 1 if pas.size else 1
    key = (prob.op_unit.astype(np.int64) * 2 + kind) * n_pass + pas
    uniq, op_group = np.unique(key, return_inverse=True)
    g_unit = uniq // (2 * n_pass)
    g_kind = (uniq // n_pass) % 2
    g_pass = uniq % n_pass
    n_seg = len(inst.seg_lo)
    ckey = ((inst.unit_mb[g_unit] * n_seg + inst.unit_seg[g_unit]) * 2 + g_kind) * n_pass + g_pass
    _, g_class = np.unique(ckey, return_inverse=True)
    return op_group.astype(np.int32), int(uniq.size), g_class.astype(np.int32)


def rollout_priorities(group_class: np.ndarray, n: int, seed: int, first: int = 0) -> np.ndarray:
    """int32 [n, n_groups]: candidate i (global index first + i) ranks the
    classes by a uniform random permutation drawn from (seed, index)."""
    group_class = np.asarray(group_class, np.int64)
    n_cls = int(group_class.max()) + 1 if group_class.size else 0
    out = np.empty((n, group_class.size), np.int32)
    for i in range(n):
        rng = np.random.default_rng(np.random.SeedSequence([seed, 77, first + i]))
        pos = rng.permutation(n_cls)          # pos[c] = position of class c
        out[i] = (n_cls - pos[group_class]).astype(np.int32)
    return out


def fifo_priorities(prob: Problem, group_class: np.ndarray, op_group: np.ndarray) -> np.ndarray:
    """int32 [n_groups]: earlier microbatches first, forward and backward
    alike (a first-in first-out base order)."""
    n_groups = int(np.max(op_group)) + 1 if len(op_group) else 0
    mb = np.zeros(n_groups, np.int64)
    mb[op_group] = prob.op_mb
    return (int(mb.max()) + 1 - mb).astype(np.int32) if n_groups else np.zeros(0, np.int32)


def expansion_draw(seed: int, iteration: int, n_untried: int) -> int:
    """Index (into the ascending list of a node's untried classes) of the child
    an MCTS expansion adds at this iteration: uniform, drawn from
    (seed, iteration)."""
    if n_untried <= 0:
        raise ValueError("nothing to expand")
    rng = np.random.default_rng(np.random.SeedSequence([seed, 93, iteration]))
    return int(rng.integers(n_untried))
