"""Independent checker: Kahn topological sort + longest path.

Builds the schedule graph straight from the high-level instance (lanes,
segments, units) -- not from the compiled CSR -- adds one edge between
consecutive ops of every rank's order, and evaluates the plain definition:
a cycle means deadlock; otherwise each op starts at the longest weighted path
into it.  Pure Python, for tiny instances only.  Shares no code with the
oracle or with the instance compiler.
"""
from __future__ import annotations

from collections import deque


def ops_of_rank(inst, r):
    """Rank-local op list in the ABI's id order: lanes ascending, units
    ascending, forward before backward."""
    out = []
    for lane in range(r, inst.L, inst.P):
        seg = next(s for s in range(len(inst.seg_lo))
                   if inst.seg_lo[s] <= lane <= inst.seg_hi[s])
        units = sorted(u for u in range(len(inst.unit_seg)) if int(inst.unit_seg[u]) == seg)
        for u in units:
            out.append(("F", u, lane))
            out.append(("B", u, lane))
    return out


def data_edges(inst):
    """(src, dst, latency) for every dependency, written from the readings:
    chain inside a segment, loss turnaround on the final lane, all-to-all
    joins between consecutive segments of one microbatch."""
    P = inst.P
    nseg = len(inst.seg_lo)
    U = len(inst.unit_seg)

    def seg_units(s, mb):
        return [u for u in range(U) if int(inst.unit_seg[u]) == s and int(inst.unit_mb[u]) == mb]

    def lat(a_lane, b_lane, value):
        return 0 if a_lane % P == b_lane % P else int(value)

    edges = []
    for u in range(U):
        s = int(inst.unit_seg[u])
        mb = int(inst.unit_mb[u])
        lo, hi = inst.seg_lo[s], inst.seg_hi[s]
        for lane in range(lo + 1, hi + 1):
            edges.append((("F", u, lane - 1), ("F", u, lane), lat(lane - 1, lane, inst.unit_comm[u])))
            edges.append((("B", u, lane), ("B", u, lane - 1), lat(lane, lane - 1, inst.unit_comm[u])))
        if s == nseg - 1:
            edges.append((("F", u, hi), ("B", u, hi), 0))
        else:
            nxt = seg_units(s + 1, mb)
            for w in nxt:
                split_down = len(nxt) > 1
                c = inst.unit_comm[w] if split_down else inst.unit_comm[u]
                lane_dn = inst.seg_lo[s + 1]
                edges.append((("F", u, hi), ("F", w, lane_dn), lat(hi, lane_dn, c)))
                edges.append((("B", w, lane_dn), ("B", u, hi), lat(lane_dn, hi, c)))
    return edges


def op_cost(inst, op):
    kind, u, lane = op
    return int(inst.fcost[lane, u] if kind == "F" else inst.bcost[lane, u])


def longest_path(inst, per_rank_orders=None):
    """Returns dict(deadlock, makespan, start, end, busy) for one candidate.
    ``per_rank_orders``: list over ranks of rank-local ids; None = data DAG only."""
    nodes = [op for r in range(inst.P) for op in ops_of_rank(inst, r)]
    succ = {n: [] for n in nodes}
    indeg = {n: 0 for n in nodes}
    for (a, b, w) in data_edges(inst):
        succ[a].append((b, w))
        indeg[b] += 1
    if per_rank_orders is not None:
        for r, order in enumerate(per_rank_orders):
            ops = ops_of_rank(inst, r)
            seq = [ops[i] for i in order]
            for a, b in zip(seq, seq[1:]):
                succ[a].append((b, 0))
                indeg[b] += 1
    start = {n: 0 for n in nodes}
    q = deque(n for n in nodes if indeg[n] == 0)
    seen = 0
    end = {}
    while q:
        n = q.popleft()
        seen += 1
        end[n] = start[n] + op_cost(inst, n)
        for (m, w) in succ[n]:
            start[m] = max(start[m], end[n] + w)
            indeg[m] -= 1
            if indeg[m] == 0:
                q.append(m)
    busy = [sum(op_cost(inst, op) for op in ops_of_rank(inst, r)) for r in range(inst.P)]
    if seen < len(nodes):
        return dict(deadlock=True, makespan=-1, start=None, end=None, busy=busy)
    return dict(deadlock=False, makespan=max(end.values()) if end else 0,
                start=start, end=end, busy=busy)
