"""CPU oracle of DIP's per-layer memory optimisation (arXiv 2504.14145,
Sec. 5.3).

TEST INFRASTRUCTURE ONLY: the test suite and the benchmark's CPU-baseline leg
are its only callers.  Plain Python.

Offline candidates (Sec. 5.3, "Offline Candidate Generation"), per stage pair:
  the exact (time, memory) Pareto front of its layers' strategy choices,
  built layer by layer (every combination of the front so far with the
  layer's strategies, dominated points dropped); then (1) its fastest point
  (least time, least memory among those), (2) its leanest point (least
  memory, least time among those), and (3) with the memory range [lo, hi]
  between them cut into S-2 equal buckets at edges lo + floor((hi-lo) k/(S-2)),
  for each bucket the multiple-choice knapsack answer for its upper edge:
  the least time (then least memory) over all choices whose memory is at
  most the edge; equal points once; listed by time ascending (memory then
  strictly descends).

Per-rank selection (Sec. 5.3, "ILP Formulation"): each stage pair i on a rank
takes one candidate; total latency is minimised subject to the memory at
every forward start staying within the rank's cap.  A pair is live at pair
k's forward start when its forward comes no later and its backward no
earlier in the rank's order (on one rank the order gives the timestamps'
order, [s_i <= s_k <= t_i]).  The paper warm-starts an ILP solver with a
greedy solution and accepts a small gap; this build computes the greedy
solution:
  every pair on its fastest candidate; then while the most loaded checkpoint
  (lowest index among equal loads) exceeds the cap, among its live pairs that
  can move to their next (leaner, slower) candidate take the one with the
  least added time per freed memory unit (compared as dt_a * dm_b < dt_b *
  dm_a; lowest pair index on ties) and move it; stop when no live pair can
  move (infeasible).
``exact`` solves the same problem by enumeration, for small cases.
"""
from __future__ import annotations

import itertools


def pareto(layers):
    """layers: [[(time, mem) per strategy] per layer] -> front sorted by memory
    ascending (time strictly descending)."""
    front = [(0, 0)]
    for opts in layers:
        pts = sorted(set((t + a, m + b) for (t, m) in front for (a, b) in opts),
                     key=lambda p: (p[1], p[0]))
        front = []
        for t, m in pts:
            if not front or t < front[-1][0]:
                if front and front[-1][1] == m:
                    continue
                front.append((t, m))
    return front


def candidates(front, S):
    """The S-candidate rule on a Pareto front (memory ascending)."""
    lean = front[0]
    fast = front[-1]
    picks = [fast, lean]
    lo, hi = lean[1], fast[1]
    if S > 2:
        edges = [lo + ((hi - lo) * k) // (S - 2) for k in range(S - 1)]
        for k in range(1, S - 1):
            fit = [p for p in front if p[1] <= edges[k]]
            picks.append(min(fit, key=lambda p: (p[0], p[1])))
    out = sorted(set(picks), key=lambda p: (p[0], p[1]))
    return out


def pair_candidates(table, S):
    """Candidate lists of every stage pair of a workloads StrategyTable."""
    out = []
    for s in range(len(table.slot_layers) - 1):
        layers = [list(zip(table.time[l].tolist(), table.mem[l].tolist()))
                  for l in range(table.slot_layers[s], table.slot_layers[s + 1])]
        out.append(candidates(pareto(layers), S))
    return out


def live_sets(order_pos_f, order_pos_b):
    n = len(order_pos_f)
    return [[i for i in range(n) if order_pos_f[i] <= order_pos_f[k] <= order_pos_b[i]]
            for k in range(n)]


def greedy_select(cands, live, cap):
    """cands[i] = [(time, mem)] time ascending; live[k] = pairs live at k.
    Returns (choice list, total time, feasible, peak)."""
    n = len(cands)
    cur = [0] * n
    load = [sum(cands[i][0][1] for i in live[k]) for k in range(n)]
    feasible = True
    while cap >= 0 and n:
        k = max(range(n), key=lambda j: (load[j], -j))
        if load[k] <= cap:
            break
        best = -1
        for i in live[k]:
            if cur[i] + 1 < len(cands[i]):
                dt = cands[i][cur[i] + 1][0] - cands[i][cur[i]][0]
                dm = cands[i][cur[i]][1] - cands[i][cur[i] + 1][1]
                if best < 0 or dt * bdm < bdt * dm:
                    best, bdt, bdm = i, dt, dm
        if best < 0:
            feasible = False
            break
        cur[best] += 1
        for j in range(n):
            if best in live[j]:
                load[j] -= bdm
    total = sum(cands[i][cur[i]][0] for i in range(n))
    return cur, total, feasible, max(load) if n else 0


def exact(cands, live, cap):
    """Least total time over every choice meeting the cap; None if none does."""
    best = None
    for choice in itertools.product(*[range(len(c)) for c in cands]):
        if cap >= 0 and any(sum(cands[i][choice[i]][1] for i in live[k]) > cap
                            for k in range(len(cands))):
            continue
        t = sum(cands[i][choice[i]][0] for i in range(len(cands)))
        if best is None or t < best:
            best = t
    return best


def rank_problem(prob, table, cands, order, r):
    """The pairs of rank r (slot order), their candidates and live sets under
    one candidate schedule's order (int16 row of the simulator's layout)."""
    base = int(prob.rank_off[r])
    nr = int(prob.rank_off[r + 1]) - base
    pos = [0] * nr
    for p in range(nr):
        pos[int(order[base + p])] = p
    slots = [s for s in range(len(cands)) if table.slot_rank[s] == r]
    pf = [pos[int(table.slot_f[s]) - base] for s in slots]
    pb = [pos[int(table.slot_b[s]) - base] for s in slots]
    return slots, [cands[s] for s in slots], live_sets(pf, pb)


def optimise(prob, table, cands, orders, caps=None):
    """Per candidate schedule and rank: (total time, feasible, peak)."""
    P = prob.n_ranks
    caps = prob.mem_cap if caps is None else caps
    out = []
    for row in orders:
        per = []
        for r in range(P):
            _, c, live = rank_problem(prob, table, cands, row, r)
            _, total, ok, peak = greedy_select(c, live, int(caps[r]))
            per.append((total, ok, peak))
        out.append(per)
    return out
