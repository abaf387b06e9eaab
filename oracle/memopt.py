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

Per-rank selection (Sec. 5.3, "ILP Formulation" and "Optimizations"): each
stage pair i on a rank takes one candidate; total latency is minimised
subject to the memory at every forward start staying within the rank's cap.
A pair is live at pair k's forward start when its forward comes no later and
its backward no earlier in the rank's order (on one rank the order gives the
timestamps' order, [s_i <= s_k <= t_i]).  The paper warm-starts an ILP
solver with a greedy solution and stops it once the solution is within 5 %
of optimal.  This build's solver, ``select``:
  1. the greedy warm start: every pair on its fastest candidate; then while
     the most loaded checkpoint (lowest index among equal loads) exceeds the
     cap, among its live pairs that can move to their next (leaner, slower)
     candidate take the one with the least added time per freed memory unit
     (compared as dt_a * dm_b < dt_b * dm_a; lowest pair index on ties) and
     move it; no live pair can move: the cap cannot be met (every live pair
     of that checkpoint is on its leanest candidate);
  2. an improvement pass: pairs in index order each go back to the fastest
     candidate that keeps every checkpoint it is live at within the cap;
     passes repeat until one changes nothing;
  3. a depth-first branch and bound from that incumbent, pairs in the order
     of their forward starts (a pair's checkpoint then involves only pairs
     already placed), candidates fastest first; a placement is dropped when
     its checkpoint exceeds the cap, and a node is cut (with the slower
     candidates after it) when its placed time plus every unplaced pair's
     fastest time, times 1.05, reaches the incumbent.  A leaf below the
     incumbent replaces it.  When the search ends every cut subtree was
     worth at least incumbent / 1.05, so the incumbent is within 5 % of the
     optimum (status 1).  The search stops early after BB_NODES placements
     examined, or is skipped for ranks of more than BB_MAX_PAIRS pairs; the
     incumbent is then returned unproven (status 3);
  4. when the search stopped early, a certificate from the Lagrangian
     relaxation of the checkpoint constraints (the dual side of the ILP's
     LP bound): for multipliers l_k >= 0, every selection within the cap
     takes at least  sum_i min_j (t_ij + m_ij * sum_{k: i live at k} l_k)
     - cap * sum_k l_k.  ``lagrangian_proof`` runs LAGR_ITERS subgradient
     steps in exact integer arithmetic (multipliers in units of 2^-F time
     per memory unit) and proves the incumbent within 5 % (status 1) once
     1.05 times that bound reaches it.
``exact`` solves the same problem by enumeration and ``exact_bb`` by the same
search without the 5 % allowance or a node limit, for small cases.
"""
from __future__ import annotations

import itertools

import numpy as np

BB_NODES = 512          # placements the branch and bound may examine per rank
BB_MAX_PAIRS = 512      # larger ranks keep the improved warm start
GAP_NUM, GAP_DEN = 105, 100   # a cut needs (placed + fastest rest) * 1.05 >= incumbent
LAGR_ITERS = 200        # subgradient steps of the certificate
LAGR_F = 20             # fraction bits of the multipliers (at most)
LAGR_LIMIT = 1 << 60    # magnitude every intermediate value stays below
LAGR_HALVE = 24         # steps between halvings of the step size


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


def tighten(cands, live, cap, cur):
    """Step 2: each pair in index order moves back to the fastest candidate
    that keeps every checkpoint it is live at within the cap; repeated until a
    pass changes nothing."""
    n = len(cands)
    cur = list(cur)
    at = [[k for k in range(n) if i in live[k]] for i in range(n)]
    load = [sum(cands[i][cur[i]][1] for i in live[k]) for k in range(n)]
    changed = True
    while changed:
        changed = False
        for i in range(n):
            # (a pair whose backward comes before its forward is live nowhere)
            top = max((load[k] for k in at[i]), default=None)
            for j in range(cur[i]):
                add = cands[i][j][1] - cands[i][cur[i]][1]
                if top is None or top + add <= cap:
                    for k in at[i]:
                        load[k] += add
                    cur[i] = j
                    changed = True
                    break
    return cur


def branch_and_bound(cands, pf, pb, cap, cur, nodes=BB_NODES, gap=(GAP_NUM, GAP_DEN)):
    """Step 3 from incumbent ``cur`` (a feasible choice): returns (choice,
    proven, placements examined).  ``nodes`` None: no limit."""
    n = len(cands)
    num, den = gap
    inc = sum(cands[i][cur[i]][0] for i in range(n))
    best = list(cur)
    order = sorted(range(n), key=lambda i: pf[i])
    rest = [0] * (n + 1)             # fastest time of the pairs at depth >= d
    for d in range(n - 1, -1, -1):
        rest[d] = rest[d + 1] + cands[order[d]][0][0]
    ch = [-1] * n
    placed = [0] * (n + 1)           # time of the pairs above depth d
    seen = 0
    d = 0
    while d >= 0:
        i = order[d]
        ch[d] += 1
        if ch[d] >= len(cands[i]):
            ch[d] = -1
            d -= 1
            continue
        seen += 1
        if nodes is not None and seen > nodes:
            return best, False, seen - 1
        t, m = cands[i][ch[d]]
        load = (m if pb[i] >= pf[i] else 0) + sum(cands[order[e]][ch[e]][1] for e in range(d)
                                                  if pb[order[e]] >= pf[i])
        if cap >= 0 and load > cap:
            continue                  # a leaner candidate may fit
        f = placed[d] + t
        if num * (f + rest[d + 1]) >= den * inc:
            ch[d] = len(cands[i])     # this and the slower candidates are cut
            continue
        if d == n - 1:
            inc = f
            for e in range(n):
                best[order[e]] = ch[e]
            continue
        placed[d + 1] = f
        d += 1
    return best, True, seen


def _bits(x):
    """Bits of a non-negative integer (0 for 0)."""
    return int(x).bit_length()


def lagrangian_values(cands, live, cap, iters=LAGR_ITERS):
    """The Lagrangian bound of every subgradient step, as (value, F): the
    bound is value / 2^F.  Multipliers l_k >= 0, one per checkpoint k (pair
    k's forward start), in units of 2^-F; pair i's price is the sum of l_k
    over the checkpoints it is live at; each step every pair takes its
    cheapest candidate under t * 2^F + m * price (the first on ties), the
    bound is the sum of those values less cap * sum_k l_k, and every
    multiplier moves by g_k * step / 2^b, b the bits of max_k |g_k| (the
    magnitude shifted down, the sign kept; kept within [0, lmax]), g_k being
    the memory those candidates put on checkpoint k less the cap;
    step = s0 / 2^(t / LAGR_HALVE) at step t (rounded down).  The constants depend on the rank's
    candidates and cap only: F = min(LAGR_F, 60 - bits(n * tmax));
    lmax = 2^60 / 2^bits(n^2 * max(1, mmax, cap)); s0 = half the largest
    (dt << F) / 2^(bits(dm) - 1) over the candidates' moves from the fastest,
    at least 1 and at most lmax -- every intermediate value stays below 2^60
    (2^61 for the bound).  Nothing when the rank has no pairs or no cap, or
    its sizes leave no such F."""
    n = len(cands)
    if n == 0 or cap < 0:
        return
    tmax = max(x[0] for c in cands for x in c)
    mmax = max(x[1] for c in cands for x in c)
    F = min(LAGR_F, 60 - _bits(n * max(tmax, 1)))
    lmax = LAGR_LIMIT >> _bits(n * n * max(1, mmax, cap))
    if F < 0 or lmax == 0:
        return
    s0 = 0
    for c in cands:
        for j in range(1, len(c)):
            s0 = max(s0, ((c[j][0] - c[0][0]) << F) >> (_bits(c[0][1] - c[j][1]) - 1))
    s0 = min(lmax, max(1, s0 >> 1))
    cover = [[k for k in range(n) if i in live[k]] for i in range(n)]
    lam = [0] * n
    for t in range(iters):
        val = -cap * sum(lam)
        mem = [0] * n
        for i in range(n):
            price = sum(lam[k] for k in cover[i])
            best = None
            for tt, mm in cands[i]:
                v = (tt << F) + mm * price
                if best is None or v < best:
                    best, mem[i] = v, mm
            val += best
        yield val, F
        g = [sum(mem[i] for i in live[k]) - cap for k in range(n)]
        sh = _bits(max(abs(x) for x in g))
        if sh == 0:
            return
        step = s0 >> (t // LAGR_HALVE)
        lam = [min(lmax, max(0, lam[k] + (1 if g[k] >= 0 else -1) * ((abs(g[k]) * step) >> sh)))
               for k in range(n)]


def lagrangian_proof(cands, live, cap, inc, iters=LAGR_ITERS, gap=(GAP_NUM, GAP_DEN)):
    """Step 4: True when, at some step, the Lagrangian bound times the gap
    reaches the incumbent's total time ``inc`` (the steps stop there)."""
    if not cands or cap < 0:
        return True
    num, den = gap
    return any(num * val >= den * (inc << F) for val, F in lagrangian_values(cands, live, cap, iters))


def select(cands, live, pf, pb, cap, nodes=BB_NODES):
    """The solver of a rank: (choice, total time, status, peak); status 1
    within the cap and proven within 5 % of optimal, 3 within the cap but
    not proven, 0 the cap cannot be met (choice where the warm start gave
    up)."""
    n = len(cands)
    cur, total, ok, peak = greedy_select(cands, live, cap)
    if not ok:
        return cur, total, 0, peak
    proven = True
    if cap >= 0 and n:
        cur = tighten(cands, live, cap, cur)
        if n <= BB_MAX_PAIRS:
            cur, proven, _ = branch_and_bound(cands, pf, pb, cap, cur, nodes)
            if not proven:
                proven = lagrangian_proof(cands, live, cap,
                                          sum(cands[i][cur[i]][0] for i in range(n)))
        else:
            proven = False
    total = sum(cands[i][cur[i]][0] for i in range(n))
    peak = max((sum(cands[i][cur[i]][1] for i in live[k]) for k in range(n)), default=0)
    return cur, total, 1 if proven else 3, peak


def exact_bb(cands, live, pf, pb, cap):
    """The optimum by the same search with no allowance and no limit, from the
    improved warm start; None when the cap cannot be met."""
    cur, _, ok, _ = greedy_select(cands, live, cap)
    if not ok:
        return None
    if cap >= 0 and cands:
        cur = tighten(cands, live, cap, cur)
        cur, _, _ = branch_and_bound(cands, pf, pb, cap, cur, None, (1, 1))
    return sum(cands[i][cur[i]][0] for i in range(len(cands)))


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


def rank_positions(prob, table, order, r):
    """Positions of rank r's pairs' forwards and backwards in its order (pairs
    in slot order, as rank_problem lists them)."""
    base = int(prob.rank_off[r])
    nr = int(prob.rank_off[r + 1]) - base
    pos = [0] * nr
    for p in range(nr):
        pos[int(order[base + p])] = p
    slots = [s for s in range(len(table.slot_rank)) if table.slot_rank[s] == r]
    return ([pos[int(table.slot_f[s]) - base] for s in slots],
            [pos[int(table.slot_b[s]) - base] for s in slots])


def optimise(prob, table, cands, orders, caps=None, nodes=BB_NODES):
    """Per candidate schedule and rank: (total time, status, peak, choice by
    pair in slot order) of ``select``."""
    P = prob.n_ranks
    caps = prob.mem_cap if caps is None else caps
    out = []
    for row in orders:
        per = []
        for r in range(P):
            _, c, live = rank_problem(prob, table, cands, row, r)
            pf, pb = rank_positions(prob, table, row, r)
            cur, total, status, peak = select(c, live, pf, pb, int(caps[r]), nodes)
            per.append((total, status, peak, cur))
        out.append(per)
    return out


def retimed_costs(prob, table, cands, per):
    """Op costs of one schedule after the selection (``per``: optimise's
    entries of its ranks): a pair's chosen time is its forward's cost plus its
    backward's, the recomputation landing in the backward; forwards keep
    their cost."""
    cost = prob.op_cost.astype(np.int64).copy()
    for r, (_, status, _, cur) in enumerate(per):
        slots = [s for s in range(len(table.slot_rank)) if table.slot_rank[s] == r]
        for i, s in enumerate(slots):
            f, b = int(table.slot_f[s]), int(table.slot_b[s])
            cost[b] = cands[s][cur[i]][0] - cost[f]
    return cost


def selected_problem(prob, table, cands, per):
    """The problem as one schedule runs it after the selection: re-timed op
    costs and each pair's activation the chosen candidate's memory."""
    import dataclasses
    act = prob.slot_act.astype(np.int64).copy()
    for r, (_, _, _, cur) in enumerate(per):
        slots = [s for s in range(len(table.slot_rank)) if table.slot_rank[s] == r]
        for i, s in enumerate(slots):
            act[s] = cands[s][cur[i]][1]
    cost = retimed_costs(prob, table, cands, per)
    return dataclasses.replace(prob, op_cost=cost.astype(prob.op_cost.dtype),
                               slot_act=act.astype(prob.slot_act.dtype))


def choice_row(table, per):
    """A schedule's choices in the library's pair numbering (rank by rank,
    slot order within a rank)."""
    out = []
    for r, (_, _, _, cur) in enumerate(per):
        out.extend(cur)
    return out

