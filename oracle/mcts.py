"""CPU oracle of DIP's MCTS segment reordering (arXiv 2504.14145, Sec. 5.1).

TEST INFRASTRUCTURE ONLY: the test suite and the benchmark's CPU-baseline leg
are its only callers; the GPU library and the package never import it.  Plain
Python, one node object per tree node, following the paper's loop:

* The searched sequence orders the n segment classes (Sec. 5.1's pipeline
  segments after its search-space reduction: the pieces of one module in one
  microbatch share a class).  The class at position i (0-based) gets priority
  n - i; a group's priority is its class's; the dual-queue interleaving of
  Sec. 5.2 (``oracle.greedy``) turns the priorities into a schedule, and the
  score (lower is better) is the iteration time: with ``memory`` given (a
  strategy table and its pair candidates), the schedule's per-layer memory
  optimisation (Sec. 5.3, ``oracle.memopt.optimise``) picks each stage pair's
  candidate and the schedule re-timed with that selection
  (``oracle.memopt.selected_problem``) is simulated; its makespan is the
  score, +inf when a rank's cap cannot be met (the re-timed run is then over
  the cap).  Without ``memory`` the score is the interleaved schedule's
  makespan, +inf over a cap.
* Tree: a node at depth d fixes the class at position d - 1; it keeps s, the
  best score seen in its subtree, and N, its visit count.
* Selection: from the root, while the node has no untried child, step to the
  child with the largest UCB  u = (s_root / s_v)^alpha + beta * sqrt(ln N_x / N_v)
  -- the paper's s_v^alpha with the score inverted so that larger is better
  (a time is minimised); a child with no finite score has first term 0;
  ties go to the lower class.  Children whose subtrees are fully explored are
  skipped; the search ends early when the root's is.
* Expansion: one untried child, drawn by ``workloads.expansion_draw``.
* Rollouts: R random completions of the node's prefix.  Rollout i of
  iteration t shuffles the remaining classes (ascending) with Durstenfeld's
  Fisher-Yates, index k in [0, j] taken as (hi32(u) * (j + 1)) >> 32 from the
  SplitMix64 stream (Steele, Lea and Flood, OOPSLA 2014) whose initial state
  is mix(mix(seed + (t + 1) G) + (i + 1) G), G = 0x9E3779B97F4A7C15.
* Backpropagation: the best rollout score (lowest index among equal ones)
  updates s and N of the new node and of every ancestor.

The two other exploration strategies the paper compares its search with
(depth-first search and random exploration, in its search-efficiency
evaluation) replace selection and expansion and keep the rollouts and the
backpropagation:

* policy "dfs": the tree is walked depth first, children in ascending class
  order: the next node expanded is the lowest untried class of the deepest
  node on the current path that still has one (after a complete sequence,
  the walk backs up);
* policy "random": every iteration rolls out from the root (random complete
  sequences; the tree does not grow).

Parallel search (Sec. 6.2: workers explore at once and merge their results
into shared tree statistics after each round of rollouts): with W workers, a
round lets worker 0, 1, ..., W-1 select and expand in turn, each adding a
virtual visit (N + 1, s unchanged) to its node and every ancestor, so that
later workers see the earlier ones' choices; the rollouts of all W nodes then
run, and their best scores update s in worker order (the virtual visits stand
as the visits).  Leaves are numbered across rounds; leaf k's expansion draw
and rollout draws use k.  W = 1 is the sequential loop above.
"""
from __future__ import annotations

import math

import numpy as np

from . import greedy as _greedy

GOLDEN = 0x9E3779B97F4A7C15
MASK64 = (1 << 64) - 1
INF = float("inf")


def mix64(z: int) -> int:
    """SplitMix64's output function."""
    z &= MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def splitmix64(state: int, count: int):
    """The first ``count`` outputs of SplitMix64 started at ``state``."""
    out = []
    for _ in range(count):
        state = (state + GOLDEN) & MASK64
        out.append(mix64(state))
    return out


def rollout_state(seed: int, draw: int, index: int) -> int:
    return mix64((mix64(seed + (draw + 1) * GOLDEN) + (index + 1) * GOLDEN) & MASK64)


def shuffled(rest, seed: int, draw: int, index: int):
    """Durstenfeld's Fisher-Yates over ``rest`` driven by the rollout's stream."""
    a = list(rest)
    m = len(a)
    u = splitmix64(rollout_state(seed, draw, index), max(m - 1, 0))
    for step, j in enumerate(range(m - 1, 0, -1)):
        k = ((u[step] >> 32) * (j + 1)) >> 32
        a[j], a[k] = a[k], a[j]
    return a


def priorities_of(sequence, group_class, n_classes):
    """Group priorities of a complete class sequence: class at position i -> n - i."""
    prio_of_class = [0] * n_classes
    for i, c in enumerate(sequence):
        prio_of_class[c] = n_classes - i
    return np.array([prio_of_class[c] for c in group_class], np.int32)


class Node:
    def __init__(self, cls, parent, n_classes):
        self.cls = cls
        self.parent = parent
        self.depth = 0 if parent is None else parent.depth + 1
        on_path = set(self.prefix())
        self.untried = [c for c in range(n_classes) if c not in on_path]
        self.children = {}
        self.N = 0
        self.s = INF
        self.done = False

    def prefix(self):
        out, v = [], self
        while v is not None and v.cls is not None:
            out.append(v.cls)
            v = v.parent
        return out[::-1]


def ucb(root_s, parent_n, child, alpha, beta):
    exploit = (root_s / child.s) ** alpha if (child.s < INF and root_s < INF) else 0.0
    return exploit + beta * math.sqrt(math.log(parent_n) / child.N)


def select(root, alpha, beta):
    x = root
    while not x.untried and x.children:
        best, best_u = None, -INF
        for c in sorted(x.children):
            v = x.children[c]
            if v.done:
                continue
            u = ucb(root.s, x.N, v, alpha, beta)
            if u > best_u:
                best, best_u = v, u
        if best is None:
            break
        x = best
    return x


def mark_done(v, n_classes):
    while v is not None:
        if v.depth == n_classes or (not v.untried and all(c.done for c in v.children.values())):
            v.done = True
            v = v.parent
        else:
            break


def score_rollouts(prob, op_group, n_groups, prio, threads=8, memory=None):
    """Scores of priority rows: the iteration time after the interleaving
    (and the memory optimisation when ``memory`` = (table, candidates)), +inf
    for a flagged schedule."""
    orders, res = _greedy(prob, op_group, n_groups, prio, threads=threads)
    if memory is None:
        return [float(m) if f == 0 else INF for m, f in zip(res.makespan, res.flags)]
    from . import evaluate
    from . import memopt as _mo
    table, cands = memory
    per_row = _mo.optimise(prob, table, cands, orders)
    out = []
    for row, per in zip(orders, per_row):
        r = evaluate(_mo.selected_problem(prob, table, cands, per), row[None, :])
        out.append(float(r.makespan[0]) if r.flags[0] == 0 else INF)
    return out


def search(prob, op_group, n_groups, group_class, iterations, rollouts, seed,
           alpha=1.0, beta=0.1, threads=8, policy="ucb", workers=1, memory=None):
    """Run the search for ``iterations`` rounds of ``workers`` leaves; returns
    (trajectory, best, root) where trajectory[k] = (prefix of leaf k, best score
    of its rollouts, index of the best rollout) and best = (score, sequence,
    leaf, index).  policy: "ucb" (the paper's MCTS), "dfs" or "random"."""
    if policy not in ("ucb", "dfs", "random"):
        raise ValueError(policy)
    if workers < 1:
        raise ValueError(workers)
    group_class = [int(c) for c in group_class]
    n = max(group_class) + 1 if group_class else 0
    root = Node(None, None, n)
    traj = []
    best = (INF, None, -1, -1)
    cursor = root                        # dfs: the node expanded last
    k = 0                                # leaves so far
    for _ in range(iterations):
        leaves = []
        for _w in range(workers):
            if root.done:
                break
            if policy == "random":
                x = root
            elif policy == "dfs":
                x = cursor
                while x is not None and not x.untried:
                    x = x.parent
                if x is None:
                    break
                c = min(x.untried)
                x.untried.remove(c)
                child = Node(c, x, n)
                x.children[c] = child
                x = cursor = child
            else:
                x = select(root, alpha, beta)
                if x.untried:
                    c = x.untried.pop(_expansion(seed, k, len(x.untried)))
                    child = Node(c, x, n)
                    x.children[c] = child
                    x = child
            v = x
            while v is not None:         # the (virtual) visit
                v.N += 1
                v = v.parent
            if x.depth == n:
                mark_done(x, n)          # a complete sequence: nothing below it
            leaves.append((x, k))
            k += 1
        if not leaves:
            break
        for x, kk in leaves:
            prefix = x.prefix()
            rest = [c for c in range(n) if c not in set(prefix)]
            seqs = [prefix + shuffled(rest, seed, kk, i) for i in range(rollouts)]
            prio = np.stack([priorities_of(q, group_class, n) for q in seqs])
            scores = score_rollouts(prob, op_group, n_groups, prio, threads, memory)
            b = min(range(rollouts), key=lambda i: (scores[i], i))
            if scores[b] == INF:
                b = -1                       # no feasible rollout
            traj.append((tuple(prefix), scores[b] if b >= 0 else INF, b))
            if b >= 0 and scores[b] < best[0]:
                best = (scores[b], seqs[b], kk, b)
            v = x
            while v is not None:
                v.s = min(v.s, scores[b] if b >= 0 else INF)
                v = v.parent
            mark_done(x, n)
    return traj, best, root


def _expansion(seed, t, n_untried):
    import workloads
    return workloads.expansion_draw(seed, t, n_untried)
