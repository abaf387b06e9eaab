"""MCTS segment reordering (DIP, arXiv 2504.14145, Sec. 5.1) with its rollouts
batched on the GPU.

The search orders the segment classes (see dip_sim_configure_rollouts); the
host keeps the tree -- a few arrays indexed by node id -- and every iteration
sends one batch of rollouts to the library: dip_sim_rollouts draws the random
completions of the selected node's prefix, interleaves them (Sec. 5.2) and
folds the best unflagged (makespan, rollout) into a 64-bit key, the only value
read back per iteration.  Tree steps, per iteration:

* selection: from the root, while a node has no untried class, step to the
  child of largest u = (s_root / s_child)^alpha + beta * sqrt(ln N_node /
  N_child), the score being the subtree's best makespan (so its ratio to the
  root's best is at most 1; a child without a feasible rollout contributes 0);
  ties to the lower class; fully explored subtrees are skipped;
* expansion: one untried class, drawn by workloads.expansion_draw;
* rollouts: n_rollouts completions (draw = iteration number);
* backpropagation: the batch's best score to the new node and its ancestors.

policy "dfs" and "random" are the two exploration strategies the paper
compares its search with: depth-first (the lowest untried class of the
deepest node on the current path that has one) and random exploration
(every batch rolled out from the root); rollouts and backpropagation stay.
"""
from __future__ import annotations

import math

import numpy as np

INF = float("inf")


class Search:
    """One search over the classes of a Sim configured for the greedy."""

    def __init__(self, sim, group_class, rollouts, seed, alpha=1.0, beta=0.1, policy="ucb"):
        import torch

        from . import configure_rollouts, OK, strerror
        import workloads

        self.torch = torch
        self.sim = sim
        self.cls_of_group = np.ascontiguousarray(group_class, np.int32)
        self.n = int(self.cls_of_group.max()) + 1
        rc = configure_rollouts(sim.h, self.n, self.cls_of_group)
        if rc != OK:
            raise RuntimeError(f"dip_sim_configure_rollouts: {strerror(rc)}")
        if policy not in ("ucb", "dfs", "random"):
            raise ValueError(policy)
        self.policy = policy
        self.cursor = 0                  # dfs: the node expanded last
        self.R = int(rollouts)
        self.seed = int(seed)
        self.alpha, self.beta = float(alpha), float(beta)
        self.draw_child = workloads.expansion_draw
        dev = torch.device("cuda", torch.cuda.current_device())
        G = self.cls_of_group.size
        self.prio = torch.empty((self.R, G), dtype=torch.int32, device=dev)
        self.ms = torch.empty(self.R, dtype=torch.int32, device=dev)
        self.fl = torch.empty(self.R, dtype=torch.uint8, device=dev)
        self.key = torch.empty(1, dtype=torch.int64, device=dev)
        # node arrays; node 0 is the root
        self.parent = [-1]
        self.cls = [-1]
        self.visits = [0]
        self.score = [INF]
        self.done = [False]
        self.kids = [{}]
        self.todo = [list(range(self.n))]
        self.depth = [0]
        self.trajectory = []
        self.best = (INF, None, -1, -1)

    def _path(self, v):
        out = []
        while v > 0:
            out.append(self.cls[v])
            v = self.parent[v]
        return out[::-1]

    def _select(self):
        v = 0
        while not self.todo[v] and self.kids[v]:
            pick, top = -1, -INF
            s_root = self.score[0]
            for c in sorted(self.kids[v]):
                w = self.kids[v][c]
                if self.done[w]:
                    continue
                s_w = self.score[w]
                exploit = (s_root / s_w) ** self.alpha if (s_w < INF and s_root < INF) else 0.0
                u = exploit + self.beta * math.sqrt(math.log(self.visits[v]) / self.visits[w])
                if u > top:
                    pick, top = w, u
            if pick < 0:
                break
            v = pick
        return v

    def _add(self, v, c):
        w = len(self.parent)
        self.parent.append(v)
        self.cls.append(c)
        self.visits.append(0)
        self.score.append(INF)
        self.done.append(False)
        self.kids.append({})
        self.depth.append(self.depth[v] + 1)
        on = set(self._path(v))
        on.add(c)
        self.todo.append([k for k in range(self.n) if k not in on])
        self.kids[v][c] = w
        return w

    def _finish(self, v):
        while v >= 0:
            if self.depth[v] == self.n or (not self.todo[v] and
                                           all(self.done[w] for w in self.kids[v].values())):
                self.done[v] = True
                v = self.parent[v]
            else:
                break

    def step(self, t):
        """One iteration (t = its number, which also names its random draws)."""
        from . import NO_KEY, decode_key, rollouts

        if self.policy == "random":
            v = 0
        elif self.policy == "dfs":
            v = self.cursor
            while v >= 0 and not self.todo[v]:
                v = self.parent[v]
            if v < 0:
                self.done[0] = True      # every sequence visited
                return
            c = min(self.todo[v])
            self.todo[v].remove(c)
            v = self.cursor = self._add(v, c)
        else:
            v = self._select()
            if self.todo[v]:
                c = self.todo[v].pop(self.draw_child(self.seed, t, len(self.todo[v])))
                v = self._add(v, c)
        prefix = self._path(v)
        self.key.fill_(-1)
        rollouts(self.sim.h, prefix, self.R, self.seed, t, self.prio, self.ms, self.fl, self.key)
        k = int(self.key.item()) & NO_KEY
        if k == NO_KEY:
            sc, idx = INF, -1
        else:
            idx, ms = decode_key(k)
            sc = float(ms)
        self.trajectory.append((tuple(prefix), sc, idx))
        if idx >= 0 and sc < self.best[0]:
            row = self.prio[idx].cpu().numpy()
            prio_of_class = np.zeros(self.n, np.int64)
            prio_of_class[self.cls_of_group] = row
            self.best = (sc, [int(c) for c in np.argsort(-prio_of_class, kind="stable")], t, idx)
        w = v
        while w >= 0:
            self.visits[w] += 1
            if sc < self.score[w]:
                self.score[w] = sc
            w = self.parent[w]
        self._finish(v)

    def run(self, iterations):
        for t in range(len(self.trajectory), iterations):
            if self.done[0]:
                break
            self.step(t)
        return self.trajectory, self.best
