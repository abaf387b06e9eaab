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

workers = W > 1 is Sec. 6.2's parallel search on one GPU: in a round, W
workers select and expand in turn, each leaving a virtual visit on its path
for the later ones; one dip_sim_rollouts_batch call rolls out all W nodes;
their best scores then update the tree in worker order.  Leaves are numbered
across rounds, and leaf k's expansion and rollout draws use k (W = 1 is the
sequential search).
"""
from __future__ import annotations

import bisect
import math

import numpy as np

INF = float("inf")


class Search:
    """One search over the classes of a Sim configured for the greedy."""

    def __init__(self, sim, group_class, rollouts, seed, alpha=1.0, beta=0.1, policy="ucb",
                 workers=1):
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
        self.W = int(workers)
        if self.W < 1:
            raise ValueError(workers)
        self.leaves = 0                  # leaves so far (names their draws)
        self.rounds = 0
        self.R = int(rollouts)
        self.seed = int(seed)
        self.alpha, self.beta = float(alpha), float(beta)
        self.draw_child = workloads.expansion_draw
        dev = torch.device("cuda", torch.cuda.current_device())
        G = self.cls_of_group.size
        self.prio = torch.empty((self.W * self.R, G), dtype=torch.int32, device=dev)
        self.ms = torch.empty(self.W * self.R, dtype=torch.int32, device=dev)
        self.fl = torch.empty(self.W * self.R, dtype=torch.uint8, device=dev)
        self.key = torch.empty(self.W, dtype=torch.int64, device=dev)
        # per node (node 0 is the root): parent, class, depth, untried classes
        # (ascending), children sorted by class (classes, node ids); visits,
        # best score and done flag in arrays, so that a selection step scores
        # all children of a node at once
        self.parent = [-1]
        self.cls = [-1]
        self.depth = [0]
        self.todo = [list(range(self.n))]
        self.kid_cls = [[]]
        self.kid_ids = [[]]
        self.nodes = 1
        self.visits = np.zeros(1024, np.int64)
        self.score = np.full(1024, INF)
        self.done = np.zeros(1024, bool)
        self.trajectory = []
        self.best = (INF, None, -1, -1)

    def _path(self, v):
        out = []
        while v > 0:
            out.append(self.cls[v])
            v = self.parent[v]
        return out[::-1]

    def _select(self):
        # the oracle's rule, evaluated per node over all children at once: the
        # same float64 operations in the same order (division and square root
        # are correctly rounded; ln N and, unless alpha is 1, the powers are
        # taken with Python floats), first maximum in class order
        v = 0
        while not self.todo[v] and self.kid_ids[v]:
            ids = np.asarray(self.kid_ids[v], np.int64)
            live = ~self.done[ids]
            if not live.any():
                break
            s_root = float(self.score[0])
            s_w = self.score[ids]
            if s_root < INF:
                fin = s_w < INF
                ratio = np.where(fin, s_root / np.where(fin, s_w, 1.0), 0.0)
                if self.alpha == 1.0:
                    exploit = ratio
                else:
                    exploit = np.array([float(r) ** self.alpha if f else 0.0
                                        for r, f in zip(ratio, fin)])
            else:
                exploit = np.zeros(ids.size)
            u = exploit + self.beta * np.sqrt(math.log(int(self.visits[v])) / self.visits[ids])
            u[~live] = -INF
            v = int(ids[int(np.argmax(u))])
        return v

    def _add(self, v, c):
        w = self.nodes
        if w == self.visits.size:
            self.visits = np.concatenate([self.visits, np.zeros(w, np.int64)])
            self.score = np.concatenate([self.score, np.full(w, INF)])
            self.done = np.concatenate([self.done, np.zeros(w, bool)])
        self.nodes += 1
        self.parent.append(v)
        self.cls.append(c)
        self.depth.append(self.depth[v] + 1)
        on = set(self._path(v))
        on.add(c)
        self.todo.append([k for k in range(self.n) if k not in on])
        self.kid_cls.append([])
        self.kid_ids.append([])
        i = bisect.bisect_left(self.kid_cls[v], c)
        self.kid_cls[v].insert(i, c)
        self.kid_ids[v].insert(i, w)
        return w

    def _finish(self, v):
        while v >= 0:
            if self.depth[v] == self.n or (not self.todo[v] and
                                           bool(np.all(self.done[self.kid_ids[v]]))):
                self.done[v] = True
                v = self.parent[v]
            else:
                break

    def _pick(self, k):
        """One worker's node (expanded if need be), or -1 if there is none."""
        if self.policy == "random":
            return 0
        if self.policy == "dfs":
            v = self.cursor
            while v >= 0 and not self.todo[v]:
                v = self.parent[v]
            if v < 0:
                return -1                # every sequence visited
            c = min(self.todo[v])
            self.todo[v].remove(c)
            v = self.cursor = self._add(v, c)
            return v
        v = self._select()
        if self.todo[v]:
            c = self.todo[v].pop(self.draw_child(self.seed, k, len(self.todo[v])))
            v = self._add(v, c)
        return v

    def step(self, t=None):
        """One round: up to W leaves, one batch of rollouts."""
        from . import NO_KEY, decode_key, rollouts_batch

        self.rounds += 1
        picked = []
        for _ in range(self.W):
            if self.done[0]:
                break
            v = self._pick(self.leaves)
            if v < 0:
                self.done[0] = True
                break
            w = v
            while w >= 0:                # the (virtual) visit
                self.visits[w] += 1
                w = self.parent[w]
            if self.depth[v] == self.n:
                self._finish(v)          # a complete sequence: nothing below it
            picked.append((v, self.leaves))
            self.leaves += 1
        if not picked:
            return
        prefixes = [self._path(v) for v, _ in picked]
        L = len(picked)
        self.key[:L].fill_(-1)
        rollouts_batch(self.sim.h, prefixes, self.R, self.seed, picked[0][1], self.prio,
                       self.ms, self.fl, self.key)
        keys = self.key[:L].cpu().tolist()
        for (v, k), prefix, key in zip(picked, prefixes, keys):
            key &= NO_KEY
            if key == NO_KEY:
                sc, idx = INF, -1
            else:
                idx, ms = decode_key(key)
                sc = float(ms)
            self.trajectory.append((tuple(prefix), sc, idx))
            if idx >= 0 and sc < self.best[0]:
                l = k - picked[0][1]
                row = self.prio[l * self.R + idx].cpu().numpy()
                prio_of_class = np.zeros(self.n, np.int64)
                prio_of_class[self.cls_of_group] = row
                self.best = (sc, [int(c) for c in np.argsort(-prio_of_class, kind="stable")], k,
                             idx)
            w = v
            while w >= 0:
                if sc < self.score[w]:
                    self.score[w] = sc
                w = self.parent[w]
            self._finish(v)

    def run(self, rounds):
        """Run rounds until ``rounds`` have been made in all (or the tree is
        exhausted); returns (trajectory, best), one trajectory entry per leaf."""
        while self.rounds < rounds and not self.done[0]:
            self.step()
        return self.trajectory, self.best
