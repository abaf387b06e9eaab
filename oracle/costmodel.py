"""CPU oracle of the operator-level cost model (DIP, arXiv 2504.14145,
Sec. 6.1) as a batched cost-table builder.

TEST INFRASTRUCTURE ONLY: the test suite and the benchmark's CPU-baseline leg
are its only callers.

An operator's latency is the largest of its three resource times,
    max(alpha_fop N_fop / F, alpha_mem N_mem / B_mem, alpha_net N_net / B_net),
read here with the per-kind coefficients c = alpha / capacity formed once per
configuration (seconds per FLOP, per byte), so a time is c * N in float64.
An item (a pipeline stage, or a data edge) runs its operators one after
another: its latency is their sum in row order.  The table entry is that sum
in whole microseconds rounded up, ceil(1e6 * t); an entry above 2^31 - 1 is
reported as -1.
"""
from __future__ import annotations

import math

import numpy as np


def item_cost(coef, rows, n_fop, n_mem, n_net, kind):
    """Microseconds of one item under one configuration (coef [kinds][3])."""
    t = 0.0
    for r in rows:
        c = coef[kind[r]]
        a = c[0] * n_fop[r]
        b = c[1] * n_mem[r]
        d = c[2] * n_net[r]
        t = t + max(max(a, b), d)
    us = math.ceil(t * 1e6)
    return us if us <= 2**31 - 1 else -1


def cost_tables(table, coef):
    """int32 [n_configs][n_items]: every item's cost under every configuration."""
    coef = np.asarray(coef, np.float64)
    n_items = len(table.item_ptr) - 1
    out = np.zeros((coef.shape[0], n_items), np.int32)
    fop, mem, net, kind = (table.n_fop.tolist(), table.n_mem.tolist(), table.n_net.tolist(),
                           table.kind.tolist())
    for b in range(coef.shape[0]):
        cb = coef[b].tolist()
        for i in range(n_items):
            out[b, i] = item_cost(cb, range(table.item_ptr[i], table.item_ptr[i + 1]),
                                  fop, mem, net, kind)
    return out
