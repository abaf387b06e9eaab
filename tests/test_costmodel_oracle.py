"""Pins of the cost-model oracle (oracle/costmodel.py, Sec. 6.1) and of the
operator counts it reads (workloads/operators.py): textbook GEMM counts, the
max over resources per operator (not per item), hand-worked tables, and
monotonicity."""
import math

import numpy as np

import oracle.costmodel as C
import workloads as W
from workloads.operators import (K_ATTN, K_COLL, K_ELEM, K_GEMM, K_P2P, N_KINDS, ModelSpec,
                                 OperatorTable, coefficient_sweep, layer_ops, operator_table)


def _table(items):
    ptr, rows = [0], []
    for ops in items:
        rows += ops
        ptr.append(len(rows))
    a = np.array(rows, np.float64).reshape(-1, 4) if rows else np.zeros((0, 4))
    return OperatorTable(np.array(ptr, np.int32), a[:, 1].copy(), a[:, 2].copy(),
                         a[:, 3].copy(), a[:, 0].astype(np.uint8), len(items), 0)


def _coef(F, Bm, Bn, alpha=(1.0, 1.0, 1.0)):
    c = np.zeros((1, N_KINDS, 3))
    c[0, :, 0] = alpha[0] / F
    c[0, :, 1] = alpha[1] / Bm
    c[0, :, 2] = alpha[2] / Bn
    return c


def test_gemm_hand_example():
    # 1024^3 GEMM: 2*1024^3 = 2,147,483,648 FLOP at 1e15 FLOP/s = 2.147 us -> 3 us;
    # its 6 MiB of traffic at 3e12 B/s is 2.1 us, below it
    tab = _table([[(K_GEMM, 2 * 1024.0 ** 3, 6 * 2 ** 20, 0.0)]])
    assert C.cost_tables(tab, _coef(1e15, 3e12, 1e11))[0, 0] == 3


def test_max_is_per_operator_not_per_item():
    # op A: 3.5 us compute, 1 us memory; op B: 1 us compute, 4.25 us memory:
    # 3.5 + 4.25 = 7.75 -> 8 us; the max of the item's totals, max(4.5, 5.25),
    # would give 6 us (values kept off whole microseconds: ceil of a float64
    # sum that lands on an integer depends on the last bit)
    tab = _table([[(K_GEMM, 3.5e9, 3e6, 0.0), (K_ELEM, 1e9, 12.75e6, 0.0)]])
    assert C.cost_tables(tab, _coef(1e15, 3e12, 1e11))[0, 0] == 8


def test_network_and_alpha():
    # 1.9e6 bytes over 1e11 B/s = 19 us, alpha_net 0.5 -> 9.5 us -> 10 us
    tab = _table([[(K_P2P, 0.0, 0.0, 1.9e6)], []])
    out = C.cost_tables(tab, _coef(1e15, 3e12, 1e11, alpha=(1.0, 1.0, 0.5)))
    assert out[0].tolist() == [10, 0]


def test_rounding_up_and_overflow():
    tab = _table([[(K_ELEM, 0.0, 1.0, 0.0)], [(K_ELEM, 0.0, 3e12 * 3000.0, 0.0)]])
    out = C.cost_tables(tab, _coef(1e15, 3e12, 1e11))
    assert out[0, 0] == 1                     # any positive time is at least 1 us
    assert out[0, 1] == -1                    # 3e9 us does not fit int32


def test_layer_counts_by_hand():
    spec = ModelSpec("t", 1, 4, 8, 2, 1, True)      # h 4, f 8, 2 heads, 1 group, gated
    ops = layer_ops(spec, 2, 1)                       # T = 2, no tensor parallelism
    # q = 4 (1 + 2 * 1/2) = 8
    assert ops[1] == (K_GEMM, 2 * 2 * 4 * 8, 2 * (2 * 4 + 4 * 8 + 2 * 8), 0.0)
    assert ops[2] == (K_ATTN, 4 * 2 * 2 * 4, 2 * (2 * 8 + 2 * 4), 0.0)
    assert ops[4] == (K_ELEM, 8 * 2 * 4, 4 * 2 * 4, 0.0)
    assert ops[5] == (K_GEMM, 2 * 2 * 4 * 8 * 2, 2 * (2 * 4 + 2 * 4 * 8 + 2 * 2 * 8), 0.0)
    assert len(ops) == 7                               # no collectives at tp = 1
    ops4 = layer_ops(spec, 2, 4)
    assert [k for (k, *_ ) in ops4].count(K_COLL) == 2
    assert ops4[4][3] == 2 * 2 * 4 * 2 * 3 / 4


def test_backward_doubles_and_tables_are_monotone():
    prob = W.make_problem(2)
    tab = operator_table(prob)
    coef = coefficient_sweep(3, seed=1)
    sub = _take(tab, 40)
    out = C.cost_tables(sub, coef)
    # F and B of one (lane, unit) are adjacent ops (ids 2 slot, 2 slot + 1)
    for i in range(0, 40, 2):
        f, b = out[:, i], out[:, i + 1]
        assert ((b >= f) & (b <= 2 * f)).all()
    slower = C.cost_tables(sub, coef * 1.5)
    assert (slower >= out).all()


def _take(tab, n):
    end = tab.item_ptr[n]
    return OperatorTable(tab.item_ptr[:n + 1].copy(), tab.n_fop[:end], tab.n_mem[:end],
                         tab.n_net[:end], tab.kind[:end], n, 0)
