"""Operator descriptors of the pipeline stages, for the operator-level cost
model (DIP, arXiv 2504.14145, Sec. 6.1).

Each stage (the forward or backward of one sub-microbatch on one lane) runs
its lane's share of the module's transformer layers; each layer is a list of
operators with a floating-point operation count N_fop, bytes of memory
traffic N_mem and bytes sent over the network N_net.  Every data edge between
different ranks is one more item: a single network operator carrying the
upstream piece's activations.  This module only counts; the latencies are the
cost model's.

Counting rules (T tokens, hidden h, FFN f, heads n, key/value groups g, head
dimension h/n, tensor-parallel degree tp, 2-byte activations and weights):
  layer norm      N_fop 8 T h / tp,              N_mem 4 T h
  QKV GEMM        2 T h q / tp,                  2 (T h + h q / tp + T q / tp),  q = h (1 + 2 g / n)
  attention       4 T^2 h / tp,                  2 (T q + T h) / tp
  output GEMM     2 T h h / tp,                  2 (T h / tp + h h / tp + T h)
  MLP in          2 T h f k / tp,                2 (T h + k h f / tp + k T f / tp), k = 2 gated, 1 not
  MLP out         2 T f h / tp,                  2 (T f / tp + f h / tp + T h)
  all-reduce      (tp > 1, after attention and after the MLP)  N_net 2 T h 2 (tp - 1) / tp
A backward stage doubles every N_fop and N_mem (gradients of inputs and of
weights) and keeps N_net.  Operator kinds: 0 GEMM, 1 attention,
2 element-wise, 3 collective, 4 point-to-point transfer.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .instance import KIND_B, Problem

K_GEMM, K_ATTN, K_ELEM, K_COLL, K_P2P = 0, 1, 2, 3, 4
N_KINDS = 5


@dataclass(frozen=True)
class ModelSpec:
    name: str
    layers: int
    hidden: int
    ffn: int
    heads: int
    groups: int
    gated: bool


# the paper's model table (layers, embedding, FFN hidden, heads, groups)
VIT_5B = ModelSpec("ViT 5B", 63, 1792, 15360, 16, 16, False)
LLAMA3_8B = ModelSpec("Llama3 8B", 32, 4096, 14336, 32, 8, True)
DIT_5B = ModelSpec("DiT 5B", 28, 3584, 10240, 28, 28, False)

SEGMENT_MODELS = {"vit": VIT_5B, "enc": VIT_5B, "llm": LLAMA3_8B, "textenc": LLAMA3_8B,
                  "dit": DIT_5B, "ditdec": DIT_5B, "vaedec": DIT_5B, "stage": LLAMA3_8B}


def layer_ops(spec: ModelSpec, T: int, tp: int):
    """[(kind, N_fop, N_mem, N_net)] of one forward layer on T tokens."""
    h, f, n, g = spec.hidden, spec.ffn, spec.heads, spec.groups
    q = h * (1 + 2 * g / n)
    k = 2 if spec.gated else 1
    ops = [(K_ELEM, 8 * T * h / tp, 4 * T * h, 0.0),
           (K_GEMM, 2 * T * h * q / tp, 2 * (T * h + h * q / tp + T * q / tp), 0.0),
           (K_ATTN, 4 * T * T * h / tp, 2 * (T * q + T * h) / tp, 0.0),
           (K_GEMM, 2 * T * h * h / tp, 2 * (T * h / tp + h * h / tp + T * h), 0.0)]
    if tp > 1:
        ops.append((K_COLL, 0.0, 0.0, 2 * T * h * 2 * (tp - 1) / tp))
    ops += [(K_ELEM, 8 * T * h / tp, 4 * T * h, 0.0),
            (K_GEMM, 2 * T * h * f * k / tp, 2 * (T * h + k * h * f / tp + k * T * f / tp), 0.0),
            (K_GEMM, 2 * T * f * h / tp, 2 * (T * f / tp + f * h / tp + T * h), 0.0)]
    if tp > 1:
        ops.append((K_COLL, 0.0, 0.0, 2 * T * h * 2 * (tp - 1) / tp))
    return ops


@dataclass
class OperatorTable:
    """Items 0 .. N-1 are the stages (global op order), N .. N+E-1 the data
    edges (pred CSR order); item i owns operator rows item_ptr[i] ..
    item_ptr[i+1]-1."""
    item_ptr: np.ndarray    # int32 [N + E + 1]
    n_fop: np.ndarray       # float64 [rows]
    n_mem: np.ndarray       # float64 [rows]
    n_net: np.ndarray       # float64 [rows]
    kind: np.ndarray        # uint8 [rows]
    n_stages: int
    n_edges: int


def operator_table(prob: Problem, tp: int = 4) -> OperatorTable:
    inst = prob.inst
    if inst is None:
        raise ValueError("needs the high-level instance")
    from .configs import CONFIGS
    names = None
    for cfg in CONFIGS.values():
        if cfg.name == inst.name:
            names = [s.name for s in cfg.segments]
    if names is None:
        names = ["stage"] * len(inst.seg_lo)
    rows, ptr = [], [0]
    lanes_of = [inst.seg_hi[s] - inst.seg_lo[s] + 1 for s in range(len(inst.seg_lo))]
    for o in range(prob.n_total):
        u = int(prob.op_unit[o])
        s = int(inst.unit_seg[u])
        spec = SEGMENT_MODELS.get(names[s], LLAMA3_8B)
        per_lane = -(-spec.layers // lanes_of[s])
        T = int(inst.unit_tok[u])
        mult = 2.0 if prob.op_kind[o] == KIND_B else 1.0
        if T > 0:
            one = layer_ops(spec, T, tp)
            for _ in range(per_lane):
                rows += [(k, mult * a, mult * b, c) for (k, a, b, c) in one]
        ptr.append(len(rows))
    # edges: activations of the upstream piece, between different ranks only
    rank = np.repeat(np.arange(prob.n_ranks), np.diff(prob.rank_off))
    for o in range(prob.n_total):
        for e in range(prob.pred_ptr[o], prob.pred_ptr[o + 1]):
            p = int(prob.pred_op[e])
            if rank[p] != rank[o]:
                u = int(prob.op_unit[p])
                spec = SEGMENT_MODELS.get(names[int(inst.unit_seg[u])], LLAMA3_8B)
                rows.append((K_P2P, 0.0, 0.0, float(2 * int(inst.unit_tok[u]) * spec.hidden)))
            ptr.append(len(rows))
    a = np.array(rows, dtype=np.float64).reshape(-1, 4) if rows else np.zeros((0, 4))
    return OperatorTable(np.array(ptr, np.int32), np.ascontiguousarray(a[:, 1]),
                         np.ascontiguousarray(a[:, 2]), np.ascontiguousarray(a[:, 3]),
                         a[:, 0].astype(np.uint8), prob.n_total, prob.n_edges)


# the capacities of one accelerator of the paper's cluster class and its links
H800_LIKE = {"flops": 989e12, "mem_bw": 3.35e12, "net_bw": 400e9}


def coefficient_sweep(n: int, seed: int, device=H800_LIKE) -> np.ndarray:
    """float64 [n][N_KINDS][3]: seconds per unit (alpha / capacity) for n
    configurations whose efficiency factors alpha are drawn uniformly in
    [0.3, 1.0] per (kind, resource) -- a calibration sweep."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 101]))
    alpha = rng.uniform(0.3, 1.0, size=(n, N_KINDS, 3))
    cap = np.array([device["flops"], device["mem_bw"], device["net_bw"]], np.float64)
    return np.ascontiguousarray(alpha / cap)
