"""Seeded synthetic instances and their compiled (CSR) form.

An instance states the scheduling problem at pipeline-stage granularity, the
granularity of DIP's interleaving and simulator (Sec. 5.2, Sec. 6.1):

* ``L = P * v`` lanes (model chunks); lane ``l`` lives on physical rank
  ``l % P``.
* Segments are contiguous lane ranges, one per modality module (Sec. 3.1).
* Units are sub-microbatches (Sec. 4): each belongs to one segment and one
  microbatch and carries a token count.
* Ops are the pipeline stages ``F(u, l)`` and ``B(u, l)`` for every lane ``l``
  of the unit's segment.

Data edges (the dependencies a pipeline stage waits for, Sec. 5.2 and the
operator DAG of Sec. 6.1), in this build's reading:

* chain inside a segment: ``F(u, l-1) -> F(u, l)`` and ``B(u, l+1) -> B(u, l)``;
* loss turnaround on the last lane of the last segment: ``F(u, l) -> B(u, l)``;
* joins between consecutive segments within one microbatch, all-to-all:
  every upstream piece's last-lane F precedes every downstream piece's
  first-lane F, and the backward edges mirror them.

Edge latency is asynchronous point-to-point transfer time (Sec. 6.3), charged
only between different physical ranks.

This module generates inputs.  It computes no start, end, makespan, bubble or
memory figure: that arithmetic belongs to the simulator and to its oracle.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .configs import WorkloadConfig, get

IMG_TOKENS = 576
VIDEO_PATCHES = 1024
FRAMES_PER_VAE_PIECE = 16
COMM_BYTES_PER_TOKEN = 4096 * 2          # hidden 4096, 2-byte activations
COMM_BYTES_PER_US = 400_000              # 400 GB/s = 4e5 bytes per microsecond

KIND_F = 0
KIND_B = 1


def op_cost_from_tokens(tok: int, a100: int, c100: int) -> int:
    """Forward cost in whole microseconds: floor(a*tok + c*tok^2/1e4)."""
    tok = int(tok)
    return (a100 * tok * 10_000 + c100 * tok * tok) // 1_000_000


def comm_from_tokens(tok: int) -> int:
    """Transfer latency, rounded up to whole microseconds."""
    return (int(tok) * COMM_BYTES_PER_TOKEN + COMM_BYTES_PER_US - 1) // COMM_BYTES_PER_US


@dataclass
class Instance:
    """High-level instance: lanes, segments, units and per-(lane, unit) costs."""

    P: int
    v: int
    seg_lo: list
    seg_hi: list
    unit_seg: np.ndarray      # [U] segment of each unit
    unit_mb: np.ndarray       # [U] microbatch of each unit
    unit_piece: np.ndarray    # [U] piece index inside (segment, microbatch)
    unit_tok: np.ndarray      # [U] tokens
    fcost: np.ndarray         # [L, U] forward cost (us); meaningful on the unit's lanes
    bcost: np.ndarray         # [L, U] backward cost (us)
    act: np.ndarray           # [L, U] activation units held from F start to B end
    unit_comm: np.ndarray     # [U] cross-rank transfer latency of the unit's activations
    mem_cap: int = -1         # per-rank cap, -1 = none
    name: str = "custom"

    @property
    def L(self) -> int:
        return self.P * self.v

    @property
    def n_seg(self) -> int:
        return len(self.seg_lo)

    def seg_of_lane(self, lane: int) -> int:
        for s in range(self.n_seg):
            if self.seg_lo[s] <= lane <= self.seg_hi[s]:
                return s
        raise ValueError(f"lane {lane} is in no segment")

    def units_of(self, seg: int, mb: int | None = None) -> list:
        sel = self.unit_seg == seg
        if mb is not None:
            sel &= self.unit_mb == mb
        return [int(u) for u in np.nonzero(sel)[0]]

    def join_comm(self, up: int, down: int) -> int:
        """Latency of the join edge between upstream piece ``up`` and
        downstream piece ``down``: the split side's tokens are what crosses
        (the upstream side's when neither side is split)."""
        s_dn = int(self.unit_seg[down])
        mb = int(self.unit_mb[down])
        if len(self.units_of(s_dn, mb)) > 1:
            return int(self.unit_comm[down])
        return int(self.unit_comm[up])


@dataclass
class Problem:
    """The compiled instance in the layout the C ABI takes (host arrays)."""

    n_ranks: int
    n_ops: np.ndarray         # int32 [P]
    rank_off: np.ndarray      # int64 [P+1]
    pred_ptr: np.ndarray      # int32 [N+1]
    pred_op: np.ndarray       # int32 [E]
    op_kind: np.ndarray       # uint8 [N]
    op_slot: np.ndarray       # int32 [N]
    n_slots: int
    mem_cap: np.ndarray       # int32 [P]
    op_cost: np.ndarray       # int32 [N]
    edge_comm: np.ndarray     # int32 [E]
    slot_act: np.ndarray      # int32 [n_slots]
    stride: int               # int16 elements per candidate
    op_lane: np.ndarray       # int32 [N] metadata (generator priorities, tests)
    op_unit: np.ndarray       # int32 [N]
    op_mb: np.ndarray         # int32 [N]
    inst: Instance | None = None

    @property
    def n_total(self) -> int:
        return int(self.rank_off[-1])

    @property
    def n_edges(self) -> int:
        return int(self.pred_ptr[-1])


def round_up(x: int, m: int) -> int:
    return (x + m - 1) // m * m


def compile_instance(inst: Instance, stride_align: int = 8) -> Problem:
    """Enumerate ops rank by rank and build the predecessor CSR.

    Rank-local op ids follow (lane ascending, unit ascending, F before B), so
    ``id = 2 * slot_local + kind``; the global index is ``rank_off[r] + id``.
    """
    P, L = inst.P, inst.L
    gid = {}                      # (kind, unit, lane) -> global op index
    n_ops = np.zeros(P, np.int32)
    lane_rows = []                # per global op: (lane, unit, kind)
    slot_of = []
    n_slots = 0
    for r in range(P):
        cnt = 0
        for lane in range(r, L, P):
            s = inst.seg_of_lane(lane)
            for u in inst.units_of(s):
                for kind in (KIND_F, KIND_B):
                    gid[(kind, u, lane)] = len(lane_rows)
                    lane_rows.append((lane, u, kind))
                    slot_of.append(n_slots)
                    cnt += 1
                n_slots += 1
        n_ops[r] = cnt
    N = len(lane_rows)
    rank_off = np.zeros(P + 1, np.int64)
    rank_off[1:] = np.cumsum(n_ops)

    def rank(lane):
        return lane % P

    preds = []
    for (lane, u, kind) in lane_rows:
        s = int(inst.unit_seg[u])
        mb = int(inst.unit_mb[u])
        lo, hi = inst.seg_lo[s], inst.seg_hi[s]
        plist = []
        if kind == KIND_F:
            if lane > lo:
                c = int(inst.unit_comm[u]) if rank(lane - 1) != rank(lane) else 0
                plist.append((gid[(KIND_F, u, lane - 1)], c))
            elif s > 0:
                up_lane = inst.seg_hi[s - 1]
                for x in inst.units_of(s - 1, mb):
                    c = inst.join_comm(x, u) if rank(up_lane) != rank(lane) else 0
                    plist.append((gid[(KIND_F, x, up_lane)], c))
        else:
            if lane < hi:
                c = int(inst.unit_comm[u]) if rank(lane + 1) != rank(lane) else 0
                plist.append((gid[(KIND_B, u, lane + 1)], c))
            elif s == inst.n_seg - 1:
                plist.append((gid[(KIND_F, u, lane)], 0))
            else:
                dn_lane = inst.seg_lo[s + 1]
                for y in inst.units_of(s + 1, mb):
                    c = inst.join_comm(u, y) if rank(dn_lane) != rank(lane) else 0
                    plist.append((gid[(KIND_B, y, dn_lane)], c))
        plist.sort()
        preds.append(plist)

    pred_ptr = np.zeros(N + 1, np.int32)
    pred_ptr[1:] = np.cumsum([len(p) for p in preds])
    pred_op = np.array([p for pl in preds for (p, _) in pl], np.int32)
    edge_comm = np.array([c for pl in preds for (_, c) in pl], np.int32)

    op_kind = np.array([k for (_, _, k) in lane_rows], np.uint8)
    op_lane = np.array([l for (l, _, _) in lane_rows], np.int32)
    op_unit = np.array([u for (_, u, _) in lane_rows], np.int32)
    op_mb = inst.unit_mb[op_unit].astype(np.int32)
    op_slot = np.array(slot_of, np.int32)
    op_cost = np.array([inst.fcost[l, u] if k == KIND_F else inst.bcost[l, u]
                        for (l, u, k) in lane_rows], np.int64)
    slot_act = np.zeros(n_slots, np.int64)
    for g, (l, u, k) in enumerate(lane_rows):
        if k == KIND_F:
            slot_act[slot_of[g]] = inst.act[l, u]
    for arr in (op_cost, slot_act):
        if arr.size and (arr.min() < 0 or arr.max() > np.iinfo(np.int32).max):
            raise ValueError("cost or activation outside int32 range")
    return Problem(
        n_ranks=P, n_ops=n_ops, rank_off=rank_off, pred_ptr=pred_ptr,
        pred_op=pred_op, op_kind=op_kind, op_slot=op_slot, n_slots=n_slots,
        mem_cap=np.full(P, inst.mem_cap, np.int32),
        op_cost=op_cost.astype(np.int32), edge_comm=edge_comm,
        slot_act=slot_act.astype(np.int32),
        stride=round_up(max(N, 1), stride_align),
        op_lane=op_lane, op_unit=op_unit, op_mb=op_mb, inst=inst)


# --------------------------------------------------------------------------
# Samplers: synthetic stand-ins for the paper's (absent) multimodal datasets.
# --------------------------------------------------------------------------

def _split_even(total: int, parts: int) -> list:
    return [total // parts + (1 if k < total % parts else 0) for k in range(parts)]


def _vlm_samples(rng, M):
    images = rng.poisson(2.0, size=M)
    text = np.clip(np.rint(rng.lognormal(6.5, 0.8, size=M)), 1, 8192).astype(np.int64)
    return images.astype(np.int64), text


def _diff_samples(rng, M):
    frames = rng.integers(8, 65, size=M).astype(np.int64)
    prompt = np.maximum(1, np.rint(rng.lognormal(5.0, 0.5, size=M))).astype(np.int64)
    return frames, prompt


def _vlm_pieces(images: int) -> list:
    """Vision pieces of one sample: clamp(#images, 1, 4), images spread evenly."""
    p = min(max(int(images), 1), 4)
    return [IMG_TOKENS * n for n in _split_even(int(images), p)]


def _vae_pieces(frames: int) -> list:
    p = (int(frames) + FRAMES_PER_VAE_PIECE - 1) // FRAMES_PER_VAE_PIECE
    return [VIDEO_PATCHES * n for n in _split_even(int(frames), p)]


def sample_units(cfg: WorkloadConfig, rng) -> list:
    """Per segment, per microbatch: the list of piece token counts."""
    M = cfg.samples
    nseg = len(cfg.segments)
    pieces = [[None] * M for _ in range(nseg)]
    if cfg.sampler == "uniform":
        for j in range(M):
            pieces[0][j] = [0]
    elif cfg.sampler == "vlm":
        images, text = _vlm_samples(rng, M)
        for j in range(M):
            pieces[0][j] = _vlm_pieces(images[j])
            pieces[1][j] = [int(text[j] + IMG_TOKENS * images[j])]
    elif cfg.sampler == "diffusion":
        frames, prompt = _diff_samples(rng, M)
        for j in range(M):
            pieces[0][j] = [int(prompt[j])]
            pieces[1][j] = [int(frames[j] * VIDEO_PATCHES)]
            pieces[2][j] = _vae_pieces(frames[j])
    elif cfg.sampler == "mixed":
        is_vlm = rng.random(M) < 0.5
        images, text = _vlm_samples(rng, M)
        frames, prompt = _diff_samples(rng, M)
        for j in range(M):
            if is_vlm[j]:
                pieces[0][j] = _vlm_pieces(images[j])
                pieces[1][j] = [int(text[j] + IMG_TOKENS * images[j])]
                pieces[2][j] = [0]
            else:
                pieces[0][j] = [0]
                pieces[1][j] = [int(prompt[j])]
                pieces[2][j] = [int(frames[j] * VIDEO_PATCHES)]
    else:
        raise ValueError(cfg.sampler)
    return pieces


def make_instance(cfg: WorkloadConfig | int, seed: int | None = None) -> Instance:
    if not isinstance(cfg, WorkloadConfig):
        cfg = get(cfg)
    seed = cfg.seed if seed is None else seed
    rng = np.random.default_rng(np.random.SeedSequence([seed, cfg.cid, 1]))
    pieces = sample_units(cfg, rng)
    useg, umb, upc, utok = [], [], [], []
    for s in range(len(cfg.segments)):
        for j in range(cfg.samples):
            for k, tok in enumerate(pieces[s][j]):
                useg.append(s)
                umb.append(j)
                upc.append(k)
                utok.append(tok)
    U = len(useg)
    L = cfg.L
    useg = np.array(useg, np.int64)
    utok = np.array(utok, np.int64)
    fcost = np.zeros((L, U), np.int64)
    act = np.zeros((L, U), np.int64)
    if cfg.sampler == "uniform":
        lo, hi = cfg.uniform_cost
        draws = rng.integers(lo, hi + 1, size=(L, cfg.samples))
        for u in range(U):
            fcost[:, u] = draws[:, umb[u]]
        act[:, :] = 1
    else:
        for u in range(U):
            seg = cfg.segments[useg[u]]
            f = op_cost_from_tokens(utok[u], seg.a100, seg.c100)
            a = int(utok[u]) * seg.layers * cfg.act_mult
            for lane in range(seg.lane_lo, seg.lane_hi + 1):
                fcost[lane, u] = f
                act[lane, u] = a
    if cfg.fixed_comm >= 0:
        ucomm = np.full(U, cfg.fixed_comm, np.int64)
    else:
        ucomm = np.array([comm_from_tokens(t) for t in utok], np.int64)
    return Instance(
        P=cfg.P, v=cfg.v,
        seg_lo=[s.lane_lo for s in cfg.segments],
        seg_hi=[s.lane_hi for s in cfg.segments],
        unit_seg=useg, unit_mb=np.array(umb, np.int64),
        unit_piece=np.array(upc, np.int64), unit_tok=utok,
        fcost=fcost, bcost=2 * fcost, act=act, unit_comm=ucomm,
        mem_cap=cfg.mem_cap_units, name=cfg.name)


def make_problem(cfg: WorkloadConfig | int, seed: int | None = None) -> Problem:
    return compile_instance(make_instance(cfg, seed))


def pipeline_instance(P: int, M: int, fcost, bcost=None, comm: int = 0,
                      act: int = 1, v: int = 1, mem_cap: int = -1) -> Instance:
    """One segment over all P*v lanes, M microbatches of one unit each.

    ``fcost`` is a scalar, or an array [L] (per lane) or [L, M].
    """
    L = P * v
    f = np.broadcast_to(np.asarray(fcost, np.int64).reshape(
        (L, 1) if np.ndim(fcost) == 1 else np.shape(fcost) or ()), (L, M)).copy()
    b = 2 * f if bcost is None else np.broadcast_to(np.asarray(bcost, np.int64).reshape(
        (L, 1) if np.ndim(bcost) == 1 else np.shape(bcost) or ()), (L, M)).copy()
    return Instance(
        P=P, v=v, seg_lo=[0], seg_hi=[L - 1],
        unit_seg=np.zeros(M, np.int64), unit_mb=np.arange(M, dtype=np.int64),
        unit_piece=np.zeros(M, np.int64), unit_tok=np.zeros(M, np.int64),
        fcost=f, bcost=b, act=np.full((L, M), act, np.int64),
        unit_comm=np.full(M, comm, np.int64), mem_cap=mem_cap,
        name=f"pipeline_P{P}_M{M}")
