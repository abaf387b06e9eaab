"""The five synthetic workloads, as data.

Every constant that shapes an instance lives here: ranks, lanes, segment lane
ranges, cost coefficients, activation model, memory caps, candidate counts and
the candidate-order recipe.  Nothing in this module computes a schedule.

Readings of the paper that these constants encode (DIP, arXiv 2504.14145):

* Separated partitioning (Sec. 3.1): each modality module owns a contiguous
  range of pipeline lanes ("segment"); lane l sits on physical rank l mod P,
  so with v lanes per rank the placement is the interleaved (virtual-stage)
  one of Megatron-LM.
* Sub-microbatches (Sec. 4, "Construct Sub-Microbatch"): a sample is split
  into modality-specific pieces; a module with nothing to do for a sample
  still gets one zero-token piece so every microbatch crosses every segment.
* Per-op cost in integer microseconds,
  F = floor((a100 * tok * 1e4 + c100 * tok^2) / 1e6), i.e. a*tok + c*tok^2/1e4
  with a = a100/100 and c = c100/100; backward costs 2*F.
* Point-to-point latency tok * hidden(4096) * 2 B / 400 GB/s, rounded up to
  whole microseconds, only between different physical ranks.
* Activation memory of a (lane, unit) pair: tokens * layers_per_lane * kappa
  units of 8 KiB (2 B * hidden 4096 per token-layer).  Layer counts follow the
  8B-scale model table (ViT 5B: 63 layers, Llama3 8B: 32, DiT 5B: 28) divided
  over the segment's lanes, rounded up.  With those counts the per-rank caps
  (64 GiB, 96 GiB) would never bind, so kappa is fixed per workload from a
  pilot of candidates so that roughly 15-20% of candidates exceed the cap.
"""
from __future__ import annotations

from dataclasses import dataclass, field

GIB_IN_UNITS = (1 << 30) // 8192  # 1 GiB expressed in 8 KiB activation units


@dataclass(frozen=True)
class SegmentSpec:
    name: str
    lane_lo: int
    lane_hi: int          # inclusive
    a100: int             # linear cost coefficient x100 (us per token)
    c100: int             # quadratic coefficient x100 (us per token^2 / 1e4)
    layers: int           # model layers per lane (activation model)


@dataclass(frozen=True)
class WorkloadConfig:
    cid: int
    name: str
    P: int                      # physical pipeline ranks
    v: int                      # lanes (virtual stages) per rank
    segments: tuple             # SegmentSpec, in pipeline order
    samples: int                # microbatches per batch
    sampler: str                # 'uniform' | 'vlm' | 'diffusion' | 'mixed'
    n_cand: int                 # candidates per batch
    order_mode: str             # '1f1b' | 'list'
    max_swaps: int              # k ~ U{0..max_swaps} random adjacent swaps
    pool: int                   # 0: fresh list order per candidate; else pool size
    mem_cap_units: int          # per-rank cap in 8 KiB units; -1 = none
    act_mult: int = 1           # kappa, integer multiplier on layers per lane
    chunk: int = 0              # candidates per streamed chunk (0 = one launch)
    seed: int = 0
    fixed_comm: int = -1        # >= 0: this latency on every cross-rank edge
    uniform_cost: tuple = (50, 500)
    notes: str = field(default="", compare=False)

    @property
    def L(self) -> int:
        return self.P * self.v


VIT = dict(a100=100, c100=25)
LLM = dict(a100=50, c100=50)
TEXTENC = dict(a100=50, c100=0)
DIT = dict(a100=10, c100=5)
VAEDEC = dict(a100=5, c100=0)

CONFIGS = {
    1: WorkloadConfig(
        cid=1, name="tiny", P=4, v=1,
        segments=(SegmentSpec("stage", 0, 3, 0, 0, 1),),
        samples=8, sampler="uniform", n_cand=1024,
        order_mode="1f1b", max_swaps=8, pool=0, mem_cap_units=-1,
        fixed_comm=10,
        notes="F ~ U{50..500} per (stage, microbatch), B = 2F, 10 us comm, act 1"),
    2: WorkloadConfig(
        cid=2, name="vlm_s8", P=8, v=1,
        segments=(SegmentSpec("vit", 0, 1, layers=32, **VIT),
                  SegmentSpec("llm", 2, 7, layers=6, **LLM)),
        samples=32, sampler="vlm", n_cand=65536,
        order_mode="list", max_swaps=2, pool=0, mem_cap_units=-1),
    3: WorkloadConfig(
        cid=3, name="vlm_interleaved_16x2", P=16, v=2,
        segments=(SegmentSpec("vit", 0, 7, layers=8, **VIT),
                  SegmentSpec("llm", 8, 31, layers=2, **LLM)),
        samples=64, sampler="vlm", n_cand=262144,
        order_mode="list", max_swaps=0, pool=0,
        mem_cap_units=64 * GIB_IN_UNITS, act_mult=48),
    4: WorkloadConfig(
        cid=4, name="diffusion_s32", P=32, v=1,
        segments=(SegmentSpec("textenc", 0, 3, layers=8, **TEXTENC),
                  SegmentSpec("dit", 4, 27, layers=2, **DIT),
                  SegmentSpec("vaedec", 28, 31, layers=1, **VAEDEC)),
        samples=128, sampler="diffusion", n_cand=1048576,
        order_mode="list", max_swaps=4, pool=1024,
        mem_cap_units=96 * GIB_IN_UNITS, act_mult=5),
    5: WorkloadConfig(
        cid=5, name="large_16x4", P=16, v=4,
        segments=(SegmentSpec("enc", 0, 7, layers=8, **VIT),
                  SegmentSpec("llm", 8, 55, layers=1, **LLM),
                  SegmentSpec("ditdec", 56, 63, layers=4, **DIT)),
        samples=256, sampler="mixed", n_cand=4194304,
        order_mode="list", max_swaps=4, pool=1024,
        mem_cap_units=96 * GIB_IN_UNITS, act_mult=11, chunk=262144),
}


def get(cid: int) -> WorkloadConfig:
    return CONFIGS[int(cid)]
