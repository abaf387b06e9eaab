#!/usr/bin/env python3
"""Throughput of batched pipeline-schedule simulation on one GPU.

One step = one pass of the hot path over one batch: simulate every candidate
of the batch (makespan, per-rank bubble, per-rank peak activation memory,
flags) and reduce the batch to its best (makespan, index).  Inputs are seeded
synthetic candidates already resident in device memory when timing starts.

Default workload: the large 16-rank x 4-virtual-stage instance (vision
encoder, LLM and DiT decoder segments, 256 mixed samples, 34,896 ops per
candidate), one resident 262,144-candidate chunk of its 4,194,304-candidate
stream per batch.  --stream additionally streams all 4,194,304 candidates
from pinned host memory (reported under its own key, host-link inclusive).

With --path mcts a step is one iteration of the MCTS segment reordering
(Sec. 5.1): tree selection and expansion on the host, then one batch of
rollouts -- random completions drawn, interleaved and scored on the GPU --
and backpropagation; the line also compares the best makespan found with
random exploration given the same number of rollouts.

With --path memopt a step is Sec. 5.3's per-layer memory optimisation of a
batch of candidate schedules: for every schedule and rank, one memory
candidate per stage pair under a cap that binds (60 % of the median
keep-everything peak).

With --path cost a step builds the operator-level cost tables (Sec. 6.1) of
a batch of configurations (efficiency factors swept per operator kind) for
every stage and cross-rank edge of the workload.

With --path greedy a step is instead the dual-queue interleaving (Sec. 5.2)
of one batch of priority vectors -- build every candidate's orders, score
them -- followed by the same argmin; the priority vectors stand in for MCTS
rollouts (a random segment sequence each) and are resident before timing.

Prints one JSON line.  Besides the throughput it carries
  roofline      the dominant kernel (the timing simulation) against the bound
                its counters show, vector (integer ALU) issue: the algorithm's
                int32 operations per launch -- 5 per simulated op -- over its
                average launch time, from HIP events the library records on
                the launch stream around each kernel, against 256 CUs x 64
                lanes x 2.4 GHz = 39.3 TOP/s; "traffic" is the HBM bytes per
                launch measured with rocprofv3 counters for the same kernel
                source (a summary under profiles/ keyed by the source hash),
                null when the source changed since;
  hbm           the same kernel's algorithmic HBM bytes per launch -- 2 bytes
                per order entry read + the outputs written -- per second,
                against the 8 TB/s HBM peak;
  issue         the committed counters' vector-issue figures for it;
  cpu_baseline  the CPU oracle timed on this host on bounded samples of the
                same workload: all host cores (the value), one core, and the
                CPU model.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "pool_kernel_traffic.md")
GREEDY_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "greedy_kernel_traffic.md")
SIM_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "sim_kernel_traffic.md")
CSRC = os.path.join(ROOT, "paper_2504_14145_amd", "csrc")
POOL_SOURCES = [os.path.join(CSRC, f) for f in ("kern_pool.hip", "internal.h", "dev_util.h")]
SIM_SOURCES = [os.path.join(CSRC, f) for f in ("kern_sim.hip", "internal.h", "dev_util.h")]
GREEDY_SOURCES = [os.path.join(CSRC, f) for f in ("kern_greedy.hip", "internal.h", "dev_util.h")]
MEMOPT_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "memopt_wave_kernel_traffic.md")
MEMOPT_SOURCES = [os.path.join(CSRC, f) for f in ("kern_memopt.hip", "internal.h", "dev_util.h")]
COST_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "cost_table_kernel_traffic.md")
COST_SOURCES = [os.path.join(CSRC, "kern_costmodel.hip"), os.path.join(ROOT, "include", "dip_sim.h")]


def source_hash(files) -> str:
    h = hashlib.sha256()
    for f in files:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def pool_source_hash() -> str:
    return source_hash(POOL_SOURCES)


def measured_traffic(workload: str, n_cand: int, slots: int, path: str = TRAFFIC_FILE,
                     sources=POOL_SOURCES):
    """HBM bytes per launch of a kernel from its committed counter summary, if
    it was taken on this kernel source, workload, batch and size parameter
    (pool slots, or the greedy's inbox size)."""
    if not os.path.exists(path):
        return None
    want = f"{source_hash(sources)} {workload} {n_cand} {slots}"
    for line in open(path):
        m = re.match(r"\s*traffic:\s*(\S+ \S+ \d+ \d+)\s+fetch_bytes=(\d+)\s+write_bytes=(\d+)", line)
        if m and m.group(1) == want:
            return int(m.group(2)) + int(m.group(3))
    return None


N_SIMD = 1024          # 256 CUs x 4 SIMDs
N_XCD = 8
VALU_CYCLES = 4        # a wave-wide vector instruction on a 16-lane SIMD


def measured_issue(workload: str, n_cand: int, slots: int, path: str = TRAFFIC_FILE,
                   sources=POOL_SOURCES):
    """Share of the launch the SIMDs spent issuing vector instructions, from
    the committed counter summary (SQ_INSTS_VALU x 4 cycles over 1,024 SIMDs
    and GRBM_GUI_ACTIVE / 8 cycles), if taken on this kernel source, workload,
    batch and size parameter."""
    if not os.path.exists(path):
        return None
    want = f"{source_hash(sources)} {workload} {n_cand} {slots}"
    for line in open(path):
        m = re.match(r"\s*issue:\s*(\S+ \S+ \d+ \d+)\s+valu_insts=(\d+)\s+salu_insts=(\d+)"
                     r"\s+gui_active=(\d+)", line)
        if m and m.group(1) == want:
            valu, salu, gui = int(m.group(2)), int(m.group(3)), int(m.group(4))
            cycles = gui / N_XCD
            return {"valu_busy": valu * VALU_CYCLES / (N_SIMD * cycles), "valu_insts": valu,
                    "salu_insts": salu, "cycles": cycles,
                    "source": os.path.relpath(path, ROOT)}
    return None


def calib_copies(args, dev):
    """Plain device copies of args.calib_copy_mib MiB (a kernel of known size
    for scaling HBM byte counters), after the timed work."""
    import torch
    if args.calib_copy_mib:
        nb = args.calib_copy_mib << 20
        src = torch.empty(nb, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copies: 3 x {nb} bytes")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


# int32 lane operations per second: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz
ALU_PEAK_INT_OPS = 256 * 64 * 2.4e9
# the algorithm's int32 operations per simulated op: add the latency, max with
# the rank's free time, add the cost, the memory delta, the running peak
INT_OPS_PER_SIM_OP = 5


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_oracle_baseline(prob, rows, seconds: float) -> dict:
    """The CPU oracle on this host's cores, on consecutive candidates of the
    batch (never repeated), each leg bounded by ``seconds`` of wall time:
    candidate-parallel on every core this process may use (the value), then
    single-threaded."""
    import oracle

    visible = len(os.sched_getaffinity(0))
    # the host's CPU share for this process: OMP_NUM_THREADS where the
    # machine sets it (one GPU's share of a shared host), else every core
    share = int(os.environ.get("OMP_NUM_THREADS", "0") or 0)
    cores = max(1, min(visible, share) if share > 0 else visible)
    n = int(rows.shape[0])

    def leg(threads, block, start):
        done, t0, i = 0, time.perf_counter(), start
        while True:
            b = min(block, n - i) if i < n else 0
            if b == 0:
                i, b = 0, min(block, n)
            oracle.evaluate(prob, rows[i:i + b], threads=threads)
            done += b
            i += b
            dt = time.perf_counter() - t0
            if dt >= seconds:
                return done, dt, i

    d_all, t_all, nxt = leg(cores, 64 * cores, 0)
    d_one, t_one, _ = leg(1, 16, nxt)
    return {"value": d_all / t_all, "unit": "candidates/s", "cores": cores, "kind": "oracle",
            "ops_per_s": d_all * prob.n_total / t_all,
            "sample": f"{d_all} consecutive candidates of the batch on {cores} threads "
                      f"({t_all:.1f} s wall)",
            "one_core": {"value": d_one / t_one, "unit": "candidates/s",
                         "ops_per_s": d_one * prob.n_total / t_one,
                         "sample": f"the next {d_one} candidates on one thread ({t_one:.1f} s)"},
            "cpu_model": cpu_model(), "host_cpus_visible": visible}


# the candidates the oracle is timed on per workload: all of the three
# smaller ones, fixed prefixes of the two larger
ORACLE_PREFIX = {1: 1024, 2: 65536, 3: 262144, 4: 65536, 5: 16384}


def run_oracle_timing(args):
    """The CPU oracle alone (no GPU work): every workload's prefix on one
    thread, then candidate-parallel on this process's share of the host's
    cores, and what a full parity sweep of the workload takes at that rate."""
    import numpy as np   # noqa: F401  (the generator's arrays)
    import oracle
    import workloads as W

    visible = len(os.sched_getaffinity(0))
    share = int(os.environ.get("OMP_NUM_THREADS", "0") or 0)
    cores = max(1, min(visible, share) if share > 0 else visible)
    per = {}
    for cid in sorted(ORACLE_PREFIX):
        cfg = W.get(cid)
        prob = W.make_problem(cfg)
        n = min(ORACLE_PREFIX[cid], args.n_cand or ORACLE_PREFIX[cid])
        rows = W.generator_for(prob, cfg).generate(0, n)
        t0 = time.perf_counter()
        one = oracle.evaluate(prob, rows, threads=1)
        t_one = time.perf_counter() - t0
        t0 = time.perf_counter()
        par = oracle.evaluate(prob, rows, threads=cores)
        t_all = time.perf_counter() - t0
        assert (one.makespan == par.makespan).all() and (one.flags == par.flags).all()
        ops = n * prob.n_total
        per[cfg.name] = {
            "candidates": n, "ops_per_candidate": int(prob.n_total),
            "one_core": {"seconds": t_one, "candidates_per_s": n / t_one, "ops_per_s": ops / t_one},
            "all_cores": {"threads": cores, "seconds": t_all, "candidates_per_s": n / t_all,
                          "ops_per_s": ops / t_all},
            "full_sweep_s_at_all_cores": cfg.n_cand / (n / t_all),
        }
        log(f"[bench] oracle on {cfg.name}: {n} candidates, one core {n / t_one:.4g}/s "
            f"({ops / t_one:.3g} ops/s), {cores} threads {n / t_all:.4g}/s; a full sweep of "
            f"{cfg.n_cand} candidates would take {cfg.n_cand / (n / t_all):.0f} s")
        if args.oracle_full and cid in args.oracle_full:
            # the whole workload, candidate-parallel, in chunks the generator
            # writes between timed oracle calls
            chunk = 65536
            t_sweep = t_gen = 0.0
            for c0 in range(0, cfg.n_cand, chunk):
                m = min(chunk, cfg.n_cand - c0)
                t0 = time.perf_counter()
                rows = W.generator_for(prob, cfg).generate(c0, m)
                t_gen += time.perf_counter() - t0
                t0 = time.perf_counter()
                oracle.evaluate(prob, rows, threads=cores)
                t_sweep += time.perf_counter() - t0
                if (c0 // chunk) % 8 == 7:
                    log(f"[bench]   full sweep of {cfg.name}: {c0 + m} candidates, "
                        f"{t_sweep:.1f} s of oracle time")
            per[cfg.name]["full_sweep"] = {"candidates": cfg.n_cand, "threads": cores,
                                           "oracle_s": t_sweep, "generator_s": t_gen}
            log(f"[bench] full sweep of {cfg.name}: {cfg.n_cand} candidates in {t_sweep:.1f} s "
                f"on {cores} threads (+ {t_gen:.1f} s generating them)")
    print(json.dumps({"metric": "oracle candidates simulated/sec", "unit": "candidates/s",
                      "kind": "oracle", "cpu_model": cpu_model(), "host_cpus_visible": visible,
                      "threads": cores, "workloads": per, "data": "synthetic"}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=0,
                    help="workload id 1-5 (default: 5 for the simulation, 2 for the other paths)")
    ap.add_argument("--n-cand", type=int, default=0, help="override candidates per batch")
    ap.add_argument("--oracle-full", type=lambda x: [int(c) for c in x.split(",")], default=[],
                    help="with --path oracle: workloads (e.g. 1,2,3,4,5) whose every candidate "
                         "the oracle also simulates, candidate-parallel, with the wall time")
    ap.add_argument("--variant", type=int, default=0)
    ap.add_argument("--wpb", type=int, default=0)
    ap.add_argument("--slots", type=int, default=0, help="pool slots per rank (pool kernel)")
    ap.add_argument("--check", type=int, default=0,
                    help="check kernel (dip_sim_configure_check mode; 0: automatic)")
    ap.add_argument("--inbox", type=int, default=0,
                    help="greedy: fix the first launch's inbox entries per kind (0: adaptive)")
    ap.add_argument("--cpu-seconds", type=float, default=6.0,
                    help="wall-time bound of each CPU oracle baseline leg (all cores, one core)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-steps", type=int, default=10,
                    help="steps re-run after the timed region with per-kernel events")
    ap.add_argument("--stream", action="store_true",
                    help="also stream the configuration's full candidate count from pinned host "
                         "memory in chunks on two streams (copy/compute overlap); reported "
                         "separately, host-link inclusive (the default for workloads larger "
                         "than one chunk)")
    ap.add_argument("--no-stream", action="store_true", help="skip that stream")
    ap.add_argument("--path", choices=("simulate", "greedy", "mcts", "search", "cost", "memopt",
                                        "oracle"),
                    default="simulate",
                    help="simulate given orders (default), build them with the greedy, "
                         "search priorities with MCTS over GPU-batched greedy rollouts, or "
                         "compare MCTS with depth-first and random exploration (search)")
    ap.add_argument("--rollouts", type=int, default=16384,
                    help="mcts: rollouts per expansion")
    ap.add_argument("--alpha", type=float, default=1.0, help="mcts/search: UCB exponent")
    ap.add_argument("--beta", type=float, default=0.1, help="mcts/search: UCB exploration weight")
    ap.add_argument("--workers", type=int, default=1,
                    help="mcts/search: tree nodes rolled out per round (parallel search)")
    ap.add_argument("--policies", default="ucb,dfs,random",
                    help="search: strategies to run (ucb, dfs, random)")
    ap.add_argument("--steady-gib", type=float, default=1.0,
                    help="simulate: also time the batch tiled to this many GiB of orders "
                         "(steady state, reported separately; 0 to skip)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after timing, run plain device copies of this many MiB (a known-size "
                         "kernel for scaling HBM byte counters)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU; "
                          f"--gpus {args.gpus} (WORLD_SIZE {world}) is not supported. "
                          "Candidates are independent, so several GPUs would each take a "
                          "contiguous candidate range and min-reduce one 64-bit key."}))
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2504_14145_amd as dip
    import workloads as W

    if not args.config:
        args.config = 5 if args.path == "simulate" else 2
    cfg = W.get(args.config)
    if args.path == "greedy":
        return run_greedy(args, cfg)
    if args.path == "mcts":
        return run_mcts(args, cfg)
    if args.path == "search":
        return run_search(args, cfg)
    if args.path == "cost":
        return run_cost(args, cfg)
    if args.path == "memopt":
        return run_memopt(args, cfg)
    if args.path == "oracle":
        return run_oracle_timing(args)
    n_cand = args.n_cand or (cfg.chunk or cfg.n_cand)
    t0 = time.time()
    prob = W.make_problem(cfg)
    gen = W.generator_for(prob, cfg)
    rows = gen.generate(0, n_cand)
    log(f"[bench] workload {cfg.name}: {n_cand} candidates x {prob.n_total} ops, "
        f"stride {prob.stride}, generated in {time.time() - t0:.1f}s")

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    orders = torch.from_numpy(rows).to(dev)
    sim = dip.Sim(prob)
    if args.check:
        rc = sim.configure_check(args.check)
        if rc != dip.OK:
            raise SystemExit(f"check kernel {args.check} unsupported: {dip.strerror(rc)}")
    if args.slots:
        rc = sim.configure_pool(args.slots)
        if rc != dip.OK:
            raise SystemExit(f"pool slots {args.slots} unsupported: {dip.strerror(rc)}")
    if args.variant or args.wpb:
        rc = sim.configure(args.variant, args.wpb)
        if rc != dip.OK:
            raise SystemExit(f"variant {args.variant}/{args.wpb} unsupported: {dip.strerror(rc)}")
    info = sim.info
    log(f"[bench] kernel config {info}")
    out = sim.outputs(n_cand)
    key = torch.empty(1, dtype=torch.int64, device=dev)
    stream = torch.cuda.current_stream()

    def step(ev_pair=None):
        key.fill_(-1)
        if ev_pair is not None:
            ev_pair[0].record(stream)
        dip.evaluate(sim.h, None, orders, n_cand, *out, stream=stream)
        if ev_pair is not None:
            ev_pair[1].record(stream)
        dip.argmin(sim.h, out[0], out[3], n_cand, 0, key, stream=stream)

    # first call uploads the costs
    dip.evaluate(sim.h, sim.costs, orders, n_cand, *out, stream=stream)
    torch.cuda.synchronize()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    events = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(args.steps):
        step(events[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    kern_ms = [a.elapsed_time(b) for a, b in events]
    kern_avg_s = sum(kern_ms) / len(kern_ms) / 1e3
    best = dip.decode_key(int(key.item()))
    flags = out[3].cpu().numpy()
    log(f"[bench] {args.steps} steps in {wall * 1e3:.2f} ms; sim kernel avg "
        f"{kern_avg_s * 1e6:.1f} us (min {min(kern_ms) * 1e3:.1f} us); best {best}; "
        f"deadlock {np.mean(flags & 1 > 0):.3f} cap {np.mean(flags & 2 > 0):.3f}")

    # per-kernel times: the library records HIP events around each kernel on
    # the launch stream
    dip.profile(sim.h, True)
    per_kernel = []
    for _ in range(max(1, args.profile_steps)):
        step()
        per_kernel.append(dip.last_profile(sim.h))
    dip.profile(sim.h, False)
    retries = dip.last_retries(sim.h) if info["variant"] >= 8 else (0, 0)
    nk = min(len(p) for p in per_kernel)
    kern_avg_ms = [sum(p[i] for p in per_kernel) / len(per_kernel) for i in range(nk)]
    names = {8: ["check", "simulate", "retry"],
             9: ["check", "simulate", "simulate_16", "simulate_32", "retry"]}.get(info["variant"],
                                                                 ["simulate"])[:nk]
    dom = names.index("simulate")
    dom_s = kern_avg_ms[dom] / 1e3
    log(f"[bench] per-kernel avg ms: " + ", ".join(f"{n} {t:.4f}" for n, t in zip(names, kern_avg_ms))
        + f"; retries {retries}")

    calib_copies(args, dev)

    # steady state: the same candidates tiled until the orders fill at least
    # args.steady_gib GiB, so the launch's fixed latency (one candidate's
    # rounds) and its tail are amortised; reported beside, never as, the value
    steady = None
    reps = int(np.ceil(args.steady_gib * (1 << 30) / orders.numel() / orders.element_size()))
    if args.steady_gib > 0 and reps > 1:
        big = orders.repeat(reps, 1)
        nb = int(big.shape[0])
        bout = sim.outputs(nb)
        for _ in range(2):
            dip.evaluate(sim.h, None, big, nb, *bout, stream=stream)
        stream.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(5)]
        for a, b in evs:
            a.record(stream)
            dip.evaluate(sim.h, None, big, nb, *bout, stream=stream)
            b.record(stream)
        stream.synchronize()
        ms = sum(a.elapsed_time(b) for a, b in evs) / len(evs)
        np.testing.assert_array_equal(bout[0][:n_cand].cpu().numpy(), out[0].cpu().numpy())
        steady = {"n_cand": nb, "orders_bytes": int(big.numel() * big.element_size()),
                  "ms_per_evaluate": ms, "value": nb / (ms / 1e3), "unit": "candidates/s",
                  "note": f"the batch tiled {reps}x on the device (same candidates); "
                          "evaluate on HIP events, 5 launches"}
        log(f"[bench] steady state: {nb} candidates ({steady['orders_bytes'] / 2**30:.2f} GiB "
            f"of orders) in {ms:.3f} ms per evaluate: {steady['value']:.3e} candidates/s")
        del big, bout

    stream_rec = None
    if (args.stream or (cfg.chunk and cfg.n_cand > n_cand and not args.n_cand)) and not args.no_stream:
        from paper_2504_14145_amd.stream import ChunkStream
        chunk = n_cand
        total = cfg.n_cand
        # two distinct host chunks, cycled: the copy and the simulation cost the
        # same whatever the orders, and the folded argmin uses global indices
        hosts = [torch.from_numpy(rows).pin_memory(),
                 torch.from_numpy(gen.generate(n_cand, n_cand)).pin_memory()]
        cs = ChunkStream(sim, chunk)
        torch.cuda.synchronize()
        t0s = time.perf_counter()
        done, k = 0, 0
        while done < total:
            n = min(chunk, total - done)
            cs.submit(hosts[k % 2][:n], done)
            done += n
            k += 1
        skey = cs.finish()
        swall = time.perf_counter() - t0s
        sbest = dip.decode_key(int(skey.item()))
        stream_rec = {"candidates": total, "chunk": chunk, "chunks": k, "wall_s": swall,
                      "candidates_per_s": total / swall,
                      "h2d_bytes": int(total) * prob.stride * 2,
                      "h2d_gb_per_s": total * prob.stride * 2 / swall / 1e9,
                      "best": {"index": sbest[0], "makespan_us": sbest[1]},
                      "note": "the workload's first two chunks of orders, pinned, cycled over "
                              "all chunk positions (copy and simulation cost the same whatever "
                              "the orders); best is over that data. The argmin over every "
                              "candidate of the workload, checked against the oracle, is "
                              "recorded in profiles/stream_large_16x4_argmin.md"}
        log(f"[bench] streamed {total} candidates in {k} chunks: {swall:.2f} s, "
            f"{total / swall:.4g} candidates/s (host link inclusive); best {sbest}")

    ms_per_step = wall / args.steps * 1e3
    cand_per_s = n_cand * args.steps / wall
    ops_per_s = cand_per_s * prob.n_total
    P = prob.n_ranks
    bytes_per_cand = 2 * prob.n_total + 4 + 4 * P + 4 * P + 1
    algo_bytes = n_cand * bytes_per_cand
    achieved_gbs = algo_bytes / dom_s / 1e9
    ops_per_launch = n_cand * prob.n_total
    kern_ops_per_s = ops_per_launch / dom_s
    slots = info.get("pool_slots", 0)
    # the counter summary of the simulation kernel that ran (variant 9: the
    # compact-record kernel, variant 8: the pool kernel)
    prof_file, prof_src = {8: (TRAFFIC_FILE, POOL_SOURCES),
                           9: (SIM_TRAFFIC_FILE, SIM_SOURCES)}.get(info["variant"], (None, None))
    traffic = measured_traffic(cfg.name, n_cand, slots, prof_file, prof_src) if prof_file else None

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_oracle_baseline(prob, rows, args.cpu_seconds)
        log(f"[bench] cpu oracle: {cpu['value']:.4g} candidates/s on {cpu['cores']} threads, "
            f"{cpu['one_core']['value']:.4g} on one ({cpu['cpu_model']})")

    rec = {
        "metric": "candidate schedules simulated/sec",
        "value": cand_per_s,
        "unit": "candidates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {"workload": cfg.name, "n_cand": n_cand, "ranks": P, "lanes": cfg.L,
                   "ops_per_candidate": prob.n_total, "microbatches": cfg.samples,
                   "parallelism": "single GPU"},
        "ops_per_s": ops_per_s,
        "evaluate_us": kern_avg_s * 1e6,
        "kernel_us": {n: t * 1e3 for n, t in zip(names, kern_avg_ms)},
        "kernel_variant": info["variant"],
        # candidates whose pools filled in the first simulation pass, and
        # those the second pass (16 slots) handed to the general kernel
        "retries": {"first_pass": retries[0], "second_pass": retries[1]},
        "pool_slots": slots,
        "best": {"index": best[0], "makespan_us": best[1]},
        # the bound the counters show: vector (integer ALU) issue; achieved
        # = the algorithm's int32 operations (INT_OPS_PER_SIM_OP per simulated
        # op) per second of the kernel, against 256 CUs x 64 lanes x 2.4 GHz
        "roofline": {"bound": "alu", "kernel": "simulate",
                     "achieved": kern_ops_per_s * INT_OPS_PER_SIM_OP / 1e12,
                     "peak": ALU_PEAK_INT_OPS / 1e12, "unit": "TOP/s",
                     "frac": kern_ops_per_s * INT_OPS_PER_SIM_OP / ALU_PEAK_INT_OPS,
                     "traffic": traffic,
                     "algorithmic_ops": ops_per_launch * INT_OPS_PER_SIM_OP,
                     "simulated_ops": ops_per_launch, "kernel_ms": dom_s * 1e3},
        # the same kernel against the HBM ceiling: algorithmic bytes (orders
        # read, outputs written) per second, and the bytes the counters saw
        "hbm": {"achieved": achieved_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved_gbs / HBM_PEAK_GBS, "traffic": traffic,
                "algorithmic_bytes": algo_bytes, "bytes_per_candidate": bytes_per_cand},
        # vector issue from the committed counters (VALU busy share)
        "issue": {"counters": measured_issue(cfg.name, n_cand, slots, prof_file, prof_src)
                  if prof_file else None},
        "steady_state": steady,
        "cpu_baseline": cpu,
    }
    if stream_rec is not None:
        rec["stream"] = stream_rec
    print(json.dumps(rec), flush=True)
    sim.close()


def run_greedy(args, cfg):
    """One step: dip_sim_greedy over a batch of priority vectors (orders and
    scores written to device memory), then dip_sim_argmin."""
    import numpy as np
    import torch

    import paper_2504_14145_amd as dip
    import workloads as W

    n_cand = args.n_cand or cfg.n_cand
    t0 = time.time()
    prob = W.make_problem(cfg)
    op_group, G, cls = W.priority_groups(prob)
    prio_np = W.rollout_priorities(cls, n_cand, seed=cfg.seed)
    log(f"[bench] greedy on {cfg.name}: {n_cand} priority vectors x {G} groups, "
        f"{prob.n_total} stages per candidate, drawn in {time.time() - t0:.1f}s")
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    prio = torch.from_numpy(prio_np).to(dev)
    sim = dip.Sim(prob)
    rc = sim.configure_greedy(G, op_group)
    if rc != dip.OK:
        raise SystemExit(f"greedy unsupported on {cfg.name}: {dip.strerror(rc)}")
    if args.inbox and dip.set_greedy_inbox(sim.h, args.inbox) != dip.OK:
        raise SystemExit(f"inbox size {args.inbox} not accepted")
    out = sim.outputs(n_cand)
    orders = torch.empty((n_cand, prob.stride), dtype=torch.int16, device=dev)
    key = torch.empty(1, dtype=torch.int64, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        key.fill_(-1)
        dip.greedy(sim.h, None, prio, n_cand, orders, *out, stream=stream)
        dip.argmin(sim.h, out[0], out[3], n_cand, 0, key, stream=stream)

    dip.greedy(sim.h, sim.costs, prio, n_cand, orders, *out, stream=stream)   # uploads costs
    torch.cuda.synchronize()
    # the inbox size adapts to the overflow counts of earlier calls, each read
    # once its call has finished: warm-up calls wait for the previous one
    for _ in range(max(args.warmup, 6)):
        step()
        torch.cuda.synchronize()
    t_start = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    best = dip.decode_key(int(key.item()))
    flags = out[3].cpu().numpy()

    dip.profile(sim.h, True)
    per_kernel = []
    for _ in range(max(1, args.profile_steps)):
        step()
        per_kernel.append(dip.last_profile(sim.h))
    dip.profile(sim.h, False)
    nk = min(len(p) for p in per_kernel)
    kern_avg_ms = [sum(p[i] for p in per_kernel) / len(per_kernel) for i in range(nk)]
    names = ["greedy", "greedy_retry"][:nk]
    info = sim.info
    log(f"[bench] {args.steps} steps in {wall * 1e3:.2f} ms; per-kernel avg ms: " +
        ", ".join(f"{n} {t:.4f}" for n, t in zip(names, kern_avg_ms)) +
        f"; inbox {info['greedy_inbox']}; best {best}; cap {np.mean(flags & 2 > 0):.3f}")

    calib_copies(args, dev)

    P = prob.n_ranks
    # per candidate: its priority vector read, its orders and scores written
    bytes_per_cand = 4 * G + 2 * prob.n_total + 4 + 8 * P + 1
    algo_bytes = n_cand * bytes_per_cand
    dom_s = kern_avg_ms[0] / 1e3
    achieved_gbs = algo_bytes / dom_s / 1e9
    kern_ops_per_s = n_cand * prob.n_total / dom_s
    cand_per_s = n_cand * args.steps / wall

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        cores = max(1, min(16, len(os.sched_getaffinity(0))))
        sample = min(n_cand, 256)
        done = 0
        tc = time.perf_counter()
        while True:
            oracle.greedy(prob, op_group, G, prio_np[:sample], stride=prob.stride, threads=cores)
            done += sample
            if time.perf_counter() - tc >= args.cpu_seconds:
                break
        dt = time.perf_counter() - tc
        cpu = {"value": done / dt, "unit": "candidates/s", "cores": cores, "kind": "oracle",
               "sample": f"first {sample} priority vectors of the batch, repeated "
                         f"{done // sample}x ({dt:.2f} s wall on {cores} threads)"}
        log(f"[bench] cpu oracle {done / dt:.0f} candidates/s on {cores} threads")

    rec = {
        "metric": "candidate schedules generated and scored/sec (dual-queue greedy)",
        "value": cand_per_s,
        "unit": "candidates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {"workload": cfg.name, "n_cand": n_cand, "ranks": P, "lanes": cfg.L,
                   "stages_per_candidate": prob.n_total, "priority_groups": G,
                   "parallelism": "single GPU"},
        "stages_per_s": cand_per_s * prob.n_total,
        "kernel_us": {n: t * 1e3 for n, t in zip(names, kern_avg_ms)},
        "greedy_inbox": info["greedy_inbox"],
        "best": {"index": best[0], "makespan_us": best[1]},
        "roofline": {"bound": "hbm", "kernel": "greedy", "achieved": achieved_gbs,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved_gbs / HBM_PEAK_GBS,
                     "traffic": measured_traffic(cfg.name, n_cand, info["greedy_inbox"],
                                                 GREEDY_TRAFFIC_FILE, GREEDY_SOURCES),
                     "algorithmic_bytes": algo_bytes},
        "issue": measured_issue(cfg.name, n_cand, info["greedy_inbox"], GREEDY_TRAFFIC_FILE,
                                GREEDY_SOURCES),
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)
    sim.close()


def run_memopt(args, cfg):
    """Steps = dip_sim_memopt over a batch of candidate schedules."""
    import numpy as np
    import torch

    import oracle
    import paper_2504_14145_amd as dip
    import workloads as W
    from workloads.strategies import strategy_table

    n_cand = args.n_cand or (cfg.chunk or cfg.n_cand)
    S = 6
    prob = W.make_problem(cfg)
    tab = strategy_table(prob)
    rows = W.generator_for(prob, cfg).generate(0, n_cand)
    # a cap that binds: 60 % of the median keep-everything peak of a sample
    peak = oracle.evaluate(prob, rows[:min(n_cand, 2048)], threads=16).peak
    prob.mem_cap[:] = int(np.median(peak) * 0.6)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    sim = dip.Sim(prob)
    rc = dip.configure_memopt(sim.h, tab.slot_layers, tab.time, tab.mem, S)
    if rc != dip.OK:
        raise SystemExit(f"memopt unsupported on {cfg.name}: {dip.strerror(rc)}")
    orders = torch.from_numpy(rows).to(dev)
    P = prob.n_ranks
    t_out = torch.empty((n_cand, P), dtype=torch.int64, device=dev)
    p_out = torch.empty((n_cand, P), dtype=torch.int32, device=dev)
    s_out = torch.empty((n_cand, P), dtype=torch.uint8, device=dev)
    log(f"[bench] memopt on {cfg.name}: {n_cand} schedules x {P} ranks, {prob.n_slots} stage "
        f"pairs, {len(tab.time)} layers, cap {prob.mem_cap[0]}, {S} candidates per pair")
    for _ in range(max(args.warmup, 1)):
        dip.memopt(sim.h, orders, n_cand, t_out, p_out, s_out)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    t0 = time.perf_counter()
    for a, b in ev:
        a.record()
        dip.memopt(sim.h, orders, n_cand, t_out, p_out, s_out)
        b.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    k_s = sum(a.elapsed_time(b) for a, b in ev) / len(ev) / 1e3
    st = s_out.cpu().numpy()
    log(f"[bench] {args.steps} steps in {wall * 1e3:.2f} ms; kernel {k_s * 1e3:.3f} ms; "
        f"within cap {np.mean((st == 1) | (st == 3)):.3f} (proven within 5 %: "
        f"{np.mean(st == 1):.3f}), out of reach {np.mean(st == 0):.3f}")
    calib_copies(args, dev)

    cpu = None
    if not args.no_cpu_baseline:
        import oracle.memopt as MO
        cands = MO.pair_candidates(tab, S)
        sample = min(n_cand, 64)
        tc = time.perf_counter()
        done = 0
        while True:
            MO.optimise(prob, tab, cands, rows[:sample])
            done += sample
            if time.perf_counter() - tc >= args.cpu_seconds:
                break
        dt = time.perf_counter() - tc
        cpu = {"value": done / dt, "unit": "schedules/s", "cores": 1, "kind": "oracle",
               "sample": f"first {sample} schedules, {done // sample}x ({dt:.2f} s, one thread)"}
        log(f"[bench] cpu oracle {done / dt:.0f} schedules/s")

    bytes_per = 2 * prob.n_total + P * (8 + 4 + 1)
    rec = {
        "metric": "candidate schedules memory-optimised/sec (per-layer strategies, Sec. 5.3)",
        "value": n_cand * args.steps / wall,
        "unit": "schedules/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {"workload": cfg.name, "n_cand": n_cand, "ranks": P,
                   "stage_pairs": prob.n_slots, "candidates_per_pair": S,
                   "cap_units": int(prob.mem_cap[0]), "parallelism": "single GPU"},
        "kernel_us": {"memopt": k_s * 1e6},
        "within_cap": float(np.mean((st == 1) | (st == 3))),
        "proven_within_5pct": float(np.mean(st == 1)),
        "roofline": {"bound": "hbm", "kernel": "memopt",
                     "achieved": n_cand * bytes_per / k_s / 1e9, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": n_cand * bytes_per / k_s / 1e9 / HBM_PEAK_GBS,
                     "traffic": measured_traffic(cfg.name, n_cand, S, MEMOPT_TRAFFIC_FILE,
                                                 MEMOPT_SOURCES),
                     "algorithmic_bytes": n_cand * bytes_per},
        "issue": measured_issue(cfg.name, n_cand, S, MEMOPT_TRAFFIC_FILE, MEMOPT_SOURCES),
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)
    sim.close()


FP64_OPS_PEAK = 78.6e12 / 2   # vector float64: 78.6 TFLOP/s counts an FMA as two


def run_cost(args, cfg):
    """Steps = dip_cost_tables over args.n_cand configurations (default 16384)."""
    import numpy as np
    import torch

    import paper_2504_14145_amd as dip
    import workloads as W
    from workloads.operators import N_KINDS, coefficient_sweep, operator_table

    n_conf = args.n_cand or 16384
    prob = W.make_problem(cfg)
    tab = operator_table(prob)
    rows, items = len(tab.kind), len(tab.item_ptr) - 1
    coef_np = coefficient_sweep(n_conf, seed=cfg.seed)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    dt = dip.DeviceOpTable(tab, N_KINDS, dev)
    coef = torch.from_numpy(coef_np).to(dev)
    out = torch.empty((n_conf, items), dtype=torch.int32, device=dev)
    log(f"[bench] cost tables on {cfg.name}: {items} items ({prob.n_total} stages, "
        f"{prob.n_edges} edges), {rows} operator rows, {n_conf} configurations")
    for _ in range(max(args.warmup, 1)):
        dip.cost_tables(dt, coef, out)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    t0 = time.perf_counter()
    for a, b in ev:
        a.record()
        dip.cost_tables(dt, coef, out)
        b.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    k_s = sum(a.elapsed_time(b) for a, b in ev) / len(ev) / 1e3
    ops = 6.0 * rows * n_conf        # per row: three products, two maxima, one sum
    log(f"[bench] {args.steps} steps in {wall * 1e3:.2f} ms; kernel {k_s * 1e3:.3f} ms; "
        f"{ops / k_s / 1e12:.2f} T float64 ops/s")
    calib_copies(args, dev)

    cpu = None
    if not args.no_cpu_baseline:
        import oracle.costmodel as OC
        sample = 2
        tc = time.perf_counter()
        done = 0
        while True:
            OC.cost_tables(tab, coef_np[:sample])
            done += sample
            if time.perf_counter() - tc >= args.cpu_seconds:
                break
        dt_c = time.perf_counter() - tc
        cpu = {"value": done * items / dt_c, "unit": "table entries/s", "cores": 1,
               "kind": "oracle",
               "sample": f"{done} configurations x {items} items ({dt_c:.2f} s wall, one thread)"}
        log(f"[bench] cpu oracle {done * items / dt_c:.0f} entries/s")

    rec = {
        "metric": "operator-level cost-table entries built/sec (Sec. 6.1)",
        "value": n_conf * items * args.steps / wall,
        "unit": "table entries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": cfg.name, "configurations": n_conf, "items": items,
                   "operator_rows": rows, "parallelism": "single GPU"},
        "kernel_us": {"cost_table": k_s * 1e6},
        "roofline": {"bound": "alu", "kernel": "cost_table", "achieved": ops / k_s / 1e12,
                     "peak": FP64_OPS_PEAK / 1e12, "unit": "T float64 ops/s",
                     "frac": ops / k_s / FP64_OPS_PEAK,
                     "traffic": measured_traffic(cfg.name, n_conf, N_KINDS, COST_TRAFFIC_FILE,
                                                 COST_SOURCES),
                     "algorithmic_bytes": n_conf * items * 4 + coef_np.nbytes + rows * 25},
        "issue": measured_issue(cfg.name, n_conf, N_KINDS, COST_TRAFFIC_FILE, COST_SOURCES),
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)


def run_mcts(args, cfg):
    """Steps = MCTS iterations with args.rollouts GPU rollouts each."""
    import numpy as np
    import torch

    import paper_2504_14145_amd as dip
    from paper_2504_14145_amd.mcts import Search
    import workloads as W

    R = args.rollouts
    prob = W.make_problem(cfg)
    op_group, G, cls = W.priority_groups(prob)
    n_cls = int(cls.max()) + 1
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    sim = dip.Sim(prob)
    rc = sim.configure_greedy(G, op_group)
    if rc != dip.OK:
        raise SystemExit(f"greedy unsupported on {cfg.name}: {dip.strerror(rc)}")
    sim.greedy(torch.zeros((1, G), dtype=torch.int32, device=dev))      # uploads the costs
    log(f"[bench] mcts on {cfg.name}: {n_cls} segment classes, {G} groups, "
        f"{prob.n_total} stages, {R} rollouts per expansion")

    search = Search(sim, cls, R, seed=cfg.seed, alpha=args.alpha, beta=args.beta,
                    workers=args.workers)
    for t in range(args.warmup):            # warm-up rounds are part of the search
        search.step(t)
    torch.cuda.synchronize()
    leaves0 = search.leaves
    t0 = time.perf_counter()
    for t in range(args.warmup, args.warmup + args.steps):
        search.step(t)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    timed_rollouts = (search.leaves - leaves0) * R
    iters = args.warmup + args.steps
    mcts_best = search.best[0]

    # per-kernel times of one more iteration's batch
    dip.profile(sim.h, True)
    key = torch.full((1,), -1, dtype=torch.int64, device=dev)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record()
    dip.rollouts(sim.h, [], R, cfg.seed, 10**6, search.prio, search.ms, search.fl, key)
    ev[1].record()
    torch.cuda.synchronize()
    k_ms = dip.last_profile(sim.h)
    batch_ms = ev[0].elapsed_time(ev[1])
    dip.profile(sim.h, False)

    # random exploration with the same number of rollouts (empty prefix)
    best_rand = float("inf")
    left, t = search.leaves * R, 0
    while left > 0:
        b = min(left, R * args.workers)
        key.fill_(-1)
        dip.rollouts(sim.h, [], b, cfg.seed + 1, t, search.prio, search.ms, search.fl, key)
        k = dip.decode_key(int(key.item()))
        if k[0] >= 0:
            best_rand = min(best_rand, float(k[1]))
        left -= b
        t += 1
    log(f"[bench] {args.steps} rounds of {args.workers} leaves in {wall * 1e3:.1f} ms; batch "
        f"{batch_ms:.3f} ms (greedy kernels {k_ms}); best makespan mcts {mcts_best} vs random "
        f"{best_rand} after {search.leaves * R} rollouts each")
    inbox = sim.info["greedy_inbox"]
    calib_copies(args, dev)

    cpu = None
    if not args.no_cpu_baseline:
        import oracle.mcts as OM
        cores = max(1, min(16, len(os.sched_getaffinity(0))))
        r_cpu = min(R, 1024)
        tc = time.perf_counter()
        it_cpu = 0
        while True:
            it_cpu += 1
            OM.search(prob, op_group, G, cls, it_cpu, r_cpu, seed=cfg.seed, threads=cores)
            if time.perf_counter() - tc >= args.cpu_seconds:
                break
        dt = time.perf_counter() - tc
        done = r_cpu * it_cpu * (it_cpu + 1) // 2      # searches of 1 .. it_cpu iterations
        cpu = {"value": done / dt, "unit": "rollouts/s", "cores": cores, "kind": "oracle",
               "sample": f"oracle searches of 1..{it_cpu} iterations x {r_cpu} rollouts "
                         f"({dt:.2f} s wall on {cores} threads)"}
        log(f"[bench] cpu oracle {done / dt:.0f} rollouts/s on {cores} threads")

    P = prob.n_ranks
    bytes_per_rollout = 4 * G + 4 + 8 * P + 1 + 4 * G     # priorities written then read, scores
    greedy_ms = k_ms[0] if k_ms else batch_ms
    rec = {
        "metric": "MCTS rollouts interleaved and scored/sec (segment reordering, Sec. 5.1)",
        "value": timed_rollouts / wall,
        "unit": "rollouts/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {"workload": cfg.name, "rollouts_per_leaf": R, "workers": args.workers, "segment_classes": n_cls,
                   "priority_groups": G, "stages_per_candidate": prob.n_total,
                   "parallelism": "single GPU"},
        "batch_ms": batch_ms,
        "greedy_inbox": inbox,
        "kernel_us": {n: t * 1e3 for n, t in zip(["greedy", "greedy_retry"], k_ms)},
        "search": {"rounds": iters, "workers": args.workers, "rollouts_each": search.leaves * R,
                   "mcts_best_makespan_us": mcts_best, "random_best_makespan_us": best_rand},
        "roofline": {"bound": "hbm", "kernel": "greedy",
                     "achieved": R * bytes_per_rollout / (greedy_ms / 1e3) / 1e9,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": R * bytes_per_rollout / (greedy_ms / 1e3) / 1e9 / HBM_PEAK_GBS,
                     "traffic": measured_traffic(cfg.name, R, inbox, GREEDY_TRAFFIC_FILE,
                                                 GREEDY_SOURCES),
                     "algorithmic_bytes": R * bytes_per_rollout},
        "issue": measured_issue(cfg.name, R, inbox, GREEDY_TRAFFIC_FILE, GREEDY_SOURCES),
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)
    sim.close()


def run_search(args, cfg):
    """The search-efficiency comparison: the segment search with MCTS (UCB),
    depth-first and random exploration, each for args.steps iterations of
    args.rollouts GPU rollouts; best makespan found against wall time."""
    import numpy as np
    import torch

    import paper_2504_14145_amd as dip
    from paper_2504_14145_amd.mcts import Search
    import workloads as W

    R = args.rollouts
    prob = W.make_problem(cfg)
    op_group, G, cls = W.priority_groups(prob)
    n_cls = int(cls.max()) + 1
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    sim = dip.Sim(prob)
    rc = sim.configure_greedy(G, op_group)
    if rc != dip.OK:
        raise SystemExit(f"greedy unsupported on {cfg.name}: {dip.strerror(rc)}")
    sim.greedy(torch.zeros((1, G), dtype=torch.int32, device=dev))      # uploads the costs
    log(f"[bench] search comparison on {cfg.name}: {n_cls} segment classes, {prob.n_total} "
        f"stages, {args.steps} iterations x {R} rollouts per strategy")
    # warm-up: one short search (kernels loaded, inbox size settled)
    Search(sim, cls, R, seed=cfg.seed + 7).run(max(args.warmup, 1))
    torch.cuda.synchronize()
    curves, final, secs, rates, iters_done = {}, {}, {}, {}, {}
    policies = [p for p in args.policies.split(",") if p]
    for policy in policies:
        srch = Search(sim, cls, R, seed=cfg.seed, alpha=args.alpha, beta=args.beta, policy=policy,
                      workers=args.workers)
        pts = []
        n_it = 0
        t0 = time.perf_counter()
        for t in range(args.steps):
            if srch.done[0]:
                break
            srch.step(t)
            b = srch.best[0] if srch.best[0] != float("inf") else None     # None: none feasible yet
            if not pts or b != pts[-1][2]:      # the points where the best improves
                pts.append([t + 1, round(time.perf_counter() - t0, 4), b])
            n_it = t + 1
        torch.cuda.synchronize()
        secs[policy] = time.perf_counter() - t0
        rates[policy] = R * srch.leaves / secs[policy]
        curves[policy] = pts
        final[policy] = srch.best[0] if srch.best[0] != float("inf") else None
        iters_done[policy] = n_it
        log(f"[bench] {policy}: best makespan {srch.best[0]} after {n_it} iterations "
            f"({secs[policy]:.2f} s, {rates[policy]:.3g} rollouts/s)")
    # the order a plain first-in first-out priority gives, for reference
    fifo = torch.from_numpy(W.fifo_priorities(prob, cls, op_group)[None, :].astype(np.int32)).to(dev)
    _, (ms, _, _, fl) = sim.greedy(fifo, orders=False)
    fifo_ms = int(ms.item()) if int(fl.item()) == 0 else None
    log(f"[bench] first-in first-out priorities: makespan {fifo_ms}")

    cpu = None
    if not args.no_cpu_baseline:
        import oracle.mcts as OM
        cores = max(1, min(16, len(os.sched_getaffinity(0))))
        tc = time.perf_counter()
        it_cpu = 0
        while True:
            it_cpu += 1
            OM.search(prob, op_group, G, cls, it_cpu, R, seed=cfg.seed, threads=cores)
            if time.perf_counter() - tc >= args.cpu_seconds:
                break
        dt = time.perf_counter() - tc
        done = R * it_cpu * (it_cpu + 1) // 2
        cpu = {"value": done / dt, "unit": "rollouts/s", "cores": cores, "kind": "oracle",
               "sample": f"oracle MCTS searches of 1..{it_cpu} iterations x {R} rollouts "
                         f"({dt:.2f} s wall on {cores} threads)"}
        log(f"[bench] cpu oracle {done / dt:.0f} rollouts/s on {cores} threads")

    # per-kernel times of one batch, for the greedy kernel's line
    dip.profile(sim.h, True)
    key = torch.full((1,), -1, dtype=torch.int64, device=dev)
    srch = Search(sim, cls, R, seed=cfg.seed)
    dip.rollouts(sim.h, [], R, cfg.seed, 10**6, srch.prio, srch.ms, srch.fl, key)
    torch.cuda.synchronize()
    k_ms = dip.last_profile(sim.h)
    dip.profile(sim.h, False)
    P = prob.n_ranks
    bytes_per_rollout = 4 * G + 4 + 8 * P + 1 + 4 * G
    greedy_ms = k_ms[0]
    achieved = R * bytes_per_rollout / (greedy_ms / 1e3) / 1e9
    rec = {
        "metric": "best makespan found by the segment search in a fixed budget "
                  "(MCTS vs depth-first vs random exploration, Sec. 5.1)",
        "value": final[policies[0]],
        "unit": "us",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": secs[policies[0]] / max(1, iters_done[policies[0]]) * 1e3,
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {"workload": cfg.name, "rollouts_per_leaf": R, "workers": args.workers,
                   "rounds": args.steps,
                   "segment_classes": n_cls, "alpha": args.alpha, "beta": args.beta,
                   "policies": policies, "parallelism": "single GPU"},
        "final_best_us": final,
        "fifo_makespan_us": fifo_ms,
        "seconds": secs,
        "rollouts_per_s": rates,
        "iterations_run": iters_done,
        "curves": {"columns": ["iteration", "seconds", "best_makespan_us"], **curves},
        "roofline": {"bound": "hbm", "kernel": "greedy", "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": None, "algorithmic_bytes": R * bytes_per_rollout},
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)
    sim.close()


if __name__ == "__main__":
    main()
