/*
 * dip_sim.h -- batched simulation of candidate pipeline schedules on one GPU.
 *
 * The problem (DIP, arXiv 2504.14145): a training iteration's pipeline is a
 * DAG of pipeline stages -- the forward or backward pass of one
 * sub-microbatch on one model chunk (Sec. 5.2) -- placed on physical
 * pipeline ranks, each of which runs one stage at a time (the per-rank t_last
 * of Sec. 5.2).  A stage may start once its rank is free and the outputs of
 * its predecessor stages have arrived; a transfer between different ranks is
 * asynchronous and adds a latency to the edge (Sec. 6.3).  A candidate
 * schedule is one action order per rank (Sec. 6.3's per-worker action list).
 * Each candidate is scored by its iteration time, under a per-rank activation
 * memory limit whose liveness is that of a stage pair, forward start to
 * backward end (Sec. 5.3's memory constraint), and the searcher keeps the
 * best candidate (Sec. 5.1's best rollout score).
 *
 * This library evaluates millions of candidates of ONE instance per call:
 *   dip_sim_create   -- validate and upload the instance's topology;
 *   dip_sim_evaluate -- simulate a batch: makespan, per-rank idle time
 *                       ("bubble"), per-rank peak activation memory, flags;
 *   dip_sim_argmin   -- fold the best (makespan, index) of a batch into a
 *                       running 64-bit key, so chunked batches reduce exactly;
 *   dip_sim_greedy   -- build candidates instead of reading them: Sec. 5.2's
 *                       dual-queue interleaving of one priority vector per
 *                       candidate, with the same outputs as evaluate;
 *   dip_sim_destroy.
 *
 * Semantics per candidate (all integers; results are exact):
 *   start(o)  = max(free(rank(o)), max over predecessors p of end(p)+comm(p,o))
 *   end(o)    = start(o) + cost(o), ops taken in each rank's order
 *   makespan  = max end(o);  bubble[r] = makespan - sum of rank r's costs
 *   peak[r]   = max over prefixes of rank r's order of the running sum of
 *               +act(slot) at each forward and -act(slot) at each backward,
 *               starting from 0 (so it is a function of the order alone)
 *   flags     = DIP_FLAG_DEADLOCK if the orders and the data edges form a
 *               cycle (the simulation stalls with ops left); makespan and
 *               bubble are then -1 while peak keeps the order-scan value;
 *             | DIP_FLAG_CAP if some rank has mem_cap[r] >= 0 and
 *               peak[r] > mem_cap[r];
 *             | DIP_FLAG_INVALID alone, if some rank's section is not a
 *               permutation of its op ids; every output is then -1.
 *
 * Threading and streams: a handle is not thread-safe; distinct handles are
 * independent.  evaluate and argmin enqueue work on the given HIP stream
 * (a hipStream_t passed as void*, NULL = the default stream) and return
 * without waiting; outputs are valid once that stream has reached the work.
 * A handle owns one device scratch area and one device copy of the costs:
 * two evaluate calls on one handle whose kernels may overlap (different
 * streams without an ordering between them) race; use one handle per stream.
 * Every call returns DIP_OK (0) or a negative DIP_E_* code; nothing throws
 * across this boundary.
 */
#ifndef DIP_SIM_H
#define DIP_SIM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DIP_SIM_ABI_VERSION 8

enum {
  DIP_OK = 0,
  DIP_E_INVAL = -1,       /* null pointer, negative count, misaligned buffer   */
  DIP_E_TOPO = -2,        /* malformed topology (ids, CSR, slots, kinds)       */
  DIP_E_RANGE = -3,       /* negative cost, or totals that could overflow int32 */
  DIP_E_UNSUPPORTED = -4, /* shape no kernel variant handles (> 64 ranks, ...) */
  DIP_E_NOMEM = -5,       /* host or device allocation failed                   */
  DIP_E_HIP = -6,         /* HIP runtime error; see dip_sim_strerror            */
  DIP_E_STATE = -7,       /* evaluate before any costs were supplied            */
  DIP_E_CAPACITY = -8     /* batch above dip_sim_evaluate_static's limit        */
};

#define DIP_FLAG_DEADLOCK 1u
#define DIP_FLAG_CAP 2u
#define DIP_FLAG_INVALID 4u

/* Opaque handle; owns only its device-side copies of the instance tables and
 * any scratch memory, released by dip_sim_destroy. */
typedef struct dip_sim dip_sim;

/* Instance topology.  Host pointers, read during dip_sim_create only.
 *
 * Ops are numbered per rank ("rank-local id" 0 .. n_ops[r]-1) and globally
 * (g = off[r] + id, off[r] = n_ops[0] + ... + n_ops[r-1]).  The workload
 * generators of this repository enumerate a rank's ops by model chunk
 * ascending, then sub-microbatch ascending, forward before backward, so
 * id = 2 * slot_local + kind; the library itself relies on no such rule. */
typedef struct {
  int32_t n_ranks;           /* P, 1 .. 64                                      */
  const int32_t *n_ops;      /* [P] ops per rank, each 0 .. 32768 (int16 ids)   */
  const int32_t *pred_ptr;   /* [N+1] CSR row pointers over global op index,
                                pred_ptr[0] = 0, non-decreasing                 */
  const int32_t *pred_op;    /* [E] global index of each predecessor, != own g  */
  const uint8_t *op_kind;    /* [N] 0 = forward (+act at start),
                                    1 = backward (-act at end)                  */
  const int32_t *op_slot;    /* [N] activation slot 0 .. n_slots-1; a forward
                                and its backward share one slot                 */
  int32_t n_slots;
  const int32_t *mem_cap;    /* [P] per-rank cap in memory units, < 0 = none    */
  int64_t cand_stride;       /* int16 elements per candidate row: >= N and a
                                multiple of 8 (16-byte rows)                    */
} dip_topology;

/* Per-batch costs.  Host pointers, read during the call that receives them. */
typedef struct {
  const int32_t *op_cost;    /* [N] microseconds, >= 0                          */
  const int32_t *edge_comm;  /* [E] microseconds, >= 0, aligned with pred_op;
                                charge only edges between different ranks       */
  const int32_t *slot_act;   /* [n_slots] memory units, >= 0                    */
} dip_costs;

/* Reported shape of a handle (what dip_sim_create chose). */
typedef struct {
  int32_t n_ranks;
  int32_t n_ops_total;       /* N */
  int32_t n_edges;           /* E */
  int32_t variant;           /* kernel variant in use, see dip_sim_configure     */
  int64_t cand_stride;
  int32_t lanes_per_group;   /* power of two >= n_ranks: lanes per candidate     */
  int32_t groups_per_wave;   /* candidates simulated side by side by one wave    */
  int32_t waves_per_block;
  int32_t lds_bytes;         /* dynamic LDS per block                            */
  int32_t max_blocks;        /* resident blocks the grid is capped at            */
  int64_t scratch_bytes;     /* device scratch owned by the handle               */
  int32_t pool_slots;        /* variant 8: end-time slots per rank pool, else 0  */
  int32_t check_kernel;      /* variants 8, 9: 1 wave per candidate, 2 tiles,
                                else 0                                         */
  int32_t greedy_inbox;      /* dip_sim_greedy: stages a rank's inbox holds in
                                its first launch (0: not configured; -1: that
                                launch is skipped); grows when many overflow  */
  int32_t greedy_lds_bytes;  /* dip_sim_greedy: LDS per block of its launch    */
  int64_t greedy_retry_ring_bytes; /* dip_sim_greedy: device memory holding the
                                second launch's inboxes where LDS cannot, else 0 */
} dip_sim_info;

/* Host-only checks, no device access: the same checks create / evaluate run
 * first.  Useful where no GPU is present. */
int dip_sim_check_topology(const dip_topology *topo);
int dip_sim_check_costs(const dip_topology *topo, const dip_costs *costs);

/* Validate the topology, copy it to the current HIP device and choose a
 * kernel variant for this device.  On success *out owns device memory. */
int dip_sim_create(const dip_topology *topo, dip_sim **out);

/* Force a kernel variant (0 = automatic choice) and waves per block
 * (0 = automatic; 1, 2, 4 or 8, and 16 for variant 9).  DIP_E_UNSUPPORTED if
 * the variant does not fit the device or the topology.
 * General kernels (any dependence DAG): 1 tables, orders and end times in
 * LDS; 2 tables in global memory, orders and end times in LDS; 3 end times
 * in LDS only; 4 nothing in LDS (end times in device scratch).
 * Variant 8 (at most 15 consumers per op, fewer than 2^16 extra edges): a
 * check kernel (permutation, peak memory, cap) followed by the pool kernel,
 * which hands end times between ranks through per-rank pools of a few
 * slots, and by a general kernel for the candidates whose pools filled up.
 * Variant 9 (the automatic choice where it fits: variant 8's topology limits,
 * a power-of-two rank count and at most 8,192 ops per rank): the same check,
 * then the simulation kernel with compact op records and the pools in LDS,
 * a second pass of it with 16 slots per pool over the candidates whose pools
 * filled, a third with 32 slots, and a general kernel for those that filled
 * again.  Costs that do not fit its records (a cost of 2^20 or more, a
 * latency of 2^11 or more) run variant 8 for that call.  Otherwise a general
 * kernel is chosen.
 * Results are the same whichever kernel runs. */
int dip_sim_configure(dip_sim *h, int32_t variant, int32_t waves_per_block);

/* Variants 8 and 9: end-time slots per rank pool, 4, 8 or 16 (0 = automatic:
 * 8), set at create time and by this call only, never by earlier calls.
 * Fewer slots keep more candidates resident; a candidate whose pools fill up
 * is re-simulated (variant 9: with 16 and then 32 slots, then by the general
 * kernel; variant 8: by the general kernel), so results never depend on it.
 * DIP_E_UNSUPPORTED if the topology does not fit variant 8. */
int dip_sim_configure_pool(dip_sim *h, int32_t slots_per_rank);

/* Variants 8 and 9: the kernel of the order-only part of the verdict
 * (permutation check, per-rank peak memory, cap flag; Sec. 5.3's memory
 * liveness).  0 = automatic (tiles when they fit), 1 = one wavefront per
 * candidate with an op-id bitmap of N bits in LDS, 2 = tiles of 64
 * candidates, one lane per candidate, the ranks split between the waves of a
 * block, each wave holding one rank's memory deltas and 64 bitmaps of (ops of
 * the rank + 1) bits in LDS; after it, for the ranks whose ops wait on an op
 * of their own rank, one wavefront per rank section tests that order from a
 * table of the section's positions.  Results are the same either way.
 * DIP_E_UNSUPPORTED if the topology does not fit variant 8 or the kernel
 * asked for does not fit the device's LDS; DIP_E_INVAL for another mode. */
int dip_sim_configure_check(dip_sim *h, int32_t mode);

int dip_sim_get_info(const dip_sim *h, dip_sim_info *info);

/* Simulate candidates orders[0 .. n_cand-1].
 *   costs      host pointers, or NULL to reuse the costs of the previous call
 *              (DIP_E_STATE if there is none).  Costs are validated (sum of
 *              all op costs and edge latencies <= INT32_MAX; per rank, the
 *              activations of its slots sum to <= INT32_MAX) and copied
 *              stream-ordered before the launch.
 *   orders     device, int16 [n_cand][cand_stride], 16-byte aligned; row c
 *              holds rank 0's order, then rank 1's, ... with no gaps; entries
 *              past N are ignored.
 *   out_*      device: makespan int32 [n_cand], bubble int32 [n_cand][P],
 *              peakmem int32 [n_cand][P], flags uint8 [n_cand].
 *   stream     hipStream_t as void*.
 * n_cand == 0 is a no-op. */
int dip_sim_evaluate(dip_sim *h, const dip_costs *costs, const int16_t *orders,
                     int64_t n_cand, int32_t *out_makespan, int32_t *out_bubble,
                     int32_t *out_peakmem, uint8_t *out_flags, void *stream);

/* dip_sim_evaluate for callers that cannot allocate memory during the call
 * (code captured into a HIP graph, serving loops, harnesses that forbid
 * allocation): the same simulation and outputs, with the costs of an earlier
 * dip_sim_evaluate call (DIP_E_STATE if there were none) and no costs
 * argument, calling no hipMalloc, hipFree or other allocating routine.  Its
 * working memory beyond inputs and outputs (retry counters and retry lists)
 * is a static device array of 64 MiB + 256 bytes that the library holds on
 * every GPU it runs on until the process ends; its tables and launch shapes
 * are the handle's, set up by dip_sim_create and the configure calls.
 * n_cand at most 4,194,304 (DIP_E_CAPACITY above).  All calls on one GPU
 * share that array: calls whose kernels may overlap on one GPU (different
 * streams without an ordering, or different handles or threads) race and
 * must be serialized by the caller.  Arguments and errors as evaluate's. */
#define DIP_SIM_STATIC_MAX_CAND 4194304
int dip_sim_evaluate_static(dip_sim *h, const int16_t *orders, int64_t n_cand,
                            int32_t *out_makespan, int32_t *out_bubble, int32_t *out_peakmem,
                            uint8_t *out_flags, void *stream);

/* Fold the lexicographic minimum of (makespan[i], index_base + i) over the
 * candidates with flags[i] == 0 into *inout_best_key (device, uint64):
 * key = (uint64)makespan << 32 | index, and the caller initialises it to
 * UINT64_MAX, which also means "no valid candidate".  Ties go to the lowest
 * index.  Requires index_base >= 0 and index_base + n_cand <= 2^32 - 1.
 * makespan and flags are device pointers (typically evaluate's outputs). */
int dip_sim_argmin(dip_sim *h, const int32_t *makespan, const uint8_t *flags,
                   int64_t n_cand, int64_t index_base, uint64_t *inout_best_key,
                   void *stream);

/* Dual-queue stage interleaving (Sec. 5.2), set-up.  op_group[N] (host,
 * read during the call) puts every op in one of n_groups priority groups --
 * Sec. 5.1's pipeline segments, which the candidates of dip_sim_greedy
 * prioritise.  A group holds ops of one kind, at most one per rank; the data
 * edges must be acyclic.  1 <= n_groups <= 65535, and at most 2048 groups of
 * either kind.  DIP_E_TOPO if a rule is broken, DIP_E_UNSUPPORTED if the
 * groups or the per-candidate tables do not fit the kernel.  Where a rank's
 * whole inboxes do not fit in LDS, the handle allocates device memory for
 * them (up to 1 GiB; dip_sim_info.greedy_retry_ring_bytes).  Replaces any
 * earlier grouping; the next dip_sim_greedy call must then pass costs. */
int dip_sim_configure_greedy(dip_sim *h, int32_t n_groups, const int32_t *op_group);

/* Stages each rank's forward and backward inbox holds in dip_sim_greedy's
 * first launch (a candidate that overflows one is simulated again by the
 * second launch, whose inboxes hold a whole rank): k a power of two from 1 to
 * 256 fixes it; k = 0 restores the default, 8 to start with and doubled by
 * a later call when more than 1/64 of a call's candidates overflowed, and,
 * once more than half of a call's candidates overflow the largest inboxes
 * that fit in LDS, later calls skip the first launch and give every
 * candidate to the second.
 * Results do not depend on k.  DIP_E_STATE before dip_sim_configure_greedy,
 * DIP_E_INVAL for another k, DIP_E_UNSUPPORTED if the inboxes do not fit in
 * LDS.  Reset by dip_sim_configure_greedy. */
int dip_sim_set_greedy_inbox(dip_sim *h, int32_t k);

/* Build and score one candidate per priority vector.
 *   prio        device, int32 [n_cand][n_groups]: larger is scheduled first;
 *               equal priorities go by group index, then by rank-local id.
 *   costs       as in evaluate (NULL reuses the last ones; DIP_E_STATE if the
 *               records of this grouping were never built).
 *   out_orders  device int16 [n_cand][cand_stride], the orders the greedy
 *               emits (evaluate's layout; entries past N untouched), or NULL.
 *   out_*       as evaluate's, for the emitted orders: the greedy's own
 *               timeline equals the simulation of those orders.
 * Per rank the greedy keeps t_last (end of its last stage) and its queued
 * stages (all predecessors scheduled), each with t_start = max over
 * predecessors of end + comm (0 without any).  A rank's next start is
 * t_min = max(t_last, least queued t_start).  If a forward and a backward
 * were both queued before t_last it alternates kinds (1F1B); otherwise it
 * takes the highest-priority stage able to start at t_min.  A forward that
 * would raise the rank's live activation (forwards scheduled, backwards not
 * yet) above a cap >= 0 disables the forward queue for that decision.  The
 * rank with the least t_min (lowest index on ties) schedules its stage; if
 * every rank is held back by its cap, the cap is lifted for one decision and
 * the result is flagged DIP_FLAG_CAP.  flags is otherwise 0.  Enqueued on
 * stream; n_cand == 0 is a no-op; n_cand <= 2^31 - 1. */
int dip_sim_greedy(dip_sim *h, const dip_costs *costs, const int32_t *prio, int64_t n_cand,
                   int16_t *out_orders, int32_t *out_makespan, int32_t *out_bubble,
                   int32_t *out_peakmem, uint8_t *out_flags, void *stream);

/* MCTS rollouts (Sec. 5.1), set-up, after dip_sim_configure_greedy:
 * group_class[n_groups] (host) puts every priority group in one of n_classes
 * segment classes -- the elements of the sequence the search orders (the
 * pieces of one module in one microbatch share a class, Sec. 5.1's search-
 * space reduction).  The class at position i of a sequence gets priority
 * n_classes - i, and every group its class's priority.  DIP_E_STATE without a
 * grouping, DIP_E_TOPO for a class out of range, DIP_E_UNSUPPORTED above 8192
 * classes.  A new grouping drops it. */
int dip_sim_configure_rollouts(dip_sim *h, int32_t n_classes, const int32_t *group_class);

/* Score n_rollouts random completions of a class prefix (Sec. 5.1's
 * rollouts), each interleaved by dip_sim_greedy, and fold the best
 * (makespan, rollout index) of the unflagged ones into *inout_best_key as
 * dip_sim_argmin does (index_base 0).
 *   prefix      host int32 [depth], distinct classes (positions 0..depth-1).
 *   seed, draw  rollout i shuffles the other classes (ascending to start)
 *               with Durstenfeld's Fisher-Yates: for j = m-1 down to 1 it
 *               swaps position j with k = (hi32(u) * (j + 1)) >> 32, u the
 *               next output of SplitMix64 (Steele, Lea, Flood 2014) started
 *               from mix(mix(seed + (draw+1)*G) + (i+1)*G), G =
 *               0x9E3779B97F4A7C15, mix = SplitMix64's output function.
 *   out_prio    device int32 [n_rollouts][n_groups]: the rollouts' priorities.
 *   out_makespan, out_flags  device [n_rollouts], as dip_sim_greedy's; once
 *               dip_sim_configure_memopt has run on the handle, a rollout is
 *               scored as Sec. 5.1 says, by its iteration time after the
 *               per-layer memory optimisation: its interleaved schedule goes
 *               through dip_sim_memopt and is re-timed with the selection
 *               (dip_sim_evaluate_selected), whose makespan and flags these
 *               are (DIP_FLAG_CAP where a rank's cap cannot be met).
 *   inout_best_key  device uint64.
 * Costs are those of the last call that passed them (DIP_E_STATE if none since
 * the grouping).  Enqueued on stream; the prefix is copied before return. */
int dip_sim_rollouts(dip_sim *h, const int32_t *prefix, int32_t depth, int64_t n_rollouts,
                     uint64_t seed, uint64_t draw, int32_t *out_prio, int32_t *out_makespan,
                     uint8_t *out_flags, uint64_t *inout_best_key, void *stream);

/* The rollouts of several tree nodes in one launch, for a search whose
 * workers (Sec. 6.2's parallel search) each pick a node per round: leaf l
 * (0 <= l < n_leaves <= 65535) has the class prefix of length depths[l]
 * (host; the prefixes concatenated in prefixes, host) and rows
 * l*per_leaf .. l*per_leaf + per_leaf - 1 of out_prio, out_makespan and
 * out_flags; its rollouts are exactly those dip_sim_rollouts makes for that
 * prefix with draw = draw_base + l.  inout_keys (device uint64 [n_leaves],
 * 8-byte aligned): key l folds in leaf l's best unflagged (makespan, rollout
 * index within the leaf).  DIP_E_INVAL for a repeated or out-of-range class
 * in a prefix, null pointers or per_leaf * n_leaves above 2^31 - 1.  Enqueued
 * on stream; the prefixes are copied before return. */
int dip_sim_rollouts_batch(dip_sim *h, int32_t n_leaves, const int32_t *depths,
                           const int32_t *prefixes, int64_t per_leaf, uint64_t seed,
                           uint64_t draw_base, int32_t *out_prio, int32_t *out_makespan,
                           uint8_t *out_flags, uint64_t *inout_keys, void *stream);

/* Per-layer memory optimisation (Sec. 5.3), set-up.  A stage pair is an
 * activation slot (its forward and backward, one rank).  Its layers are
 * slot_layers[s] .. slot_layers[s+1]-1 (host, [n_slots+1], from 0), and layer
 * l's strategies cost layer_time[l][k] microseconds (forward and backward
 * together) and hold layer_mem[l][k] memory units (host int64, >= 0,
 * k < n_strategies).  Per pair the library keeps up to n_candidates (2 .. 8)
 * candidates: the exact (time, memory) Pareto front of its layers' choices,
 * its fastest point, its leanest point, and for each of the n_candidates - 2
 * equal buckets of the memory range between them the least time whose memory
 * is at most the bucket's upper edge lo + floor((hi - lo) k / (n - 2))
 * (Sec. 5.3's multiple-choice knapsack); equal points once, by time.
 * bb_nodes bounds the branch and bound of dip_sim_memopt: the placements it
 * may examine per (schedule, rank), 0 for 512.
 * DIP_E_TOPO unless every slot has one forward and one backward on one rank;
 * DIP_E_RANGE for a negative entry, a candidate memory above 2^31 - 1, a
 * candidate time above 2^40, or fastest memories of a rank summing above
 * 2^31 - 1;
 * DIP_E_INVAL for bb_nodes < 0; DIP_E_UNSUPPORTED for a rank of 16384 pairs
 * or more. */
int dip_sim_configure_memopt(dip_sim *h, const int32_t *slot_layers, const int64_t *layer_time,
                             const int64_t *layer_mem, int32_t n_strategies,
                             int32_t n_candidates, int32_t bb_nodes);

/* For every candidate schedule (orders as dip_sim_evaluate reads them) and
 * rank, choose one candidate per stage pair of the rank so that the memory at
 * every forward start -- the pairs whose forward comes no later and whose
 * backward no earlier in the rank's order -- stays within mem_cap[r] (none if
 * negative), with the least total time (Sec. 5.3's ILP, solved to within the
 * 5 % gap the paper accepts):
 *   1. the greedy warm start: every pair on its fastest candidate; while the
 *      most loaded forward start (the earliest pair among equal loads) is over
 *      the cap, move the live pair whose next candidate adds the least time
 *      per memory unit freed (lowest pair on ties); stop when none can move;
 *   2. pairs in index order each go back to the fastest candidate that keeps
 *      every forward start it is live at within the cap, until nothing moves;
 *   3. a depth-first branch and bound, pairs by forward position, candidates
 *      fastest first, a node cut when 1.05 x (its placed time + the unplaced
 *      pairs' fastest times) reaches the incumbent; it ends proven (the
 *      incumbent is within 5 % of the optimum) or after bb_nodes placements
 *      examined; ranks of more than 512 pairs skip it;
 *   4. when the search stopped early, a certificate: 200 steps of integer
 *      subgradient ascent on the Lagrangian relaxation of the forward-start
 *      constraints (for multipliers l_k >= 0 every selection within the cap
 *      takes at least sum_i min_j (t_ij + m_ij * sum_{k: i live at k} l_k)
 *      - cap * sum_k l_k); the incumbent is proven once 1.05 x that bound
 *      reaches it.
 * Outputs, device [n_cand][P]: out_time (int64, the rank's total pair time),
 * out_peak (memory at the most loaded forward start), out_status (1 within
 * the cap and proven within 5 %, 3 within the cap but not proven, 0 the cap
 * cannot be met, 2 the rank's section is not a permutation: time and peak -1);
 * out_choice (device [n_cand][n_pairs] uint8, or null): the chosen candidate
 * of every pair, pairs numbered rank by rank and within a rank in slot order
 * (candidates by time ascending; undefined for status 2).  Enqueued on
 * stream; DIP_E_STATE before dip_sim_configure_memopt, DIP_E_INVAL for null
 * or misaligned outputs, DIP_E_UNSUPPORTED when a rank's state does not fit
 * in LDS. */
int dip_sim_memopt(dip_sim *h, const int16_t *orders, int64_t n_cand, int64_t *out_time,
                   int32_t *out_peak, uint8_t *out_status, uint8_t *out_choice, void *stream);

/* dip_sim_evaluate of schedules re-timed with a memory selection (Sec. 5.3,
 * then Sec. 5.1's iteration time): pair p of schedule i runs candidate
 * choice[i][p] (dip_sim_memopt's out_choice layout) -- its backward costs
 * its op_cost plus the candidate's time less the pair's fastest time (the
 * recomputation runs inside the backward), and its activation is the
 * candidate's memory -- with the costs and latencies of the last
 * dip_sim_evaluate call.  Outputs and flags as dip_sim_evaluate's (the peak
 * and the cap flag from the chosen memories); a choice beyond a pair's
 * candidates makes its schedule invalid (DIP_FLAG_INVALID, outputs -1).
 * DIP_E_STATE before dip_sim_configure_memopt or before any costs,
 * DIP_E_RANGE when a re-timed backward could exceed 2^31 - 1 microseconds,
 * DIP_E_INVAL for null or misaligned pointers. */
int dip_sim_evaluate_selected(dip_sim *h, const int16_t *orders, const uint8_t *choice,
                              int64_t n_cand, int32_t *out_makespan, int32_t *out_bubble,
                              int32_t *out_peakmem, uint8_t *out_flags, void *stream);

/* Operator-level cost tables (Sec. 6.1), independent of any handle.  An item
 * (a pipeline stage, a data edge, ...) is a run of operator rows; each row
 * has a FLOP count, bytes of memory traffic, bytes sent, and a kind.  For
 * configuration b, coef[b][kind] = {c_fop, c_mem, c_net} are seconds per
 * unit (alpha / capacity: the efficiency factor over the FLOP rate, memory
 * bandwidth, network bandwidth).  A row's latency is
 * max(c_fop N_fop, c_mem N_mem, c_net N_net); an item's entry is
 * ceil(1e6 * the sum of its rows' latencies in row order) microseconds,
 * computed in float64 without fused multiply-adds; -1 if above 2^31 - 1 or
 * if a row's kind is >= n_kinds.  Rows outside [0, n_rows) are ignored. */
typedef struct {
  int32_t n_items;
  int32_t n_rows;
  int32_t n_kinds;           /* 1 .. 256                                       */
  const int32_t *item_ptr;   /* device [n_items+1] row range of each item      */
  const double *n_fop;       /* device [n_rows], 8-byte aligned                */
  const double *n_mem;       /* device [n_rows]                                */
  const double *n_net;       /* device [n_rows]                                */
  const uint8_t *kind;       /* device [n_rows]                                */
} dip_op_table;

/* out: device int32 [n_configs][n_items]; coef: device double
 * [n_configs][n_kinds][3].  Enqueued on stream; DIP_E_INVAL for bad sizes
 * (n_configs above 65535 * 256), null or misaligned pointers. */
int dip_cost_tables(const dip_op_table *t, int64_t n_configs, const double *coef, int32_t *out,
                    void *stream);

/* Per-kernel timing of evaluate (for measurement).  With enable != 0, each
 * later evaluate records HIP events on its stream around each kernel it
 * launches; dip_sim_last_profile then waits for the last of them and writes
 * the kernel times in milliseconds, in launch order, to out_ms[0 .. *n_out-1]
 * (out_ms must hold DIP_SIM_PROFILE_MAX floats; n_out <= 5: variant 8 launches the check, pool and retry kernels;
 * variant 9 the check kernel, the simulation kernel, its passes with 16-
 * and 32-slot pools over the candidates whose pools filled (a pass that
 * does not run reports about 0), and the retry kernel; variants 1-4 one
 * kernel; dip_sim_greedy records its two launches the same way).  *n_out = 0
 * if the last evaluate recorded nothing. */
#define DIP_SIM_PROFILE_MAX 8
int dip_sim_profile(dip_sim *h, int32_t enable);
int dip_sim_last_profile(dip_sim *h, float *out_ms, int32_t *n_out);

/* Diagnostics of the last evaluate (variants 8 and 9): *out_first = the
 * candidates whose pools filled in the first simulation pass; *out_second =
 * those left to the general kernel (variant 9: the ones its passes with 16-
 * and 32-slot pools could not finish either).  Waits for that call's
 * stream. */
int dip_sim_last_retries(dip_sim *h, int64_t *out_first, int64_t *out_second);

/* Release the handle's device memory.  Waits for the device first. */
void dip_sim_destroy(dip_sim *h);

/* Static description of a return code; for DIP_E_HIP, the last HIP error
 * seen by this thread. */
const char *dip_sim_strerror(int code);

int dip_sim_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DIP_SIM_H */
