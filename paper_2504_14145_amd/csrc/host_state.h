// host_state.h -- the handle behind the C ABI of include/dip_sim.h and the
// helpers that the host files share: host.hip (handle life cycle, evaluate,
// argmin), host_plan.hip (kernel-variant choice and launch shapes),
// host_tables.hip (cost-dependent device tables), host_next.hip (the greedy
// interleaving, MCTS rollouts and memory selection entry points) and
// host_check.cpp (host-side validation, plain C++).
//
// Kernel families (see kern_general.hip, kern_pool.hip, kern_sim.hip):
//   variants 1-4  general kernel, any predecessor count, tables placed per
//                 variant (all in LDS ... end times in device scratch);
//   variant 8     check kernel (permutation, memory) + pool kernel (end times
//                 handed between ranks through small per-rank slot pools, op
//                 records through the caches) + the general kernel in list
//                 mode for candidates whose pools filled up;
//   variant 9     as 8 with the simulation kernel of kern_sim.hip in place of
//                 the pool kernel: compact op records resident in LDS and the
//                 orders staged through per-lane LDS rings, then a second
//                 pass with 16 pool slots before the general kernel.  It
//                 needs a power-of-two rank count, at most 8192 ops per rank,
//                 and per call costs below 2^20 and latencies below 2^11
//                 (checked whenever costs change; a call outside them runs
//                 variant 8).
#pragma once

#include <algorithm>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <unordered_map>
#include <vector>

#include "dip_sim.h"
#include "host_limits.h"
#include "internal.h"

namespace dipsim_host {

// the HIP error behind the last DIP_E_HIP of this thread
extern thread_local hipError_t g_last_hip;

constexpr int64_t kScratchCap = int64_t(2) << 30;  // device scratch ceiling
// simulation-kernel records up to this size are stored one per op, larger
// tables as deduplicated pages (one more LDS read per record)
constexpr int64_t kSimDirectMax = 32768;
// tables (records, extra edges) up to this size go to each block's LDS,
// beside the pools of up to 16 waves
constexpr int64_t kPoolTabLimit = 131072;

#define DIP_HIP(expr)          \
  do {                         \
    hipError_t e_ = (expr);    \
    if (e_ != hipSuccess) {    \
      g_last_hip = e_;         \
      return DIP_E_HIP;        \
    }                          \
  } while (0)

inline int ceil_pow2_log2(int p) {
  int l = 0;
  while ((1 << l) < p) ++l;
  return l;
}

}  // namespace dipsim_host

struct dip_sim {
  int device = 0;
  int32_t P = 0, N = 0, E = 0, n_slots = 0;
  int64_t stride = 0;
  std::vector<int32_t> n_ops, rank_off, pred_ptr, pred_op, op_slot, cap;
  std::vector<uint8_t> kind;
  int32_t pwl = 0, G = 0;
  std::vector<int32_t> rank_of;        // [N] rank running each op
  // own-rank predecessors: the tile check verifies their order, and the
  // simulation kernel then drops those edges when their latency is zero
  bool self_ok = false;                // at most one own-rank predecessor per op
  uint64_t self_ranks = 0;             // bit r: rank r has ops with one
  std::vector<int32_t> self_pred;      // [N] its local id + 1, 0 if none
  int32_t *d_selfp = nullptr;
  bool sim_drop_self = false;          // the current sim tables dropped them
  std::vector<int32_t> last_cost, last_comm, last_act;   // the last costs (host copies)
  std::vector<int32_t> n_cons;         // [N] consumers of each op
  bool pool_ok = false;                // topology fits the pool kernel
  int32_t n_extra = 0;                 // pool kernel: edges after each op's first
  bool pool_tab = false;               // pool kernel: tables copied into LDS
  int64_t pool_tab_bytes = 0;          // their bytes (records, then extra edges)
  int pool_slots = 8, forced_pool_slots = 0;   // slots per rank pool (variants 8, 9)
  // simulation kernel (variant 9)
  bool sim_ok = false;                 // topology fits it
  bool sim_costs_ok = false;           // the last costs fit its records
  bool sim_paged = false;              // records stored as deduplicated pages
  int32_t sim_n_extra = 0;             // extra-edge words (edges of multi-predecessor ops)
  int64_t sim_tab_cap = 0;             // bytes of d_sim_tab
  int32_t sim_tab_vec = 0;             // 16-byte units of the current table image
  uint32_t sim_off_pmap = 0, sim_off_extra = 0;
  uint4 *d_sim_tab = nullptr;          // LDS image: records, page map, extra edges
  int4 *d_sim_lane = nullptr;          // [P] {first op, ops, busy, record base}
  int sim_wpb = 1, sim_max_blocks = 1;
  int64_t sim_lds = 0;
  int64_t sim_state_base = 0;
  // second pass over the first pass's retry list, with 16-slot pools
  bool sim2_ok = false;
  int sim2_wpb = 1, sim2_max_blocks = 1;
  int64_t sim2_lds = 0;
  int64_t *d_retry2 = nullptr;         // candidates the second pass could not hold
  // third pass over what the earlier ones could not hold, with 32-slot pools
  bool sim3_ok = false;
  int sim3_wpb = 1, sim3_max_blocks = 1;
  int64_t sim3_lds = 0;
  hipStream_t last_stream = nullptr;   // stream of the last evaluate (diagnostics)
  uint32_t *last_counts = nullptr;     // its retry counters
  void *d_static = nullptr;            // this device's address of the static scratch array
  int last_general = 0;                // counter (index) of the list its general kernel took
  int4 *d_pool_rec = nullptr;          // pool records [N][2]
  int2 *d_pool_edge = nullptr;         // pool edges [E]
  int64_t *d_retry = nullptr;          // candidates re-run by the general kernel
  uint32_t *d_retry_count = nullptr;   // [2] retry count, on-demand candidate counter
  int64_t retry_cap = 0;
  int check_blocks_per_cu = 1;
  bool wc_ok = false;                  // the wave-per-candidate check fits
  int check_mode = 0;                  // 0 automatic, 1 wave per candidate, 2 tiles
  // tile check (lane = candidate, waves splitting the ranks)
  struct TilePlan {
    int nw = 1;                        // waves per block
    int32_t max_nr = 0;
    int64_t lds = 0;
    int blocks_per_cu = 1;
    int32_t *d_plan = nullptr;         // [nw+1] offsets, then the ranks
  };
  bool tc_ok = false;                  // the main pass (every rank)
  TilePlan tc;
  // order kernel after the tile check (ranks with own-rank predecessors):
  // one wave per section, a block per rank and chunk of candidates
  bool to_ok = false;
  int oc_wpb = 4;                      // waves per block
  int oc_per_wave = 1;                 // candidates per wave and block (for large batches)
  int oc_blocks_per_cu = 1;
  int64_t oc_lds = 0;
  int32_t oc_tab_bytes = 0;
  int32_t oc_n_ranks = 0;
  int32_t *d_oc_ranks = nullptr;       // [oc_n_ranks]
  void *d_scratch_fb = nullptr;        // general kernel (list mode) end tables
  int fb_variant = 4;                  // retry kernel: 3 (end times in LDS) when they fit, else 4
  int64_t fb_lds = 0;
  int64_t scratch_fb_bytes = 0;
  int fb_blocks = 1;
  // device tables
  int4 *d_rec = nullptr;               // general records [N]
  int2 *d_edge = nullptr;              // general edges [E]
  int32_t *d_md = nullptr;             // memory deltas [N] (+act at F, -act at B)
  int32_t *d_rank_off = nullptr, *d_busy = nullptr, *d_cap = nullptr;
  void *d_scratch_gen = nullptr;       // variant 4: end tables per resident wave
  int64_t scratch_gen_bytes = 0;
  // pinned staging for cost uploads
  unsigned char *h_stage = nullptr;
  int64_t stage_bytes = 0;
  hipEvent_t stage_done = nullptr;
  // optional per-kernel timing of evaluate: events before each kernel and after the last
  bool profile = false;
  hipEvent_t prof_ev[6] = {nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};
  int prof_n = 0;                      // events recorded by the last evaluate
  bool stage_pending = false;
  bool costs_set = false;
  // launch configuration of the chosen variant
  int variant = 0, wpb = 1;
  int64_t lds_bytes = 0;
  int max_blocks = 1;
  int n_cu = 1;
  int64_t lds_block_max = 65536;
  int forced_variant = 0, forced_wpb = 0;
  // general configuration (always available)
  int gen_variant = 0, gen_wpb = 1, gen_max_blocks = 1;
  int64_t gen_lds = 0;
  // greedy stage interleaving (dip_sim_configure_greedy / dip_sim_greedy)
  bool gr_ok = false;                  // groups configured
  bool gr_costs_ok = false;            // records hold the current costs
  int32_t gr_G = 0, gr_GF = 0, gr_J = 0, gr_max_nr = 0;
  int gr_pwl = 3, gr_nw = 1;
  std::vector<int32_t> gr_op;          // [G*P] global op of (internal group, rank), -1 none
  std::vector<int32_t> gr_ig;          // [N] internal group of each op
  std::vector<int32_t> gr_join;        // [N] join index of an op with several predecessors
  std::vector<int32_t> gr_succ_ptr;    // [N+1] successors of each op ...
  std::vector<int32_t> gr_succ_op;     // ... and the edge they come through
  std::vector<int32_t> gr_succ_edge;
  int32_t gr_n_extra = 0;              // successors after each op's first
  int32_t *d_gr_caller = nullptr;      // [G]
  int32_t *d_gr_src = nullptr;         // [P+1] offsets, then the source groups
  int4 *d_gr_rec = nullptr;            // [G*P*2]
  int4 *d_gr_succ = nullptr;           // [max(extra, 1)]
  unsigned char *h_gr_stage = nullptr; // pinned staging of the records
  int64_t *d_gr_retry = nullptr;
  uint32_t *d_gr_retry_count = nullptr;
  int64_t gr_retry_cap = 0;
  // adaptive inbox size: a call's retry count is copied back asynchronously
  // and read by a later call, which doubles the inboxes when more than 1/64
  // of its candidates needed the second launch
  int gr_K = 16;
  bool gr_K_fixed = false;             // dip_sim_set_greedy_inbox fixed it
  bool gr_direct = false;              // later calls run only the whole-rank-inbox launch
  uint32_t *h_gr_seen = nullptr;       // pinned
  hipEvent_t gr_seen_ev = nullptr;
  bool gr_seen_pending = false;
  int64_t gr_seen_n = 0;
  struct GrLaunch {
    int pwl = 3, wpb = 1, K = 8, blocks_per_cu = 1;
    bool gring = false;                // inboxes in device memory (d_gr_ring)
    int max_blocks = 0;                // gring: blocks the ring memory has slots for
    int32_t cand_bytes = 0, off_pend = 0, off_npend = 0, off_join = 0, off_gpos = 0,
            off_ord = 0, off_grk = 0;
    int64_t lds = 0;
  } gr_main, gr_retry;
  int32_t gr_meta_bytes = 0;
  uint64_t *d_gr_ring = nullptr;       // retry launch's inboxes when LDS cannot hold them
  int64_t gr_ring_bytes = 0;
  // MCTS rollouts (dip_sim_configure_rollouts / dip_sim_rollouts)
  bool rl_ok = false;
  int32_t rl_n = 0;                    // classes
  std::vector<int32_t> rl_class;       // [G] caller-indexed class of each group
  int32_t *d_rl_class = nullptr;       // [G]
  int32_t *d_rl_seq = nullptr;         // [leaves][n] prefix, then the other classes; [leaves] depths
  int32_t *h_rl_seq = nullptr;         // pinned staging of it
  int32_t rl_leaf_cap = 0;             // leaves the two hold
  hipEvent_t rl_seq_ev = nullptr;
  bool rl_seq_pending = false;
  int32_t *d_rl_bub = nullptr, *d_rl_peak = nullptr;  // [cap][P] greedy outputs
  int64_t rl_cap = 0;
  // rollouts scored after the memory selection: the orders, the selection's
  // outputs and choices
  int16_t *d_rl_orders = nullptr;
  int64_t *d_rl_mo_time = nullptr;
  int32_t *d_rl_mo_peak = nullptr;
  uint8_t *d_rl_mo_status = nullptr, *d_rl_choice = nullptr;
  int64_t rl_mo_cap = 0;
  // per-layer memory optimisation (dip_sim_configure_memopt / dip_sim_memopt)
  bool mo_ok = false;
  int32_t mo_max_pairs = 0, mo_n_pairs = 0, mo_bb_nodes = 512;
  int64_t mo_max_extra = 0;            // largest slowest-less-fastest time of a pair
  std::vector<int32_t> mo_pair_b;      // the backward op of every pair (pair order)
  std::vector<int64_t> mo_pair_extra;  // its slowest time less its fastest
  int32_t *d_mo_pair_off = nullptr, *d_mo_lid_pair = nullptr;
  int64_t *d_mo_time = nullptr;
  int32_t *d_mo_mem = nullptr, *d_mo_dm = nullptr;
  uint32_t *d_mo_key = nullptr;
};

namespace dipsim_host {

using namespace dipsim;

struct GenBytes {
  int64_t tab, ord, end;
};

struct Pick {
  int v = 0, wpb = 0, nb = 0, waves = 0;
};

struct StageLayout {
  int64_t rec, edge, busy, md, prec8, pedge, stab, slane, total;
};

GenBytes general_bytes(const dip_sim *h, int v);
int64_t lds_for(const dip_sim *h, int v, int wpb);
const void *kernel_ptr(const dip_sim *h, int v);
int blocks_per_cu(dip_sim *h, int v, int wpb);
int64_t scratch_need(const dip_sim *h, int v, int wpb, int blocks);
int ensure_scratch(dip_sim *h, int64_t need);
bool plan_tiles(dip_sim *h, const std::vector<int32_t> &rks, bool order, dip_sim::TilePlan *T);
int plan_tile_check(dip_sim *h);
int ensure_fallback(dip_sim *h);
// the check kernel evaluate runs: 1 wave per candidate, 2 tiles
int check_kind(const dip_sim *h);
// evaluate's check tests the order of own-rank edges (the simulation
// kernel's tables may then drop those of zero latency)
bool order_checked(const dip_sim *h);
int run_tile_check(dip_sim *h, const int16_t *orders, int64_t n_cand, int32_t *out_ms,
                   int32_t *out_bub, int32_t *out_peak, uint8_t *out_flags, hipStream_t stream,
                   uint32_t *counts);
int run_wave_check(dip_sim *h, const int16_t *orders, int64_t n_cand, int32_t *out_ms,
                   int32_t *out_bub, int32_t *out_peak, uint8_t *out_flags, hipStream_t stream,
                   uint32_t *counts);
int ensure_retry(dip_sim *h, int64_t n);
Pick best_of(dip_sim *h, int v_lo, int v_hi, int forced_wpb);
int apply_pick(dip_sim *h, const Pick &p, int *variant, int *wpb, int *max_blocks,
               int64_t *lds);
bool sim_shape(dip_sim *h, int slots, int forced_wpb, int *wpb, int *max_blocks, int64_t *lds_out);
int sim_plan(dip_sim *h);
int choose_config(dip_sim *h);
int64_t sim_tab_bound(const dip_sim *h);
StageLayout stage_layout(const dip_sim *h);
int upload_greedy_records(dip_sim *h, const dip_costs *c, hipStream_t stream);
int upload_sim_tables(dip_sim *h, const dip_costs *c, const int32_t *busy, const StageLayout &L,
                      hipStream_t stream);
int upload_costs(dip_sim *h, const dip_costs *c, hipStream_t stream);
bool greedy_layout(const dip_sim *h, int K, int pwl, dip_sim::GrLaunch *L, bool gring = false);
void release_rollout_memopt(dip_sim *h);
void release_rollouts(dip_sim *h);
void release_memopt(dip_sim *h);
void release_greedy(dip_sim *h);
void release(dip_sim *h);

}  // namespace dipsim_host
