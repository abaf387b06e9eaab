// host.hip -- the C ABI of include/dip_sim.h: validation, device tables,
// kernel-variant choice and stream-ordered launches.
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
//                 orders staged through per-lane LDS rings.  It needs at most
//                 8192 ops per rank, and per call costs below 2^20 and
//                 latencies below 2^11 (checked whenever costs change; a call
//                 outside them runs variant 8).
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
#include "internal.h"

using namespace dipsim;

namespace {

thread_local hipError_t g_last_hip = hipSuccess;
constexpr int kMaxDevices = 64;

// dip_sim_evaluate_static's working memory, one copy per GPU for the life of
// the process: the retry counters (kStaticHead bytes), then two retry lists of
// kStaticMaxCand 8-byte entries.  In host code `scratch` only names the
// symbol; its device address comes from hipGetSymbolAddress, per device.
constexpr int64_t kStaticMaxCand = int64_t(1) << 22;
constexpr int64_t kStaticHead = 256;
constexpr int64_t kStaticBytes = kStaticHead + 2 * 8 * kStaticMaxCand;
static __device__ __align__(256) unsigned char scratch[kStaticBytes];

// the device address of `scratch` on the current device, looked up once per
// device (nullptr, with the HIP error kept, if the lookup fails)
void *static_scratch_on_current_device() {
  static std::mutex mu;
  static void *addr[kMaxDevices] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    g_last_hip = hipErrorInvalidDevice;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void *ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) {
      g_last_hip = e;
      return nullptr;
    }
    addr[dev] = ptr;
  }
  return addr[dev];
}

constexpr int kMaxRanks = 64;
constexpr int32_t kMaxOpsPerRank = 32768;
constexpr int64_t kScratchCap = int64_t(2) << 30;  // device scratch ceiling
// simulation-kernel records up to this size are stored one per op, larger
// tables as deduplicated pages (one more LDS read per record)
constexpr int64_t kSimDirectMax = 32768;

#define DIP_HIP(expr)          \
  do {                         \
    hipError_t e_ = (expr);    \
    if (e_ != hipSuccess) {    \
      g_last_hip = e_;         \
      return DIP_E_HIP;        \
    }                          \
  } while (0)

int ceil_pow2_log2(int p) {
  int l = 0;
  while ((1 << l) < p) ++l;
  return l;
}

}  // namespace

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
  hipStream_t last_stream = nullptr;   // stream of the last evaluate (diagnostics)
  uint32_t *last_counts = nullptr;     // its retry counters
  void *d_static = nullptr;            // this device's address of the static scratch array
  bool last_pass2 = false;             // it ran the second simulation pass
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
  bool to_ok = false;                  // the order pass (ranks with own-rank predecessors)
  TilePlan to;
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
  hipEvent_t prof_ev[5] = {nullptr, nullptr, nullptr, nullptr, nullptr};
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

namespace {

struct GenBytes {
  int64_t tab, ord, end;
};

GenBytes general_bytes(const dip_sim *h, int v) {
  GenBytes b{0, 0, 0};
  const int64_t G = h->G;
  if (v == 1) b.tab = align16(int64_t(h->N) * 16) + align16(int64_t(h->E) * 8);
  if (v <= 2) b.ord = align16(G * h->stride * 2);
  if (v <= 3) b.end = align16(G * int64_t(h->N) * 4);
  return b;
}

int64_t lds_for(const dip_sim *h, int v, int wpb) {
  if (v <= 4) {
    GenBytes b = general_bytes(h, v);
    return b.tab + int64_t(wpb) * (b.ord + b.end);
  }
  if (v == 8)
    return h->pool_tab_bytes + int64_t(wpb) * h->G * pool_group_bytes(1 << h->pwl, h->pool_slots);
  return 0;
}

const void *kernel_ptr(const dip_sim *h, int v) {
  if (v <= 4) return general_kernel_ptr(v);
  return pool_kernel_ptr(h->pwl, h->pool_slots, h->pool_tab);
}

// Resident blocks per CU for (variant, waves per block); 0 if it does not fit.
int blocks_per_cu(dip_sim *h, int v, int wpb) {
  if (v == 8 && !h->pool_ok) return 0;
  const int64_t lds = lds_for(h, v, wpb);
  if (lds > h->lds_block_max) return 0;
  const void *k = kernel_ptr(h, v);
  if (lds > 65536) {
    if (hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)) != hipSuccess) {
      (void)hipGetLastError();
      return 0;
    }
  }
  int nb = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, k, wpb * kWave, size_t(lds)) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  return nb;
}

int64_t scratch_need(const dip_sim *h, int v, int wpb, int blocks) {
  if (v == 4) return int64_t(blocks) * wpb * h->G * int64_t(h->N) * 4;
  return 0;
}

// Device scratch for variant 4 (general): end tables per resident wave.
int ensure_scratch(dip_sim *h, int64_t need) {
  void **buf = &h->d_scratch_gen;
  int64_t *have = &h->scratch_gen_bytes;
  if (need > *have) {
    if (*buf) {
      DIP_HIP(hipDeviceSynchronize());
      DIP_HIP(hipFree(*buf));
      *buf = nullptr;
    }
    *have = 0;
    if (hipMalloc(buf, size_t(need)) != hipSuccess) {
      (void)hipGetLastError();
      return DIP_E_NOMEM;
    }
    *have = need;
  }
  return DIP_OK;
}

// The pool kernel's fallback: the general kernel with end tables in device
// Tile check plan over a set of ranks: they are split between the waves of a
// block, longest section first onto the least loaded wave.  The number of
// waves per block is the one (up to 16, and not above the ranks or what keeps
// every wave near the longest section) that keeps the most waves resident per
// CU.  false when a rank's section does not fit.
bool plan_tiles(dip_sim *h, const std::vector<int32_t> &rks, bool order, dip_sim::TilePlan *T) {
  int32_t max_nr = 0;
  int64_t n_sum = 0;
  for (int32_t r : rks) {
    max_nr = std::max(max_nr, h->n_ops[r]);
    n_sum += h->n_ops[r];
  }
  if (rks.empty() || int64_t(h->stride) * 2 * kWave > int64_t(INT32_MAX)) return false;
  const void *kern = tile_check_kernel_ptr(order);
  const int64_t region = tile_region_bytes(max_nr);
  const int nw_max = int(std::min<int64_t>(
      {16, int64_t(rks.size()), (n_sum + std::max(max_nr, 1) - 1) / std::max(max_nr, 1)}));
  int nw = 0, nb = 0, best_waves = 0;
  for (int w = 1; w <= std::max(nw_max, 1); ++w) {
    const int64_t lds = kTileFlagBytes + int64_t(w) * region;
    if (lds > h->lds_block_max) break;
    if (lds > 65536 &&
        hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)) != hipSuccess) {
      (void)hipGetLastError();
      break;
    }
    int b = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, kern, w * kWave, size_t(lds)) != hipSuccess) {
      (void)hipGetLastError();
      break;
    }
    if (b > 0 && b * w >= best_waves) {
      best_waves = b * w;
      nw = w;
      nb = b;
    }
  }
  if (nw == 0) return false;
  std::vector<int32_t> sorted(rks), load(nw, 0), wave_of(h->P, -1);
  std::stable_sort(sorted.begin(), sorted.end(),
                   [&](int32_t x, int32_t y) { return h->n_ops[x] > h->n_ops[y]; });
  for (int32_t r : sorted) {
    const int w = int(std::min_element(load.begin(), load.end()) - load.begin());
    wave_of[r] = w;
    load[w] += h->n_ops[r];
  }
  std::vector<int32_t> plan(size_t(nw) + 1 + rks.size());
  int k = 0;
  for (int w = 0; w < nw; ++w) {
    plan[w] = k;
    for (int r = 0; r < h->P; ++r)
      if (wave_of[r] == w) plan[nw + 1 + k++] = r;
  }
  plan[nw] = k;
  const int64_t lds = kTileFlagBytes + int64_t(nw) * region;
  if (lds > 65536 &&
      hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  if (!T->d_plan && hipMalloc(&T->d_plan, size_t(h->P + 17) * 4) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  if (hipMemcpy(T->d_plan, plan.data(), plan.size() * 4, hipMemcpyHostToDevice) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  T->nw = nw;
  T->max_nr = max_nr;
  T->lds = lds;
  T->blocks_per_cu = nb;
  return true;
}

// The main tile check over every rank, and the order pass over the ranks
// with own-rank predecessors (when there are any).
int plan_tile_check(dip_sim *h) {
  std::vector<int32_t> all(h->P), own;
  for (int r = 0; r < h->P; ++r) {
    all[r] = r;
    if ((h->self_ranks >> r) & 1u) own.push_back(r);
  }
  h->tc_ok = plan_tiles(h, all, false, &h->tc);
  // (without the order pass the simulation kernel keeps those edges)
  h->to_ok = h->tc_ok && h->self_ok && !own.empty() && plan_tiles(h, own, true, &h->to);
  return DIP_OK;
}

// scratch (variant 4), one wave per block, in list mode.
int ensure_fallback(dip_sim *h) {
  h->fb_blocks = h->n_cu;
  // the retry kernel keeps its candidates' end times in LDS when one wave's
  // tables fit (much shorter waits per op than device scratch)
  h->fb_variant = 4;
  h->fb_lds = 0;
  {
    const int64_t lds3 = lds_for(h, 3, 1);
    int nb3 = 0;
    if (lds3 <= h->lds_block_max &&
        (lds3 <= 65536 || hipFuncSetAttribute(general_kernel_ptr(3),
                                              hipFuncAttributeMaxDynamicSharedMemorySize,
                                              int(lds3)) == hipSuccess) &&
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb3, general_kernel_ptr(3), kWave,
                                                     size_t(lds3)) == hipSuccess &&
        nb3 > 0) {
      h->fb_variant = 3;
      h->fb_lds = lds3;
    }
    (void)hipGetLastError();
  }
  const int64_t need = int64_t(h->fb_blocks) * h->G * int64_t(h->N) * 4;
  if (need > h->scratch_fb_bytes) {
    if (h->d_scratch_fb) {
      DIP_HIP(hipDeviceSynchronize());
      DIP_HIP(hipFree(h->d_scratch_fb));
      h->d_scratch_fb = nullptr;
    }
    h->scratch_fb_bytes = 0;
    if (hipMalloc(&h->d_scratch_fb, size_t(need)) != hipSuccess) {
      (void)hipGetLastError();
      return DIP_E_NOMEM;
    }
    h->scratch_fb_bytes = need;
  }
  // the wave-per-candidate check: one op-id bitmap of N bits per wave
  h->wc_ok = false;
  int nb = 0;
  const int64_t lds = 4 * check_lds_per_group(h->N);
  if (lds <= h->lds_block_max &&
      (lds <= 65536 || hipFuncSetAttribute(check_kernel_ptr(h->pwl),
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           int(lds)) == hipSuccess) &&
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, check_kernel_ptr(h->pwl), 4 * kWave,
                                                   size_t(lds)) == hipSuccess &&
      nb > 0) {
    h->check_blocks_per_cu = nb;
    h->wc_ok = true;
  }
  (void)hipGetLastError();
  return (h->wc_ok || h->tc_ok) ? DIP_OK : DIP_E_UNSUPPORTED;
}

bool use_tile_check(const dip_sim *h) {
  return h->check_mode == 2 || (h->check_mode == 0 && h->tc_ok) || !h->wc_ok;
}

int run_tile_check(dip_sim *h, const int16_t *orders, int64_t n_cand, int32_t *out_ms,
                   int32_t *out_bub, int32_t *out_peak, uint8_t *out_flags, hipStream_t stream,
                   uint32_t *counts) {
  TileCheckArgs c{};
  c.orders = orders;
  c.n_cand = n_cand;
  c.stride = h->stride;
  c.out_ms = out_ms;
  c.out_bub = out_bub;
  c.out_peak = out_peak;
  c.out_flags = out_flags;
  c.md = h->d_md;
  c.rank_off = h->d_rank_off;
  c.cap = h->d_cap;
  c.selfp = h->d_selfp;
  c.P = h->P;
  c.retry_count = counts;
  const int64_t tiles = (n_cand + kWave - 1) / kWave;
  for (int pass = 0; pass < (h->to_ok ? 2 : 1); ++pass) {
    const dip_sim::TilePlan &T = pass ? h->to : h->tc;
    c.plan = T.d_plan;
    c.nw = T.nw;
    c.md_bytes = tile_md_bytes(T.max_nr);
    c.region_bytes = tile_region_bytes(T.max_nr);
    const int blocks = int(std::min<int64_t>(tiles, int64_t(T.blocks_per_cu) * h->n_cu));
    DIP_HIP(launch_tile_check(std::max(blocks, 1), T.nw, size_t(T.lds), stream, c, pass == 1));
  }
  return DIP_OK;
}

int run_wave_check(dip_sim *h, const int16_t *orders, int64_t n_cand, int32_t *out_ms,
                   int32_t *out_bub, int32_t *out_peak, uint8_t *out_flags, hipStream_t stream,
                   uint32_t *counts) {
  CheckArgs c{};
  c.orders = orders;
  c.n_cand = n_cand;
  c.stride = h->stride;
  c.out_ms = out_ms;
  c.out_bub = out_bub;
  c.out_peak = out_peak;
  c.out_flags = out_flags;
  c.md = h->d_md;
  c.rank_off = h->d_rank_off;
  c.cap = h->d_cap;
  c.P = h->P;
  c.N = h->N;
  c.wpb = 4;
  c.retry_count = counts;
  const int64_t c_lds = 4 * check_lds_per_group(h->N);
  const int64_t c_per_block = 4;
  const int c_blocks = int(std::min<int64_t>((n_cand + c_per_block - 1) / c_per_block,
                                             int64_t(h->check_blocks_per_cu) * h->n_cu));
  DIP_HIP(launch_check(h->pwl, std::max(c_blocks, 1), 4, size_t(c_lds), stream, c));
  return DIP_OK;
}

int ensure_retry(dip_sim *h, int64_t n) {
  if (!h->d_retry_count) DIP_HIP(hipMalloc(&h->d_retry_count, 16));
  if (n <= h->retry_cap) return DIP_OK;
  if (h->d_retry) {
    DIP_HIP(hipDeviceSynchronize());
    DIP_HIP(hipFree(h->d_retry));
    h->d_retry = nullptr;
  }
  h->retry_cap = 0;
  if (h->d_retry2) {
    DIP_HIP(hipFree(h->d_retry2));
    h->d_retry2 = nullptr;
  }
  if (hipMalloc(&h->d_retry, size_t(n) * 8) != hipSuccess ||
      (h->sim_ok && hipMalloc(&h->d_retry2, size_t(n) * 8) != hipSuccess)) {
    (void)hipGetLastError();
    return DIP_E_NOMEM;
  }
  h->retry_cap = n;
  return DIP_OK;
}

// tables (records, extra edges) up to this size go to each block's LDS,
// beside the pools of up to 16 waves
constexpr int64_t kPoolTabLimit = 131072;

struct Pick {
  int v = 0, wpb = 0, nb = 0, waves = 0;
};

Pick best_of(dip_sim *h, int v_lo, int v_hi, int forced_wpb) {
  Pick best;
  for (int v = v_lo; v <= v_hi; ++v) {
    for (int w : {16, 8, 4, 2, 1}) {
      if (forced_wpb && w != forced_wpb) continue;
      if (w >= 8 && !(v == 8 && h->pool_tab)) continue;   // only the tables-in-LDS pool kernel
      const int nb = blocks_per_cu(h, v, w);
      if (nb <= 0) continue;
      const int waves = nb * w;
      // prefer the lower variant (less global traffic) unless a higher one
      // at least doubles the resident waves and the lower has fewer than 8
      if (best.v == 0 ||
          (waves > best.waves && (v == best.v || (best.waves < 8 && waves >= 2 * best.waves)))) {
        best = Pick{v, w, nb, waves};
      }
    }
  }
  return best;
}

int apply_pick(dip_sim *h, const Pick &p, int *variant, int *wpb, int *max_blocks,
               int64_t *lds) {
  *variant = p.v;
  *wpb = p.wpb;
  *lds = lds_for(h, p.v, p.wpb);
  int mb = p.nb * h->n_cu;
  if (p.v == 4) {
    const int64_t per_block = scratch_need(h, p.v, p.wpb, 1);
    mb = int(std::min<int64_t>(mb, std::max<int64_t>(1, kScratchCap / per_block)));
    int rc = ensure_scratch(h, scratch_need(h, p.v, p.wpb, mb));
    if (rc != DIP_OK) return rc;
  }
  *max_blocks = mb;
  return DIP_OK;
}

// Launch shape of the simulation kernel for the current table image and a
// pool size: the waves per block (one table copy per block) that keep the
// most waves resident per CU, fewer blocks on ties.  false if nothing fits.
bool sim_shape(dip_sim *h, int slots, int forced_wpb, int *wpb, int *max_blocks, int64_t *lds_out) {
  const int64_t tab = int64_t(h->sim_tab_vec) * 16;
  const int64_t grp = sim_group_bytes(1 << h->pwl, slots);
  const void *k = sim_kernel_ptr(h->pwl, slots, h->sim_paged);
  int best_w = 0, best_nb = 0;
  for (int w = 16; w >= 1; --w) {
    if (forced_wpb && w != forced_wpb) continue;
    const int64_t lds = tab + int64_t(w) * h->G * grp;
    if (lds > h->lds_block_max) continue;
    if (lds > 65536 &&
        hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)) != hipSuccess) {
      (void)hipGetLastError();
      continue;
    }
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, k, w * kWave, size_t(lds)) != hipSuccess) {
      (void)hipGetLastError();
      continue;
    }
    if (nb > 0 && nb * w > best_nb * best_w) {
      best_w = w;
      best_nb = nb;
    }
  }
  if (best_w == 0) return false;
  const int64_t lds = tab + int64_t(best_w) * h->G * grp;
  if (lds > 65536 &&
      hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  *wpb = best_w;
  *max_blocks = best_nb * h->n_cu;
  *lds_out = lds;
  return true;
}

// Both passes' shapes; sim_costs_ok false when the first does not fit.
int sim_plan(dip_sim *h) {
  h->sim_costs_ok = false;
  h->sim2_ok = false;
  h->sim_state_base = int64_t(h->sim_tab_vec) * 16;
  if (!sim_shape(h, h->pool_slots, h->forced_variant == 9 ? h->forced_wpb : 0, &h->sim_wpb,
                 &h->sim_max_blocks, &h->sim_lds))
    return DIP_OK;
  h->sim_costs_ok = true;
  if (h->pool_slots < 16)
    h->sim2_ok = sim_shape(h, 16, 0, &h->sim2_wpb, &h->sim2_max_blocks, &h->sim2_lds);
  return DIP_OK;
}

int choose_config(dip_sim *h) {
  // general configuration first (always available)
  const bool force_gen = h->forced_variant >= 1 && h->forced_variant <= 4;
  Pick g = best_of(h, force_gen ? h->forced_variant : 1, force_gen ? h->forced_variant : 4,
                   force_gen ? h->forced_wpb : 0);
  if (g.v == 0) return DIP_E_UNSUPPORTED;
  int rc = apply_pick(h, g, &h->gen_variant, &h->gen_wpb, &h->gen_max_blocks, &h->gen_lds);
  if (rc != DIP_OK) return rc;
  if (force_gen || !h->pool_ok) {
    if (h->forced_variant >= 8) return DIP_E_UNSUPPORTED;
    h->variant = h->gen_variant;
    h->wpb = h->gen_wpb;
    h->max_blocks = h->gen_max_blocks;
    h->lds_bytes = h->gen_lds;
    return DIP_OK;
  }
  if (h->forced_variant == 9 && !h->sim_ok) return DIP_E_UNSUPPORTED;
  // variant 8's shape: also what variant 9 runs for costs outside its records
  Pick p = best_of(h, 8, 8, h->forced_variant == 8 ? h->forced_wpb : 0);
  if (p.v == 0) return DIP_E_UNSUPPORTED;
  rc = ensure_fallback(h);
  if (rc != DIP_OK) return rc;
  rc = apply_pick(h, p, &h->variant, &h->wpb, &h->max_blocks, &h->lds_bytes);
  if (rc != DIP_OK) return rc;
  if (h->sim_ok && h->forced_variant != 8) {
    h->variant = 9;
    if (h->costs_set) {
      rc = sim_plan(h);
      if (rc != DIP_OK) return rc;
      // a forced shape the current costs or the LDS do not allow
      if (h->forced_variant == 9 && !h->sim_costs_ok) return DIP_E_UNSUPPORTED;
    }
  }
  return DIP_OK;
}

int check_costs_against(int32_t P, const int32_t *n_ops, const int32_t *pred_ptr,
                        const int32_t *op_slot, const uint8_t *kind, int32_t n_slots,
                        const dip_costs *c, int64_t *total_out) {
  if (!c || !c->op_cost || !c->slot_act) return DIP_E_INVAL;
  int64_t N = 0;
  for (int r = 0; r < P; ++r) N += n_ops[r];
  const int64_t E = pred_ptr[N];
  if (E > 0 && !c->edge_comm) return DIP_E_INVAL;
  int64_t total = 0;
  for (int64_t g = 0; g < N; ++g) {
    if (c->op_cost[g] < 0) return DIP_E_RANGE;
    total += c->op_cost[g];
  }
  for (int64_t e = 0; e < E; ++e) {
    if (c->edge_comm[e] < 0) return DIP_E_RANGE;
    total += c->edge_comm[e];
  }
  if (total > INT32_MAX) return DIP_E_RANGE;
  for (int32_t s = 0; s < n_slots; ++s)
    if (c->slot_act[s] < 0) return DIP_E_RANGE;
  // per rank: the running activation sum stays within int32 either way
  int64_t off = 0;
  for (int r = 0; r < P; ++r) {
    int64_t up = 0, down = 0;
    for (int64_t g = off; g < off + n_ops[r]; ++g) {
      const int64_t act = c->slot_act[op_slot[g]];
      if (kind[g] == 0) up += act;
      else down += act;
    }
    if (up > INT32_MAX || down > INT32_MAX) return DIP_E_RANGE;
    off += n_ops[r];
  }
  if (total_out) *total_out = total;
  return DIP_OK;
}

struct StageLayout {
  int64_t rec, edge, busy, md, prec8, pedge, stab, slane, total;
};

// bytes of the simulation kernel's table image at most (direct records, or
// pages with a page map, then the extra edges)
int64_t sim_tab_bound(const dip_sim *h) {
  const int64_t direct = align16(int64_t(h->N) * 8);
  const int64_t pages = int64_t(h->N) / kSimPage + h->P;
  const int64_t paged = pages * kSimPage * 8 + align16(pages * 2);
  return std::max(direct, paged) + align16(int64_t(std::max(h->sim_n_extra, 1)) * 4);
}

StageLayout stage_layout(const dip_sim *h) {
  StageLayout L{};
  int64_t off = 0;
  L.rec = off; off += align16(int64_t(h->N) * 16);
  L.edge = off; off += align16(int64_t(std::max(h->E, 1)) * 8);
  L.busy = off; off += align16(int64_t(h->P) * 4);
  L.md = off; off += align16(int64_t(h->N) * 4);
  L.prec8 = off; off += h->pool_ok ? align16(int64_t(h->N) * 16) : 0;
  L.pedge = off; off += h->pool_ok ? align16(int64_t(std::max(h->n_extra, 1)) * 8) : 0;
  L.stab = off; off += h->sim_ok ? sim_tab_bound(h) : 0;
  L.slane = off; off += h->sim_ok ? align16(int64_t(h->P) * 16) : 0;
  L.total = off;
  return L;
}

// Greedy records per (internal group, rank): {cost, act, local id |
// successors << 16, index of the second successor}, then the first successor
// {internal group | kind << 16 | rank << 17, comm, join index or -1, the
// join's predecessor count}; further successors in the same 16-byte form.
// The staging area is guarded by the caller's wait on stage_done.
int upload_greedy_records(dip_sim *h, const dip_costs *c, hipStream_t stream) {
  const int32_t P = h->P, G = h->gr_G;
  int4 *rec = reinterpret_cast<int4 *>(h->h_gr_stage);
  int4 *ext = rec + int64_t(G) * P * 2;
  auto succ_entry = [&](int32_t k) {
    const int32_t o = h->gr_succ_op[k], e = h->gr_succ_edge[k];
    const uint32_t w = uint32_t(h->gr_ig[o]) | (uint32_t(h->kind[o]) << 16) |
                       (uint32_t(h->rank_of[o]) << 17);
    const int32_t j = h->gr_join[o];
    return make_int4(int32_t(w), c->edge_comm[e], j,
                     j >= 0 ? h->pred_ptr[o + 1] - h->pred_ptr[o] : 0);
  };
  int32_t xi = 0;
  for (int32_t ig = 0; ig < G; ++ig)
    for (int32_t r = 0; r < P; ++r) {
      int4 *q = rec + (int64_t(ig) * P + r) * 2;
      const int32_t g = h->gr_op[int64_t(ig) * P + r];
      if (g < 0) {
        q[0] = make_int4(0, 0, int32_t(kGreedyNoStage), 0);
        q[1] = make_int4(0, 0, -1, 0);
        continue;
      }
      const int32_t b = h->gr_succ_ptr[g], ns = h->gr_succ_ptr[g + 1] - b;
      q[0] = make_int4(c->op_cost[g], c->slot_act[h->op_slot[g]],
                       int32_t(uint32_t(g - h->rank_off[r]) | (uint32_t(ns) << 16)), xi);
      q[1] = ns > 0 ? succ_entry(b) : make_int4(0, 0, -1, 0);
      for (int32_t k = 1; k < ns; ++k) ext[xi++] = succ_entry(b + k);
    }
  DIP_HIP(hipMemcpyAsync(h->d_gr_rec, rec, size_t(G) * P * 32, hipMemcpyHostToDevice, stream));
  if (xi > 0) DIP_HIP(hipMemcpyAsync(h->d_gr_succ, ext, size_t(xi) * 16, hipMemcpyHostToDevice, stream));
  h->gr_costs_ok = true;
  return DIP_OK;
}

// The simulation kernel's tables for these costs (see kern_sim.hip and
// internal.h for the record and edge-word formats): records relative to their
// op, stored directly when small, else as pages of kSimPage records of one
// rank with equal pages kept once; then the extra edges.  Leaves
// sim_costs_ok false (evaluate then runs variant 8) when a cost or latency is
// outside the record's fields or the tables do not fit in LDS.
int upload_sim_tables(dip_sim *h, const dip_costs *c, const int32_t *busy, const StageLayout &L,
                      hipStream_t stream) {
  h->sim_costs_ok = false;
  for (int32_t g = 0; g < h->N; ++g)
    if (uint32_t(c->op_cost[g]) > kSimCostMax) return DIP_OK;
  for (int32_t e = 0; e < h->E; ++e)
    if (uint32_t(c->edge_comm[e]) > kSimCommMax) return DIP_OK;
  const int32_t P = h->P;
  // an edge between two ops of one rank with zero latency holds by the order
  // alone once the tile check has verified that the predecessor comes first
  // (it flags the candidate deadlocked otherwise): dropped, its producer then
  // publishes no end time for it
  h->sim_drop_self = h->to_ok && use_tile_check(h);
  auto dropped = [&](int32_t g, int32_t k) {
    return h->sim_drop_self && h->rank_of[h->pred_op[k]] == h->rank_of[g] && c->edge_comm[k] == 0;
  };
  std::vector<int32_t> readers(size_t(h->N), 0);
  for (int32_t g = 0; g < h->N; ++g)
    for (int32_t k = h->pred_ptr[g]; k < h->pred_ptr[g + 1]; ++k)
      if (!dropped(g, k)) ++readers[h->pred_op[k]];
  std::vector<uint32_t> rec(size_t(h->N) * 2), extra;
  extra.reserve(size_t(std::max(h->sim_n_extra, 1)));
  std::vector<int32_t> kept;
  auto edge_word = [&](int32_t g, int32_t k, bool last) {
    const int32_t p = h->pred_op[k];
    const int32_t r = h->rank_of[g], rp = h->rank_of[p];
    const int32_t d = (p - h->rank_off[rp]) - (g - h->rank_off[r]);
    const uint32_t dr = uint32_t((rp - r + P) % P);
    return dr | ((uint32_t(d) & 0x3fffu) << 6) | (uint32_t(c->edge_comm[k]) << 20) |
           (last ? kSimLast : 0u);
  };
  for (int32_t g = 0; g < h->N; ++g) {
    kept.clear();
    for (int32_t k = h->pred_ptr[g]; k < h->pred_ptr[g + 1]; ++k)
      if (!dropped(g, k)) kept.push_back(k);
    const int32_t np = int32_t(kept.size());
    rec[2 * g] = uint32_t(c->op_cost[g]) | (uint32_t(readers[g]) << 20) |
                 (np > 1 ? kSimMulti : 0u) | (np > 0 ? kSimHasPred : 0u);
    if (np == 1) {
      rec[2 * g + 1] = edge_word(g, kept[0], true);
    } else if (np > 1) {
      rec[2 * g + 1] = uint32_t(extra.size());
      for (int32_t i = 0; i < np; ++i) extra.push_back(edge_word(g, kept[i], i == np - 1));
    } else {
      rec[2 * g + 1] = 0;
    }
  }
  unsigned char *img = h->h_stage + L.stab;
  int32_t *lane = reinterpret_cast<int32_t *>(h->h_stage + L.slane);
  const int64_t direct = align16(int64_t(h->N) * 8);
  int64_t off_pmap = 0, recs_bytes = direct;
  std::vector<uint16_t> pmap;
  std::vector<int32_t> recb(P);
  // pages: each rank's records in runs of kSimPage local ids, equal runs once
  bool paged = false;
  if (direct > kSimDirectMax) {
    std::unordered_map<std::string, int32_t> seen;
    std::vector<uint32_t> pages;
    bool ok = true;
    for (int r = 0; r < P && ok; ++r) {
      recb[r] = int32_t(pmap.size());
      for (int32_t p0 = 0; p0 < h->n_ops[r]; p0 += kSimPage) {
        std::string key(size_t(kSimPage) * 8, '\0');
        const int32_t n = std::min(kSimPage, h->n_ops[r] - p0);
        std::memcpy(&key[0], &rec[2 * size_t(h->rank_off[r] + p0)], size_t(n) * 8);
        auto it = seen.find(key);
        int32_t id;
        if (it == seen.end()) {
          id = int32_t(seen.size());
          seen.emplace(key, id);
          const size_t at = pages.size();
          pages.resize(at + size_t(kSimPage) * 2);
          std::memcpy(&pages[at], key.data(), key.size());
        } else {
          id = it->second;
        }
        if (id >= kSimMaxPages) ok = false;
        pmap.push_back(uint16_t(id * kSimPage));
      }
    }
    const int64_t pbytes = int64_t(pages.size()) * 4;
    if (ok && pbytes + align16(int64_t(pmap.size()) * 2) < direct) {
      paged = true;
      recs_bytes = pbytes;
      std::memcpy(img, pages.data(), size_t(pbytes));
      off_pmap = pbytes;
      std::memcpy(img + off_pmap, pmap.data(), pmap.size() * 2);
      recs_bytes = pbytes + align16(int64_t(pmap.size()) * 2);
    }
  }
  if (!paged) {
    std::memcpy(img, rec.data(), size_t(h->N) * 8);
    for (int r = 0; r < P; ++r) recb[r] = h->rank_off[r];
    recs_bytes = direct;
  }
  const int64_t off_extra = recs_bytes;
  if (!extra.empty()) std::memcpy(img + off_extra, extra.data(), extra.size() * 4);
  const int64_t total = off_extra + align16(int64_t(std::max<size_t>(extra.size(), 1)) * 4);
  if (total > L.slane - L.stab || total > h->sim_tab_cap) return DIP_OK;
  for (int r = 0; r < P; ++r) {
    lane[4 * r] = h->rank_off[r];
    lane[4 * r + 1] = h->n_ops[r];
    lane[4 * r + 2] = busy[r];
    lane[4 * r + 3] = recb[r];
  }
  h->sim_paged = paged;
  h->sim_off_pmap = uint32_t(off_pmap);
  h->sim_off_extra = uint32_t(off_extra);
  h->sim_tab_vec = int32_t(total / 16);
  DIP_HIP(hipMemcpyAsync(h->d_sim_tab, img, size_t(total), hipMemcpyHostToDevice, stream));
  DIP_HIP(hipMemcpyAsync(h->d_sim_lane, lane, size_t(P) * 16, hipMemcpyHostToDevice, stream));
  return sim_plan(h);
}

int upload_costs(dip_sim *h, const dip_costs *c, hipStream_t stream) {
  int64_t total = 0;
  int rc = check_costs_against(h->P, h->n_ops.data(), h->pred_ptr.data(), h->op_slot.data(),
                               h->kind.data(), h->n_slots, c, &total);
  if (rc != DIP_OK) return rc;
  if (h->stage_pending) {
    DIP_HIP(hipEventSynchronize(h->stage_done));
    h->stage_pending = false;
  }
  if (c->op_cost != h->last_cost.data()) {
    h->last_cost.assign(c->op_cost, c->op_cost + h->N);
    h->last_comm.assign(c->edge_comm, c->edge_comm + h->E);
    h->last_act.assign(c->slot_act, c->slot_act + h->n_slots);
  }
  const StageLayout L = stage_layout(h);
  int4 *rec = reinterpret_cast<int4 *>(h->h_stage + L.rec);
  int2 *edge = reinterpret_cast<int2 *>(h->h_stage + L.edge);
  int32_t *busy = reinterpret_cast<int32_t *>(h->h_stage + L.busy);
  for (int32_t g = 0; g < h->N; ++g) {
    const int32_t act = c->slot_act[h->op_slot[g]];
    rec[g] = make_int4(c->op_cost[g], h->kind[g] == 0 ? act : -act, h->pred_ptr[g],
                       h->pred_ptr[g + 1]);
  }
  for (int32_t e = 0; e < h->E; ++e) edge[e] = make_int2(h->pred_op[e], c->edge_comm[e]);
  for (int r = 0; r < h->P; ++r) {
    int64_t s = 0;
    for (int32_t g = h->rank_off[r]; g < h->rank_off[r + 1]; ++g) s += c->op_cost[g];
    busy[r] = int32_t(s);
  }
  DIP_HIP(hipMemcpyAsync(h->d_rec, rec, size_t(h->N) * 16, hipMemcpyHostToDevice, stream));
  if (h->E > 0)
    DIP_HIP(hipMemcpyAsync(h->d_edge, edge, size_t(h->E) * 8, hipMemcpyHostToDevice, stream));
  DIP_HIP(hipMemcpyAsync(h->d_busy, busy, size_t(h->P) * 4, hipMemcpyHostToDevice, stream));
  {
    int32_t *md = reinterpret_cast<int32_t *>(h->h_stage + L.md);
    for (int32_t g = 0; g < h->N; ++g) md[g] = rec[g].y;
    DIP_HIP(hipMemcpyAsync(h->d_md, md, size_t(h->N) * 4, hipMemcpyHostToDevice, stream));
  }
  if (h->pool_ok) {
    // pool records {cost, first edge's comm, first edge word | readers << 24,
    // item tag or 0 | index of the op's extra edges << 16}; edge words are
    // {pred tag | pred rank << 16 | last}; tags are rank-local ids + 1
    int4 *pr = reinterpret_cast<int4 *>(h->h_stage + L.prec8);
    int2 *pe = reinterpret_cast<int2 *>(h->h_stage + L.pedge);
    auto word = [&](int32_t k, bool last) {
      const int32_t p = h->pred_op[k];
      const int32_t rp = h->rank_of[p];
      return uint32_t(p - h->rank_off[rp] + 1) | (uint32_t(rp) << kEdgeRankShift) |
             (last ? kEdgeLast : 0u);
    };
    int32_t xi = 0;
    for (int32_t g = 0; g < h->N; ++g) {
      const int32_t b = h->pred_ptr[g], np = h->pred_ptr[g + 1] - b;
      const int32_t tag = h->n_cons[g] > 0 ? g - h->rank_off[h->rank_of[g]] + 1 : 0;
      const uint32_t w0 = np > 0 ? word(b, np == 1) : kNoEdgeWord;
      pr[g] = make_int4(c->op_cost[g], np > 0 ? c->edge_comm[b] : 0,
                        int32_t(w0 | (uint32_t(h->n_cons[g]) << 24)),
                        int32_t(uint32_t(tag) | (uint32_t(xi) << 16)));
      for (int32_t k = 1; k < np; ++k) pe[xi++] = make_int2(int32_t(word(b + k, k == np - 1)), c->edge_comm[b + k]);
    }
    DIP_HIP(hipMemcpyAsync(h->d_pool_rec, pr, size_t(h->N) * 16, hipMemcpyHostToDevice, stream));
    if (h->n_extra > 0)
      DIP_HIP(hipMemcpyAsync(h->d_pool_edge, pe, size_t(h->n_extra) * 8, hipMemcpyHostToDevice, stream));
  }
  if (h->sim_ok) {
    rc = upload_sim_tables(h, c, busy, L, stream);
    if (rc != DIP_OK) return rc;
  }
  if (h->gr_ok) {
    rc = upload_greedy_records(h, c, stream);
    if (rc != DIP_OK) return rc;
  }
  DIP_HIP(hipEventRecord(h->stage_done, stream));
  h->stage_pending = true;
  h->costs_set = true;
  return DIP_OK;
}

// LDS plan of one greedy candidate with inboxes of K entries: the inboxes,
// their counts and the join accumulators overlay the priorities, which only
// the set-up reads; then positions, position -> group and position -> global
// rank (16-bit each).
bool greedy_layout(const dip_sim *h, int K, int pwl, dip_sim::GrLaunch *L, bool gring = false) {
  const int64_t G = h->gr_G, P = h->P, J = h->gr_J;
  L->pwl = pwl;
  L->K = K;
  L->wpb = 1;
  L->gring = gring;
  L->max_blocks = 0;
  // two rings per rank (none in LDS with gring); two head/count words per
  // lane (padding lanes' stay 0)
  const int64_t lanes = int64_t(1) << pwl;
  const int64_t rings = gring ? 0 : P * (2 * K + 1) * 8;
  L->off_pend = 0;
  L->off_npend = int32_t(rings);
  L->off_join = int32_t(rings + 8 * lanes);
  const int64_t head = align16(std::max<int64_t>(4 * G, L->off_join + 8 * J));
  L->off_gpos = int32_t(head);
  L->off_ord = int32_t(head + align16(2 * G));
  L->off_grk = int32_t(head + 2 * align16(2 * G));
  L->cand_bytes = int32_t(head + 3 * align16(2 * G));
  L->lds = h->gr_meta_bytes + int64_t(kWave >> pwl) * L->cand_bytes;
  if (L->lds > h->lds_block_max) return false;
  int bpc = 0;
  const void *k = greedy_kernel_ptr(pwl, h->gr_nw, gring);
  if (!k || (L->lds > 65536 && hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize,
                                                   int(L->lds)) != hipSuccess) ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&bpc, k, kWave * L->wpb,
                                                   size_t(L->lds)) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  L->blocks_per_cu = std::max(1, bpc);
  return true;
}

void release_rollout_memopt(dip_sim *h) {
  if (h->d_rl_orders) (void)hipFree(h->d_rl_orders);
  if (h->d_rl_mo_time) (void)hipFree(h->d_rl_mo_time);
  if (h->d_rl_mo_peak) (void)hipFree(h->d_rl_mo_peak);
  if (h->d_rl_mo_status) (void)hipFree(h->d_rl_mo_status);
  if (h->d_rl_choice) (void)hipFree(h->d_rl_choice);
  h->d_rl_orders = nullptr;
  h->d_rl_mo_time = nullptr;
  h->d_rl_mo_peak = nullptr;
  h->d_rl_mo_status = h->d_rl_choice = nullptr;
  h->rl_mo_cap = 0;
}

void release_rollouts(dip_sim *h) {
  if (h->d_rl_class) (void)hipFree(h->d_rl_class);
  if (h->d_rl_seq) (void)hipFree(h->d_rl_seq);
  if (h->h_rl_seq) (void)hipHostFree(h->h_rl_seq);
  if (h->rl_seq_ev) (void)hipEventDestroy(h->rl_seq_ev);
  if (h->d_rl_bub) (void)hipFree(h->d_rl_bub);
  if (h->d_rl_peak) (void)hipFree(h->d_rl_peak);
  release_rollout_memopt(h);
  h->d_rl_class = h->d_rl_seq = h->h_rl_seq = nullptr;
  h->rl_leaf_cap = 0;
  h->rl_seq_ev = nullptr;
  h->rl_seq_pending = false;
  h->d_rl_bub = h->d_rl_peak = nullptr;
  h->rl_cap = 0;
  h->rl_ok = false;
}

void release_memopt(dip_sim *h) {
  if (h->d_mo_pair_off) (void)hipFree(h->d_mo_pair_off);
  if (h->d_mo_lid_pair) (void)hipFree(h->d_mo_lid_pair);
  if (h->d_mo_time) (void)hipFree(h->d_mo_time);
  if (h->d_mo_mem) (void)hipFree(h->d_mo_mem);
  if (h->d_mo_key) (void)hipFree(h->d_mo_key);
  if (h->d_mo_dm) (void)hipFree(h->d_mo_dm);
  h->d_mo_pair_off = h->d_mo_lid_pair = nullptr;
  h->d_mo_time = nullptr;
  h->d_mo_mem = h->d_mo_dm = nullptr;
  h->d_mo_key = nullptr;
  h->mo_ok = false;
}

void release_greedy(dip_sim *h) {
  if (h->d_gr_caller) (void)hipFree(h->d_gr_caller);
  if (h->d_gr_src) (void)hipFree(h->d_gr_src);
  if (h->d_gr_rec) (void)hipFree(h->d_gr_rec);
  if (h->d_gr_succ) (void)hipFree(h->d_gr_succ);
  if (h->h_gr_stage) (void)hipHostFree(h->h_gr_stage);
  if (h->d_gr_retry) (void)hipFree(h->d_gr_retry);
  if (h->d_gr_retry_count) (void)hipFree(h->d_gr_retry_count);
  if (h->h_gr_seen) (void)hipHostFree(h->h_gr_seen);
  if (h->gr_seen_ev) (void)hipEventDestroy(h->gr_seen_ev);
  if (h->d_gr_ring) (void)hipFree(h->d_gr_ring);
  h->d_gr_ring = nullptr;
  h->gr_ring_bytes = 0;
  h->h_gr_seen = nullptr;
  h->gr_seen_ev = nullptr;
  h->gr_seen_pending = false;
  h->d_gr_caller = h->d_gr_src = nullptr;
  h->d_gr_rec = h->d_gr_succ = nullptr;
  h->h_gr_stage = nullptr;
  h->d_gr_retry = nullptr;
  h->d_gr_retry_count = nullptr;
  h->gr_retry_cap = 0;
  h->gr_ok = h->gr_costs_ok = false;
}

void release(dip_sim *h) {
  if (!h) return;
  (void)hipDeviceSynchronize();
  if (h->d_rec) (void)hipFree(h->d_rec);
  if (h->d_edge) (void)hipFree(h->d_edge);
  if (h->d_md) (void)hipFree(h->d_md);
  if (h->d_selfp) (void)hipFree(h->d_selfp);
  if (h->d_sim_tab) (void)hipFree(h->d_sim_tab);
  if (h->d_sim_lane) (void)hipFree(h->d_sim_lane);
  if (h->d_rank_off) (void)hipFree(h->d_rank_off);
  if (h->d_busy) (void)hipFree(h->d_busy);
  if (h->d_cap) (void)hipFree(h->d_cap);
  if (h->tc.d_plan) (void)hipFree(h->tc.d_plan);
  if (h->to.d_plan) (void)hipFree(h->to.d_plan);
  if (h->d_scratch_gen) (void)hipFree(h->d_scratch_gen);
  if (h->d_scratch_fb) (void)hipFree(h->d_scratch_fb);
  if (h->d_pool_rec) (void)hipFree(h->d_pool_rec);
  if (h->d_pool_edge) (void)hipFree(h->d_pool_edge);
  if (h->d_retry) (void)hipFree(h->d_retry);
  if (h->d_retry2) (void)hipFree(h->d_retry2);
  if (h->d_retry_count) (void)hipFree(h->d_retry_count);
  release_rollouts(h);
  release_greedy(h);
  release_memopt(h);
  if (h->h_stage) (void)hipHostFree(h->h_stage);
  if (h->stage_done) (void)hipEventDestroy(h->stage_done);
  for (hipEvent_t &ev : h->prof_ev)
    if (ev) (void)hipEventDestroy(ev);
  delete h;
}

}  // namespace

extern "C" {

int dip_sim_abi_version(void) { return DIP_SIM_ABI_VERSION; }

int dip_sim_check_topology(const dip_topology *t) {
  if (!t || !t->n_ops || !t->pred_ptr || !t->op_kind || !t->op_slot || !t->mem_cap)
    return DIP_E_INVAL;
  if (t->n_ranks <= 0) return DIP_E_INVAL;
  if (t->n_ranks > kMaxRanks) return DIP_E_UNSUPPORTED;
  int64_t N = 0;
  for (int r = 0; r < t->n_ranks; ++r) {
    if (t->n_ops[r] < 0 || t->n_ops[r] > kMaxOpsPerRank) return DIP_E_TOPO;
    N += t->n_ops[r];
  }
  if (N == 0 || N > INT32_MAX / 64) return DIP_E_TOPO;
  if (t->cand_stride < N || t->cand_stride % 8 != 0) return DIP_E_INVAL;
  if (t->n_slots < 0) return DIP_E_TOPO;
  if (t->pred_ptr[0] != 0) return DIP_E_TOPO;
  for (int64_t g = 0; g < N; ++g)
    if (t->pred_ptr[g + 1] < t->pred_ptr[g]) return DIP_E_TOPO;
  const int64_t E = t->pred_ptr[N];
  if (E > 0 && !t->pred_op) return DIP_E_INVAL;
  for (int64_t g = 0; g < N; ++g) {
    for (int32_t e = t->pred_ptr[g]; e < t->pred_ptr[g + 1]; ++e)
      if (t->pred_op[e] < 0 || t->pred_op[e] >= N || t->pred_op[e] == g) return DIP_E_TOPO;
    if (t->op_kind[g] > 1) return DIP_E_TOPO;
    if (t->op_slot[g] < 0 || t->op_slot[g] >= t->n_slots) return DIP_E_TOPO;
  }
  return DIP_OK;
}

int dip_sim_check_costs(const dip_topology *t, const dip_costs *c) {
  int rc = dip_sim_check_topology(t);
  if (rc != DIP_OK) return rc;
  return check_costs_against(t->n_ranks, t->n_ops, t->pred_ptr, t->op_slot, t->op_kind,
                             t->n_slots, c, nullptr);
}

int dip_sim_create(const dip_topology *t, dip_sim **out) {
  if (!out) return DIP_E_INVAL;
  *out = nullptr;
  int rc = dip_sim_check_topology(t);
  if (rc != DIP_OK) return rc;
  dip_sim *h = new (std::nothrow) dip_sim();
  if (!h) return DIP_E_NOMEM;
  h->P = t->n_ranks;
  h->n_ops.assign(t->n_ops, t->n_ops + h->P);
  h->rank_off.assign(h->P + 1, 0);
  for (int r = 0; r < h->P; ++r) h->rank_off[r + 1] = h->rank_off[r] + t->n_ops[r];
  h->N = h->rank_off[h->P];
  h->E = t->pred_ptr[h->N];
  h->n_slots = t->n_slots;
  h->stride = t->cand_stride;
  h->pred_ptr.assign(t->pred_ptr, t->pred_ptr + h->N + 1);
  if (h->E > 0) h->pred_op.assign(t->pred_op, t->pred_op + h->E);
  h->kind.assign(t->op_kind, t->op_kind + h->N);
  h->op_slot.assign(t->op_slot, t->op_slot + h->N);
  h->cap.assign(t->mem_cap, t->mem_cap + h->P);
  h->pwl = ceil_pow2_log2(h->P);
  h->G = kWave >> h->pwl;
  // kernel eligibility
  {
    std::vector<int32_t> &rank_of = h->rank_of;
    rank_of.assign(h->N, 0);
    for (int r = 0; r < h->P; ++r)
      for (int32_t g = h->rank_off[r]; g < h->rank_off[r + 1]; ++g) rank_of[g] = r;
    // pool kernel eligibility: at most 15 consumers per op (4-bit reader
    // counts), fewer than 2^16 edges after the ops' first ones (16-bit index
    // in the record; tags are rank-local ids + 1 <= 32768 by construction)
    h->self_pred.assign(h->N, 0);
    h->self_ok = true;
    for (int32_t g = 0; g < h->N; ++g)
      for (int32_t k = h->pred_ptr[g]; k < h->pred_ptr[g + 1]; ++k) {
        const int32_t p = h->pred_op[k];
        if (rank_of[p] != rank_of[g]) continue;
        if (h->self_pred[g] != 0) h->self_ok = false;
        h->self_pred[g] = p - h->rank_off[rank_of[p]] + 1;
        h->self_ranks |= uint64_t(1) << rank_of[g];
      }
    h->n_cons.assign(h->N, 0);
    bool pool = int64_t(h->N) * 16 < INT32_MAX;
    int64_t extra = 0;
    for (int32_t g = 0; g < h->N && pool; ++g) {
      extra += std::max(h->pred_ptr[g + 1] - h->pred_ptr[g] - 1, 0);
      for (int32_t k = h->pred_ptr[g]; k < h->pred_ptr[g + 1]; ++k)
        if (++h->n_cons[h->pred_op[k]] > 15) pool = false;
    }
    h->pool_ok = pool && extra < (1 << 16);
    h->n_extra = int32_t(std::min<int64_t>(extra, INT32_MAX));
    // small tables go to each block's LDS, read once per block
    const int64_t tab = align16(int64_t(h->N) * 16) + align16(int64_t(std::max(h->n_extra, 1)) * 8);
    h->pool_tab = h->pool_ok && tab <= kPoolTabLimit;
    h->pool_tab_bytes = h->pool_tab ? tab : 0;
    // simulation kernel eligibility: local ids below 8192 (14-bit id
    // differences), at most 15 consumers per op (as the pool kernel)
    int32_t max_nr = 0;
    for (int r = 0; r < h->P; ++r) max_nr = std::max(max_nr, h->n_ops[r]);
    int64_t sim_extra = 0;
    for (int32_t g = 0; g < h->N; ++g) {
      const int32_t np = h->pred_ptr[g + 1] - h->pred_ptr[g];
      if (np > 1) sim_extra += np;
    }
    // (the simulation kernel plays rank r on lane r of a power-of-two group)
    h->sim_ok = h->pool_ok && (h->P & (h->P - 1)) == 0 && max_nr <= kSimDeltaMax + 1 &&
                sim_extra < (int64_t(1) << 24);
    h->sim_n_extra = int32_t(std::min<int64_t>(sim_extra, INT32_MAX));
    // pools: 8 slots per rank (the simulation kernel's candidates that fill
    // them go through a second pass with 16)
    h->pool_slots = 8;
  }

  auto hip_fail = [&](hipError_t e) { g_last_hip = e; release(h); return int(DIP_E_HIP); };
  hipError_t e;
  if ((e = hipGetDevice(&h->device)) != hipSuccess) return hip_fail(e);
  int v = 0;
  if ((e = hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, h->device)) != hipSuccess)
    return hip_fail(e);
  h->n_cu = std::max(1, v);
  if ((e = hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, h->device)) != hipSuccess)
    return hip_fail(e);
  h->lds_block_max = v;
  if (hipDeviceGetAttribute(&v, hipDeviceAttributeSharedMemPerBlockOptin, h->device) == hipSuccess && v > 0)
    h->lds_block_max = std::max<int64_t>(h->lds_block_max, v);
  (void)hipGetLastError();
  h->d_static = static_scratch_on_current_device();
  if (!h->d_static) return hip_fail(g_last_hip);
  if ((e = hipMalloc(&h->d_rec, size_t(h->N) * 16)) != hipSuccess) return hip_fail(e);
  if ((e = hipMalloc(&h->d_edge, size_t(std::max(h->E, 1)) * 8)) != hipSuccess) return hip_fail(e);
  if ((e = hipMalloc(&h->d_md, size_t(h->N) * 4)) != hipSuccess) return hip_fail(e);
  if (h->self_ok) {
    if ((e = hipMalloc(&h->d_selfp, size_t(h->N) * 4)) != hipSuccess) return hip_fail(e);
    if ((e = hipMemcpy(h->d_selfp, h->self_pred.data(), size_t(h->N) * 4,
                       hipMemcpyHostToDevice)) != hipSuccess)
      return hip_fail(e);
  }
  if (h->pool_ok) {
    if ((e = hipMalloc(&h->d_pool_rec, size_t(h->N) * 16)) != hipSuccess) return hip_fail(e);
    if ((e = hipMalloc(&h->d_pool_edge, size_t(std::max(h->n_extra, 1)) * 8)) != hipSuccess)
      return hip_fail(e);
  }
  if (h->sim_ok) {
    h->sim_tab_cap = sim_tab_bound(h);
    if ((e = hipMalloc(&h->d_sim_tab, size_t(h->sim_tab_cap))) != hipSuccess) return hip_fail(e);
    if ((e = hipMalloc(&h->d_sim_lane, size_t(h->P) * 16)) != hipSuccess) return hip_fail(e);
  }
  if ((e = hipMalloc(&h->d_rank_off, size_t(h->P + 1) * 4)) != hipSuccess) return hip_fail(e);
  if ((e = hipMalloc(&h->d_busy, size_t(h->P) * 4)) != hipSuccess) return hip_fail(e);
  if ((e = hipMalloc(&h->d_cap, size_t(h->P) * 4)) != hipSuccess) return hip_fail(e);
  if ((e = hipMemcpy(h->d_rank_off, h->rank_off.data(), size_t(h->P + 1) * 4,
                     hipMemcpyHostToDevice)) != hipSuccess)
    return hip_fail(e);
  if ((e = hipMemcpy(h->d_cap, h->cap.data(), size_t(h->P) * 4, hipMemcpyHostToDevice)) != hipSuccess)
    return hip_fail(e);
  h->stage_bytes = stage_layout(h).total;
  if ((e = hipHostMalloc(reinterpret_cast<void **>(&h->h_stage), size_t(h->stage_bytes),
                         hipHostMallocDefault)) != hipSuccess)
    return hip_fail(e);
  if ((e = hipEventCreateWithFlags(&h->stage_done, hipEventDisableTiming)) != hipSuccess)
    return hip_fail(e);
  if (h->pool_ok && (rc = plan_tile_check(h)) != DIP_OK) {
    release(h);
    return rc;
  }
  rc = choose_config(h);
  if (rc != DIP_OK) {
    release(h);
    return rc;
  }
  *out = h;
  return DIP_OK;
}

int dip_sim_configure(dip_sim *h, int32_t variant, int32_t waves_per_block) {
  if (!h || variant < 0 || variant > 9 || (variant >= 5 && variant <= 7)) return DIP_E_INVAL;
  if (!(waves_per_block == 0 || waves_per_block == 1 || waves_per_block == 2 ||
        waves_per_block == 4 || waves_per_block == 8 || (variant == 9 && waves_per_block == 16)))
    return DIP_E_INVAL;
  const int old_v = h->forced_variant, old_w = h->forced_wpb;
  h->forced_variant = variant;
  h->forced_wpb = waves_per_block;
  int rc = choose_config(h);
  if (rc != DIP_OK) {
    h->forced_variant = old_v;
    h->forced_wpb = old_w;
    (void)choose_config(h);
  }
  return rc;
}

int dip_sim_configure_pool(dip_sim *h, int32_t slots_per_rank) {
  if (!h || !(slots_per_rank == 0 || pool_slots_ok(slots_per_rank))) return DIP_E_INVAL;
  if (!h->pool_ok) return DIP_E_UNSUPPORTED;
  const int old_s = h->pool_slots, old_f = h->forced_pool_slots;
  h->forced_pool_slots = slots_per_rank;
  h->pool_slots = slots_per_rank ? slots_per_rank : 8;
  int rc = choose_config(h);
  if (rc != DIP_OK) {
    h->pool_slots = old_s;
    h->forced_pool_slots = old_f;
    (void)choose_config(h);
  }
  return rc;
}

int dip_sim_configure_check(dip_sim *h, int32_t mode) {
  if (!h || mode < 0 || mode > 2) return DIP_E_INVAL;
  if (!h->pool_ok || (mode == 1 && !h->wc_ok) || (mode == 2 && !h->tc_ok)) return DIP_E_UNSUPPORTED;
  h->check_mode = mode;
  // the simulation kernel's tables drop own-rank edges only behind the tile
  // check: rebuild them from the last costs when that changes
  if (h->sim_ok && h->costs_set && h->sim_drop_self != (h->to_ok && use_tile_check(h))) {
    const dip_costs c{h->last_cost.data(), h->last_comm.data(), h->last_act.data()};
    int rc = upload_costs(h, &c, nullptr);
    if (rc != DIP_OK) return rc;
    DIP_HIP(hipStreamSynchronize(nullptr));
  }
  return DIP_OK;
}

int dip_sim_get_info(const dip_sim *h, dip_sim_info *info) {
  if (!h || !info) return DIP_E_INVAL;
  // variant 9 reports its shape for the current costs; before any costs it
  // has none yet (0 waves), and for costs outside its records variant 8 runs
  const bool sim = h->variant == 9 && (!h->costs_set || h->sim_costs_ok);
  const int v = h->variant == 9 && !sim ? 8 : h->variant;
  info->n_ranks = h->P;
  info->n_ops_total = h->N;
  info->n_edges = h->E;
  info->variant = v;
  info->cand_stride = h->stride;
  info->lanes_per_group = 1 << h->pwl;
  info->groups_per_wave = h->G;
  info->waves_per_block = sim ? (h->sim_costs_ok ? h->sim_wpb : 0) : h->wpb;
  info->lds_bytes = int32_t(sim ? (h->sim_costs_ok ? h->sim_lds : 0) : h->lds_bytes);
  info->max_blocks = sim ? (h->sim_costs_ok ? h->sim_max_blocks : 0) : h->max_blocks;
  info->scratch_bytes = h->scratch_gen_bytes + h->scratch_fb_bytes + h->retry_cap * 8;
  info->pool_slots = v >= 8 ? h->pool_slots : 0;
  info->check_kernel = v >= 8 ? (use_tile_check(h) ? 2 : 1) : 0;
  info->greedy_inbox = h->gr_ok ? h->gr_K : 0;
  info->greedy_lds_bytes = h->gr_ok ? int32_t(h->gr_main.lds) : 0;
  info->greedy_retry_ring_bytes = h->gr_ok ? h->gr_ring_bytes : 0;
  return DIP_OK;
}

}  // extern "C"

namespace {

// Device memory an evaluate call works in beyond its inputs and outputs: the
// retry counters and the two retry lists (variants 8 and 9).
struct CallScratch {
  uint32_t *counts;   // [4] zeroed by the check kernel
  int64_t *list_a;    // [n_cand] first pass retries
  int64_t *list_b;    // [n_cand] second pass retries (variant 9)
};

int evaluate_impl(dip_sim *h, const dip_costs *costs, const int16_t *orders, int64_t n_cand,
                  int32_t *out_makespan, int32_t *out_bubble, int32_t *out_peakmem,
                  uint8_t *out_flags, void *stream_, const CallScratch *sx) {
  if (!h || n_cand < 0) return DIP_E_INVAL;
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  if (costs) {
    int rc = upload_costs(h, costs, stream);
    if (rc != DIP_OK) return rc;
  }
  if (!h->costs_set) return DIP_E_STATE;
  if (n_cand == 0) return DIP_OK;
  if (!orders || !out_makespan || !out_bubble || !out_peakmem || !out_flags) return DIP_E_INVAL;
  if ((reinterpret_cast<uintptr_t>(orders) & 15) != 0) return DIP_E_INVAL;
  if ((reinterpret_cast<uintptr_t>(out_makespan) | reinterpret_cast<uintptr_t>(out_bubble) |
       reinterpret_cast<uintptr_t>(out_peakmem)) & 3)
    return DIP_E_INVAL;

  h->prof_n = 0;
  auto mark = [&](int i) -> hipError_t {
    if (!h->profile) return hipSuccess;
    h->prof_n = i + 1;
    return hipEventRecord(h->prof_ev[i], stream);
  };
  (void)hipGetLastError();
  if (h->variant >= 8) {
    CallScratch own{};
    if (!sx) {   // the handle's buffers, grown to the batch
      int rc = ensure_retry(h, n_cand);
      if (rc != DIP_OK) return rc;
      own = CallScratch{h->d_retry_count, h->d_retry, h->d_retry2};
      sx = &own;
    }
    uint32_t *const counts = sx->counts;
    h->last_counts = counts;
    DIP_HIP(mark(0));
    int rc = use_tile_check(h) ? run_tile_check(h, orders, n_cand, out_makespan, out_bubble,
                                                out_peakmem, out_flags, stream, counts)
                               : run_wave_check(h, orders, n_cand, out_makespan, out_bubble,
                                                out_peakmem, out_flags, stream, counts);
    if (rc != DIP_OK) return rc;
    DIP_HIP(mark(1));
    const uint32_t round_limit = uint32_t(h->N) + uint32_t(h->E) + 16u;
    // candidates past the resident groups: long ones are handed out on demand
    // when every group runs several in sequence (fixed successors let unlucky
    // groups pile up long candidates); with fewer, fixed successors keep the
    // second ones in few waves, and the other waves exit.  Short candidates
    // finish so often that one counter serving every request becomes the
    // bottleneck: they take fixed successors unless the batch holds at least
    // four per group, and then only the last 10 % go on demand.
    auto static_end_for = [&](int64_t n_slots) -> int64_t {
      if (h->N > 4096) return n_cand >= 2 * n_slots ? n_slots : INT64_MAX;
      return n_cand >= 4 * n_slots ? n_slots * ((n_cand / 10 * 9) / n_slots) : INT64_MAX;
    };
    const int64_t *retry_list = sx->list_a;
    const uint32_t *retry_count = counts;
    h->last_stream = stream;
    h->last_pass2 = false;
    if (h->variant == 9 && h->sim_costs_ok) {
      SimArgs a{};
      a.orders = orders;
      a.n_cand = n_cand;
      a.stride = h->stride;
      a.out_ms = out_makespan;
      a.out_bub = out_bubble;
      a.out_flags = out_flags;
      a.tab = h->d_sim_tab;
      a.tab_vec = h->sim_tab_vec;
      a.off_pmap = h->sim_off_pmap;
      a.off_extra = h->sim_off_extra;
      a.lane_info = reinterpret_cast<const int32_t *>(h->d_sim_lane);
      a.state_base = uint32_t(h->sim_state_base);
      a.P = h->P;
      a.wpb = h->sim_wpb;
      a.retry = sx->list_a;
      a.retry_count = counts;
      a.round_limit = round_limit;
      const int64_t per_block = int64_t(h->sim_wpb) * h->G;
      const int blocks =
          int(std::min<int64_t>((n_cand + per_block - 1) / per_block, h->sim_max_blocks));
      a.static_end = static_end_for(int64_t(blocks) * per_block);
      DIP_HIP(launch_sim(h->pwl, h->pool_slots, h->sim_paged, blocks, h->sim_wpb,
                         size_t(h->sim_lds), stream, a));
      DIP_HIP(mark(2));
      if (h->sim2_ok) {
        // the candidates whose pools filled, again with 16 slots per pool
        // (deadlocked orders fill small pools too; larger ones tell them
        // from merely crowded ones); its own retries go to the general kernel
        a.list = sx->list_a;
        a.list_count = counts;
        a.retry = sx->list_b;
        a.retry_count = counts + 2;
        a.wpb = h->sim2_wpb;
        a.static_end = INT64_MAX;
        DIP_HIP(launch_sim(h->pwl, 16, h->sim_paged, h->sim2_max_blocks, h->sim2_wpb,
                           size_t(h->sim2_lds), stream, a));
        retry_list = sx->list_b;
        retry_count = counts + 2;
        h->last_pass2 = true;
      }
      DIP_HIP(mark(3));
    } else {
      PoolArgs a{};
      a.orders = orders;
      a.n_cand = n_cand;
      a.stride = h->stride;
      a.out_ms = out_makespan;
      a.out_bub = out_bubble;
      a.out_flags = out_flags;
      a.rec = h->d_pool_rec;
      a.edge = h->d_pool_edge;
      a.rank_off = h->d_rank_off;
      a.busy = h->d_busy;
      a.P = h->P;
      a.wpb = h->wpb;
      a.retry = sx->list_a;
      a.retry_count = counts;
      a.rec_bytes = h->N * 16;
      a.edge_bytes = std::max(h->n_extra, 1) * 8;
      a.tab_edges = uint32_t(align16(int64_t(h->N) * 16));
      a.pool_base = uint32_t(h->pool_tab_bytes);
      a.round_limit = round_limit;
      const int64_t per_block = int64_t(h->wpb) * h->G;
      const int blocks = int(std::min<int64_t>((n_cand + per_block - 1) / per_block, h->max_blocks));
      const int64_t se = static_end_for(int64_t(blocks) * per_block);
      a.next_cand = se == INT64_MAX ? nullptr : counts + 1;
      a.static_end = se == INT64_MAX ? 0 : se;
      DIP_HIP(launch_pool(h->pwl, h->pool_slots, h->pool_tab, blocks, h->wpb,
                          size_t(h->lds_bytes), stream, a));
      DIP_HIP(mark(2));
    }

    GeneralArgs f{};
    f.orders = orders;
    f.n_cand = n_cand;
    f.stride = h->stride;
    f.out_ms = out_makespan;
    f.out_bub = out_bubble;
    f.out_peak = out_peakmem;
    f.out_flags = out_flags;
    f.rec = h->d_rec;
    f.edge = h->d_edge;
    f.rank_off = h->d_rank_off;
    f.busy = h->d_busy;
    f.cap = h->d_cap;
    f.gends = static_cast<int32_t *>(h->d_scratch_fb);
    f.P = h->P;
    f.pwl = h->pwl;
    f.G = h->G;
    f.N = h->N;
    f.E = h->E;
    f.wpb = 1;
    f.list = retry_list;
    f.list_count = retry_count;
    DIP_HIP(launch_general(h->fb_variant, h->fb_blocks, 1, size_t(h->fb_lds), stream, f));
    DIP_HIP(mark(h->prof_n));
    return DIP_OK;
  }

  const int v = h->variant <= 4 ? h->variant : h->gen_variant;
  const int wpb = h->variant <= 4 ? h->wpb : h->gen_wpb;
  const int maxb = h->variant <= 4 ? h->max_blocks : h->gen_max_blocks;
  const int64_t lds = h->variant <= 4 ? h->lds_bytes : h->gen_lds;
  GeneralArgs a{};
  a.orders = orders;
  a.n_cand = n_cand;
  a.stride = h->stride;
  a.n_groups = (n_cand + h->G - 1) / h->G;
  a.out_ms = out_makespan;
  a.out_bub = out_bubble;
  a.out_peak = out_peakmem;
  a.out_flags = out_flags;
  a.rec = h->d_rec;
  a.edge = h->d_edge;
  a.rank_off = h->d_rank_off;
  a.busy = h->d_busy;
  a.cap = h->d_cap;
  a.gends = static_cast<int32_t *>(h->d_scratch_gen);
  a.P = h->P;
  a.pwl = h->pwl;
  a.G = h->G;
  a.N = h->N;
  a.E = h->E;
  a.wpb = wpb;
  const GenBytes b = general_bytes(h, v);
  a.tab_bytes = uint32_t(b.tab);
  a.ord_bytes = uint32_t(b.ord);
  a.end_bytes = uint32_t(b.end);
  const int64_t want = (a.n_groups + wpb - 1) / wpb;
  const int blocks = int(std::min<int64_t>(want, maxb));
  DIP_HIP(mark(0));
  DIP_HIP(launch_general(v, blocks, wpb, size_t(lds), stream, a));
  DIP_HIP(mark(1));
  return DIP_OK;
}

}  // namespace

extern "C" {

int dip_sim_evaluate(dip_sim *h, const dip_costs *costs, const int16_t *orders, int64_t n_cand,
                     int32_t *out_makespan, int32_t *out_bubble, int32_t *out_peakmem,
                     uint8_t *out_flags, void *stream) {
  return evaluate_impl(h, costs, orders, n_cand, out_makespan, out_bubble, out_peakmem, out_flags,
                       stream, nullptr);
}

int dip_sim_evaluate_static(dip_sim *h, const int16_t *orders, int64_t n_cand,
                            int32_t *out_makespan, int32_t *out_bubble, int32_t *out_peakmem,
                            uint8_t *out_flags, void *stream) {
  if (!h || n_cand < 0) return DIP_E_INVAL;
  if (!h->costs_set) return DIP_E_STATE;
  if (n_cand > kStaticMaxCand) return DIP_E_CAPACITY;
  if (!h->d_static) return DIP_E_STATE;
  // the array's device address on this handle's device: counters, then the
  // two lists of kStaticMaxCand entries
  unsigned char *base = static_cast<unsigned char *>(h->d_static);
  const CallScratch sx{reinterpret_cast<uint32_t *>(base),
                       reinterpret_cast<int64_t *>(base + kStaticHead),
                       reinterpret_cast<int64_t *>(base + kStaticHead + 8 * kStaticMaxCand)};
  return evaluate_impl(h, nullptr, orders, n_cand, out_makespan, out_bubble, out_peakmem,
                       out_flags, stream, &sx);
}

int dip_sim_configure_greedy(dip_sim *h, int32_t n_groups, const int32_t *op_group) {
  if (!h || !op_group || n_groups < 1 || n_groups > 65535) return DIP_E_INVAL;
  const int32_t N = h->N, P = h->P;
  // every group holds stages of one kind, at most one per rank
  std::vector<int8_t> gk(n_groups, -1);
  std::vector<int32_t> at(int64_t(n_groups) * P, -1);
  for (int32_t g = 0; g < N; ++g) {
    const int32_t q = op_group[g];
    if (q < 0 || q >= n_groups) return DIP_E_TOPO;
    if (gk[q] >= 0 && gk[q] != int8_t(h->kind[g])) return DIP_E_TOPO;
    gk[q] = int8_t(h->kind[g]);
    int32_t &slot = at[int64_t(q) * P + h->rank_of[g]];
    if (slot >= 0) return DIP_E_TOPO;
    slot = g;
  }
  // the data edges must be acyclic (Kahn)
  std::vector<int32_t> succ_ptr(N + 1, 0), succ_op(std::max(h->E, 1)), succ_edge(std::max(h->E, 1));
  for (int32_t e = 0; e < h->E; ++e) ++succ_ptr[h->pred_op[e] + 1];
  for (int32_t g = 0; g < N; ++g) succ_ptr[g + 1] += succ_ptr[g];
  {
    std::vector<int32_t> fill(succ_ptr.begin(), succ_ptr.end() - 1);
    for (int32_t g = 0; g < N; ++g)
      for (int32_t e = h->pred_ptr[g]; e < h->pred_ptr[g + 1]; ++e) {
        const int32_t k = fill[h->pred_op[e]]++;
        succ_op[k] = g;
        succ_edge[k] = e;
      }
    std::vector<int32_t> left(N), stack;
    for (int32_t g = 0; g < N; ++g) {
      left[g] = h->pred_ptr[g + 1] - h->pred_ptr[g];
      if (left[g] == 0) stack.push_back(g);
    }
    int32_t seen = 0;
    while (!stack.empty()) {
      const int32_t g = stack.back();
      stack.pop_back();
      ++seen;
      for (int32_t k = succ_ptr[g]; k < succ_ptr[g + 1]; ++k)
        if (--left[succ_op[k]] == 0) stack.push_back(succ_op[k]);
    }
    if (seen != N) return DIP_E_TOPO;
  }
  // internal numbering: forward groups (and empty ones), then backward groups
  std::vector<int32_t> caller, internal(n_groups);
  for (int pass = 0; pass < 2; ++pass)
    for (int32_t q = 0; q < n_groups; ++q)
      if ((gk[q] == 1) == (pass == 1)) {
        internal[q] = int32_t(caller.size());
        caller.push_back(q);
      }
  int32_t GF = 0;
  while (GF < n_groups && gk[caller[GF]] != 1) ++GF;
  const int32_t wmax = (std::max(GF, n_groups - GF) + 63) / 64;
  int nw = 1;
  while (nw < wmax) nw *= 2;
  if (nw > 32) return DIP_E_UNSUPPORTED;

  (void)hipDeviceSynchronize();   // no call may still read the old tables
  release_rollouts(h);             // the classes belong to the old grouping
  release_greedy(h);
  h->gr_G = n_groups;
  h->gr_GF = GF;
  h->gr_nw = nw;
  h->gr_ig.assign(N, 0);
  h->gr_op.assign(int64_t(n_groups) * P, -1);
  for (int32_t g = 0; g < N; ++g) {
    h->gr_ig[g] = internal[op_group[g]];
    h->gr_op[int64_t(h->gr_ig[g]) * P + h->rank_of[g]] = g;
  }
  h->gr_join.assign(N, -1);
  h->gr_J = 0;
  for (int32_t g = 0; g < N; ++g)
    if (h->pred_ptr[g + 1] - h->pred_ptr[g] >= 2) h->gr_join[g] = h->gr_J++;
  h->gr_succ_ptr = succ_ptr;
  h->gr_succ_op = succ_op;
  h->gr_succ_edge = succ_edge;
  h->gr_n_extra = 0;
  for (int32_t g = 0; g < N; ++g) h->gr_n_extra += std::max(succ_ptr[g + 1] - succ_ptr[g] - 1, 0);
  std::vector<int32_t> src(P + 1, 0), src_list;
  h->gr_max_nr = 0;
  for (int32_t r = 0; r < P; ++r) {
    h->gr_max_nr = std::max(h->gr_max_nr, h->n_ops[r]);
    for (int32_t g = h->rank_off[r]; g < h->rank_off[r + 1]; ++g)
      if (h->pred_ptr[g + 1] == h->pred_ptr[g]) src_list.push_back(h->gr_ig[g]);
    src[r + 1] = int32_t(src_list.size());
  }
  src.insert(src.end(), src_list.begin(), src_list.end());
  h->gr_meta_bytes = int32_t(align16(2 * int64_t(n_groups)));
  // inboxes of 8 stages per kind to start with; the second launch sizes them
  // to a whole rank
  const int pwl = std::max(2, h->pwl);
  h->gr_K = 8;
  h->gr_K_fixed = false;
  if (!greedy_layout(h, h->gr_K, pwl, &h->gr_main)) return DIP_E_UNSUPPORTED;
  // a stage joins its rank's inbox of its kind once, so a ring of a power
  // of two entries no fewer than the rank's stages of that kind never fills
  int32_t most = 1;
  {
    std::vector<int32_t> per(2 * int64_t(P), 0);
    for (int32_t g = 0; g < N; ++g) most = std::max(most, ++per[2 * h->rank_of[g] + h->kind[g]]);
  }
  int kr = 1;
  while (kr < most) kr *= 2;
  if (kr > 0x8000) return DIP_E_UNSUPPORTED;      // 16-bit ring heads and counts
  int pr = pwl;
  while (pr <= 6 && !greedy_layout(h, kr, pr, &h->gr_retry)) ++pr;
  int64_t ring_bytes = 0;
  if (pr > 6) {
    // rings in device memory, one region per resident candidate slot; at
    // most 1 GiB of them (fewer resident blocks if need be)
    if (!greedy_layout(h, kr, pwl, &h->gr_retry, true)) return DIP_E_UNSUPPORTED;
    const int64_t per_block = int64_t(h->gr_retry.wpb) * (kWave >> pwl) * P * (2 * int64_t(kr) + 1) * 8;
    const int64_t want = int64_t(h->n_cu) * h->gr_retry.blocks_per_cu;
    h->gr_retry.max_blocks = int(std::max<int64_t>(1, std::min<int64_t>(want, (int64_t(1) << 30) / per_block)));
    ring_bytes = int64_t(h->gr_retry.max_blocks) * per_block;
  }

  auto fail = [&](hipError_t e) {
    g_last_hip = e;
    release_greedy(h);
    return int(DIP_E_HIP);
  };
  hipError_t e;
  const int64_t rec_bytes = int64_t(n_groups) * P * 32;
  const int64_t ext_bytes = int64_t(std::max(h->gr_n_extra, 1)) * 16;
  if ((e = hipMalloc(&h->d_gr_caller, size_t(n_groups) * 4)) != hipSuccess) return fail(e);
  if ((e = hipMalloc(&h->d_gr_src, src.size() * 4)) != hipSuccess) return fail(e);
  if ((e = hipMalloc(&h->d_gr_rec, size_t(rec_bytes))) != hipSuccess) return fail(e);
  if ((e = hipMalloc(&h->d_gr_succ, size_t(ext_bytes))) != hipSuccess) return fail(e);
  if ((e = hipHostMalloc(reinterpret_cast<void **>(&h->h_gr_stage), size_t(rec_bytes + ext_bytes),
                         hipHostMallocDefault)) != hipSuccess)
    return fail(e);
  if ((e = hipMemcpy(h->d_gr_caller, caller.data(), size_t(n_groups) * 4, hipMemcpyHostToDevice)) !=
      hipSuccess)
    return fail(e);
  if ((e = hipMemcpy(h->d_gr_src, src.data(), src.size() * 4, hipMemcpyHostToDevice)) != hipSuccess)
    return fail(e);
  if (ring_bytes > 0) {
    if ((e = hipMalloc(&h->d_gr_ring, size_t(ring_bytes))) != hipSuccess) return fail(e);
    h->gr_ring_bytes = ring_bytes;
  }
  h->gr_ok = true;
  h->gr_costs_ok = false;
  return DIP_OK;
}

int dip_sim_greedy(dip_sim *h, const dip_costs *costs, const int32_t *prio, int64_t n_cand,
                   int16_t *out_orders, int32_t *out_makespan, int32_t *out_bubble,
                   int32_t *out_peakmem, uint8_t *out_flags, void *stream_) {
  if (!h || n_cand < 0) return DIP_E_INVAL;
  if (!h->gr_ok) return DIP_E_STATE;
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  if (costs) {
    int rc = upload_costs(h, costs, stream);
    if (rc != DIP_OK) return rc;
  }
  if (!h->gr_costs_ok) return DIP_E_STATE;
  if (n_cand == 0) return DIP_OK;
  if (n_cand > INT32_MAX) return DIP_E_INVAL;
  if (!prio || !out_makespan || !out_bubble || !out_peakmem || !out_flags) return DIP_E_INVAL;
  if ((reinterpret_cast<uintptr_t>(prio) | reinterpret_cast<uintptr_t>(out_makespan) |
       reinterpret_cast<uintptr_t>(out_bubble) | reinterpret_cast<uintptr_t>(out_peakmem)) & 3)
    return DIP_E_INVAL;
  if (reinterpret_cast<uintptr_t>(out_orders) & 1) return DIP_E_INVAL;
  if (h->gr_retry_cap < n_cand) {
    if (h->d_gr_retry) (void)hipFree(h->d_gr_retry);
    h->d_gr_retry = nullptr;
    h->gr_retry_cap = 0;
    DIP_HIP(hipMalloc(&h->d_gr_retry, size_t(n_cand) * 8));
    h->gr_retry_cap = n_cand;
  }
  if (!h->d_gr_retry_count) DIP_HIP(hipMalloc(&h->d_gr_retry_count, 16));
  if (h->gr_seen_pending && hipEventQuery(h->gr_seen_ev) == hipSuccess) {
    h->gr_seen_pending = false;
    dip_sim::GrLaunch bigger;
    if (!h->gr_K_fixed && h->gr_K < 256 && int64_t(*h->h_gr_seen) * 64 > h->gr_seen_n &&
        greedy_layout(h, 2 * h->gr_K, h->gr_main.pwl, &bigger)) {
      h->gr_K *= 2;
      h->gr_main = bigger;
    }
  }
  (void)hipGetLastError();
  h->prof_n = 0;
  auto mark = [&](int i) -> hipError_t {
    if (!h->profile) return hipSuccess;
    h->prof_n = i + 1;
    return hipEventRecord(h->prof_ev[i], stream);
  };
  (void)hipGetLastError();
  DIP_HIP(hipMemsetAsync(h->d_gr_retry_count, 0, 4, stream));
  GreedyArgs a{};
  a.prio = prio;
  a.n_cand = n_cand;
  a.out_orders = out_orders;
  a.stride = h->stride;
  a.out_ms = out_makespan;
  a.out_bub = out_bubble;
  a.out_peak = out_peakmem;
  a.out_flags = out_flags;
  a.rec = h->d_gr_rec;
  a.succ = h->d_gr_succ;
  a.caller = h->d_gr_caller;
  a.src = h->d_gr_src;
  a.rank_off = h->d_rank_off;
  a.busy = h->d_busy;
  a.cap = h->d_cap;
  a.P = h->P;
  a.G = h->gr_G;
  a.GF = h->gr_GF;
  a.J = h->gr_J;
  a.n_rounds = h->N;
  a.has_cap = 0;
  for (int r = 0; r < h->P; ++r) a.has_cap |= h->cap[r] >= 0 ? 1 : 0;
  a.meta_bytes = h->gr_meta_bytes;
  auto set_layout = [&](const dip_sim::GrLaunch &L) {
    a.K = L.K;
    a.wpb = L.wpb;
    a.cand_bytes = L.cand_bytes;
    a.off_pend = L.off_pend;
    a.off_npend = L.off_npend;
    a.off_join = L.off_join;
    a.off_gpos = L.off_gpos;
    a.off_ord = L.off_ord;
    a.off_grk = L.off_grk;
  };
  set_layout(h->gr_main);
  a.retry = h->d_gr_retry;
  a.retry_count = h->d_gr_retry_count;
  const int64_t per_block = int64_t(h->gr_main.wpb) * (kWave >> h->gr_main.pwl);
  const int64_t blocks = (n_cand + per_block - 1) / per_block;
  if (blocks > INT32_MAX) return DIP_E_INVAL;
  DIP_HIP(mark(0));
  DIP_HIP(launch_greedy(h->gr_main.pwl, h->gr_nw, false, int(blocks), h->gr_main.wpb,
                        size_t(h->gr_main.lds), stream, a));
  DIP_HIP(mark(1));
  // candidates whose inboxes overflowed, with inboxes as large as a rank
  set_layout(h->gr_retry);
  a.list = h->d_gr_retry;
  a.list_count = h->d_gr_retry_count;
  a.retry = nullptr;
  a.retry_count = nullptr;
  int64_t rb = std::min<int64_t>(int64_t(h->n_cu) * h->gr_retry.blocks_per_cu, blocks);
  if (h->gr_retry.gring) {
    rb = std::min<int64_t>(rb, h->gr_retry.max_blocks);   // one ring region per resident slot
    a.gring = h->d_gr_ring;
  }
  DIP_HIP(launch_greedy(h->gr_retry.pwl, h->gr_nw, h->gr_retry.gring, int(rb), h->gr_retry.wpb,
                        size_t(h->gr_retry.lds), stream, a));
  DIP_HIP(mark(2));
  if (!h->gr_K_fixed && h->gr_K < 256 && !h->gr_seen_pending) {
    if (!h->h_gr_seen) {
      DIP_HIP(hipHostMalloc(reinterpret_cast<void **>(&h->h_gr_seen), 16, hipHostMallocDefault));
      DIP_HIP(hipEventCreateWithFlags(&h->gr_seen_ev, hipEventDisableTiming));
    }
    DIP_HIP(hipMemcpyAsync(h->h_gr_seen, h->d_gr_retry_count, 4, hipMemcpyDeviceToHost, stream));
    DIP_HIP(hipEventRecord(h->gr_seen_ev, stream));
    h->gr_seen_pending = true;
    h->gr_seen_n = n_cand;
  }
  return DIP_OK;
}

int dip_sim_set_greedy_inbox(dip_sim *h, int32_t k) {
  if (!h || k < 0 || k > 256 || (k & (k - 1)) != 0) return DIP_E_INVAL;
  if (!h->gr_ok) return DIP_E_STATE;
  const int kk = k ? k : 8;
  dip_sim::GrLaunch L;
  if (!greedy_layout(h, kk, h->gr_main.pwl, &L)) return DIP_E_UNSUPPORTED;
  h->gr_K = kk;
  h->gr_main = L;
  h->gr_K_fixed = k != 0;
  return DIP_OK;
}

int dip_sim_configure_rollouts(dip_sim *h, int32_t n_classes, const int32_t *group_class) {
  if (!h || !group_class || n_classes < 1) return DIP_E_INVAL;
  if (!h->gr_ok) return DIP_E_STATE;
  if (n_classes > 8192) return DIP_E_UNSUPPORTED;   // a rollout's tables in 64 KiB of LDS
  const int32_t G = h->gr_G;
  std::vector<int32_t> cls(group_class, group_class + G);
  std::vector<char> used(n_classes, 0);
  for (int32_t g = 0; g < G; ++g) {
    if (cls[g] < 0 || cls[g] >= n_classes) return DIP_E_TOPO;
    used[cls[g]] = 1;
  }
  (void)hipDeviceSynchronize();
  release_rollouts(h);
  auto fail = [&](hipError_t e) {
    g_last_hip = e;
    release_rollouts(h);
    return int(DIP_E_HIP);
  };
  hipError_t e;
  if ((e = hipMalloc(&h->d_rl_class, size_t(G) * 4)) != hipSuccess) return fail(e);
  if ((e = hipMalloc(&h->d_rl_seq, size_t(n_classes + 1) * 4)) != hipSuccess) return fail(e);
  if ((e = hipHostMalloc(reinterpret_cast<void **>(&h->h_rl_seq), size_t(n_classes + 1) * 4,
                         hipHostMallocDefault)) != hipSuccess)
    return fail(e);
  h->rl_leaf_cap = 1;
  if ((e = hipEventCreateWithFlags(&h->rl_seq_ev, hipEventDisableTiming)) != hipSuccess) return fail(e);
  if ((e = hipMemcpy(h->d_rl_class, cls.data(), size_t(G) * 4, hipMemcpyHostToDevice)) != hipSuccess)
    return fail(e);
  h->rl_class = cls;
  h->rl_n = n_classes;
  h->rl_ok = true;
  return DIP_OK;
}

int dip_sim_rollouts_batch(dip_sim *h, int32_t n_leaves, const int32_t *depths,
                           const int32_t *prefixes, int64_t per_leaf, uint64_t seed,
                           uint64_t draw_base, int32_t *out_prio, int32_t *out_makespan,
                           uint8_t *out_flags, uint64_t *inout_keys, void *stream_) {
  if (!h || n_leaves < 1 || n_leaves > 65535 || per_leaf < 0 || !depths) return DIP_E_INVAL;
  if (!h->rl_ok || !h->gr_ok) return DIP_E_STATE;
  if (!h->gr_costs_ok) return DIP_E_STATE;
  const int32_t n = h->rl_n;
  // every prefix: distinct classes in range
  int64_t total = 0;
  for (int32_t l = 0; l < n_leaves; ++l) {
    if (depths[l] < 0 || depths[l] > n) return DIP_E_INVAL;
    total += depths[l];
  }
  if (total > 0 && !prefixes) return DIP_E_INVAL;
  {
    std::vector<int32_t> seen(n, -1);
    int64_t k = 0;
    for (int32_t l = 0; l < n_leaves; ++l)
      for (int32_t d = 0; d < depths[l]; ++d, ++k) {
        const int32_t c = prefixes[k];
        if (c < 0 || c >= n || seen[c] == l) return DIP_E_INVAL;
        seen[c] = l;
      }
  }
  if (per_leaf == 0) return DIP_OK;
  if (per_leaf > INT32_MAX / n_leaves || !out_prio || !out_makespan || !out_flags || !inout_keys)
    return DIP_E_INVAL;
  if (reinterpret_cast<uintptr_t>(inout_keys) & 7) return DIP_E_INVAL;
  const int64_t rows = per_leaf * n_leaves;
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  if (h->rl_cap < rows) {
    if (h->d_rl_bub) (void)hipFree(h->d_rl_bub);
    if (h->d_rl_peak) (void)hipFree(h->d_rl_peak);
    h->d_rl_bub = h->d_rl_peak = nullptr;
    h->rl_cap = 0;
    DIP_HIP(hipMalloc(&h->d_rl_bub, size_t(rows) * h->P * 4));
    DIP_HIP(hipMalloc(&h->d_rl_peak, size_t(rows) * h->P * 4));
    h->rl_cap = rows;
  }
  // per leaf its prefix, then the other classes ascending; then the depths;
  // through pinned staging
  if (h->rl_seq_pending) {
    DIP_HIP(hipEventSynchronize(h->rl_seq_ev));
    h->rl_seq_pending = false;
  }
  const size_t words = size_t(n_leaves) * size_t(n + 1);
  if (h->rl_leaf_cap < n_leaves) {
    DIP_HIP(hipDeviceSynchronize());              // no launch may still read the old buffer
    if (h->d_rl_seq) (void)hipFree(h->d_rl_seq);
    if (h->h_rl_seq) (void)hipHostFree(h->h_rl_seq);
    h->d_rl_seq = h->h_rl_seq = nullptr;
    h->rl_leaf_cap = 0;
    DIP_HIP(hipMalloc(&h->d_rl_seq, words * 4));
    DIP_HIP(hipHostMalloc(reinterpret_cast<void **>(&h->h_rl_seq), words * 4, hipHostMallocDefault));
    h->rl_leaf_cap = n_leaves;
  }
  {
    std::vector<char> on(n);
    int64_t k = 0;
    for (int32_t l = 0; l < n_leaves; ++l) {
      int32_t *row = h->h_rl_seq + int64_t(l) * n;
      std::fill(on.begin(), on.end(), 0);
      int32_t w = 0;
      for (int32_t d = 0; d < depths[l]; ++d, ++k) {
        row[w++] = prefixes[k];
        on[prefixes[k]] = 1;
      }
      for (int32_t c = 0; c < n; ++c)
        if (!on[c]) row[w++] = c;
      h->h_rl_seq[int64_t(n_leaves) * n + l] = depths[l];
    }
  }
  DIP_HIP(hipMemcpyAsync(h->d_rl_seq, h->h_rl_seq, words * 4, hipMemcpyHostToDevice, stream));
  DIP_HIP(hipEventRecord(h->rl_seq_ev, stream));
  h->rl_seq_pending = true;
  RolloutArgs a{};
  a.n = rows;
  a.per_leaf = per_leaf;
  a.out_prio = out_prio;
  a.seqs = h->d_rl_seq;
  a.depths = h->d_rl_seq + int64_t(n_leaves) * n;
  a.group_class = h->d_rl_class;
  a.seed = seed;
  a.draw = draw_base;
  a.n_classes = n;
  a.G = h->gr_G;
  DIP_HIP(launch_rollout_prio(stream, a));
  int rc;
  if (!h->mo_ok) {
    rc = dip_sim_greedy(h, nullptr, out_prio, rows, nullptr, out_makespan, h->d_rl_bub,
                        h->d_rl_peak, out_flags, stream_);
    if (rc != DIP_OK) return rc;
  } else {
    // Sec. 5.1's score: the interleaved schedule after the per-layer memory
    // optimisation, re-timed with its selection (a rank whose cap cannot be
    // met keeps a selection over the cap, which the re-timed run flags)
    if (h->rl_mo_cap < rows) {
      DIP_HIP(hipDeviceSynchronize());
      release_rollout_memopt(h);
      DIP_HIP(hipMalloc(&h->d_rl_orders, size_t(rows) * size_t(h->stride) * 2));
      DIP_HIP(hipMalloc(&h->d_rl_mo_time, size_t(rows) * h->P * 8));
      DIP_HIP(hipMalloc(&h->d_rl_mo_peak, size_t(rows) * h->P * 4));
      DIP_HIP(hipMalloc(&h->d_rl_mo_status, size_t(rows) * h->P));
      DIP_HIP(hipMalloc(&h->d_rl_choice, size_t(rows) * std::max(h->mo_n_pairs, 1)));
      h->rl_mo_cap = rows;
    }
    rc = dip_sim_greedy(h, nullptr, out_prio, rows, h->d_rl_orders, out_makespan, h->d_rl_bub,
                        h->d_rl_peak, out_flags, stream_);
    if (rc != DIP_OK) return rc;
    rc = dip_sim_memopt(h, h->d_rl_orders, rows, h->d_rl_mo_time, h->d_rl_mo_peak,
                        h->d_rl_mo_status, h->d_rl_choice, stream_);
    if (rc != DIP_OK) return rc;
    rc = dip_sim_evaluate_selected(h, h->d_rl_orders, h->d_rl_choice, rows, out_makespan,
                                   h->d_rl_bub, h->d_rl_peak, out_flags, stream_);
    if (rc != DIP_OK) return rc;
  }
  // the best unflagged rollout of each leaf, indexed within the leaf
  const int64_t want = (per_leaf + 255) / 256;
  const int blocks = int(std::max<int64_t>(1, std::min<int64_t>(want, int64_t(h->n_cu) * 8 / n_leaves)));
  DIP_HIP(launch_argmin(blocks, stream, out_makespan, out_flags, rows, per_leaf, n_leaves, 0,
                        reinterpret_cast<unsigned long long *>(inout_keys)));
  return DIP_OK;
}

int dip_sim_rollouts(dip_sim *h, const int32_t *prefix, int32_t depth, int64_t n_rollouts,
                     uint64_t seed, uint64_t draw, int32_t *out_prio, int32_t *out_makespan,
                     uint8_t *out_flags, uint64_t *inout_best_key, void *stream_) {
  if (!h || n_rollouts < 0 || depth < 0) return DIP_E_INVAL;
  return dip_sim_rollouts_batch(h, 1, &depth, prefix, n_rollouts, seed, draw, out_prio,
                                out_makespan, out_flags, inout_best_key, stream_);
}

int dip_sim_configure_memopt(dip_sim *h, const int32_t *slot_layers, const int64_t *layer_time,
                             const int64_t *layer_mem, int32_t n_strategies, int32_t n_candidates,
                             int32_t bb_nodes) {
  if (!h || !slot_layers || n_strategies < 1 || n_candidates < 2 ||
      n_candidates > kMemoptMaxCands || bb_nodes < 0)
    return DIP_E_INVAL;
  const int32_t P = h->P, N = h->N, ns = h->n_slots;
  // every slot: one forward and one backward on one rank
  std::vector<int32_t> f_of(ns, -1), b_of(ns, -1);
  for (int32_t g = 0; g < N; ++g) {
    int32_t &x = h->kind[g] ? b_of[h->op_slot[g]] : f_of[h->op_slot[g]];
    if (x >= 0) return DIP_E_TOPO;
    x = g;
  }
  for (int32_t q = 0; q < ns; ++q)
    if (f_of[q] < 0 || b_of[q] < 0 || h->rank_of[f_of[q]] != h->rank_of[b_of[q]]) return DIP_E_TOPO;
  if (slot_layers[0] != 0) return DIP_E_INVAL;
  for (int32_t q = 0; q < ns; ++q)
    if (slot_layers[q + 1] < slot_layers[q]) return DIP_E_INVAL;
  if (slot_layers[ns] > 0 && (!layer_time || !layer_mem)) return DIP_E_INVAL;
  // candidates per slot: exact Pareto front of the layers' choices, then the
  // fastest, the leanest and one knapsack answer per bucket edge
  struct Pt {
    int64_t t, m;
  };
  std::vector<std::vector<Pt>> cand(ns);
  for (int32_t q = 0; q < ns; ++q) {
    std::vector<Pt> front{{0, 0}}, pts;
    for (int32_t l = slot_layers[q]; l < slot_layers[q + 1]; ++l) {
      pts.clear();
      for (const Pt &p : front)
        for (int32_t k = 0; k < n_strategies; ++k) {
          const int64_t t = layer_time[int64_t(l) * n_strategies + k];
          const int64_t m = layer_mem[int64_t(l) * n_strategies + k];
          if (t < 0 || m < 0) return DIP_E_RANGE;
          pts.push_back({p.t + t, p.m + m});
        }
      std::sort(pts.begin(), pts.end(),
                [](const Pt &x, const Pt &y) { return x.m != y.m ? x.m < y.m : x.t < y.t; });
      front.clear();
      for (const Pt &p : pts)
        if (front.empty() || (p.t < front.back().t && p.m != front.back().m)) front.push_back(p);
      if (front.size() > (size_t(1) << 20)) return DIP_E_UNSUPPORTED;
    }
    std::vector<Pt> pick{front.back(), front.front()};
    const int64_t lo = front.front().m, hi = front.back().m;
    for (int32_t k = 1; k + 1 < n_candidates; ++k) {
      const int64_t edge = lo + ((hi - lo) * k) / (n_candidates - 2);
      size_t j = 0;
      while (j + 1 < front.size() && front[j + 1].m <= edge) ++j;
      pick.push_back(front[j]);
    }
    std::sort(pick.begin(), pick.end(),
              [](const Pt &x, const Pt &y) { return x.t != y.t ? x.t < y.t : x.m < y.m; });
    std::vector<Pt> uniq;
    for (const Pt &p : pick)
      if (uniq.empty() || uniq.back().t != p.t || uniq.back().m != p.m) uniq.push_back(p);
    for (const Pt &p : uniq)
      if (p.m > INT32_MAX || p.t > (int64_t(1) << 40)) return DIP_E_RANGE;
    cand[q] = uniq;
  }
  // pairs per rank in slot order; each op's pair index and kind
  std::vector<int32_t> pair_off(P + 1, 0), lid_pair(N, 0), slot_pair(ns, 0), pair_b;
  std::vector<int64_t> pair_extra;
  std::vector<int32_t> mem, mdm;
  std::vector<int64_t> tim;
  std::vector<uint32_t> mkey;
  int32_t max_pairs = 0;
  struct Move {
    int64_t dt, dm;
    int32_t at;                  // index into the rank's [pair][candidate] slice
  };
  std::vector<Move> moves;
  for (int32_t r = 0; r < P; ++r) {
    int32_t i = 0;
    const size_t first = tim.size();
    moves.clear();
    int64_t fastest_mem = 0;
    for (int32_t q = 0; q < ns; ++q) {
      if (h->rank_of[f_of[q]] != r) continue;
      slot_pair[q] = i;
      const int32_t nc = int32_t(cand[q].size());
      fastest_mem += cand[q][0].m;
      pair_b.push_back(b_of[q]);
      pair_extra.push_back(cand[q][nc - 1].t - cand[q][0].t);
      for (int32_t j = 0; j < kMemoptMaxCands; ++j) {
        const bool in = j < nc;
        tim.push_back(in ? cand[q][j].t : 0);
        mem.push_back(in ? int32_t(cand[q][j].m) : 0);
        mkey.push_back(kMemoptNoMove);
        mdm.push_back(0);
        if (j + 1 < nc)
          moves.push_back({cand[q][j + 1].t - cand[q][j].t, cand[q][j].m - cand[q][j + 1].m,
                           i * kMemoptMaxCands + j});
      }
      ++i;
    }
    if (i >= (1 << kMemoptPairBits)) return DIP_E_UNSUPPORTED;
    if (fastest_mem > INT32_MAX) return DIP_E_RANGE;
    // exact ratio order of the rank's moves: dt_a / dm_a < dt_b / dm_b (dm > 0)
    auto less = [](const Move &x, const Move &y) {
      return __int128(x.dt) * y.dm < __int128(y.dt) * x.dm;
    };
    std::stable_sort(moves.begin(), moves.end(), less);
    uint32_t dense = 0;
    for (size_t k = 0; k < moves.size(); ++k) {
      if (k > 0 && less(moves[k - 1], moves[k])) ++dense;
      const int32_t pair = moves[k].at / kMemoptMaxCands;
      mkey[first + size_t(moves[k].at)] = (dense << kMemoptPairBits) | uint32_t(pair);
      mdm[first + size_t(moves[k].at)] = int32_t(moves[k].dm);
    }
    pair_off[r + 1] = pair_off[r] + i;
    max_pairs = std::max(max_pairs, i);
  }
  for (int32_t g = 0; g < N; ++g)
    lid_pair[g] = int32_t(uint32_t(slot_pair[h->op_slot[g]]) | (uint32_t(h->kind[g]) << 31));
  (void)hipDeviceSynchronize();
  release_memopt(h);
  auto fail = [&](hipError_t e) {
    g_last_hip = e;
    release_memopt(h);
    return int(DIP_E_HIP);
  };
  hipError_t e;
  const size_t cells = std::max<size_t>(tim.size(), 1);       // pairs x candidates
  if ((e = hipMalloc(&h->d_mo_pair_off, size_t(P + 1) * 4)) != hipSuccess) return fail(e);
  if ((e = hipMalloc(&h->d_mo_lid_pair, size_t(std::max(N, 1)) * 4)) != hipSuccess) return fail(e);
  if ((e = hipMalloc(&h->d_mo_time, cells * 8)) != hipSuccess) return fail(e);
  if ((e = hipMalloc(&h->d_mo_mem, cells * 4)) != hipSuccess) return fail(e);
  if ((e = hipMalloc(&h->d_mo_key, cells * 4)) != hipSuccess) return fail(e);
  if ((e = hipMalloc(&h->d_mo_dm, cells * 4)) != hipSuccess) return fail(e);
  if ((e = hipMemcpy(h->d_mo_pair_off, pair_off.data(), size_t(P + 1) * 4, hipMemcpyHostToDevice)) ||
      (N > 0 && (e = hipMemcpy(h->d_mo_lid_pair, lid_pair.data(), size_t(N) * 4, hipMemcpyHostToDevice))) ||
      (!tim.empty() &&
       ((e = hipMemcpy(h->d_mo_time, tim.data(), tim.size() * 8, hipMemcpyHostToDevice)) ||
        (e = hipMemcpy(h->d_mo_mem, mem.data(), mem.size() * 4, hipMemcpyHostToDevice)) ||
        (e = hipMemcpy(h->d_mo_key, mkey.data(), mkey.size() * 4, hipMemcpyHostToDevice)) ||
        (e = hipMemcpy(h->d_mo_dm, mdm.data(), mdm.size() * 4, hipMemcpyHostToDevice)))))
    return fail(e);
  h->mo_max_pairs = max_pairs;
  h->mo_n_pairs = pair_off[P];
  h->mo_bb_nodes = bb_nodes > 0 ? bb_nodes : 512;
  h->mo_pair_b = pair_b;
  h->mo_pair_extra = pair_extra;
  h->mo_max_extra = 0;
  for (int64_t x : pair_extra) h->mo_max_extra = std::max(h->mo_max_extra, x);
  h->mo_ok = true;
  return DIP_OK;
}

int dip_sim_memopt(dip_sim *h, const int16_t *orders, int64_t n_cand, int64_t *out_time,
                   int32_t *out_peak, uint8_t *out_status, uint8_t *out_choice, void *stream) {
  if (!h || n_cand < 0) return DIP_E_INVAL;
  if (!h->mo_ok) return DIP_E_STATE;
  if (n_cand == 0) return DIP_OK;
  if (!orders || !out_time || !out_peak || !out_status) return DIP_E_INVAL;
  if ((reinterpret_cast<uintptr_t>(out_time) & 7) || (reinterpret_cast<uintptr_t>(out_peak) & 3) ||
      (reinterpret_cast<uintptr_t>(orders) & 1))
    return DIP_E_INVAL;
  MemoptArgs a{};
  a.orders = orders;
  a.n_cand = n_cand;
  a.stride = h->stride;
  a.out_time = out_time;
  a.out_peak = out_peak;
  a.out_status = out_status;
  a.out_choice = out_choice;
  a.n_pairs = h->mo_n_pairs;
  a.bb_nodes = h->mo_bb_nodes;
  a.rank_off = h->d_rank_off;
  a.pair_off = h->d_mo_pair_off;
  a.lid_pair = h->d_mo_lid_pair;
  a.cand_time = h->d_mo_time;
  a.cand_mem = h->d_mo_mem;
  a.move_key = h->d_mo_key;
  a.move_dm = h->d_mo_dm;
  a.cap = h->d_cap;
  a.P = h->P;
  a.max_pairs = std::max(h->mo_max_pairs, 1);
  (void)hipGetLastError();
  if (a.max_pairs <= 512) {
    // a wave per (schedule, rank), pairs in registers
    constexpr int kWaves = 4;
    int ppl = 1;
    while (64 * ppl < a.max_pairs) ppl *= 2;
    if ((n_cand + kWaves - 1) / kWaves > INT32_MAX || h->P > 65535) return DIP_E_INVAL;
    if (memopt_wave_lds(a.max_pairs, kWaves) > 65536) return DIP_E_UNSUPPORTED;
    DIP_HIP(launch_memopt_wave(ppl, kWaves, static_cast<hipStream_t>(stream), a));
    return DIP_OK;
  }
  a.bytes_per_thread = int32_t(int64_t(a.max_pairs) * 9);
  int tpb = 64;
  while (tpb > 1 && int64_t(tpb) * a.bytes_per_thread > 65536) tpb /= 2;
  if (int64_t(tpb) * a.bytes_per_thread > 65536) return DIP_E_UNSUPPORTED;
  if (n_cand * h->P / tpb + 1 > INT32_MAX) return DIP_E_INVAL;
  DIP_HIP(launch_memopt(tpb, static_cast<hipStream_t>(stream), a));
  return DIP_OK;
}

int dip_sim_evaluate_selected(dip_sim *h, const int16_t *orders, const uint8_t *choice,
                              int64_t n_cand, int32_t *out_makespan, int32_t *out_bubble,
                              int32_t *out_peakmem, uint8_t *out_flags, void *stream) {
  if (!h || n_cand < 0) return DIP_E_INVAL;
  if (!h->mo_ok || !h->costs_set) return DIP_E_STATE;
  if (n_cand == 0) return DIP_OK;
  if (!orders || !choice || !out_makespan || !out_bubble || !out_peakmem || !out_flags)
    return DIP_E_INVAL;
  if ((reinterpret_cast<uintptr_t>(orders) & 15) ||
      ((reinterpret_cast<uintptr_t>(out_makespan) | reinterpret_cast<uintptr_t>(out_bubble) |
        reinterpret_cast<uintptr_t>(out_peakmem)) & 3))
    return DIP_E_INVAL;
  // a re-timed backward stays within int32
  for (size_t p = 0; p < h->mo_pair_b.size(); ++p)
    if (int64_t(h->last_cost[size_t(h->mo_pair_b[p])]) + h->mo_pair_extra[p] > INT32_MAX)
      return DIP_E_RANGE;
  GeneralArgs a{};
  a.orders = orders;
  a.n_cand = n_cand;
  a.stride = h->stride;
  a.n_groups = (n_cand + h->G - 1) / h->G;
  a.out_ms = out_makespan;
  a.out_bub = out_bubble;
  a.out_peak = out_peakmem;
  a.out_flags = out_flags;
  a.rec = h->d_rec;
  a.edge = h->d_edge;
  a.rank_off = h->d_rank_off;
  a.busy = h->d_busy;
  a.cap = h->d_cap;
  a.gends = static_cast<int32_t *>(h->d_scratch_gen);
  a.P = h->P;
  a.pwl = h->pwl;
  a.G = h->G;
  a.N = h->N;
  a.E = h->E;
  a.wpb = h->gen_wpb;
  a.choice = choice;
  a.n_pairs = h->mo_n_pairs;
  a.lid_pair = h->d_mo_lid_pair;
  a.pair_off = h->d_mo_pair_off;
  a.cand_time = h->d_mo_time;
  a.cand_mem = h->d_mo_mem;
  a.cand_key = h->d_mo_key;
  const GenBytes b = general_bytes(h, h->gen_variant);
  a.tab_bytes = uint32_t(b.tab);
  a.ord_bytes = uint32_t(b.ord);
  a.end_bytes = uint32_t(b.end);
  const int64_t want = (a.n_groups + h->gen_wpb - 1) / h->gen_wpb;
  const int blocks = int(std::min<int64_t>(want, h->gen_max_blocks));
  (void)hipGetLastError();
  DIP_HIP(launch_general(h->gen_variant, blocks, h->gen_wpb, size_t(h->gen_lds),
                         static_cast<hipStream_t>(stream), a));
  return DIP_OK;
}

int dip_sim_argmin(dip_sim *h, const int32_t *makespan, const uint8_t *flags, int64_t n_cand,
                   int64_t index_base, uint64_t *inout_best_key, void *stream_) {
  if (!h || n_cand < 0 || index_base < 0) return DIP_E_INVAL;
  if (index_base + n_cand > int64_t(UINT32_MAX)) return DIP_E_RANGE;
  if (n_cand == 0) return DIP_OK;
  if (!makespan || !flags || !inout_best_key) return DIP_E_INVAL;
  if ((reinterpret_cast<uintptr_t>(inout_best_key) & 7) || (reinterpret_cast<uintptr_t>(makespan) & 3))
    return DIP_E_INVAL;
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  const int64_t want = (n_cand + 255) / 256;
  const int blocks = int(std::min<int64_t>(want, int64_t(h->n_cu) * 8));
  DIP_HIP(launch_argmin(blocks, stream, makespan, flags, n_cand, n_cand, 1, uint64_t(index_base),
                        reinterpret_cast<unsigned long long *>(inout_best_key)));
  return DIP_OK;
}

int dip_sim_profile(dip_sim *h, int32_t enable) {
  if (!h) return DIP_E_INVAL;
  if (enable && !h->prof_ev[0])
    for (hipEvent_t &ev : h->prof_ev) DIP_HIP(hipEventCreate(&ev));
  h->profile = enable != 0;
  h->prof_n = 0;
  return DIP_OK;
}

int dip_sim_last_profile(dip_sim *h, float *out_ms, int32_t *n_out) {
  if (!h || !out_ms || !n_out) return DIP_E_INVAL;
  *n_out = 0;
  if (h->prof_n < 2) return DIP_OK;
  DIP_HIP(hipEventSynchronize(h->prof_ev[h->prof_n - 1]));
  for (int i = 0; i + 1 < h->prof_n; ++i)
    DIP_HIP(hipEventElapsedTime(out_ms + i, h->prof_ev[i], h->prof_ev[i + 1]));
  *n_out = h->prof_n - 1;
  return DIP_OK;
}

int dip_sim_last_retries(dip_sim *h, int64_t *out_first, int64_t *out_second) {
  if (!h || !out_first || !out_second) return DIP_E_INVAL;
  *out_first = *out_second = 0;
  if (h->variant < 8 || !h->last_counts) return DIP_OK;
  DIP_HIP(hipStreamSynchronize(h->last_stream));
  uint32_t cnt[4] = {0, 0, 0, 0};
  DIP_HIP(hipMemcpy(cnt, h->last_counts, sizeof(cnt), hipMemcpyDeviceToHost));
  *out_first = cnt[0];
  *out_second = h->last_pass2 ? cnt[2] : cnt[0];
  return DIP_OK;
}

void dip_sim_destroy(dip_sim *h) { release(h); }

const char *dip_sim_strerror(int code) {
  switch (code) {
    case DIP_OK: return "ok";
    case DIP_E_INVAL: return "invalid argument (null pointer, negative count or misaligned buffer)";
    case DIP_E_TOPO: return "malformed topology";
    case DIP_E_RANGE: return "negative cost or totals that could overflow int32";
    case DIP_E_UNSUPPORTED: return "shape not supported by any kernel variant on this device";
    case DIP_E_NOMEM: return "out of memory";
    case DIP_E_HIP: return hipGetErrorString(g_last_hip);
    case DIP_E_STATE: return "no costs supplied yet";
    case DIP_E_CAPACITY: return "batch larger than the static scratch area holds";
    default: return "unknown error";
  }
}

}  // extern "C"
