// host.hip -- the handle's life cycle (create, configure, destroy), evaluate
// and its allocation-free variant, argmin, profiling and error strings.
#include "host_state.h"

using namespace dipsim;
using namespace dipsim_host;

namespace dipsim_host {

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
  if (h->d_oc_ranks) (void)hipFree(h->d_oc_ranks);
  if (h->d_sim_tab) (void)hipFree(h->d_sim_tab);
  if (h->d_sim_lane) (void)hipFree(h->d_sim_lane);
  if (h->d_rank_off) (void)hipFree(h->d_rank_off);
  if (h->d_busy) (void)hipFree(h->d_busy);
  if (h->d_cap) (void)hipFree(h->d_cap);
  if (h->tc.d_plan) (void)hipFree(h->tc.d_plan);
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

}  // namespace dipsim_host

extern "C" {

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
  // the simulation kernel's tables drop own-rank edges only behind a check
  // that tests their order: rebuild them from the last costs when that changes
  if (h->sim_ok && h->costs_set && h->sim_drop_self != order_checked(h)) {
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
  info->check_kernel = v >= 8 ? check_kind(h) : 0;
  info->greedy_inbox = h->gr_ok ? (h->gr_direct ? -1 : h->gr_K) : 0;
  info->greedy_lds_bytes = h->gr_ok ? int32_t(h->gr_main.lds) : 0;
  info->greedy_retry_ring_bytes = h->gr_ok ? h->gr_ring_bytes : 0;
  return DIP_OK;
}

}  // extern "C"

namespace {

// Device memory an evaluate call works in beyond its inputs and outputs: the
// retry counters and the two retry lists (variants 8 and 9).
struct CallScratch {
  uint32_t *counts;   // [kRetryCounters] zeroed by the check kernel
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
    int rc = check_kind(h) == 2 ? run_tile_check(h, orders, n_cand, out_makespan, out_bubble,
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
    h->last_general = 0;
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
      // The candidates whose pools filled, again with 16 and then 32 slots
      // per pool (deadlocked orders fill small pools too; larger ones tell
      // them from merely crowded ones), each pass in list mode over the
      // previous one's retries, the two lists taking turns; what the last
      // pass leaves goes to the general kernel.  (A pass that does not run
      // still records its event: the profile keeps one entry per pass.)
      auto pass = [&](bool run, int slots, int wpb, int max_blocks, int64_t lds, int next) -> int {
        if (run) {
          int64_t *out = retry_list == sx->list_a ? sx->list_b : sx->list_a;
          a.list = retry_list;
          a.list_count = retry_count;
          a.retry = out;
          a.retry_count = counts + next;
          a.wpb = wpb;
          a.static_end = INT64_MAX;
          DIP_HIP(launch_sim(h->pwl, slots, h->sim_paged, max_blocks, wpb, size_t(lds), stream, a));
          retry_list = out;
          retry_count = counts + next;
          h->last_general = next;
        }
        return DIP_OK;
      };
      if ((rc = pass(h->sim2_ok, 16, h->sim2_wpb, h->sim2_max_blocks, h->sim2_lds, 2)) != DIP_OK)
        return rc;
      DIP_HIP(mark(3));
      if ((rc = pass(h->sim3_ok, 32, h->sim3_wpb, h->sim3_max_blocks, h->sim3_lds, 4)) != DIP_OK)
        return rc;
      DIP_HIP(mark(4));
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
  uint32_t cnt[kRetryCounters] = {};
  DIP_HIP(hipMemcpy(cnt, h->last_counts, sizeof(cnt), hipMemcpyDeviceToHost));
  *out_first = cnt[0];
  *out_second = cnt[h->last_general];
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
