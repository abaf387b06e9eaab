// host_next.hip -- entry points beyond the simulation: the dual-queue greedy
// interleaving (Sec. 5.2), MCTS rollouts scored on the GPU (Sec. 5.1) and the
// per-layer memory selection with the re-timed evaluate (Sec. 5.3).
#include "host_state.h"

using namespace dipsim;
using namespace dipsim_host;

namespace dipsim_host {

bool greedy_layout(const dip_sim *h, int K, int pwl, dip_sim::GrLaunch *L, bool gring) {
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
  // (wide E sets, 32 words, sit in LDS after the tables: each lane
  // of the candidate two sets of gr_nw words)
  const int64_t ebits = h->gr_nw >= 32 ? lanes * 16 * int64_t(h->gr_nw) : 0;
  L->cand_bytes = int32_t(head + 3 * align16(2 * G) + ebits);
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

}  // namespace dipsim_host

extern "C" {

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
  h->gr_direct = false;
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
    // an earlier call's overflow count: more than 1/64 of its candidates
    // doubles the first launch's inboxes while they fit LDS; more than half of
    // them at the largest inbox that fits makes later calls skip the first
    // launch (it would run them all only for the second to run them again)
    h->gr_seen_pending = false;
    dip_sim::GrLaunch bigger;
    const int64_t seen = int64_t(*h->h_gr_seen);
    if (!h->gr_K_fixed && seen * 64 > h->gr_seen_n) {
      if (h->gr_K < 256 && greedy_layout(h, 2 * h->gr_K, h->gr_main.pwl, &bigger)) {
        h->gr_K *= 2;
        h->gr_main = bigger;
      } else if (seen * 2 > h->gr_seen_n) {
        h->gr_direct = true;
      }
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
  DIP_HIP(launch_zero_words(h->d_gr_retry_count, 1, stream));
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
  if (!h->gr_direct)
    DIP_HIP(launch_greedy(h->gr_main.pwl, h->gr_nw, false, int(blocks), h->gr_main.wpb,
                          size_t(h->gr_main.lds), stream, a));
  DIP_HIP(mark(1));
  // candidates whose inboxes overflowed (or, skipping the first launch, all
  // of them), with inboxes as large as a rank
  set_layout(h->gr_retry);
  a.list = h->gr_direct ? nullptr : h->d_gr_retry;
  a.list_count = h->gr_direct ? nullptr : h->d_gr_retry_count;
  a.retry = nullptr;
  a.retry_count = nullptr;
  const int64_t per_block_r = int64_t(h->gr_retry.wpb) * (kWave >> h->gr_retry.pwl);
  int64_t rb = std::min<int64_t>(int64_t(h->n_cu) * h->gr_retry.blocks_per_cu,
                                 h->gr_direct ? (n_cand + per_block_r - 1) / per_block_r : blocks);
  if (h->gr_retry.gring) {
    rb = std::min<int64_t>(rb, h->gr_retry.max_blocks);   // one ring region per resident slot
    a.gring = h->d_gr_ring;
  }
  DIP_HIP(launch_greedy(h->gr_retry.pwl, h->gr_nw, h->gr_retry.gring, int(rb), h->gr_retry.wpb,
                        size_t(h->gr_retry.lds), stream, a));
  DIP_HIP(mark(2));
  if (!h->gr_K_fixed && !h->gr_direct && !h->gr_seen_pending) {
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
  h->gr_direct = false;
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
    // a wave per (schedule, rank), pairs in registers; four waves per block
    // where their LDS fits, else two, else one
    int waves = 4;
    while (waves > 1 && memopt_wave_lds(a.max_pairs, waves) > 65536) waves /= 2;
    int ppl = 1;
    while (64 * ppl < a.max_pairs) ppl *= 2;
    if ((n_cand + waves - 1) / waves > INT32_MAX || h->P > 65535) return DIP_E_INVAL;
    if (memopt_wave_lds(a.max_pairs, waves) > 65536) return DIP_E_UNSUPPORTED;
    DIP_HIP(launch_memopt_wave(ppl, waves, static_cast<hipStream_t>(stream), a));
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

}  // extern "C"
