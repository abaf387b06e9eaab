// host_plan.hip -- kernel-variant choice and launch shapes: occupancy of the
// general kernel's variants, device scratch, the tile check's wave plans,
// the simulation kernel's shapes for both pool sizes, and the check and
// retry launches an evaluate call makes.
#include "host_state.h"

using namespace dipsim;
using namespace dipsim_host;

namespace dipsim_host {

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
// Tile check plan: the ranks are split between the waves of a block,
// longest section first onto the least loaded wave.  The number of waves per
// block is the one (up to kTileMaxWaves, and not above the ranks or what
// keeps every wave near the longest section) that keeps the most waves
// resident per CU.  false when a rank's section does not fit.
bool plan_tiles(dip_sim *h, dip_sim::TilePlan *T) {
  int32_t max_nr = 0;
  int64_t n_sum = 0;
  for (int r = 0; r < h->P; ++r) {
    max_nr = std::max(max_nr, h->n_ops[r]);
    n_sum += h->n_ops[r];
  }
  if (int64_t(h->stride) * 2 * kWave > int64_t(INT32_MAX)) return false;
  const void *kern = tile_check_kernel_ptr();
  const int64_t region = tile_region_bytes(max_nr);
  const int nw_max = int(std::min<int64_t>(
      {int64_t(kTileMaxWaves), int64_t(h->P), (n_sum + std::max(max_nr, 1) - 1) / std::max(max_nr, 1)}));
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
  std::vector<int32_t> sorted(size_t(h->P)), load(nw, 0), wave_of(h->P, -1);
  for (int r = 0; r < h->P; ++r) sorted[r] = r;
  std::stable_sort(sorted.begin(), sorted.end(),
                   [&](int32_t x, int32_t y) { return h->n_ops[x] > h->n_ops[y]; });
  for (int32_t r : sorted) {
    const int w = int(std::min_element(load.begin(), load.end()) - load.begin());
    wave_of[r] = w;
    load[w] += h->n_ops[r];
  }
  std::vector<int32_t> plan(size_t(nw) + 1 + size_t(h->P));
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
  if (!T->d_plan && hipMalloc(&T->d_plan, size_t(h->P + kTileMaxWaves + 1) * 4) != hipSuccess) {
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

// The order kernel over the ranks with own-rank predecessors: the waves per
// block are the count (4, 8 or 16) that keeps the most waves resident per
// CU, the larger on ties (fewer table copies).  false when nothing fits.
bool plan_order_check(dip_sim *h, const std::vector<int32_t> &rks) {
  int32_t max_nr = 0;
  int64_t n_sum = 0;
  for (int32_t r : rks) {
    max_nr = std::max(max_nr, h->n_ops[r]);
    n_sum += h->n_ops[r];
  }
  const int32_t tab = order_table_bytes(max_nr);
  const void *kern = order_check_kernel_ptr();
  int best = 0;
  for (int w : {4, 8, 16}) {
    const int64_t lds = int64_t(tab) * (w + 1);
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
    if (b > 0 && b * w >= best) {
      best = b * w;
      h->oc_wpb = w;
      h->oc_blocks_per_cu = b;
      h->oc_lds = lds;
    }
  }
  if (best == 0) return false;
  if (h->oc_lds > 65536 && hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                                               int(h->oc_lds)) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  if (!h->d_oc_ranks && hipMalloc(&h->d_oc_ranks, size_t(h->P) * 4) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  if (hipMemcpy(h->d_oc_ranks, rks.data(), rks.size() * 4, hipMemcpyHostToDevice) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  // candidates per wave and block: about 64 KB of a mean section's ids, so
  // that the table copy at a block's start stays a few percent of its work
  const int64_t mean_bytes = std::max<int64_t>(2 * n_sum / int64_t(rks.size()), 1);
  h->oc_per_wave = int(std::min<int64_t>(64, std::max<int64_t>(2, 65536 / mean_bytes)));
  h->oc_tab_bytes = tab;
  h->oc_n_ranks = int32_t(rks.size());
  return true;
}

// The tile check over every rank, and the order kernel over the ranks with
// own-rank predecessors (when there are any and each op has at most one).
int plan_tile_check(dip_sim *h) {
  std::vector<int32_t> own;
  for (int r = 0; r < h->P; ++r)
    if ((h->self_ranks >> r) & 1u) own.push_back(r);
  h->tc_ok = plan_tiles(h, &h->tc);
  // (without the order kernel the simulation kernel keeps those edges)
  h->to_ok = h->tc_ok && h->self_ok && !own.empty() && plan_order_check(h, own);
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

int check_kind(const dip_sim *h) {
  if (h->check_mode != 0) return h->check_mode;
  return h->tc_ok ? 2 : 1;
}

bool order_checked(const dip_sim *h) { return check_kind(h) == 2 && h->to_ok; }

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
  c.P = h->P;
  c.retry_count = counts;
  const int64_t tiles = (n_cand + kWave - 1) / kWave;
  const dip_sim::TilePlan &T = h->tc;
  c.plan = T.d_plan;
  c.nw = T.nw;
  c.md_bytes = tile_md_bytes(T.max_nr);
  c.region_bytes = tile_region_bytes(T.max_nr);
  const int blocks = int(std::min<int64_t>(tiles, int64_t(T.blocks_per_cu) * h->n_cu));
  DIP_HIP(launch_tile_check(std::max(blocks, 1), T.nw, size_t(T.lds), stream, c));
  if (!h->to_ok) return DIP_OK;
  OrderCheckArgs o{};
  o.orders = orders;
  o.n_cand = n_cand;
  o.stride = h->stride;
  o.out_ms = out_ms;
  o.out_bub = out_bub;
  o.out_flags = out_flags;
  o.selfp = h->d_selfp;
  o.rank_off = h->d_rank_off;
  o.ranks = h->d_oc_ranks;
  o.P = h->P;
  o.n_ranks = h->oc_n_ranks;
  o.wpb = h->oc_wpb;
  o.tab_bytes = h->oc_tab_bytes;
  o.wave_bytes = h->oc_tab_bytes;
  // fewer candidates per wave for batches too small to give every resident
  // block slot four chunks of each rank
  const int64_t resident = int64_t(h->oc_blocks_per_cu) * h->n_cu;
  const int64_t want_chunks = std::max<int64_t>(1, 4 * resident / o.n_ranks);
  const int64_t per_wave =
      (n_cand + int64_t(o.wpb) * want_chunks - 1) / (int64_t(o.wpb) * want_chunks);
  o.per_wave = int32_t(std::max<int64_t>(1, std::min<int64_t>(h->oc_per_wave, per_wave)));
  const int64_t per_block = int64_t(o.per_wave) * o.wpb;
  o.n_chunks = (n_cand + per_block - 1) / per_block;
  const int64_t blocks_o = order_blocks(o.n_chunks, o.n_ranks);
  if (blocks_o > int64_t(INT32_MAX)) return DIP_E_INVAL;
  DIP_HIP(launch_order_check(blocks_o, o.wpb, size_t(h->oc_lds), stream, o));
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
  if (!h->d_retry_count) DIP_HIP(hipMalloc(&h->d_retry_count, kRetryCounters * 4));
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

// The passes' shapes (the configured pools, then 16 and 32 slots for the
// candidates whose pools filled); sim_costs_ok false when the first does not
// fit.
int sim_plan(dip_sim *h) {
  h->sim_costs_ok = false;
  h->sim2_ok = false;
  h->sim3_ok = false;
  h->sim_state_base = int64_t(h->sim_tab_vec) * 16;
  if (!sim_shape(h, h->pool_slots, h->forced_variant == 9 ? h->forced_wpb : 0, &h->sim_wpb,
                 &h->sim_max_blocks, &h->sim_lds))
    return DIP_OK;
  h->sim_costs_ok = true;
  if (h->pool_slots < 16)
    h->sim2_ok = sim_shape(h, 16, 0, &h->sim2_wpb, &h->sim2_max_blocks, &h->sim2_lds);
  h->sim3_ok = sim_shape(h, 32, 0, &h->sim3_wpb, &h->sim3_max_blocks, &h->sim3_lds);
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

}  // namespace dipsim_host
