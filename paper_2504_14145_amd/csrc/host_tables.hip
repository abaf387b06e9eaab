// host_tables.hip -- device tables that depend on the costs: the staging
// layout, the general and pool kernels' records, the greedy's records and the
// simulation kernel's compact records (direct or paged), uploaded whenever a
// call brings new costs.
#include "host_state.h"

using namespace dipsim;
using namespace dipsim_host;

namespace dipsim_host {

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
  // alone once the check kernel has verified that the predecessor comes first
  // (it flags the candidate deadlocked otherwise): dropped, its producer then
  // publishes no end time for it
  h->sim_drop_self = order_checked(h);
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

}  // namespace dipsim_host
