// host_check.cpp -- host-side validation of instances and costs (the checks
// dip_sim_check_topology and dip_sim_check_costs document).  Plain C++ with
// no HIP dependency, so that a CPU test can build it with sanitizers.
#include <cstdint>

#include "dip_sim.h"
#include "host_limits.h"

namespace dipsim_host {

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

}  // namespace dipsim_host

using namespace dipsim_host;

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

}  // extern "C"
