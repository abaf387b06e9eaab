// host_limits.h -- shape limits of the handle and the host-side validation
// of instances and costs (plain C++, shared by the library and the CPU
// sanitizer build of the validation).
#pragma once

#include <cstdint>

#include "dip_sim.h"

namespace dipsim_host {

constexpr int kMaxRanks = 64;
constexpr int32_t kMaxOpsPerRank = 32768;

// DIP_OK or the code dip_sim_check_costs documents, for costs c of an
// instance of P ranks (n_ops[P], CSR pred_ptr, op_slot and kind per op,
// n_slots); *total_out (if given) the sum of all costs and latencies
int check_costs_against(int32_t P, const int32_t *n_ops, const int32_t *pred_ptr,
                        const int32_t *op_slot, const uint8_t *kind, int32_t n_slots,
                        const dip_costs *c, int64_t *total_out);

}  // namespace dipsim_host
