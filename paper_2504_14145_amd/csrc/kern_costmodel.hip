// kern_costmodel.hip -- operator-level cost tables (DIP, arXiv 2504.14145,
// Sec. 6.1) for many configurations at once.
//
// An operator's latency is its largest resource time, read with per-kind
// coefficients c = alpha / capacity (seconds per FLOP, per byte of memory
// traffic, per byte sent): max(c_fop N_fop, c_mem N_mem, c_net N_net).  An
// item (a pipeline stage, a data edge) runs its operators in sequence; its
// entry is ceil(1e6 * sum) microseconds, -1 if that exceeds 2^31 - 1 or if an
// operator's kind is out of range.  One lane per configuration; float64
// throughout, without fused multiply-adds, so the sums are the float64 sums in
// row order.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "dip_sim.h"

namespace {

constexpr int kConfigsPerBlock = 256;
constexpr int kItemsPerBlock = 8;
constexpr int kLdsKinds = 16;     // kinds whose coefficients fit the block's LDS

// Lane = configuration, 256 per block; a block walks kItemsPerBlock items, and
// all its lanes read the same operator row at a time (one broadcast load).
// The block's coefficients sit in LDS as [kind][resource][lane].
__global__ __launch_bounds__(256) void cost_table_kernel(dip_op_table t, int64_t n_configs,
                                                         const double *coef, int32_t *out) {
#pragma clang fp contract(off)
  extern __shared__ double cl[];          // [kind][resource][lane] when it fits
  const int64_t b0 = int64_t(blockIdx.y) * kConfigsPerBlock;
  const int64_t b = b0 + threadIdx.x;
  const bool live = b < n_configs;
  const int K = t.n_kinds;
  const bool lds = K <= kLdsKinds;
  if (lds) {
    for (int j = threadIdx.x; j < K * 3 * kConfigsPerBlock; j += blockDim.x) {
      const int lane = j % kConfigsPerBlock, kr = j / kConfigsPerBlock;   // kr = kind * 3 + resource
      const int64_t bb = b0 + lane;
      cl[j] = bb < n_configs ? coef[bb * K * 3 + kr] : 0.0;
    }
    __syncthreads();
  }
  const double *cg = coef + (live ? b : 0) * int64_t(K) * 3;
  const int32_t i0 = int32_t(blockIdx.x) * kItemsPerBlock;
  for (int32_t i = i0; i < i0 + kItemsPerBlock && i < t.n_items; ++i) {
    const int32_t r0 = max(t.item_ptr[i], 0), r1 = min(t.item_ptr[i + 1], t.n_rows);
    double s = 0.0;
    bool bad = false;
#pragma unroll 4
    for (int32_t r = r0; r < r1; ++r) {
      const int32_t k = t.kind[r];
      if (k >= K) {
        bad = true;
        break;
      }
      double cf, cm, cn;
      if (lds) {
        cf = cl[(3 * k) * kConfigsPerBlock + threadIdx.x];
        cm = cl[(3 * k + 1) * kConfigsPerBlock + threadIdx.x];
        cn = cl[(3 * k + 2) * kConfigsPerBlock + threadIdx.x];
      } else {
        cf = cg[3 * k];
        cm = cg[3 * k + 1];
        cn = cg[3 * k + 2];
      }
      const double a = cf * t.n_fop[r];
      const double m = cm * t.n_mem[r];
      const double n = cn * t.n_net[r];
      s = s + fmax(fmax(a, m), n);
    }
    const double us = ceil(s * 1e6);
    if (live) out[b * t.n_items + i] = (bad || !(us <= 2147483647.0)) ? -1 : int32_t(us);
  }
}

}  // namespace

extern "C" int dip_cost_tables(const dip_op_table *t, int64_t n_configs, const double *coef,
                               int32_t *out, void *stream) {
  if (!t || n_configs < 0 || t->n_items < 0 || t->n_rows < 0 || t->n_kinds < 1 ||
      t->n_kinds > 256)
    return DIP_E_INVAL;
  if (n_configs == 0 || t->n_items == 0) return DIP_OK;
  if (!t->item_ptr || !coef || !out || (t->n_rows > 0 && (!t->n_fop || !t->n_mem || !t->n_net ||
                                                          !t->kind)))
    return DIP_E_INVAL;
  if ((reinterpret_cast<uintptr_t>(coef) | reinterpret_cast<uintptr_t>(t->n_fop) |
       reinterpret_cast<uintptr_t>(t->n_mem) | reinterpret_cast<uintptr_t>(t->n_net)) & 7)
    return DIP_E_INVAL;
  if ((reinterpret_cast<uintptr_t>(out) | reinterpret_cast<uintptr_t>(t->item_ptr)) & 3)
    return DIP_E_INVAL;
  const int64_t gx = (int64_t(t->n_items) + kItemsPerBlock - 1) / kItemsPerBlock;
  const int64_t gy = (n_configs + kConfigsPerBlock - 1) / kConfigsPerBlock;
  if (gx > INT32_MAX || gy > 65535) return DIP_E_INVAL;
  const dim3 grid{unsigned(gx), unsigned(gy), 1u};
  const size_t lds = t->n_kinds <= kLdsKinds ? size_t(t->n_kinds) * 3 * kConfigsPerBlock * 8 : 0;
  hipLaunchKernelGGL(cost_table_kernel, grid, dim3(256), lds, static_cast<hipStream_t>(stream), *t,
                     n_configs, coef, out);
  return hipGetLastError() == hipSuccess ? DIP_OK : DIP_E_HIP;
}
