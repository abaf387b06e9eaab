// kern_costmodel.hip -- operator-level cost tables (DIP, arXiv 2504.14145,
// Sec. 6.1) for many configurations at once.
//
// An operator's latency is its largest resource time, read with per-kind
// coefficients c = alpha / capacity (seconds per FLOP, per byte of memory
// traffic, per byte sent): max(c_fop N_fop, c_mem N_mem, c_net N_net).  An
// item (a pipeline stage, a data edge) runs its operators in sequence; its
// entry is ceil(1e6 * sum) microseconds, -1 if that exceeds 2^31 - 1 or if an
// operator's kind is out of range.  One thread per (configuration, item);
// float64 throughout, without fused multiply-adds, so the sums are the
// float64 sums in row order.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "dip_sim.h"

namespace {

__global__ __launch_bounds__(256) void cost_table_kernel(dip_op_table t, int64_t n_configs,
                                                         const double *coef, int32_t *out) {
#pragma clang fp contract(off)
  const int32_t i = int32_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= t.n_items) return;
  const int32_t r0 = max(t.item_ptr[i], 0), r1 = min(t.item_ptr[i + 1], t.n_rows);
  for (int64_t b = blockIdx.y; b < n_configs; b += gridDim.y) {
    const double *cb = coef + b * int64_t(t.n_kinds) * 3;
    double s = 0.0;
    bool bad = false;
    for (int32_t r = r0; r < r1; ++r) {
      const int32_t k = t.kind[r];
      if (k >= t.n_kinds) {
        bad = true;
        break;
      }
      const double a = cb[3 * k] * t.n_fop[r];
      const double m = cb[3 * k + 1] * t.n_mem[r];
      const double n = cb[3 * k + 2] * t.n_net[r];
      s = s + fmax(fmax(a, m), n);
    }
    const double us = ceil(s * 1e6);
    out[b * t.n_items + i] = (bad || !(us <= 2147483647.0)) ? -1 : int32_t(us);
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
  const dim3 grid(unsigned((t->n_items + 255) / 256), unsigned(n_configs < 65535 ? n_configs : 65535));
  hipLaunchKernelGGL(cost_table_kernel, grid, dim3(256), 0, static_cast<hipStream_t>(stream), *t,
                     n_configs, coef, out);
  return hipGetLastError() == hipSuccess ? DIP_OK : DIP_E_HIP;
}
