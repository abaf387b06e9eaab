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
// all its lanes read the same operator row at a time (scalar loads).  With
// LDS, the block's coefficients sit there as [kind][resource][lane]; else each
// lane reads its own from global memory.  A row's kind byte is taken from the
// aligned 32-bit word that holds it (a word that holds a valid byte lies in a
// valid page, so the wider read cannot fault), which a scalar load can serve;
// an out-of-range kind marks the item and is clamped, so the row loop has no
// early exit and its unrolled iterations overlap.
template <bool LDS>
__global__ __launch_bounds__(256) void cost_table_kernel(dip_op_table t, int64_t n_configs,
                                                         const double *coef, int32_t *out) {
#pragma clang fp contract(off)
  extern __shared__ double cl[];          // [kind][resource][lane]
  const int64_t b0 = int64_t(blockIdx.y) * kConfigsPerBlock;
  const int64_t b = b0 + threadIdx.x;
  const bool live = b < n_configs;
  const int K = t.n_kinds;
  if constexpr (LDS) {
    for (int j = threadIdx.x; j < K * 3 * kConfigsPerBlock; j += blockDim.x) {
      const int lane = j % kConfigsPerBlock, kr = j / kConfigsPerBlock;   // kr = kind * 3 + resource
      const int64_t bb = b0 + lane;
      cl[j] = bb < n_configs ? coef[bb * K * 3 + kr] : 0.0;
    }
    __syncthreads();
  }
  const double *cg = coef + (live ? b : 0) * int64_t(K) * 3;
  const uintptr_t kaddr = reinterpret_cast<uintptr_t>(t.kind);
  // read-only for the whole launch: the constant address space lets the
  // uniform word reads go through the scalar cache
  using ConstWord = const __attribute__((address_space(4))) uint32_t;
  ConstWord *kw = reinterpret_cast<ConstWord *>(kaddr & ~uintptr_t(3));
  const uint32_t k0 = uint32_t(kaddr & 3);
  const int32_t i0 = int32_t(blockIdx.x) * kItemsPerBlock;
  for (int32_t i = i0; i < i0 + kItemsPerBlock && i < t.n_items; ++i) {
    const int32_t r0 = max(t.item_ptr[i], 0), r1 = min(t.item_ptr[i + 1], t.n_rows);
    double s = 0.0;
    bool bad = false;
    // one row: its coefficients (kind kc, already clamped) times its counts,
    // the largest of the three added to the running sum
    auto row = [&](int32_t r, uint32_t kc) {
      double cf, cm, cn;
      if constexpr (LDS) {
        cf = cl[(3 * kc) * kConfigsPerBlock + threadIdx.x];
        cm = cl[(3 * kc + 1) * kConfigsPerBlock + threadIdx.x];
        cn = cl[(3 * kc + 2) * kConfigsPerBlock + threadIdx.x];
      } else {
        cf = cg[3 * kc];
        cm = cg[3 * kc + 1];
        cn = cg[3 * kc + 2];
      }
      const double a = cf * t.n_fop[r];
      const double m = cm * t.n_mem[r];
      const double n = cn * t.n_net[r];
      s = s + fmax(fmax(a, m), n);
    };
    int32_t r = r0;
    // eight rows at a time: their kind bytes from the aligned words holding
    // the first, the fifth and the last of them (each holds a valid byte;
    // the last two are the same word when the first is aligned)
    for (; r + 7 < r1; r += 8) {
      const uint32_t at = k0 + uint32_t(r), sh = (at & 3u) * 8u;
      const uint64_t wa = kw[at >> 2], wb = kw[(at >> 2) + 1], wc = kw[(at + 7) >> 2];
      const uint64_t k8 = uint64_t(uint32_t((wa | (wb << 32)) >> sh)) |
                          (uint64_t(uint32_t((wb | (wc << 32)) >> sh)) << 32);
      uint32_t kc[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t k = uint32_t(k8 >> (8 * j)) & 0xffu;
        bad |= k >= uint32_t(K);
        kc[j] = min(k, uint32_t(K - 1));
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) row(r + j, kc[j]);
    }
    for (; r < r1; ++r) {
      const uint32_t at = k0 + uint32_t(r);
      const uint32_t k = (kw[at >> 2] >> ((at & 3u) * 8u)) & 0xffu;
      bad |= k >= uint32_t(K);
      row(r, min(k, uint32_t(K - 1)));
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
  if (t->n_kinds <= kLdsKinds)
    hipLaunchKernelGGL(cost_table_kernel<true>, grid, dim3(256),
                       size_t(t->n_kinds) * 3 * kConfigsPerBlock * 8, static_cast<hipStream_t>(stream),
                       *t, n_configs, coef, out);
  else
    hipLaunchKernelGGL(cost_table_kernel<false>, grid, dim3(256), 0, static_cast<hipStream_t>(stream),
                       *t, n_configs, coef, out);
  return hipGetLastError() == hipSuccess ? DIP_OK : DIP_E_HIP;
}
