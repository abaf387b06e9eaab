// kern_memopt.hip -- per-layer memory optimisation (DIP, arXiv 2504.14145,
// Sec. 5.3) of many candidate schedules at once.
//
// For every (candidate schedule, rank), each stage pair of the rank takes one
// of its memory candidates (time ascending, memory strictly descending) so
// that the live memory at every forward start stays within the rank's cap,
// with the least total time the greedy warm start of Sec. 5.3's ILP finds:
// all pairs on their fastest candidate; while the most loaded checkpoint
// (lowest index among equal loads) is over the cap, move the live pair with
// the least added time per freed memory unit (dt_a * dm_b < dt_b * dm_a,
// lowest pair index on ties) to its next candidate; give up when no live
// pair can move.  Pair i is live at pair k's forward start when its forward
// comes no later and its backward no earlier in the rank's order.
//
// One thread per (schedule, rank); its forward and backward positions,
// checkpoint loads and choices sit in LDS.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "internal.h"

namespace dipsim {

namespace {

__global__ __launch_bounds__(256) void memopt_kernel(MemoptArgs a) {
  extern __shared__ __align__(16) unsigned char sh[];
  const int64_t id = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (id >= a.n_cand * a.P) return;
  const int64_t c = id / a.P;
  const int r = int(id % a.P);
  const int32_t np = a.pair_off[r + 1] - a.pair_off[r];
  const int32_t pbase = a.pair_off[r];
  unsigned char *mine = sh + int64_t(threadIdx.x) * a.bytes_per_thread;
  int32_t *load = reinterpret_cast<int32_t *>(mine);
  uint16_t *pf = reinterpret_cast<uint16_t *>(mine + 4 * a.max_pairs);
  uint16_t *pb = pf + a.max_pairs;
  uint8_t *cur = reinterpret_cast<uint8_t *>(pb + a.max_pairs);
  for (int32_t i = 0; i < np; ++i) {
    pf[i] = 0xffffu;
    pb[i] = 0xffffu;
    cur[i] = 0;
  }
  // positions of each pair's forward and backward in the rank's order
  const int32_t base = a.rank_off[r], nr = a.rank_off[r + 1] - base;
  const int16_t *row = a.orders + c * a.stride + base;
  bool valid = true;
  for (int32_t p = 0; p < nr; ++p) {
    const int32_t lid = row[p];
    if (lid < 0 || lid >= nr) {
      valid = false;
      break;
    }
    const uint32_t w = uint32_t(a.lid_pair[base + lid]);
    uint16_t *slot = (w >> 31) ? pb : pf;
    const uint32_t i = w & 0x7fffffffu;
    if (slot[i] != 0xffffu) {
      valid = false;
      break;
    }
    slot[i] = uint16_t(p);
  }
  const int64_t o = c * a.P + r;
  if (!valid) {
    a.out_time[o] = -1;
    a.out_peak[o] = -1;
    a.out_status[o] = 2;
    return;
  }
  const int64_t *ct = a.cand_time + int64_t(pbase) * kMemoptMaxCands;
  const int32_t *cm = a.cand_mem + int64_t(pbase) * kMemoptMaxCands;
  const int32_t *nc = a.n_cands + pbase;
  for (int32_t k = 0; k < np; ++k) {
    int32_t s = 0;
    for (int32_t i = 0; i < np; ++i)
      if (pf[i] <= pf[k] && pf[k] <= pb[i]) s += cm[i * kMemoptMaxCands];
    load[k] = s;
  }
  const int32_t cap = a.cap[r];
  bool ok = true;
  if (cap >= 0) {
    for (;;) {
      int32_t kk = 0;
      for (int32_t k = 1; k < np; ++k)
        if (load[k] > load[kk]) kk = k;
      if (np == 0 || load[kk] <= cap) break;
      int32_t best = -1;
      int64_t bdt = 0, bdm = 1;
      for (int32_t i = 0; i < np; ++i) {
        if (!(pf[i] <= pf[kk] && pf[kk] <= pb[i])) continue;
        const int32_t j = cur[i];
        if (j + 1 >= nc[i]) continue;
        const int64_t dt = ct[i * kMemoptMaxCands + j + 1] - ct[i * kMemoptMaxCands + j];
        const int64_t dm = int64_t(cm[i * kMemoptMaxCands + j]) - cm[i * kMemoptMaxCands + j + 1];
        if (best < 0 || dt * bdm < bdt * dm) {
          best = i;
          bdt = dt;
          bdm = dm;
        }
      }
      if (best < 0) {
        ok = false;
        break;
      }
      cur[best] += 1;
      for (int32_t k = 0; k < np; ++k)
        if (pf[best] <= pf[k] && pf[k] <= pb[best]) load[k] -= int32_t(bdm);
    }
  }
  int64_t total = 0;
  int32_t peak = 0;
  for (int32_t i = 0; i < np; ++i) {
    total += ct[i * kMemoptMaxCands + cur[i]];
    peak = max(peak, load[i]);
  }
  a.out_time[o] = total;
  a.out_peak[o] = peak;
  a.out_status[o] = ok ? 1 : 0;
}

}  // namespace

hipError_t launch_memopt(int threads_per_block, hipStream_t s, const MemoptArgs &a) {
  const int64_t n = a.n_cand * a.P;
  const int64_t blocks = (n + threads_per_block - 1) / threads_per_block;
  hipLaunchKernelGGL(memopt_kernel, dim3(unsigned(blocks)), dim3(threads_per_block),
                     size_t(threads_per_block) * a.bytes_per_thread, s, a);
  return hipGetLastError();
}

}  // namespace dipsim
