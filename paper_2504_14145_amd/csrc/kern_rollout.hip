// kern_rollout.hip -- priority vectors of MCTS rollouts (DIP, arXiv
// 2504.14145, Sec. 5.1).
//
// A rollout completes the search tree's class prefix at random and hands the
// sequence to the interleaving as priorities: the class at position i of n
// gets priority n - i, and every group takes its class's priority.  Rollout i
// of draw d shuffles the classes not in the prefix (ascending order to
// start) with Durstenfeld's Fisher-Yates; for j = m-1 down to 1 the swap
// partner k in [0, j] is (hi32(u) * (j + 1)) >> 32, u the next output of
// SplitMix64 (Steele, Lea and Flood, OOPSLA 2014) started from
// mix(mix(seed + (d + 1) G) + (i + 1) G), G = 0x9E3779B97F4A7C15.
// One thread per rollout; its working arrays sit in device scratch.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "internal.h"

namespace dipsim {

namespace {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;

__device__ __forceinline__ uint64_t mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__global__ __launch_bounds__(256) void rollout_prio_kernel(RolloutArgs a) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= a.n) return;
  const int32_t m = a.m, n = a.n_classes;
  int32_t *seq = a.scratch + i * 2 * int64_t(n);
  int32_t *prio_of = seq + m;
  for (int32_t k = 0; k < m; ++k) seq[k] = a.rest[k];
  uint64_t st = mix(mix(a.seed + (a.draw + 1) * kGolden) + uint64_t(i + 1) * kGolden);
  for (int32_t j = m - 1; j >= 1; --j) {
    st += kGolden;
    const uint64_t u = mix(st);
    const int32_t k = int32_t(((u >> 32) * uint64_t(j + 1)) >> 32);
    const int32_t t = seq[j];
    seq[j] = seq[k];
    seq[k] = t;
  }
  for (int32_t d = 0; d < a.depth; ++d) prio_of[a.prefix[d]] = n - d;
  for (int32_t k = 0; k < m; ++k) prio_of[seq[k]] = n - (a.depth + k);
  int32_t *out = a.out_prio + i * a.G;
  for (int32_t g = 0; g < a.G; ++g) out[g] = prio_of[a.group_class[g]];
}

}  // namespace

hipError_t launch_rollout_prio(hipStream_t s, const RolloutArgs &a) {
  const int64_t blocks = (a.n + 255) / 256;
  hipLaunchKernelGGL(rollout_prio_kernel, dim3(unsigned(blocks)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace dipsim
