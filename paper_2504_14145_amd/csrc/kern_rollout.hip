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
// One thread per rollout; its working arrays sit in LDS.
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

// A block of B threads handles B consecutive rollouts: each thread shuffles
// its rollout's classes and fills its class-priority table in LDS, then the
// block writes the B priority rows with consecutive threads on consecutive
// groups.
__global__ __launch_bounds__(64) void rollout_prio_kernel(RolloutArgs a) {
  extern __shared__ __align__(16) int32_t sh[];
  const int32_t m = a.m, n = a.n_classes, B = blockDim.x;
  const int64_t first = int64_t(blockIdx.x) * B;
  const int64_t i = first + threadIdx.x;
  int32_t *seq = sh + int64_t(threadIdx.x) * (m + n);
  int32_t *prio_of = seq + m;
  if (i < a.n) {
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
  }
  __syncthreads();
  const int64_t rows = a.n - first < B ? a.n - first : B;
  for (int64_t rr = 0; rr < rows; ++rr) {
    const int32_t *po = sh + rr * (m + n) + m;
    int32_t *out = a.out_prio + (first + rr) * a.G;
    for (int32_t g = threadIdx.x; g < a.G; g += B) out[g] = po[a.group_class[g]];
  }
}

}  // namespace

hipError_t launch_rollout_prio(hipStream_t s, const RolloutArgs &a) {
  // rollouts per block: a power of two up to 64 whose tables fit 64 KiB
  const int64_t per = int64_t(a.m + a.n_classes) * 4;
  int B = 64;
  while (B > 1 && B * per > 65536) B /= 2;
  if (B * per > 65536) return hipErrorInvalidValue;
  const int64_t blocks = (a.n + B - 1) / B;
  hipLaunchKernelGGL(rollout_prio_kernel, dim3(unsigned(blocks)), dim3(B), size_t(B * per), s, a);
  return hipGetLastError();
}

}  // namespace dipsim
