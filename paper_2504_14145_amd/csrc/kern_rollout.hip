// kern_rollout.hip -- priority vectors of MCTS rollouts (DIP, arXiv
// 2504.14145, Sec. 5.1).
//
// A rollout completes a search-tree node's class prefix at random and hands
// the sequence to the interleaving as priorities: the class at position i of
// n gets priority n - i, and every group takes its class's priority.  Rollout
// i of draw d shuffles the classes not in the prefix (ascending order to
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

// A block of B threads handles B consecutive rollouts (rows): row r belongs
// to leaf r / per_leaf, whose template is its class prefix followed by the
// other classes ascending, and is that leaf's rollout r % per_leaf, drawn with
// the leaf's draw number.  Each thread shuffles its row's classes and fills
// its class-priority table in LDS, then the block writes the B priority rows
// with consecutive threads on consecutive groups.
__global__ __launch_bounds__(64) void rollout_prio_kernel(RolloutArgs a) {
  extern __shared__ __align__(16) int32_t sh[];
  const int32_t n = a.n_classes, B = blockDim.x;
  const int64_t first = int64_t(blockIdx.x) * B;
  const int64_t i = first + threadIdx.x;
  int32_t *seq = sh + int64_t(threadIdx.x) * 2 * n;
  int32_t *prio_of = seq + n;
  if (i < a.n) {
    const int64_t leaf = i / a.per_leaf, ri = i % a.per_leaf;
    const int32_t dep = a.depths[leaf], m = n - dep;
    const int32_t *tmpl = a.seqs + leaf * n;
    for (int32_t k = 0; k < m; ++k) seq[k] = tmpl[dep + k];
    const uint64_t draw = a.draw + uint64_t(leaf);
    uint64_t st = mix(mix(a.seed + (draw + 1) * kGolden) + uint64_t(ri + 1) * kGolden);
    for (int32_t j = m - 1; j >= 1; --j) {
      st += kGolden;
      const uint64_t u = mix(st);
      const int32_t k = int32_t(((u >> 32) * uint64_t(j + 1)) >> 32);
      const int32_t t = seq[j];
      seq[j] = seq[k];
      seq[k] = t;
    }
    for (int32_t d = 0; d < dep; ++d) prio_of[tmpl[d]] = n - d;
    for (int32_t k = 0; k < m; ++k) prio_of[seq[k]] = n - (dep + k);
  }
  __syncthreads();
  const int64_t rows = a.n - first < B ? a.n - first : B;
  for (int64_t rr = 0; rr < rows; ++rr) {
    const int32_t *po = sh + rr * 2 * n + n;
    int32_t *out = a.out_prio + (first + rr) * a.G;
    for (int32_t g = threadIdx.x; g < a.G; g += B) out[g] = po[a.group_class[g]];
  }
}

}  // namespace

hipError_t launch_rollout_prio(hipStream_t s, const RolloutArgs &a) {
  // rollouts per block: a power of two up to 64 whose tables fit 64 KiB
  const int64_t per = int64_t(2 * a.n_classes) * 4;
  int B = 64;
  while (B > 1 && B * per > 65536) B /= 2;
  if (B * per > 65536) return hipErrorInvalidValue;
  const int64_t blocks = (a.n + B - 1) / B;
  hipLaunchKernelGGL(rollout_prio_kernel, dim3(unsigned(blocks)), dim3(B), size_t(B * per), s, a);
  return hipGetLastError();
}

}  // namespace dipsim
