// kern_argmin.hip -- best (makespan, index) over a batch of simulated
// candidates: the lexicographic minimum of packed 64-bit keys, folded into a
// running key so that chunked batches reduce exactly.
#include "internal.h"

namespace dipsim {
namespace {

// Argmin: packed key (makespan << 32 | index) per valid candidate; wave
// reduction with cross-lane shuffles, block reduction through LDS, then one
// 64-bit atomic min per block into the caller's running key.
__global__ __launch_bounds__(256) void argmin_kernel(const int32_t *ms, const uint8_t *flags,
                                                     int64_t n, int64_t seg_len, uint64_t base,
                                                     unsigned long long *key) {
  __shared__ unsigned long long s_best[256 / kWave];
  unsigned long long best = ~0ull;
  const int64_t s0 = int64_t(blockIdx.y) * seg_len;
  const int64_t s1 = n - s0 < seg_len ? n : s0 + seg_len;
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t i = s0 + int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < s1; i += stride) {
    if (flags[i] == 0) {
      const unsigned long long k =
          (static_cast<unsigned long long>(static_cast<uint32_t>(ms[i])) << 32) |
          static_cast<uint32_t>(base + uint64_t(i - s0));
      best = k < best ? k : best;
    }
  }
  for (int off = kWave / 2; off > 0; off >>= 1) {
    const unsigned lo = __shfl_xor(static_cast<unsigned>(best), off, kWave);
    const unsigned hi = __shfl_xor(static_cast<unsigned>(best >> 32), off, kWave);
    const unsigned long long other = (static_cast<unsigned long long>(hi) << 32) | lo;
    best = other < best ? other : best;
  }
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  if (lane == 0) s_best[wave] = best;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long b = s_best[0];
    for (int w = 1; w < int(blockDim.x / kWave); ++w) b = s_best[w] < b ? s_best[w] : b;
    if (b != ~0ull) atomicMin(key + blockIdx.y, b);
  }
}

}  // namespace

hipError_t launch_argmin(int blocks, hipStream_t s, const int32_t *ms, const uint8_t *flags,
                         int64_t n, int64_t seg_len, int n_seg, uint64_t base,
                         unsigned long long *key) {
  argmin_kernel<<<dim3(unsigned(blocks), unsigned(n_seg)), dim3(256), 0, s>>>(ms, flags, n, seg_len,
                                                                             base, key);
  return hipGetLastError();
}

}  // namespace dipsim
