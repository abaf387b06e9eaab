// dev_util.h -- small device helpers shared by the kernel translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace dipsim {

// Lane 0 of every group of 2^PWL lanes.
template <int PWL>
__host__ __device__ constexpr uint64_t group_low_lanes() {
  uint64_t low = 1;
  for (int s = 1 << PWL; s < 64; s <<= 1) low |= low << s;
  return low;
}

// Bit (g << PWL) of the result is set iff some lane of group g is set in m.
template <int PWL>
__device__ __forceinline__ uint64_t any_in_group(uint64_t m) {
#pragma unroll
  for (int s = 1; s < (1 << PWL); s <<= 1) m |= m >> s;
  return m & group_low_lanes<PWL>();
}

// Waits for this wave's outstanding LDS (and scalar-load) operations.
__device__ __forceinline__ void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Orders the LDS accesses of the lanes of one wave around this point.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

}  // namespace dipsim
