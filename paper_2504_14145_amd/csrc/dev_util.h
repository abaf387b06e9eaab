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

// Every lane of group g is set iff bit (g << PWL) of m is (m holds group bits
// only, as any_in_group returns them).
template <int PWL>
__device__ __forceinline__ uint64_t any_lane_of_group(uint64_t m) {
#pragma unroll
  for (int s = 1; s < (1 << PWL); s <<= 1) m |= m << s;
  return m;
}

// Waits for this wave's outstanding LDS (and scalar-load) operations.
__device__ __forceinline__ void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Keeps this wave's LDS accesses on either side of this point in program
// order (the LDS serves one wave's instructions in issue order), without the
// wait for outstanding global loads that a workgroup-scope fence brings.
__device__ __forceinline__ void wave_lds_order() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Orders the LDS accesses of the lanes of one wave around this point.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// min / max of one value over all 64 lanes of a wave, returned to every lane
// as a uniform value: quad permutations and the half-row and row mirrors
// reduce each row of 16 lanes, then the four row results are read out.
// Every lane of the wave must be active.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_row(uint32_t v) {
  return uint32_t(__builtin_amdgcn_update_dpp(0, int(v), CTRL, 0xf, 0xf, false));
}
template <bool MAX>
__device__ __forceinline__ uint32_t wave_reduce_u32(uint32_t v) {
  auto op = [](uint32_t x, uint32_t y) { return MAX ? max(x, y) : min(x, y); };
  v = op(v, dpp_row<0xb1>(v));    // quad_perm [1,0,3,2]
  v = op(v, dpp_row<0x4e>(v));    // quad_perm [2,3,0,1]
  v = op(v, dpp_row<0x141>(v));   // row_half_mirror
  v = op(v, dpp_row<0x140>(v));   // row_mirror
  const uint32_t r0 = uint32_t(__builtin_amdgcn_readlane(int(v), 0));
  const uint32_t r1 = uint32_t(__builtin_amdgcn_readlane(int(v), 16));
  const uint32_t r2 = uint32_t(__builtin_amdgcn_readlane(int(v), 32));
  const uint32_t r3 = uint32_t(__builtin_amdgcn_readlane(int(v), 48));
  return op(op(r0, r1), op(r2, r3));
}
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) { return wave_reduce_u32<false>(v); }
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) { return wave_reduce_u32<true>(v); }

}  // namespace dipsim
