// kern_check.hip -- the order-only part of a candidate's verdict, run before
// the timing simulation of the pool kernel:
//
//   * every rank section must be a permutation of that rank's op ids
//     (an id out of range or repeated makes the candidate invalid, and every
//     output of an invalid candidate is -1);
//   * peak activation memory per rank: the running sum of +act at each
//     forward and -act at each backward along the rank's order, starting from
//     0, and its maximum -- the liveness of a stage pair's activation from its
//     forward to its backward (Sec. 5.3), which depends on the order only;
//   * the cap flag: some rank's peak exceeds its cap.
//
// One wavefront per candidate.  A rank section is read 64 ids at a time
// (coalesced 128-byte loads); duplicates are caught with an atomic OR into a
// bitmap of all op ids in the wave's LDS, and the running sum is a wave
// prefix scan carried from chunk to chunk.
#include "dip_sim.h"
#include "dev_util.h"
#include "internal.h"

namespace dipsim {
namespace {

extern __shared__ __align__(16) unsigned char c_lds[];

__global__ __launch_bounds__(256) void check_kernel(CheckArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int bm_words = (a.N + 31) / 32;
  uint32_t *bm = reinterpret_cast<uint32_t *>(c_lds) + wave * ((bm_words + 3) & ~3);
  if (a.retry_count && blockIdx.x == 0 && threadIdx.x == 0) *a.retry_count = 0u;

  int cap_l = -1, rb_l = 0;
  if (lane < a.P) {
    cap_l = a.cap[lane];
    rb_l = a.rank_off[lane];
  }
  const int64_t n_waves = int64_t(gridDim.x) * a.wpb;
  for (int64_t cand = int64_t(blockIdx.x) * a.wpb + wave; cand < a.n_cand; cand += n_waves) {
    for (int i = lane; i < bm_words; i += kWave) bm[i] = 0u;
    bool bad = false;
    int my_peak = 0;
    const int16_t *row = a.orders + cand * a.stride;
    for (int r = 0; r < a.P; ++r) {
      const int rb = __shfl(rb_l, r, kWave);
      const int n = a.rank_off[r + 1] - rb;
      int carry = 0, run_max = 0;
      for (int i0 = 0; i0 < n; i0 += kWave) {
        const int i = i0 + lane;
        const bool live = i < n;
        const int id = live ? int(row[rb + i]) : 0;
        const bool ok = live && unsigned(id) < unsigned(n);
        const int g = rb + (ok ? id : 0);
        int d = 0;
        if (ok) {
          const uint32_t bit = 1u << (g & 31);
          const uint32_t old = atomicOr(bm + (g >> 5), bit);
          bad = bad || (old & bit) != 0u;
          d = a.md[g];
        }
        bad = bad || (live && !ok);
        // inclusive prefix sum of the memory deltas over the 64 lanes
        int x = d;
#pragma unroll
        for (int off = 1; off < kWave; off <<= 1) {
          const int y = __shfl_up(x, off, kWave);
          if (lane >= off) x += y;
        }
        x += carry;
        if (live) run_max = max(run_max, x);
        carry = __shfl(x, kWave - 1, kWave);
      }
#pragma unroll
      for (int off = 1; off < kWave; off <<= 1) run_max = max(run_max, __shfl_xor(run_max, off, kWave));
      if (lane == r) my_peak = run_max;
    }
    const bool invalid = __builtin_amdgcn_ballot_w64(bad) != 0ull;
    const bool over = lane < a.P && cap_l >= 0 && my_peak > cap_l;
    const bool capped = __builtin_amdgcn_ballot_w64(over) != 0ull;
    if (lane < a.P) {
      a.out_peak[cand * a.P + lane] = invalid ? -1 : my_peak;
      if (invalid) a.out_bub[cand * a.P + lane] = -1;
    }
    if (lane == 0) {
      a.out_flags[cand] = invalid ? uint8_t(DIP_FLAG_INVALID) : uint8_t(capped ? DIP_FLAG_CAP : 0u);
      if (invalid) a.out_ms[cand] = -1;
    }
  }
}

}  // namespace

const void *check_kernel_ptr() { return reinterpret_cast<const void *>(check_kernel); }

hipError_t launch_check(int blocks, int wpb, size_t lds, hipStream_t s, const CheckArgs &a) {
  check_kernel<<<dim3(blocks), dim3(wpb * kWave), lds, s>>>(a);
  return hipGetLastError();
}

}  // namespace dipsim
