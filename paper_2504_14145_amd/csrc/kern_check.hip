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
// Same layout as the simulation: G = 64 / PW candidates per wavefront, lane r
// of a group walks rank r's section, sixteen ids per step (their loads, the
// duplicate checks and the memory-delta loads each issued together).
// Duplicates are caught by an atomic OR into the group's bitmap of all op
// ids in LDS.
#include "dip_sim.h"
#include "dev_util.h"
#include "internal.h"

namespace dipsim {
namespace {

extern __shared__ __align__(16) unsigned char c_lds[];

template <int PWL>
__global__ __launch_bounds__(256) void check_kernel(CheckArgs a) {
  constexpr int PW = 1 << PWL;
  constexpr int G = kWave / PW;
  constexpr int U = 16;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int grp = lane >> PWL;
  const int r = lane & (PW - 1);
  const bool on = r < a.P;
  const int gbit = grp << PWL;
  const int wpg = int(check_lds_per_group(a.N) / 4);
  uint32_t *bm = reinterpret_cast<uint32_t *>(c_lds) + (wave * G + grp) * wpg;
  if (a.retry_count && blockIdx.x == 0 && threadIdx.x == 0) *a.retry_count = 0u;

  int rb = 0, nr = 0, cap_r = -1;
  if (on) {
    rb = a.rank_off[r];
    nr = a.rank_off[r + 1] - rb;
    cap_r = a.cap[r];
  }
  const int64_t n_slots = int64_t(gridDim.x) * a.wpb * G;
  for (int64_t base = (int64_t(blockIdx.x) * a.wpb + wave) * G; base < a.n_cand; base += n_slots) {
    const int64_t cand = base + grp;
    const bool live = cand < a.n_cand;
    for (int i = r; i < wpg; i += PW) bm[i] = 0u;
    bool bad = false;
    int mem = 0, peak = 0;
    if (live && on && nr > 0) {
      // branch-free steps: every id load, bitmap OR and delta load of a step
      // is issued before any result is used
      const int16_t *row = a.orders + cand * a.stride + rb;
      for (int i0 = 0; i0 < nr; i0 += U) {
        int id[U];
#pragma unroll
        for (int k = 0; k < U; ++k) id[k] = row[min(i0 + k, nr - 1)];
        uint32_t old[U], bit[U];
        int d[U];
#pragma unroll
        for (int k = 0; k < U; ++k) {
          const bool in = i0 + k < nr;
          const bool ok = unsigned(id[k]) < unsigned(nr);
          bad = bad || (in && !ok);
          const int g = rb + (ok ? id[k] : 0);
          bit[k] = (in && ok) ? 1u << (g & 31) : 0u;
          old[k] = atomicOr(bm + (g >> 5), bit[k]);
          d[k] = a.md[g];
          d[k] = (in && ok) ? d[k] : 0;
        }
#pragma unroll
        for (int k = 0; k < U; ++k) {
          bad = bad || (old[k] & bit[k]) != 0u;
          mem += d[k];
          peak = max(peak, mem);
        }
      }
    }
    const bool g_bad = (any_in_group<PWL>(__builtin_amdgcn_ballot_w64(bad)) >> gbit) & 1;
    const bool over = live && on && cap_r >= 0 && peak > cap_r;
    const bool g_cap = (any_in_group<PWL>(__builtin_amdgcn_ballot_w64(over)) >> gbit) & 1;
    if (live && on) {
      a.out_peak[cand * a.P + r] = g_bad ? -1 : peak;
      if (g_bad) a.out_bub[cand * a.P + r] = -1;
      if (r == 0) {
        a.out_flags[cand] = g_bad ? uint8_t(DIP_FLAG_INVALID) : uint8_t(g_cap ? DIP_FLAG_CAP : 0u);
        if (g_bad) a.out_ms[cand] = -1;
      }
    }
  }
}

}  // namespace

const void *check_kernel_ptr(int pwl) {
  switch (pwl) {
    case 0: return reinterpret_cast<const void *>(check_kernel<0>);
    case 1: return reinterpret_cast<const void *>(check_kernel<1>);
    case 2: return reinterpret_cast<const void *>(check_kernel<2>);
    case 3: return reinterpret_cast<const void *>(check_kernel<3>);
    case 4: return reinterpret_cast<const void *>(check_kernel<4>);
    case 5: return reinterpret_cast<const void *>(check_kernel<5>);
    default: return reinterpret_cast<const void *>(check_kernel<6>);
  }
}

hipError_t launch_check(int pwl, int blocks, int wpb, size_t lds, hipStream_t s,
                        const CheckArgs &a) {
  const dim3 grid(blocks), block(wpb * kWave);
  switch (pwl) {
    case 0: check_kernel<0><<<grid, block, lds, s>>>(a); break;
    case 1: check_kernel<1><<<grid, block, lds, s>>>(a); break;
    case 2: check_kernel<2><<<grid, block, lds, s>>>(a); break;
    case 3: check_kernel<3><<<grid, block, lds, s>>>(a); break;
    case 4: check_kernel<4><<<grid, block, lds, s>>>(a); break;
    case 5: check_kernel<5><<<grid, block, lds, s>>>(a); break;
    default: check_kernel<6><<<grid, block, lds, s>>>(a); break;
  }
  return hipGetLastError();
}

}  // namespace dipsim
