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
// One wavefront per candidate reads the candidate's row 64 positions at a
// time (one coalesced 128-byte load per step).  Rank sections are contiguous
// in the row, so a step covers one rank, or a few when section boundaries
// fall inside it; a scalar loop walks those boundaries.  Duplicates are caught
// by an atomic OR into a bitmap of all op ids in the wave's LDS.  The running
// memory of a rank is a prefix sum: one DPP scan of the step's deltas gives
// every lane the sum from the start of the step, and a rank's part of it is
// that scan minus its value just before the rank's first lane, plus what the
// rank had accumulated in earlier steps.  The rank's peak is then a masked
// DPP max over its lanes.
#include "dip_sim.h"
#include "dev_util.h"
#include "internal.h"

namespace dipsim {
namespace {

extern __shared__ __align__(16) unsigned char c_lds[];

// DPP controls (GFX9 family): shift right within a row of 16 lanes, and the
// broadcasts of lane 15 / lane 31 to the following rows
constexpr int kRowShr = 0x110;
constexpr int kRowBcast15 = 0x142;
constexpr int kRowBcast31 = 0x143;

// inclusive prefix sum over the 64 lanes
__device__ __forceinline__ int wave_scan_add(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, kRowShr + 1, 0xf, 0xf, true);
  x += __builtin_amdgcn_update_dpp(0, x, kRowShr + 2, 0xf, 0xf, true);
  x += __builtin_amdgcn_update_dpp(0, x, kRowShr + 4, 0xf, 0xf, true);
  x += __builtin_amdgcn_update_dpp(0, x, kRowShr + 8, 0xf, 0xf, true);
  x += __builtin_amdgcn_update_dpp(0, x, kRowBcast15, 0xa, 0xf, false);
  x += __builtin_amdgcn_update_dpp(0, x, kRowBcast31, 0xc, 0xf, false);
  return x;
}

// maximum over the 64 lanes of non-negative values
__device__ __forceinline__ int wave_max_nonneg(int x) {
  x = max(x, __builtin_amdgcn_update_dpp(0, x, kRowShr + 1, 0xf, 0xf, true));
  x = max(x, __builtin_amdgcn_update_dpp(0, x, kRowShr + 2, 0xf, 0xf, true));
  x = max(x, __builtin_amdgcn_update_dpp(0, x, kRowShr + 4, 0xf, 0xf, true));
  x = max(x, __builtin_amdgcn_update_dpp(0, x, kRowShr + 8, 0xf, 0xf, true));
  x = max(x, __builtin_amdgcn_update_dpp(0, x, kRowBcast15, 0xa, 0xf, false));
  x = max(x, __builtin_amdgcn_update_dpp(0, x, kRowBcast31, 0xc, 0xf, false));
  return __builtin_amdgcn_readlane(x, kWave - 1);
}

__global__ __launch_bounds__(256) void check_kernel(CheckArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int wpw = int(check_lds_per_group(a.N) / 4);
  uint32_t *bm = reinterpret_cast<uint32_t *>(c_lds) + wave * wpw;
  if (a.retry_count && blockIdx.x == 0 && threadIdx.x == 0) *a.retry_count = 0u;

  const int cap_l = lane < a.P ? a.cap[lane] : -1;
  // section offsets in a register, lane k holding rank_off[k] (read with
  // readlane instead of scalar loads inside the boundary loops)
  const int ro_v = a.rank_off[min(lane, a.P)];
  auto ro = [&](int k) { return k < kWave ? __builtin_amdgcn_readlane(ro_v, k) : a.N; };
  const int64_t n_waves = int64_t(gridDim.x) * a.wpb;
  for (int64_t cand = int64_t(blockIdx.x) * a.wpb + wave; cand < a.n_cand; cand += n_waves) {
    for (int i = lane; i < wpw; i += kWave) bm[i] = 0u;
    const int16_t *row = a.orders + cand * a.stride;
    bool bad = false;
    int peak_l = 0;   // lane r: the peak of rank r
    int r = 0;        // rank of the step's first position
    int rb = ro(0), re = ro(1);   // its section [rb, re)
    int carry = 0;    // running memory of rank r before the step
    // one step: the 64 positions from p0, whose ids were loaded one step ahead
    auto step = [&](int p0, int id) {
      while (re <= p0 && r + 1 < a.P) {   // ranks that ended at the previous step's end
        ++r;
        rb = re;
        re = ro(r + 1);
        carry = 0;
      }
      const int p = p0 + lane;
      const bool live = p < a.N;
      // the section holding p: walk the boundaries inside the step
      int s_b = rb, s_e = re;
      {
        int rr = r, e = re;
        while (e < p0 + kWave && rr + 1 < a.P) {
          ++rr;
          const int nb = e, ne = ro(rr + 1);
          if (p >= nb) {
            s_b = nb;
            s_e = ne;
          }
          e = ne;
        }
      }
      const bool ok = live && unsigned(id) < unsigned(s_e - s_b);
      bad = bad || (live && !ok);
      const int g = s_b + (ok ? id : 0);
      const uint32_t bit = ok ? 1u << (g & 31) : 0u;
      const uint32_t old = atomicOr(bm + (g >> 5), bit);
      const int d = ok ? a.md[g] : 0;
      bad = bad || (old & bit) != 0u;
      const int S = wave_scan_add(d);

      // each rank with positions in this step: its running memory and peak
      int seg_lo = 0;
      for (;;) {
        const int seg_hi = min(re - p0, kWave);   // lanes [seg_lo, seg_hi) belong to rank r
        if (seg_hi > seg_lo) {
          const int before = seg_lo > 0 ? __builtin_amdgcn_readlane(S, seg_lo - 1) : 0;
          const bool in = lane >= seg_lo && lane < seg_hi;
          const int x = S - before + carry;
          const int mx = wave_max_nonneg(in ? max(x, 0) : 0);
          peak_l = lane == r ? max(peak_l, mx) : peak_l;
          carry = __builtin_amdgcn_readlane(x, seg_hi - 1);
        }
        if (re >= p0 + kWave || r + 1 >= a.P) break;   // rank r continues into the next step
        seg_lo = seg_hi;
        ++r;
        rb = re;
        re = ro(r + 1);
        carry = 0;
      }
    };
    auto load_id = [&](int p) { return int(row[p < a.N ? p : 0]); };
    // two steps per iteration, each step's ids loaded one step earlier
    int id_a = load_id(lane);
    for (int p0 = 0; p0 < a.N; p0 += 2 * kWave) {
      const int id_b = load_id(p0 + kWave + lane);
      step(p0, id_a);
      id_a = load_id(p0 + 2 * kWave + lane);
      if (p0 + kWave < a.N) step(p0 + kWave, id_b);
    }
    const bool invalid = __builtin_amdgcn_ballot_w64(bad) != 0ull;
    const bool over = lane < a.P && cap_l >= 0 && peak_l > cap_l;
    const bool capped = __builtin_amdgcn_ballot_w64(over) != 0ull;
    if (lane < a.P) {
      a.out_peak[cand * a.P + lane] = invalid ? -1 : peak_l;
      if (invalid) a.out_bub[cand * a.P + lane] = -1;
    }
    if (lane == 0) {
      a.out_flags[cand] = invalid ? uint8_t(DIP_FLAG_INVALID) : uint8_t(capped ? DIP_FLAG_CAP : 0u);
      if (invalid) a.out_ms[cand] = -1;
    }
  }
}

}  // namespace

const void *check_kernel_ptr(int) { return reinterpret_cast<const void *>(check_kernel); }

hipError_t launch_check(int, int blocks, int wpb, size_t lds, hipStream_t s, const CheckArgs &a) {
  check_kernel<<<dim3(blocks), dim3(wpb * kWave), lds, s>>>(a);
  return hipGetLastError();
}

}  // namespace dipsim
