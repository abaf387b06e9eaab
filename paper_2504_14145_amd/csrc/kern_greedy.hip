// kern_greedy.hip -- dual-queue stage interleaving (DIP, arXiv 2504.14145,
// Sec. 5.2) of many candidate priority vectors at once.
//
// Per candidate the kernel builds each rank's stage order the way Sec. 5.2's
// greedy does, and the timeline that comes with it:
//   * a stage is queued on its rank once all its predecessors are scheduled,
//     with t_start = max over them of end + comm (0 without predecessors);
//   * a rank can next start at t_min = max(t_last, smallest queued t_start);
//     if both a forward and a backward were queued before t_last, it takes the
//     kind opposite to its last stage (1F1B); otherwise it takes any stage
//     that can start at t_min; within that set the highest priority wins
//     (priority, then group index, then rank-local id);
//   * a forward that would raise the rank's live activation above its cap
//     disables the forward queue for that decision (Sec. 5.2's memory rule);
//   * the rank with the smallest t_min (lowest index on ties) commits its
//     choice; when every rank is held back by its cap, the cap is lifted for
//     one decision.
// Every round commits exactly one stage of every candidate, so a candidate
// takes N rounds.
//
// Mapping: a group of PW = 2^PWL lanes per candidate, lane = rank; 64 / PW
// candidates per wave.  A rank's queued stages are kept by priority position
// (the group's rank among groups of its kind under the candidate's
// priorities):
//   E  bitmap (registers) of queued stages with t_start <  t_last,
//   Z  bitmap (registers) of queued stages with t_start == t_last,
//   inbox (LDS) of stages whose t_start is still ahead: (t_start, kind, pos).
// Lanes touch only their own bitmaps; the committing lane appends the stages
// its commit completes to the target ranks' inboxes, and each lane sorts its
// inbox into E / Z at the start of the next round.  A group min over the
// lanes' t_min picks the committing rank.  An inbox that fills up sends the
// candidate to a list that a second launch, with inboxes as large as a rank's
// stage count, simulates again.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "dip_sim.h"
#include "dev_util.h"
#include "internal.h"

namespace dipsim {

namespace {

constexpr uint32_t kNoPos = 0xffffu;
constexpr uint32_t kNever = 0xffffffffu;

// A set of priority positions 0 .. 64 * NW - 1, held in registers; indexes are
// resolved by selects so that the words never leave registers.
template <int NW>
struct Bits {
  uint64_t w[NW];
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int i = 0; i < NW; ++i) w[i] = 0;
  }
  __device__ __forceinline__ void set(uint32_t p) {
    const uint32_t k = p >> 6;
    const uint64_t b = uint64_t(1) << (p & 63u);
#pragma unroll
    for (int i = 0; i < NW; ++i) w[i] |= uint32_t(i) == k ? b : uint64_t(0);
  }
  __device__ __forceinline__ void clear(uint32_t p) {
    const uint32_t k = p >> 6;
    const uint64_t b = ~(uint64_t(1) << (p & 63u));
#pragma unroll
    for (int i = 0; i < NW; ++i) w[i] &= uint32_t(i) == k ? b : ~uint64_t(0);
  }
  __device__ __forceinline__ bool any() const {
    uint64_t m = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) m |= w[i];
    return m != 0;
  }
  // this |= z, z = {}
  __device__ __forceinline__ void absorb(Bits &z) {
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      w[i] |= z.w[i];
      z.w[i] = 0;
    }
  }
};

// lowest position in a | b, kNoPos if both are empty
template <int NW>
__device__ __forceinline__ uint32_t first_of(const Bits<NW> &a, const Bits<NW> &b) {
  uint32_t r = kNoPos;
#pragma unroll
  for (int i = NW - 1; i >= 0; --i) {
    const uint64_t m = a.w[i] | b.w[i];
    if (m != 0) r = uint32_t(i) * 64u + uint32_t(__builtin_ctzll(m));
  }
  return r;
}

template <int PWL>
__device__ __forceinline__ uint32_t group_min(uint32_t v) {
#pragma unroll
  for (int s = 1; s < (1 << PWL); s <<= 1) v = min(v, uint32_t(__shfl_xor(int(v), s)));
  return v;
}

template <int PWL>
__device__ __forceinline__ uint32_t group_max(uint32_t v) {
#pragma unroll
  for (int s = 1; s < (1 << PWL); s <<= 1) v = max(v, uint32_t(__shfl_xor(int(v), s)));
  return v;
}

// bits of this lane's group in a wave-wide mask, lowest rank at bit 0
template <int PWL>
__device__ __forceinline__ uint64_t group_bits(uint64_t m, int grp) {
  constexpr uint64_t low = (1 << PWL) == 64 ? ~uint64_t(0) : (uint64_t(1) << (1 << PWL)) - 1;
  return (m >> (grp << PWL)) & low;
}

// One rank's choice: start time, priority position, kind (0 forward, 1
// backward) and, for a stage still in the inbox, its inbox index.
struct Choice {
  uint32_t tau, pos, kind, slot;
};

}  // namespace

template <int PWL, int NW>
__global__ __launch_bounds__(256) void greedy_kernel(GreedyArgs a) {
  constexpr int PW = 1 << PWL;
  constexpr int GW = kWave >> PWL;
  extern __shared__ __align__(16) unsigned char lds[];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int grp = lane >> PWL;
  const int r = lane & (PW - 1);
  const int G = a.G, GF = a.GF, P = a.P, K = a.K;

  uint16_t *meta = reinterpret_cast<uint16_t *>(lds);
  for (int i = threadIdx.x; i < G; i += blockDim.x) meta[i] = uint16_t(a.caller[i]);
  __syncthreads();

  unsigned char *cb = lds + a.meta_bytes + int64_t(wave * GW + grp) * a.cand_bytes;
  int32_t *prio = reinterpret_cast<int32_t *>(cb);               // setup only ...
  uint64_t *pend0 = reinterpret_cast<uint64_t *>(cb + a.off_pend);  // ... then inboxes
  uint64_t *pend = pend0 + int64_t(r) * K;
  uint32_t *npend = reinterpret_cast<uint32_t *>(cb + a.off_npend);
  uint32_t *jtab = reinterpret_cast<uint32_t *>(cb + a.off_join);
  uint16_t *gpos = reinterpret_cast<uint16_t *>(cb + a.off_gpos);
  uint16_t *ord = reinterpret_cast<uint16_t *>(cb + a.off_ord);
  uint16_t *grk = reinterpret_cast<uint16_t *>(cb + a.off_grk);

  const int64_t n_slots = int64_t(gridDim.x) * a.wpb * GW;
  for (int64_t slot = (int64_t(blockIdx.x) * a.wpb + wave) * GW + grp;; slot += n_slots) {
    int64_t cand = -1;
    if (a.list) {
      if (slot < int64_t(*a.list_count)) cand = a.list[slot];
    } else if (slot < a.n_cand) {
      cand = slot;
    }
    const bool has = cand >= 0;
    if (!__any(has)) break;
    const bool real = has && r < P;

    // ---- setup: positions of the groups under this candidate's priorities
    if (has) {
      const int32_t *pv = a.prio + cand * G;
      for (int g = r; g < G; g += PW) prio[g] = pv[meta[g]];
    }
    wave_sync();
    if (has) {
      for (int g = r; g < G; g += PW) {
        const int32_t pg = prio[g];
        const uint32_t cg = meta[g];
        const bool fg = g < GF;
        uint32_t before = 0, same = 0;
        for (int h = 0; h < G; ++h) {
          const int32_t ph = prio[h];
          const bool ahead = ph > pg || (ph == pg && uint32_t(meta[h]) < cg);
          before += ahead ? 1u : 0u;
          same += (ahead && ((h < GF) == fg)) ? 1u : 0u;
        }
        gpos[g] = uint16_t(same);
        const int at = fg ? int(same) : GF + int(same);
        ord[at] = uint16_t(g);
        grk[at] = uint16_t(before);
      }
    }
    wave_sync();
    if (has) {
      for (int j = r; j < 2 * a.J; j += PW) jtab[j] = 0;
      if (r < P) npend[r] = 0;
    }
    Bits<NW> eF, eB, zF, zB;
    eF.zero();
    eB.zero();
    zF.zero();
    zB.zero();
    if (real) {
      // stages without predecessors: queued at t_start 0 = t_last
      const int32_t *src_list = a.src + P + 1;
      for (int s = a.src[r]; s < a.src[r + 1]; ++s) {
        const int g = src_list[s];
        if (g < GF) zF.set(gpos[g]);
        else zB.set(gpos[g]);
      }
    }
    wave_sync();

    uint32_t t_last = 0, tl_seen = 0, last_kind = 0, n_emit = 0;
    int32_t live = 0, peak = 0;
    bool ovf = false, stuck = false;
    const int32_t capr = real ? a.cap[r] : -1;
    const int64_t row = real ? cand * a.stride + a.rank_off[r] : 0;
    const uint32_t n_own = real ? uint32_t(a.rank_off[r + 1] - a.rank_off[r]) : 0u;

    for (int it = 0; it < a.n_rounds; ++it) {
      // ---- 1. inbox: stages whose t_start has come move into E / Z
      uint32_t pmF = kNever, pmB = kNever, ppF = kNoPos, ppB = kNoPos, psF = 0, psB = 0;
      if (real) {
        if (t_last != tl_seen) {
          eF.absorb(zF);
          eB.absorb(zB);
          tl_seen = t_last;
        }
        const uint32_t n = npend[r];
        uint32_t j = 0;
        for (uint32_t i = 0; i < n; ++i) {
          const uint64_t e = pend[i];
          const uint32_t t = uint32_t(e >> 17);
          const uint32_t p = uint32_t(e) & 0xffffu;
          const bool bk = ((uint32_t(e) >> 16) & 1u) != 0;
          if (t < t_last) {
            if (bk) eB.set(p);
            else eF.set(p);
          } else if (t == t_last) {
            if (bk) zB.set(p);
            else zF.set(p);
          } else {
            if (j != i) pend[j] = e;
            if (bk) {
              if (t < pmB || (t == pmB && p < ppB)) {
                pmB = t;
                ppB = p;
                psB = j;
              }
            } else if (t < pmF || (t == pmF && p < ppF)) {
              pmF = t;
              ppF = p;
              psF = j;
            }
            ++j;
          }
        }
        if (j != n) npend[r] = j;
      }

      // ---- 2. this rank's choice
      const uint32_t fF = first_of(eF, zF), fB = first_of(eB, zB);
      const bool xF = eF.any(), xB = eB.any();
      uint32_t gF = kNoPos, gB = kNoPos, hF = kNoPos, hB = kNoPos;
      if (real) {
        if (fF != kNoPos) gF = grk[fF];
        if (fB != kNoPos) gB = grk[GF + fB];
        if (ppF != kNoPos) hF = grk[ppF];
        if (ppB != kNoPos) hB = grk[GF + ppB];
      }
      auto decide = [&](bool fw) {
        Choice c;
        const bool nF = fw && fF != kNoPos, nB = fB != kNoPos;
        c.slot = kNever;
        if (nF || nB) {
          c.tau = t_last;
          if (fw && xF && xB) c.kind = last_kind ^ 1u;
          else c.kind = (nF && (!nB || gF < gB)) ? 0u : 1u;
          c.pos = c.kind ? fB : fF;
        } else {
          const uint32_t tF = fw ? pmF : kNever;
          c.tau = min(tF, pmB);
          if (c.tau == kNever) {
            c.pos = kNoPos;
            c.kind = 0;
          } else {
            c.kind = (tF == c.tau && (pmB != c.tau || hF < hB)) ? 0u : 1u;
            c.pos = c.kind ? ppB : ppF;
            c.slot = c.kind ? psB : psF;
          }
        }
        return c;
      };
      const Choice ce = decide(true);
      Choice cd = ce;
      int4 q0e = make_int4(0, 0, 0, 0), q1e = q0e;
      bool have_e = false;
      if (a.has_cap && real && ce.pos != kNoPos && ce.kind == 0 && capr >= 0) {
        const int4 *rp = a.rec + (int64_t(ord[ce.pos]) * P + r) * 2;
        q0e = rp[0];
        q1e = rp[1];
        have_e = true;
        if (live + q0e.y > capr) cd = decide(false);   // forward queue disabled
      }

      // ---- 3. the rank with the smallest t_min commits
      const uint32_t key_d = (real && cd.pos != kNoPos) ? cd.tau : kNever;
      uint32_t m = group_min<PWL>(key_d);
      uint32_t key = key_d;
      bool forced = false;
      if (__any(has && m == kNever)) {
        const uint32_t key_e = (real && ce.pos != kNoPos) ? ce.tau : kNever;
        const uint32_t m2 = group_min<PWL>(key_e);
        if (m == kNever) {
          forced = true;
          m = m2;
          key = key_e;
        }
      }
      if (has && m == kNever) stuck = true;   // only a cyclic data graph gets here
      const uint64_t mine = group_bits<PWL>(__ballot(real && m != kNever && key == m), grp);
      const bool win = mine != 0 && r == __builtin_ctzll(mine);

      if (win) {
        const Choice c = forced ? ce : cd;
        int4 q0, q1;
        if (have_e && c.kind == ce.kind && c.pos == ce.pos) {
          q0 = q0e;
          q1 = q1e;
        } else {
          const int4 *rp = a.rec + (int64_t(ord[c.kind ? GF + c.pos : c.pos]) * P + r) * 2;
          q0 = rp[0];
          q1 = rp[1];
        }
        const uint32_t end = c.tau + uint32_t(q0.x);
        if (c.slot == kNever) {
          if (c.kind) {
            eB.clear(c.pos);
            zB.clear(c.pos);
          } else {
            eF.clear(c.pos);
            zF.clear(c.pos);
          }
        } else {
          const uint32_t n = npend[r] - 1;
          if (c.slot != n) pend[c.slot] = pend[n];
          npend[r] = n;
        }
        t_last = end;
        last_kind = c.kind;
        if (c.kind == 0) {
          live += q0.y;
          peak = max(peak, live);
        } else {
          live -= q0.y;
        }
        if (n_emit < n_own) {
          if (a.out_orders) a.out_orders[row + n_emit] = int16_t(q0.z & 0xffff);
        } else {
          ovf = true;     // more commits than stages: never with consistent tables
        }
        ++n_emit;
        // successors whose last predecessor this was join the target inboxes
        const uint32_t ns = uint32_t(q0.z) >> 16;
        for (uint32_t s = 0; s < ns; ++s) {
          const int4 e = s == 0 ? q1 : a.succ[q0.w + int32_t(s) - 1];
          uint32_t t = end + uint32_t(e.y);
          if (e.z >= 0) {
            uint32_t *jb = jtab + 2 * e.z;
            const uint32_t acc = max(jb[0], t), cnt = jb[1] + 1u;
            jb[0] = acc;
            jb[1] = cnt;
            if (cnt < uint32_t(e.w)) continue;
            t = acc;
          }
          const uint32_t w = uint32_t(e.x);
          const uint32_t tr = (w >> 17) & 63u;
          const uint32_t k = npend[tr];
          if (k >= uint32_t(K)) {
            ovf = true;
            continue;
          }
          pend0[int64_t(tr) * K + k] =
              (uint64_t(t) << 17) | (uint64_t((w >> 16) & 1u) << 16) | uint64_t(gpos[w & 0xffffu]);
          npend[tr] = k + 1;
        }
      }
      wave_sync();
    }

    // ---- outputs
    const uint32_t T = group_max<PWL>(real ? t_last : 0u);
    const uint64_t wcap = __ballot(real && capr >= 0 && peak > capr);
    const uint64_t wovf = __ballot(ovf);
    const bool gcap = group_bits<PWL>(wcap, grp) != 0;
    const bool govf = group_bits<PWL>(wovf, grp) != 0;
    if (has) {
      if (govf && a.retry) {
        if (r == 0) a.retry[atomicAdd(a.retry_count, 1u)] = cand;
      } else if (govf) {      // cannot happen with inboxes as large as a rank
        if (real) {
          a.out_bub[cand * P + r] = -1;
          a.out_peak[cand * P + r] = -1;
        }
        if (r == 0) {
          a.out_ms[cand] = -1;
          a.out_flags[cand] = DIP_FLAG_INVALID;
        }
      } else {
        if (real) {
          a.out_bub[cand * P + r] = stuck ? -1 : int32_t(T) - a.busy[r];
          a.out_peak[cand * P + r] = peak;
        }
        if (r == 0) {
          a.out_ms[cand] = stuck ? -1 : int32_t(T);
          a.out_flags[cand] = uint8_t((stuck ? DIP_FLAG_DEADLOCK : 0u) | (gcap ? DIP_FLAG_CAP : 0u));
        }
      }
    }
    wave_sync();
  }
}

namespace {

template <int PWL>
const void *ptr_nw(int nw) {
  switch (nw) {
    case 1: return reinterpret_cast<const void *>(&greedy_kernel<PWL, 1>);
    case 2: return reinterpret_cast<const void *>(&greedy_kernel<PWL, 2>);
    case 4: return reinterpret_cast<const void *>(&greedy_kernel<PWL, 4>);
    case 8: return reinterpret_cast<const void *>(&greedy_kernel<PWL, 8>);
    default: return nullptr;
  }
}

template <int PWL>
hipError_t launch_nw(int nw, int blocks, int wpb, size_t lds, hipStream_t s, const GreedyArgs &a) {
  const dim3 grid(blocks), block(wpb * kWave);
  switch (nw) {
    case 1: hipLaunchKernelGGL((greedy_kernel<PWL, 1>), grid, block, lds, s, a); break;
    case 2: hipLaunchKernelGGL((greedy_kernel<PWL, 2>), grid, block, lds, s, a); break;
    case 4: hipLaunchKernelGGL((greedy_kernel<PWL, 4>), grid, block, lds, s, a); break;
    case 8: hipLaunchKernelGGL((greedy_kernel<PWL, 8>), grid, block, lds, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

const void *greedy_kernel_ptr(int pwl, int nw) {
  switch (pwl) {
    case 2: return ptr_nw<2>(nw);
    case 3: return ptr_nw<3>(nw);
    case 4: return ptr_nw<4>(nw);
    case 5: return ptr_nw<5>(nw);
    case 6: return ptr_nw<6>(nw);
    default: return nullptr;
  }
}

hipError_t launch_greedy(int pwl, int nw, int blocks, int wpb, size_t lds, hipStream_t s,
                         const GreedyArgs &a) {
  switch (pwl) {
    case 2: return launch_nw<2>(nw, blocks, wpb, lds, s, a);
    case 3: return launch_nw<3>(nw, blocks, wpb, lds, s, a);
    case 4: return launch_nw<4>(nw, blocks, wpb, lds, s, a);
    case 5: return launch_nw<5>(nw, blocks, wpb, lds, s, a);
    case 6: return launch_nw<6>(nw, blocks, wpb, lds, s, a);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace dipsim
