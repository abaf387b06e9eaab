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
//   E      bitmap (registers) of queued stages with t_start < t_last (and the
//          stages without predecessors while t_last is 0);
//   inbox  two rings (LDS), forward and backward, of the other queued
//          stages, sorted by (t_start, position): a ring's front is its
//          kind's least t_start and, among equal ones, its best priority.
// Lanes touch only their own bitmaps; the committing lane inserts the stages
// its commit completes into the target ranks' inboxes, and each lane moves
// the entries that came due into E at the start of the next round.  A group min over the
// lanes' t_min picks the committing rank.  An inbox that fills up sends the
// candidate to a list that a second launch, with inboxes as large as a rank's
// stage count of that kind, simulates again; where such inboxes do not fit in
// LDS, that launch keeps them in device memory (GRING), one region per
// resident candidate slot.
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
  __device__ __forceinline__ void clear(uint32_t p) {
    const uint32_t k = p >> 6;
    const uint64_t b = ~(uint64_t(1) << (p & 63u));
#pragma unroll
    for (int i = 0; i < NW; ++i) w[i] &= uint32_t(i) == k ? b : ~uint64_t(0);
  }
};

// lowest position in a, kNoPos if empty
template <int NW>
__device__ __forceinline__ uint32_t first_in(const Bits<NW> &a) {
  uint32_t r = kNoPos;
#pragma unroll
  for (int i = NW - 1; i >= 0; --i)
    if (a.w[i] != 0) r = uint32_t(i) * 64u + uint32_t(__builtin_ctzll(a.w[i]));
  return r;
}

// sets position p in f (kind 0) or b (kind 1) without branching
template <int NW>
__device__ __forceinline__ void set_kind(Bits<NW> &f, Bits<NW> &b, uint32_t kind, uint32_t p) {
  const uint32_t k = p >> 6;
  const uint64_t bit = uint64_t(1) << (p & 63u);
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const uint64_t m = uint32_t(i) == k ? bit : uint64_t(0);
    f.w[i] |= kind ? uint64_t(0) : m;
    b.w[i] |= kind ? m : uint64_t(0);
  }
}

// The two E sets of one rank (forward, backward).  Up to 16 words a set they
// live in registers; 32-word sets (every set or clear would touch every word
// through selects) live in the lane's own LDS words, with a register mask of
// the words that are not zero, so that a set, a clear and the first
// position each take one or two LDS accesses.
template <int NW, bool IN_LDS = (NW >= 32)>
struct EPair {
  Bits<NW> f, b;
  __device__ __forceinline__ void init(uint64_t *) {
    f.zero();
    b.zero();
  }
  __device__ __forceinline__ void set(uint32_t kind, uint32_t p) { set_kind(f, b, kind, p); }
  // clears position p of a kind; the kind's new first position
  __device__ __forceinline__ uint32_t clear_first(uint32_t kind, uint32_t p) {
    if (kind) {
      b.clear(p);
      return first_in(b);
    }
    f.clear(p);
    return first_in(f);
  }
  __device__ __forceinline__ uint32_t first(uint32_t kind) const { return first_in(kind ? b : f); }
};

template <int NW>
struct EPair<NW, true> {
  static_assert(NW <= 32, "one summary bit per word");
  uint64_t *w;        // [2][NW] this lane's words: forward, then backward
  uint32_t nz[2];     // words that are not zero, per kind
  __device__ __forceinline__ void init(uint64_t *words) {
    w = words;
#pragma unroll
    for (int i = 0; i < 2 * NW; ++i) w[i] = 0;
    nz[0] = nz[1] = 0;
  }
  __device__ __forceinline__ void set(uint32_t kind, uint32_t p) {
    const uint32_t k = p >> 6;
    __hip_atomic_fetch_or(w + kind * NW + k, uint64_t(1) << (p & 63u), __ATOMIC_RELAXED,
                          __HIP_MEMORY_SCOPE_WAVEFRONT);
    nz[kind] |= 1u << k;
  }
  __device__ __forceinline__ uint32_t first(uint32_t kind) const {
    if (nz[kind] == 0) return kNoPos;
    const uint32_t k = uint32_t(__builtin_ctz(nz[kind]));
    return k * 64u + uint32_t(__builtin_ctzll(w[kind * NW + k]));
  }
  __device__ __forceinline__ uint32_t clear_first(uint32_t kind, uint32_t p) {
    const uint32_t k = p >> 6;
    const uint64_t bit = uint64_t(1) << (p & 63u);
    const uint64_t old = __hip_atomic_fetch_and(w + kind * NW + k, ~bit, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_WAVEFRONT);
    if ((old & ~bit) == 0) nz[kind] &= ~(1u << k);
    return first(kind);
  }
};

template <int CTRL>
__device__ __forceinline__ uint32_t dpp(uint32_t v) {
  return uint32_t(__builtin_amdgcn_update_dpp(0, int(v), CTRL, 0xf, 0xf, false));
}

// min / max over the 2^PWL lanes of a group: quad permutations, then the
// half-row and row mirrors (each lane meets the other half), then shuffles
template <int PWL, bool MAX>
__device__ __forceinline__ uint32_t group_reduce(uint32_t v) {
  auto op = [](uint32_t x, uint32_t y) { return MAX ? max(x, y) : min(x, y); };
  if constexpr (PWL >= 1) v = op(v, dpp<0xb1>(v));    // quad_perm [1,0,3,2]
  if constexpr (PWL >= 2) v = op(v, dpp<0x4e>(v));    // quad_perm [2,3,0,1]
  if constexpr (PWL >= 3) v = op(v, dpp<0x141>(v));   // row_half_mirror
  if constexpr (PWL >= 4) v = op(v, dpp<0x140>(v));   // row_mirror
  if constexpr (PWL >= 5) v = op(v, uint32_t(__shfl_xor(int(v), 16)));
  if constexpr (PWL >= 6) v = op(v, uint32_t(__shfl_xor(int(v), 32)));
  return v;
}
template <int PWL>
__device__ __forceinline__ uint32_t group_min(uint32_t v) { return group_reduce<PWL, false>(v); }
template <int PWL>
__device__ __forceinline__ uint32_t group_max(uint32_t v) { return group_reduce<PWL, true>(v); }

// Orders the LDS accesses of the wave's lanes around this point without
// waiting for its global stores.
__device__ __forceinline__ void lds_sync() {
  lds_wait();
  __builtin_amdgcn_wave_barrier();
}

// ranking key: priority, then lower caller index first
__device__ __forceinline__ uint64_t rank_key(int32_t prio, uint32_t caller) {
  return (uint64_t(uint32_t(prio) ^ 0x80000000u) << 32) | uint64_t(0xffffu - caller);
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

template <int PWL, int NW, bool GRING>
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
  // ... then the inboxes: per rank a forward ring and a backward ring of K
  // entries each (and one spare entry); per lane (padding lanes included) a
  // word {head, count << 16} per kind
  // rank stride 2K + 1 entries, so that the lanes' rings start in different banks
  const int64_t rstride = 2 * int64_t(K) + 1;
  uint64_t *ring0;
  if constexpr (GRING)
    ring0 = a.gring + ((int64_t(blockIdx.x) * a.wpb + wave) * GW + grp) * P * rstride;
  else
    ring0 = reinterpret_cast<uint64_t *>(cb + a.off_pend);
  uint64_t *ringF = ring0 + int64_t(r < P ? r : 0) * rstride;
  uint64_t *ringB = ringF + K;
  uint32_t *hcw = reinterpret_cast<uint32_t *>(cb + a.off_npend);
  uint32_t *jtab = reinterpret_cast<uint32_t *>(cb + a.off_join);
  uint16_t *gpos = reinterpret_cast<uint16_t *>(cb + a.off_gpos);
  uint16_t *ord = reinterpret_cast<uint16_t *>(cb + a.off_ord);
  uint16_t *grk = reinterpret_cast<uint16_t *>(cb + a.off_grk);
  // wide E sets: each lane's 2 NW words at the end of its candidate's region
  uint64_t *ebits = reinterpret_cast<uint64_t *>(cb + a.cand_bytes) - int64_t(PW - r) * 2 * NW;

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
      // rank of every group among all groups and among its kind, eight of
      // this lane's groups against each group in turn
      constexpr int B = 8;
      for (int g0 = r; g0 < G; g0 += B * PW) {
        uint64_t kg[B];
        uint32_t nf[B], nb[B];
#pragma unroll
        for (int t = 0; t < B; ++t) {
          const int g = g0 + t * PW;
          kg[t] = g < G ? rank_key(prio[g], meta[g]) : ~uint64_t(0);
          nf[t] = nb[t] = 0;
        }
        for (int h = 0; h < GF; ++h) {
          const uint64_t kh = rank_key(prio[h], meta[h]);
#pragma unroll
          for (int t = 0; t < B; ++t) nf[t] += kh > kg[t] ? 1u : 0u;
        }
        for (int h = GF; h < G; ++h) {
          const uint64_t kh = rank_key(prio[h], meta[h]);
#pragma unroll
          for (int t = 0; t < B; ++t) nb[t] += kh > kg[t] ? 1u : 0u;
        }
#pragma unroll
        for (int t = 0; t < B; ++t) {
          const int g = g0 + t * PW;
          if (g < G) {
            const bool fg = g < GF;
            const uint32_t same = fg ? nf[t] : nb[t];
            gpos[g] = uint16_t(same);
            const int at = fg ? int(same) : GF + int(same);
            ord[at] = uint16_t(g);
            grk[at] = uint16_t(nf[t] + nb[t]);
          }
        }
      }
    }
    wave_sync();
    if (has)
      for (int j = r; j < 2 * a.J; j += PW) jtab[j] = 0;
    hcw[2 * r] = 0;
    hcw[2 * r + 1] = 0;
    // E: queued stages with t_start < t_last (and the stages without
    // predecessors while t_last is still 0, their t_start); a stage with
    // t_start >= t_last waits in its kind's inbox
    EPair<NW> e;
    e.init(ebits);
    if (real) {
      const int32_t *src_list = a.src + P + 1;
      for (int s = a.src[r]; s < a.src[r + 1]; ++s) {
        const int g = src_list[s];
        e.set(g < GF ? 0u : 1u, gpos[g]);
      }
    }
    // first (best) position in each E, kept up to date: an entry moving in
    // can only lower it; the commit that takes it looks again
    uint32_t eF1 = e.first(0u), eB1 = e.first(1u);
    wave_sync();

    uint32_t t_last = 0, last_kind = 0, n_emit = 0;
    uint32_t rec_key = kNever;
    int4 q0 = make_int4(0, 0, 0, 0), q1 = q0;
    int32_t live = 0, peak = 0;
    bool ovf = false, stuck = false;
    const int32_t capr = real ? a.cap[r] : -1;
    const int64_t row = real ? cand * a.stride + a.rank_off[r] : 0;
    const uint32_t n_own = real ? uint32_t(a.rank_off[r + 1] - a.rank_off[r]) : 0u;
    const uint32_t mask = uint32_t(K) - 1u;

    for (int it = 0; it < a.n_rounds; ++it) {
      // ---- 1. inboxes: entries that came due move into E; the fronts are
      // each kind's least t_start (best position among equal ones)
      const uint32_t cF0 = hcw[2 * r], cB0 = hcw[2 * r + 1];
      uint32_t hF = cF0 & 0xffffu, nF = cF0 >> 16, hB = cB0 & 0xffffu, nB = cB0 >> 16;
      uint64_t frF = ~uint64_t(0), frB = ~uint64_t(0);
      for (; nF > 0; ++hF, --nF) {
        frF = ringF[hF & mask];
        if (uint32_t(frF >> 17) >= t_last) break;
        const uint32_t p = uint32_t(frF >> 1) & 0xffffu;
        e.set(0u, p);
        eF1 = min(eF1, p);
        frF = ~uint64_t(0);
      }
      for (; nB > 0; ++hB, --nB) {
        frB = ringB[hB & mask];
        if (uint32_t(frB >> 17) >= t_last) break;
        const uint32_t p = uint32_t(frB >> 1) & 0xffffu;
        e.set(1u, p);
        eB1 = min(eB1, p);
        frB = ~uint64_t(0);
      }
      const uint32_t cF = (hF & 0xffffu) | (nF << 16), cB = (hB & 0xffffu) | (nB << 16);
      if (cF != cF0) hcw[2 * r] = cF;
      if (cB != cB0) hcw[2 * r + 1] = cB;
      const uint32_t pmF = nF ? uint32_t(frF >> 17) : kNever, pmB = nB ? uint32_t(frB >> 17) : kNever;
      const uint32_t ppF = nF ? uint32_t(frF >> 1) & 0xffffu : kNoPos;
      const uint32_t ppB = nB ? uint32_t(frB >> 1) & 0xffffu : kNoPos;

      // ---- 2. this rank's choice
      const uint32_t fF = eF1, fB = eB1;
      const bool xF = fF != kNoPos && t_last > 0, xB = fB != kNoPos && t_last > 0;
      // the best stage of each kind able to start at tau: E's first (E is
      // non-empty only when tau == t_last) or the inbox front if due then
      auto decide = [&](bool fw) {
        Choice c;
        const uint32_t eF_ = fw ? fF : kNoPos, pF = fw ? pmF : kNever;
        const bool anyE = eF_ != kNoPos || fB != kNoPos;
        c.tau = anyE ? t_last : min(pF, pmB);
        const bool inF = pF == c.tau && ppF < eF_;
        const bool inB = pmB == c.tau && ppB < fB;
        const uint32_t bF = inF ? ppF : eF_, bB = inB ? ppB : fB;
        const uint32_t gF = grk[bF < uint32_t(GF) ? bF : 0u];
        const uint32_t gB = grk[bB < uint32_t(G - GF) ? GF + bB : 0u];
        const bool alt = fw && xF && xB;                           // 1F1B
        const uint32_t k = bF == kNoPos ? 1u : (bB == kNoPos ? 0u : (gF < gB ? 0u : 1u));
        c.kind = alt ? (last_kind ^ 1u) : k;
        c.pos = c.kind ? bB : bF;
        c.slot = (c.kind ? inB : inF) ? 1u : 0u;    // 1: the kind's inbox front
        return c;
      };
      // the record of a choice: {cost, act, local id | successors << 16,
      // second successor's index}, {first successor}; kept while the choice
      // stays the same
      auto fetch = [&](const Choice &c) {
        const uint32_t k = (c.kind << 16) | c.pos;
        if (k != rec_key) {
          const int4 *rp = a.rec + (int64_t(ord[c.kind ? GF + c.pos : c.pos]) * P + r) * 2;
          q0 = rp[0];
          q1 = rp[1];
          rec_key = k;
        }
      };
      const Choice ce = decide(true);
      Choice cd = ce;
      if (ce.pos != kNoPos) {
        fetch(ce);
        if (a.has_cap && ce.kind == 0 && capr >= 0 && live + q0.y > capr) {
          cd = decide(false);                   // forward queue disabled
          if (cd.pos != kNoPos) fetch(cd);
        }
      }

      // ---- 3. the rank with the smallest t_min commits
      const uint32_t key_d = cd.pos != kNoPos ? cd.tau : kNever;
      uint32_t m = group_min<PWL>(key_d);
      uint32_t key = key_d;
      bool forced = false;
      if (__any(has && m == kNever)) {
        const uint32_t key_e = ce.pos != kNoPos ? ce.tau : kNever;
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
        if (forced) fetch(c);
        const uint32_t end = c.tau + uint32_t(q0.x);
        if (c.slot == 0) {
          if (c.kind)
            eB1 = e.clear_first(1u, c.pos);
          else
            eF1 = e.clear_first(0u, c.pos);
        } else {
          // the kind's inbox front: one step on
          const uint32_t hw = hcw[2 * r + c.kind];
          hcw[2 * r + c.kind] = (((hw & 0xffffu) + 1u) & 0xffffu) | ((hw >> 16) - 1u) << 16;
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
        // successors whose last predecessor this was join the target inboxes,
        // kept sorted by (t_start, position)
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
          const uint32_t tr = (w >> 17) & 63u, tk = (w >> 16) & 1u;
          const uint32_t h = hcw[2 * tr + tk];
          const uint32_t head = h & 0xffffu, n = h >> 16;
          if (n >= uint32_t(K)) {
            ovf = true;
            continue;
          }
          uint64_t *rt = ring0 + int64_t(tr) * rstride + (tk ? K : 0);
          const uint64_t x = (uint64_t(t) << 17) | (uint64_t(gpos[w & 0xffffu]) << 1) | uint64_t(tk);
          uint32_t i = n;
          for (; i > 0; --i) {
            const uint64_t prev = rt[(head + i - 1) & mask];
            if (prev <= x) break;
            rt[(head + i) & mask] = prev;
          }
          rt[(head + i) & mask] = x;
          hcw[2 * tr + tk] = h + (1u << 16);
        }
      }
      if constexpr (GRING)
        wave_sync();      // the inboxes' device-memory writes too
      else
        lds_sync();
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

template <int PWL, bool GRING>
const void *ptr_nw(int nw) {
  switch (nw) {
    case 1: return reinterpret_cast<const void *>(&greedy_kernel<PWL, 1, GRING>);
    case 2: return reinterpret_cast<const void *>(&greedy_kernel<PWL, 2, GRING>);
    case 4: return reinterpret_cast<const void *>(&greedy_kernel<PWL, 4, GRING>);
    case 8: return reinterpret_cast<const void *>(&greedy_kernel<PWL, 8, GRING>);
    case 16: return reinterpret_cast<const void *>(&greedy_kernel<PWL, 16, GRING>);
    case 32: return reinterpret_cast<const void *>(&greedy_kernel<PWL, 32, GRING>);
    default: return nullptr;
  }
}

template <int PWL>
const void *ptr_pwl(int nw, bool gring) {
  return gring ? ptr_nw<PWL, true>(nw) : ptr_nw<PWL, false>(nw);
}

}  // namespace

__global__ void zero_words_kernel(uint32_t *p, int n) {
  if (int(threadIdx.x) < n) p[threadIdx.x] = 0u;
}

hipError_t launch_zero_words(uint32_t *p, int n, hipStream_t s) {
  zero_words_kernel<<<1, 64, 0, s>>>(p, n);
  return hipGetLastError();
}

const void *greedy_kernel_ptr(int pwl, int nw, bool gring) {
  switch (pwl) {
    case 2: return ptr_pwl<2>(nw, gring);
    case 3: return ptr_pwl<3>(nw, gring);
    case 4: return ptr_pwl<4>(nw, gring);
    case 5: return ptr_pwl<5>(nw, gring);
    case 6: return ptr_pwl<6>(nw, gring);
    default: return nullptr;
  }
}

hipError_t launch_greedy(int pwl, int nw, bool gring, int blocks, int wpb, size_t lds,
                         hipStream_t s, const GreedyArgs &a) {
  const void *k = greedy_kernel_ptr(pwl, nw, gring);
  if (!k) return hipErrorInvalidValue;
  void *args[] = {const_cast<GreedyArgs *>(&a)};
  return hipLaunchKernel(k, dim3(unsigned(blocks)), dim3(unsigned(wpb * kWave)), args, lds, s);
}

}  // namespace dipsim
