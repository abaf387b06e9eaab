// kern_memopt.hip -- per-layer memory optimisation (DIP, arXiv 2504.14145,
// Sec. 5.3) of many candidate schedules at once.
//
// For every (candidate schedule, rank), each stage pair of the rank takes one
// of its memory candidates (time ascending, memory strictly descending) so
// that the live memory at every forward start stays within the rank's cap,
// with the least total time (Sec. 5.3's ILP, solved to within 5 %):
//   1. the greedy warm start: all pairs on their fastest candidate; while the
//      most loaded checkpoint (lowest index among equal loads) is over the
//      cap, move the live pair with the least added time per freed memory
//      unit (dt_a * dm_b < dt_b * dm_a, lowest pair index on ties) to its
//      next candidate; give up when no live pair can move;
//   2. an improvement pass: pairs in index order each go back to the fastest
//      candidate that keeps every checkpoint it is live at within the cap,
//      until a pass changes nothing;
//   3. a depth-first branch and bound from there, pairs in the order of their
//      forward starts, candidates fastest first: a placement whose own
//      checkpoint exceeds the cap is dropped, a node whose placed time plus
//      the unplaced pairs' fastest times, times 1.05, reaches the incumbent
//      is cut with its slower siblings, and a complete placement below the
//      incumbent replaces it.  A finished search proves the incumbent within
//      5 % of the optimum (status 1); after bb_nodes placements examined, or
//      on ranks of more than 512 pairs (no search), status 3;
//   4. when the search stopped early, a certificate from the Lagrangian
//      relaxation of the checkpoint constraints (the dual side of the ILP's
//      LP bound), by exact integer subgradient steps: status 1 once 1.05
//      times the bound reaches the incumbent.
// Pair i is live at pair k's forward start when its forward comes no later
// and its backward no earlier in the rank's order.
//
// The comparison of moves depends on the candidates only, not on the
// schedule, so the host ranks every move of a rank once (exact 128-bit cross
// products) and hands each a 32-bit key: the least key is the greedy's
// choice.  Two kernels:
//   memopt_wave_kernel  a wave per (schedule, rank), lane j owning pairs
//                       j, j + 64, ... in registers; the most loaded
//                       checkpoint and the best move are one DPP wave
//                       reduction each; a block holds schedules of one rank
//                       and shares that rank's move tables in LDS.  In the
//                       search, lane j also holds the stack entries of
//                       depths j, j + 64, ... (candidate, placed time,
//                       fastest time of the rest), and a checkpoint's load
//                       is one wave sum over the placed pairs.
//   memopt_kernel       a thread per (schedule, rank), for ranks of more
//                       than 512 pairs (steps 1 and 2); its state sits in
//                       LDS, element-major across the block.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "dev_util.h"
#include "internal.h"

namespace dipsim {

namespace {

// the Lagrangian certificate: subgradient steps, fraction bits of the
// multipliers (at most), and the magnitude every value stays below
constexpr int kMemoptLagrIters = 200;
constexpr int kMemoptLagrF = 20;
constexpr int kMemoptLagrLimitBits = 60;
constexpr int kMemoptLagrHalve = 24;   // steps between halvings of the step size

// bits of a non-negative value (0 for 0)
__device__ __forceinline__ int bits64(int64_t x) { return x ? 64 - __clzll(x) : 0; }

__device__ __forceinline__ void lds_sync_wave() {
  lds_wait();
  __builtin_amdgcn_wave_barrier();
}

// min / max of one value over the 64 lanes of a wave, read out of lane 63:
// the row reduction of dpp_row, then the row broadcasts (lane 15 of each row
// into the next row, lane 31 into rows 2 and 3), rows outside the mask
// keeping their value (the identity as the old value)
template <bool MAX>
__device__ __forceinline__ uint32_t wave_reduce63(uint32_t v) {
  auto op = [](uint32_t x, uint32_t y) { return MAX ? max(x, y) : min(x, y); };
  constexpr int kId = MAX ? 0 : -1;
  v = op(v, dpp_row<0xb1>(v));    // quad_perm [1,0,3,2]
  v = op(v, dpp_row<0x4e>(v));    // quad_perm [2,3,0,1]
  v = op(v, dpp_row<0x141>(v));   // row_half_mirror
  v = op(v, dpp_row<0x140>(v));   // row_mirror
  v = op(v, uint32_t(__builtin_amdgcn_update_dpp(kId, int(v), 0x142, 0xa, 0xf, false)));  // row_bcast:15
  v = op(v, uint32_t(__builtin_amdgcn_update_dpp(kId, int(v), 0x143, 0xc, 0xf, false)));  // row_bcast:31
  return uint32_t(__builtin_amdgcn_readlane(int(v), 63));
}

// sum of one value over the 64 lanes of a wave (wrapping), the same in every lane
__device__ __forceinline__ int32_t wave_sum(int32_t v) {
  v += int32_t(dpp_row<0xb1>(uint32_t(v)));    // quad_perm [1,0,3,2]
  v += int32_t(dpp_row<0x4e>(uint32_t(v)));    // quad_perm [2,3,0,1]
  v += int32_t(dpp_row<0x141>(uint32_t(v)));   // row_half_mirror
  v += int32_t(dpp_row<0x140>(uint32_t(v)));   // row_mirror
  return __builtin_amdgcn_readlane(v, 0) + __builtin_amdgcn_readlane(v, 16) +
         __builtin_amdgcn_readlane(v, 32) + __builtin_amdgcn_readlane(v, 48);
}

__device__ __forceinline__ int64_t wave_sum64(int64_t v) {
#pragma unroll
  for (int s = 1; s < 64; s <<= 1)
    v += (int64_t(__shfl_xor(int(v >> 32), s)) << 32) | uint32_t(__shfl_xor(int(uint32_t(v)), s));
  return v;
}

__device__ __forceinline__ void write_out(const MemoptArgs &a, int64_t o, int64_t t, int32_t pk,
                                          uint8_t st) {
  a.out_time[o] = t;
  a.out_peak[o] = pk;
  a.out_status[o] = st;
}

// ---------------------------------------------------------------- thread per problem

__global__ __launch_bounds__(256) void memopt_kernel(MemoptArgs a) {
  extern __shared__ __align__(16) unsigned char sh[];
  const int64_t id = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (id >= a.n_cand * a.P) return;
  const int64_t c = id / a.P;
  const int r = int(id % a.P);
  const int32_t np = a.pair_off[r + 1] - a.pair_off[r];
  const int32_t pbase = a.pair_off[r];
  // element-major arrays, [element][thread], so that the lanes of a wave
  // touch consecutive words
  const int T = blockDim.x, t = threadIdx.x;
  const int64_t m = a.max_pairs;
  int32_t *load_ = reinterpret_cast<int32_t *>(sh) + t;
  uint16_t *pf_ = reinterpret_cast<uint16_t *>(sh + 4 * m * T) + t;
  uint16_t *pb_ = pf_ + m * T;
  uint8_t *cur_ = reinterpret_cast<uint8_t *>(sh + 8 * m * T) + t;
#define load(i) load_[int64_t(i) * T]
#define pf(i) pf_[int64_t(i) * T]
#define pb(i) pb_[int64_t(i) * T]
#define cur(i) cur_[int64_t(i) * T]
  for (int32_t i = 0; i < np; ++i) {
    pf(i) = 0xffffu;
    pb(i) = 0xffffu;
    cur(i) = 0;
  }
  // positions of each pair's forward and backward in the rank's order
  const int32_t base = a.rank_off[r], nr = a.rank_off[r + 1] - base;
  const int16_t *row = a.orders + c * a.stride + base;
  bool valid = true;
  for (int32_t p = 0; p < nr; ++p) {
    const int32_t lid = row[p];
    if (lid < 0 || lid >= nr) {
      valid = false;
      break;
    }
    const uint32_t w = uint32_t(a.lid_pair[base + lid]);
    uint16_t *slot = ((w >> 31) ? pb_ : pf_) + int64_t(w & 0x7fffffffu) * T;
    if (*slot != 0xffffu) {
      valid = false;
      break;
    }
    *slot = uint16_t(p);
  }
  const int64_t o = c * a.P + r;
  if (!valid) {
    write_out(a, o, -1, -1, 2);
    return;
  }
  const int64_t *ct = a.cand_time + int64_t(pbase) * kMemoptMaxCands;
  const int32_t *cm = a.cand_mem + int64_t(pbase) * kMemoptMaxCands;
  const uint32_t *mk = a.move_key + int64_t(pbase) * kMemoptMaxCands;
  const int32_t *md = a.move_dm + int64_t(pbase) * kMemoptMaxCands;
  for (int32_t k = 0; k < np; ++k) {
    int32_t s = 0;
    for (int32_t i = 0; i < np; ++i)
      if (pf(i) <= pf(k) && pf(k) <= pb(i)) s += cm[i * kMemoptMaxCands];
    load(k) = s;
  }
  const int32_t cap = a.cap[r];
  bool ok = true;
  if (cap >= 0) {
    for (;;) {
      int32_t kk = 0;
      for (int32_t k = 1; k < np; ++k)
        if (load(k) > load(kk)) kk = k;
      if (np == 0 || load(kk) <= cap) break;
      uint32_t best = kMemoptNoMove;
      for (int32_t i = 0; i < np; ++i)
        if (pf(i) <= pf(kk) && pf(kk) <= pb(i)) best = min(best, mk[i * kMemoptMaxCands + cur(i)]);
      if (best == kMemoptNoMove) {
        ok = false;
        break;
      }
      const int32_t bi = int32_t(best & ((1u << kMemoptPairBits) - 1));
      const int32_t dm = md[bi * kMemoptMaxCands + cur(bi)];
      cur(bi) += 1;
      for (int32_t k = 0; k < np; ++k)
        if (pf(bi) <= pf(k) && pf(k) <= pb(bi)) load(k) -= dm;
    }
  }
  uint8_t status = ok ? 1 : 0;
  if (ok && cap >= 0 && np > 0) {
    // step 2; no search on ranks this large
    for (bool changed = true; changed;) {
      changed = false;
      for (int32_t i = 0; i < np; ++i) {
        int32_t top = INT32_MIN;
        for (int32_t k = 0; k < np; ++k)
          if (pf(i) <= pf(k) && pf(k) <= pb(i)) top = max(top, load(k));
        const int32_t ci = cur(i);
        const int32_t mc = cm[i * kMemoptMaxCands + ci];
        for (int32_t j = 0; j < ci; ++j) {
          const int32_t add = cm[i * kMemoptMaxCands + j] - mc;
          if (int64_t(top) + add <= int64_t(cap)) {
            for (int32_t k = 0; k < np; ++k)
              if (pf(i) <= pf(k) && pf(k) <= pb(i)) load(k) += add;
            cur(i) = uint8_t(j);
            changed = true;
            break;
          }
        }
      }
    }
    status = 3;
  }
  int64_t total = 0;
  int32_t peak = 0;
  for (int32_t i = 0; i < np; ++i) {
    total += ct[i * kMemoptMaxCands + cur(i)];
    peak = max(peak, load(i));
    if (a.out_choice) a.out_choice[c * a.n_pairs + pbase + i] = cur(i);
  }
  write_out(a, o, total, peak, status);
}
#undef load
#undef pf
#undef pb
#undef cur

// ---------------------------------------------------------------- wave per problem

template <int PPL>
__global__ __launch_bounds__(256) void memopt_wave_kernel(MemoptArgs a) {
  extern __shared__ __align__(16) unsigned char sh[];
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int r = blockIdx.y;
  const int64_t c = int64_t(blockIdx.x) * nw + wv;
  const int32_t pbase = a.pair_off[r];
  const int32_t np = a.pair_off[r + 1] - pbase;
  const int64_t mp = a.max_pairs;
  // the rank's tables, shared by the block: move keys and freed memory
  // [pair][candidate], memory of the fastest candidate [pair]
  uint32_t *tkey = reinterpret_cast<uint32_t *>(sh);
  int32_t *tdm = reinterpret_cast<int32_t *>(sh + 32 * mp);
  int32_t *tm0 = reinterpret_cast<int32_t *>(sh + 64 * mp);
  // this wave's positions of each pair's forward and backward, its pairs in
  // the order of their forwards, and the final choice of each pair
  uint16_t *pfa = reinterpret_cast<uint16_t *>(sh + 68 * mp) + int64_t(wv) * 3 * mp;
  uint16_t *pba = pfa + mp;
  uint16_t *orda = pba + mp;
  uint8_t *sela = sh + 68 * mp + 6 * mp * nw + int64_t(wv) * mp;
  // the certificate's arrays over the checkpoints in forward order: prefix
  // sums of the multipliers, memory differences, multipliers
  int64_t *lps = reinterpret_cast<int64_t *>(sh + ((68 + 7 * nw) * mp + 7) / 8 * 8) +
                 int64_t(wv) * 3 * (mp + 1);
  {
    const uint32_t *gk = a.move_key + int64_t(pbase) * kMemoptMaxCands;
    const int32_t *gd = a.move_dm + int64_t(pbase) * kMemoptMaxCands;
    const int32_t *gm = a.cand_mem + int64_t(pbase) * kMemoptMaxCands;
    for (int32_t x = threadIdx.x; x < np * kMemoptMaxCands; x += blockDim.x) {
      tkey[x] = gk[x];
      tdm[x] = gd[x];
    }
    for (int32_t i = threadIdx.x; i < np; i += blockDim.x) tm0[i] = gm[i * kMemoptMaxCands];
  }
  __syncthreads();
  if (c >= a.n_cand) return;                        // whole waves, after the last barrier
  for (int32_t i = lane; i < np; i += 64) {
    pfa[i] = 0xffffu;
    pba[i] = 0xffffu;
  }
  lds_sync_wave();
  const int32_t base = a.rank_off[r], nr = a.rank_off[r + 1] - base;
  const int16_t *row = a.orders + c * a.stride + base;
  bool bad = false;
  for (int32_t p = lane; p < nr; p += 64) {
    const int32_t lid = row[p];
    if (lid < 0 || lid >= nr) {
      bad = true;
      continue;
    }
    const uint32_t w = uint32_t(a.lid_pair[base + lid]);
    ((w >> 31) ? pba : pfa)[w & 0x7fffffffu] = uint16_t(p);
  }
  lds_sync_wave();
  // every rank op is one end of one pair, so with all nr ids in range a
  // repeated id leaves some end unfilled
  for (int32_t i = lane; i < np; i += 64)
    if (pfa[i] == 0xffffu || pba[i] == 0xffffu) bad = true;
  const int64_t o = c * a.P + r;
  if (__any(bad)) {
    if (lane == 0) write_out(a, o, -1, -1, 2);
    return;
  }
  // own pairs: positions, current candidate, its next move (key, freed
  // memory), load of the own checkpoint under the fastest candidates
  uint32_t pf[PPL], pb[PPL], key[PPL];
  int32_t cur[PPL], dm[PPL], load[PPL];
#pragma unroll
  for (int q = 0; q < PPL; ++q) {
    const int32_t i = lane + 64 * q;
    const bool own = i < np;
    pf[q] = own ? pfa[i] : 0xffffu;
    pb[q] = own ? pba[i] : 0u;
    cur[q] = 0;
    key[q] = own ? tkey[i * kMemoptMaxCands] : kMemoptNoMove;
    dm[q] = own ? tdm[i * kMemoptMaxCands] : 0;
    int32_t s = 0;
    if (own)
      for (int32_t j = 0; j < np; ++j)
        if (pfa[j] <= pf[q] && pf[q] <= pba[j]) s += tm0[j];
    load[q] = s;
  }
  const int32_t cap = a.cap[r];
  bool ok = true;
  if (cap >= 0) {
    for (;;) {
      // most loaded checkpoint (order-preserving unsigned image of the load)
      uint32_t mx = 0;
#pragma unroll
      for (int q = 0; q < PPL; ++q)
        if (lane + 64 * q < np) mx = max(mx, uint32_t(load[q]) ^ 0x80000000u);
      mx = wave_reduce63<true>(mx);
      const int32_t top = int32_t(mx ^ 0x80000000u);
      if (np == 0 || top <= cap) break;
      // its forward position: the lowest pair index holding that load
      uint32_t pfk = 0;
      bool found = false;
#pragma unroll
      for (int q = 0; q < PPL; ++q) {
        const uint64_t b = __ballot(lane + 64 * q < np && load[q] == top);
        if (!found && b) {
          pfk = uint32_t(__builtin_amdgcn_readlane(int(pf[q]), __builtin_ctzll(b)));
          found = true;
        }
      }
      // best move among the pairs live there
      uint32_t m = kMemoptNoMove;
#pragma unroll
      for (int q = 0; q < PPL; ++q)
        if (pf[q] <= pfk && pfk <= pb[q]) m = min(m, key[q]);
      m = wave_reduce63<false>(m);
      if (m == kMemoptNoMove) {
        ok = false;
        break;
      }
      const int32_t bi = int32_t(m & ((1u << kMemoptPairBits) - 1));
      const int qb = bi >> 6, ob = bi & 63;
      // the moved pair's positions from the wave's tables, its freed memory
      // from its owner lane
      const uint32_t spf = pfa[bi], spb = pba[bi];
      int32_t sdm = 0;
#pragma unroll
      for (int q = 0; q < PPL; ++q)
        if (q == qb) sdm = dm[q];
      sdm = __builtin_amdgcn_readlane(sdm, ob);
      // every checkpoint the moved pair is live at drops; its owner steps on
#pragma unroll
      for (int q = 0; q < PPL; ++q) {
        if (spf <= pf[q] && pf[q] <= spb) load[q] -= sdm;
        if (q == qb && lane == ob) {
          const int32_t x = bi * kMemoptMaxCands + ++cur[q];
          key[q] = tkey[x];
          dm[q] = tdm[x];
        }
      }
    }
  }
  const int64_t *ct = a.cand_time + int64_t(pbase) * kMemoptMaxCands;
  const int32_t *cmem = a.cand_mem + int64_t(pbase) * kMemoptMaxCands;
  // the register of slot q of every lane as one value, and its update in one lane
  auto pick = [](const auto (&v)[PPL], int qd) {
    auto x = v[0];
#pragma unroll
    for (int q = 1; q < PPL; ++q)
      if (q == qd) x = v[q];
    return x;
  };
  auto own = [&](int q) { return lane + 64 * q < np; };
  uint8_t status = ok ? 1 : 0;
  if (ok && cap >= 0 && np > 0) {
    // ---- step 2: back to faster candidates where every checkpoint allows
    for (bool changed = true; changed;) {
      changed = false;
      for (int32_t i = 0; i < np; ++i) {
        const uint32_t spf = pfa[i], spb = pba[i];
        uint32_t mx = 0;
#pragma unroll
        for (int q = 0; q < PPL; ++q)
          if (own(q) && spf <= pf[q] && pf[q] <= spb) mx = max(mx, uint32_t(load[q]) ^ 0x80000000u);
        const int64_t top = int32_t(wave_reduce63<true>(mx) ^ 0x80000000u);
        const int qi = i >> 6, li = i & 63;
        const int32_t ci = __builtin_amdgcn_readlane(pick(cur, qi), li);
        const int32_t mc = cmem[i * kMemoptMaxCands + ci];
        int32_t nj = ci;
        for (int32_t j = 0; j < ci; ++j)
          if (top + (cmem[i * kMemoptMaxCands + j] - mc) <= int64_t(cap)) {
            nj = j;
            break;
          }
        if (nj < ci) {
          const int32_t add = cmem[i * kMemoptMaxCands + nj] - mc;
#pragma unroll
          for (int q = 0; q < PPL; ++q) {
            if (own(q) && spf <= pf[q] && pf[q] <= spb) load[q] += add;
            if (q == qi && lane == li) cur[q] = nj;
          }
          changed = true;
        }
      }
    }

    // ---- step 3: branch and bound, pairs by forward position
    // depth of each own pair: the pairs whose forward comes earlier
#pragma unroll
    for (int q = 0; q < PPL; ++q)
      if (own(q)) {
        int32_t dep = 0;
        for (int32_t j = 0; j < np; ++j) dep += pfa[j] < pf[q] ? 1 : 0;
        orda[dep] = uint16_t(lane + 64 * q);
      }
    lds_sync_wave();
    // stack entries of depths lane + 64 q: pair, candidate, placed time
    // above the depth, fastest time of the pairs from the depth on
    int32_t dpair[PPL], dch[PPL];
    int64_t dplaced[PPL], drest[PPL];
    // own pairs: candidate and memory of the current placement, best choice
    int32_t pcur[PPL], pmem[PPL], best[PPL];
#pragma unroll
    for (int q = 0; q < PPL; ++q) {
      dpair[q] = own(q) ? orda[lane + 64 * q] : 0;
      dch[q] = -1;
      dplaced[q] = 0;
      drest[q] = 0;
      pcur[q] = 0;
      pmem[q] = 0;
      best[q] = cur[q];
    }
    {
      int64_t rest = 0;
      for (int32_t d = np - 1; d >= 0; --d) {
        rest += ct[int32_t(orda[d]) * kMemoptMaxCands];
#pragma unroll
        for (int q = 0; q < PPL; ++q)
          if (q == (d >> 6) && lane == (d & 63)) drest[q] = rest;
      }
    }
    int64_t inc = 0;
#pragma unroll
    for (int q = 0; q < PPL; ++q)
      if (own(q)) inc += ct[(lane + 64 * q) * kMemoptMaxCands + cur[q]];
    inc = wave_sum64(inc);
    bool proven = true;
    uint32_t seen = 0;
    int32_t d = 0;
    while (d >= 0) {
      const int qd = d >> 6, ld = d & 63;
      const int32_t i = __builtin_amdgcn_readlane(pick(dpair, qd), ld);
      const int32_t c = __builtin_amdgcn_readlane(pick(dch, qd), ld) + 1;
      // candidate c of pair i exists when the move into it does
      const bool has = c < kMemoptMaxCands && (c == 0 || tkey[i * kMemoptMaxCands + c - 1] != kMemoptNoMove);
      if (!has) {
#pragma unroll
        for (int q = 0; q < PPL; ++q)
          if (q == qd && lane == ld) dch[q] = -1;
        --d;
        continue;
      }
#pragma unroll
      for (int q = 0; q < PPL; ++q)
        if (q == qd && lane == ld) dch[q] = c;
      if (++seen > uint32_t(a.bb_nodes)) {
        proven = false;
        break;
      }
      const int64_t t = ct[i * kMemoptMaxCands + c];
      const int32_t m = cmem[i * kMemoptMaxCands + c];
      // its checkpoint: the placed pairs (forward earlier) still live there
      const uint32_t spf = pfa[i];
      int32_t part = 0;
#pragma unroll
      for (int q = 0; q < PPL; ++q)
        if (own(q) && pf[q] < spf && pb[q] >= spf) part += pmem[q];
      // (a pair whose backward comes before its forward is live nowhere)
      const int64_t own_m = pba[i] >= spf ? int64_t(m) : 0;
      if (own_m + wave_sum(part) > int64_t(cap)) continue;   // a leaner one may fit
      const int64_t f =
          int64_t(uint32_t(__builtin_amdgcn_readlane(int(uint32_t(pick(dplaced, qd))), ld))) |
          (int64_t(__builtin_amdgcn_readlane(int(pick(dplaced, qd) >> 32), ld)) << 32);
      const int64_t f_t = f + t;
      int64_t rest = 0;
      if (d + 1 < np) {
        const int q1 = (d + 1) >> 6, l1 = (d + 1) & 63;
        rest = int64_t(uint32_t(__builtin_amdgcn_readlane(int(uint32_t(pick(drest, q1))), l1))) |
               (int64_t(__builtin_amdgcn_readlane(int(pick(drest, q1) >> 32), l1)) << 32);
      }
      if (__int128(105) * (f_t + rest) >= __int128(100) * inc) {   // cut, with the slower ones
#pragma unroll
        for (int q = 0; q < PPL; ++q)
          if (q == qd && lane == ld) dch[q] = kMemoptMaxCands;
        continue;
      }
      const int qi = i >> 6, li = i & 63;
#pragma unroll
      for (int q = 0; q < PPL; ++q)
        if (q == qi && lane == li) {
          pcur[q] = c;
          pmem[q] = m;
        }
      if (d == np - 1) {   // every pair placed, below the incumbent
        inc = f_t;
#pragma unroll
        for (int q = 0; q < PPL; ++q) best[q] = pcur[q];
        continue;
      }
      const int q1 = (d + 1) >> 6, l1 = (d + 1) & 63;
#pragma unroll
      for (int q = 0; q < PPL; ++q)
        if (q == q1 && lane == l1) dplaced[q] = f_t;
      ++d;
    }
    status = proven ? 1 : 3;
    // the final choice and its checkpoint loads
#pragma unroll
    for (int q = 0; q < PPL; ++q) {
      cur[q] = best[q];
      if (own(q)) sela[lane + 64 * q] = uint8_t(cur[q]);
    }
    lds_sync_wave();
#pragma unroll
    for (int q = 0; q < PPL; ++q) {
      int32_t s = 0;
      if (own(q))
        for (int32_t j = 0; j < np; ++j)
          if (pfa[j] <= pf[q] && pf[q] <= pba[j]) s += cmem[j * kMemoptMaxCands + sela[j]];
      load[q] = s;
    }
    if (!proven) {
      // ---- step 4 (after the final choice, whose loads are set): the
      // Lagrangian certificate.  Multipliers l_k >= 0 (units
      // of 2^-F time per memory unit), one per checkpoint k (pair k's
      // forward start).  Each step: a pair's price is the sum of the
      // multipliers of the checkpoints it is live at; it takes its cheapest
      // candidate under t * 2^F + m * price (the first on ties); the bound
      // (times 2^F) is the sum of those values less cap * sum_k l_k, and
      // proves the incumbent once 1.05 times it reaches the incumbent;
      // otherwise each multiplier moves by g_k * step / 2^b, b the bits of
      // max |g| (the magnitude shifted down, the sign kept; kept in [0,
      // lmax]), g_k being the memory of the taken candidates live at
      // checkpoint k less the cap, step = s0 / 2^(t / 24).  F = min(20, 60 -
      // bits(np * tmax)), lmax = 2^60 / 2^bits(np^2 * max(1, mmax, cap)) and
      // s0 = half the largest (dt << F) / 2^(bits(dm) - 1) over the moves
      // from each pair's fastest candidate (at least 1, at most lmax) keep
      // every value below 2^61, with no division.  A pair is live exactly at the
      // checkpoints whose forward order lies in [its own, the number of
      // forwards not after its backward), so both sums are differences of
      // prefix sums over the checkpoints in forward order, kept in the
      // wave's LDS.  Integer arithmetic: the same values as any other order
      // of summation.
      auto has = [&](int32_t i, int32_t j) {
        return j < kMemoptMaxCands && (j == 0 || tkey[i * kMemoptMaxCands + j - 1] != kMemoptNoMove);
      };
      auto shfl64 = [](int64_t v, int src) {
        return (int64_t(__shfl(int(v >> 32), src)) << 32) | uint32_t(__shfl(int(uint32_t(v)), src));
      };
      auto wave_max64 = [](int64_t v) {
#pragma unroll
        for (int s = 1; s < 64; s <<= 1)
          v = max(v, (int64_t(__shfl_xor(int(v >> 32), s)) << 32) |
                         uint32_t(__shfl_xor(int(uint32_t(v)), s)));
        return v;
      };
      // inclusive prefix sum over the 64 lanes
      auto wave_scan64 = [&](int64_t v) {
#pragma unroll
        for (int s = 1; s < 64; s <<= 1) {
          const int64_t y = shfl64(v, lane >= s ? lane - s : lane);
          if (lane >= s) v += y;
        }
        return v;
      };
      int64_t tmx = 0, mmx = 0, s0 = 0;
#pragma unroll
      for (int q = 0; q < PPL; ++q)
        if (own(q)) {
          const int32_t i = lane + 64 * q;
          for (int32_t j = 0; has(i, j); ++j) {
            tmx = max(tmx, ct[i * kMemoptMaxCands + j]);
            mmx = max(mmx, int64_t(cmem[i * kMemoptMaxCands + j]));
          }
        }
      tmx = wave_max64(tmx);
      mmx = wave_max64(mmx);
      const int F = min(kMemoptLagrF, kMemoptLagrLimitBits - bits64(int64_t(np) * max(tmx, int64_t(1))));
      const int lb = bits64(int64_t(np) * np * max(max(int64_t(1), mmx), int64_t(cap)));
      const int64_t lmax = lb <= kMemoptLagrLimitBits ? int64_t(1) << (kMemoptLagrLimitBits - lb) : 0;
      if (F >= 0 && lmax > 0) {
#pragma unroll
        for (int q = 0; q < PPL; ++q)
          if (own(q)) {
            const int32_t i = lane + 64 * q;
            const int64_t t0 = ct[i * kMemoptMaxCands];
            const int64_t m0 = cmem[i * kMemoptMaxCands];
            for (int32_t j = 1; has(i, j); ++j)
              s0 = max(s0, ((ct[i * kMemoptMaxCands + j] - t0) << F) >>
                               (bits64(m0 - cmem[i * kMemoptMaxCands + j]) - 1));
          }
        s0 = min(lmax, max(int64_t(1), wave_max64(s0) >> 1));
        // own pairs: the forward-order range [lo, hi) of the checkpoints
        // they are live at
        int32_t lo[PPL], hi[PPL];
#pragma unroll
        for (int q = 0; q < PPL; ++q) {
          int32_t x = 0, y = 0;
          if (own(q))
            for (int32_t j = 0; j < np; ++j) {
              x += pfa[j] < pf[q] ? 1 : 0;
              y += pfa[j] <= pb[q] ? 1 : 0;
            }
          lo[q] = x;
          hi[q] = y;
        }
        int64_t *ps = lps;                   // [np + 1] prefix sums of the multipliers
        int64_t *dif = lps + (mp + 1);       // [np + 1] memory differences, then g
        int64_t *lam = lps + 2 * (mp + 1);   // [np] multipliers, by forward order
        for (int32_t d = lane; d < np; d += 64) lam[d] = 0;
        lds_sync_wave();
        for (int t = 0; t < kMemoptLagrIters; ++t) {
          // prefix sums of the multipliers; the difference array cleared
          int64_t carry = 0;
#pragma unroll
          for (int q = 0; q < PPL; ++q) {
            if (64 * q >= np) continue;
            const int32_t d = lane + 64 * q;
            const int64_t v = wave_scan64(d < np ? lam[d] : 0) + carry;
            if (d < np) ps[d + 1] = v;
            if (d <= np) dif[d] = 0;
            carry = shfl64(v, 63);
          }
          if (lane == 0) ps[0] = 0;
          if (np % 64 == 0 && lane == 0) dif[np] = 0;
          lds_sync_wave();
          int64_t part = 0;
#pragma unroll
          for (int q = 0; q < PPL; ++q)
            if (own(q)) {
              const int32_t i = lane + 64 * q;
              const int64_t price = hi[q] > lo[q] ? ps[hi[q]] - ps[lo[q]] : 0;
              int64_t bv = 0;
              int32_t bm = 0;
              for (int32_t j = 0; has(i, j); ++j) {
                const int64_t v = (ct[i * kMemoptMaxCands + j] << F) +
                                  int64_t(cmem[i * kMemoptMaxCands + j]) * price;
                if (j == 0 || v < bv) {
                  bv = v;
                  bm = cmem[i * kMemoptMaxCands + j];
                }
              }
              part += bv;
              if (hi[q] > lo[q]) {
                atomicAdd(reinterpret_cast<unsigned long long *>(dif + lo[q]),
                          static_cast<unsigned long long>(int64_t(bm)));
                atomicAdd(reinterpret_cast<unsigned long long *>(dif + hi[q]),
                          static_cast<unsigned long long>(-int64_t(bm)));
              }
            }
          const int64_t val = wave_sum64(part) - int64_t(cap) * carry;
          if (__int128(105) * val >= __int128(100) * (__int128(inc) << F)) {
            status = 1;
            break;
          }
          lds_sync_wave();
          // g at every depth: the running sum of the differences less the
          // cap, written over the differences
          int64_t gabs = 0, run = 0;
#pragma unroll
          for (int q = 0; q < PPL; ++q) {
            if (64 * q >= np) continue;
            const int32_t d = lane + 64 * q;
            const int64_t v = wave_scan64(d < np ? dif[d] : 0) + run;
            run = shfl64(v, 63);
            const int64_t g = v - int64_t(cap);
            if (d < np) {
              dif[d] = g;
              gabs = max(gabs, g < 0 ? -g : g);
            }
          }
          const int sh = bits64(wave_max64(gabs));
          if (sh == 0) break;
          const int64_t step = s0 >> (t / kMemoptLagrHalve);
          for (int32_t d = lane; d < np; d += 64) {
            const int64_t g = dif[d];
            const int64_t mv = ((g < 0 ? -g : g) * step) >> sh;
            lam[d] = min(lmax, max(int64_t(0), lam[d] + (g < 0 ? -mv : mv)));
          }
          lds_sync_wave();   // (the next step rewrites the arrays)
        }
      }
    }
  }
  int64_t total = 0;
  uint32_t pk = 0x80000000u;                        // image of load 0
#pragma unroll
  for (int q = 0; q < PPL; ++q) {
    const int32_t i = lane + 64 * q;
    if (i < np) {
      total += ct[i * kMemoptMaxCands + cur[q]];
      pk = max(pk, uint32_t(load[q]) ^ 0x80000000u);
      if (a.out_choice) a.out_choice[c * a.n_pairs + pbase + i] = uint8_t(cur[q]);
    }
  }
  pk = wave_reduce63<true>(pk);
#pragma unroll
  for (int s = 1; s < 64; s <<= 1)
    total += (int64_t(__shfl_xor(int(total >> 32), s)) << 32) |
             uint32_t(__shfl_xor(int(uint32_t(total)), s));
  if (lane == 0) write_out(a, o, total, int32_t(pk ^ 0x80000000u), status);
}

}  // namespace

size_t memopt_wave_lds(int32_t max_pairs, int waves_per_block) {
  // the rank's tables and the waves' positions and choices, then (8-byte
  // aligned) each wave's two certificate arrays of max_pairs + 1 words
  const size_t head = size_t(max_pairs) * (68 + 7 * size_t(waves_per_block));
  return (head + 7) / 8 * 8 + size_t(waves_per_block) * 24 * (size_t(max_pairs) + 1);
}

hipError_t launch_memopt_wave(int ppl, int waves_per_block, hipStream_t s, const MemoptArgs &a) {
  const int64_t bx = (a.n_cand + waves_per_block - 1) / waves_per_block;
  const size_t lds = memopt_wave_lds(a.max_pairs, waves_per_block);
  const dim3 grid{unsigned(bx), unsigned(a.P)}, block{unsigned(64 * waves_per_block)};
  switch (ppl) {
    case 1: hipLaunchKernelGGL(memopt_wave_kernel<1>, grid, block, lds, s, a); break;
    case 2: hipLaunchKernelGGL(memopt_wave_kernel<2>, grid, block, lds, s, a); break;
    case 4: hipLaunchKernelGGL(memopt_wave_kernel<4>, grid, block, lds, s, a); break;
    case 8: hipLaunchKernelGGL(memopt_wave_kernel<8>, grid, block, lds, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_memopt(int threads_per_block, hipStream_t s, const MemoptArgs &a) {
  const int64_t n = a.n_cand * a.P;
  const int64_t blocks = (n + threads_per_block - 1) / threads_per_block;
  const size_t lds = size_t(threads_per_block) * size_t(a.bytes_per_thread);
  hipLaunchKernelGGL(memopt_kernel, dim3(unsigned(blocks)), dim3(unsigned(threads_per_block)), lds,
                     s, a);
  return hipGetLastError();
}

}  // namespace dipsim
