// kern_check.hip -- the order-only part of a candidate's verdict, run before
// the timing simulation (one wave per candidate, or tiles of 64 candidates
// with lane = candidate followed by the order kernel):
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
#include <type_traits>

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
  if (a.retry_count && blockIdx.x == 0 && threadIdx.x < kRetryCounters) a.retry_count[threadIdx.x] = 0u;

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

// ---------------------------------------------------------------- tile check
// Lane = candidate: the 64 lanes of a wave hold 64 consecutive candidates and
// walk one rank's section of their rows in lockstep, so section boundaries
// are the same for every lane and only the ids differ.
//
//   * A section is a permutation of 0 .. n_r-1 iff its n_r ids set n_r
//     distinct bits of a map of bits 0 .. n_r, with an id above n_r - 1
//     clamped to the overflow bit n_r and that bit left clear (n_r ids, all
//     in range and pairwise distinct).  A lane's map lives in LDS word-major
//     (word w of lane l at 64 w + l), so the 64 lanes of one OR touch 64
//     distinct words and no two of them share a bank within a half-wave.
//   * The running memory is the sum of the deltas of the ops taken so far,
//     read from the wave's copy of the rank's deltas in LDS; the peak is its
//     maximum, starting from 0 (Sec. 5.3).
// The verdict of a candidate needs all of its ranks: each wave ORs its
// findings into the candidates' flag words in LDS, and after a block barrier
// the outputs of an invalid candidate are overwritten with -1.  (The order of
// ops that wait on an op of their own rank is the order kernel's, below.)

__global__ __launch_bounds__(kTileMaxWaves * kWave) void tile_check_kernel(TileCheckArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  uint32_t *flg = reinterpret_cast<uint32_t *>(c_lds);
  unsigned char *region = c_lds + kTileFlagBytes + wave * a.region_bytes;
  int32_t *mdl = reinterpret_cast<int32_t *>(region);   // the rank's deltas
  uint32_t *bm = reinterpret_cast<uint32_t *>(region + a.md_bytes) + lane;   // word w at bm[64 w]
  // staging of 8 units of the 64 rows (8 KB), unit k of row l at slot
  // k ^ (l & 7) of the row's 8, so the reads of one unit by 8 lanes hit 8
  // distinct bank groups
  unsigned char *stg = region + a.region_bytes - kTileStageBytes;
  if (a.retry_count && blockIdx.x == 0 && threadIdx.x < kRetryCounters) a.retry_count[threadIdx.x] = 0u;

  const int kb = a.plan[wave], ke = a.plan[wave + 1];
  const int32_t *ranks = a.plan + a.nw + 1;
  const int64_t n_tiles = (a.n_cand + kWave - 1) / kWave;
  const uint32_t row_bytes = uint32_t(a.stride) * 2u;
  for (int64_t tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
    if (wave == 0) flg[lane] = 0u;
    __syncthreads();
    const int64_t c0 = tile * kWave;
    const int n_live = int(min<int64_t>(a.n_cand - c0, kWave));
    const bool live = lane < n_live;
    const int64_t cand = c0 + lane;
    // the tile's rows behind one buffer descriptor; a lane past the end of
    // the batch reads the last row
    const uint64_t base = reinterpret_cast<uint64_t>(a.orders + c0 * a.stride);
    const uint64_t base_u = uint64_t(uint32_t(__builtin_amdgcn_readfirstlane(uint32_t(base)))) |
                            (uint64_t(uint32_t(__builtin_amdgcn_readfirstlane(uint32_t(base >> 32)))) << 32);
    const __amdgpu_buffer_rsrc_t rows = __builtin_amdgcn_make_buffer_rsrc(
        reinterpret_cast<void *>(base_u), 0,
        __builtin_amdgcn_readfirstlane(int(uint32_t(n_live) * row_bytes)), kBufferWord3);
    uint32_t fl = 0;
    for (int k = kb; k < ke; ++k) {
      const int r = ranks[k];
      const int rb = a.rank_off[r], re = a.rank_off[r + 1];
      const int nr = re - rb;
      const int n_words = (nr + 32) >> 5;   // bits 0 .. nr
      const int32_t *src = a.md;
      // the rank's deltas into the wave's region (entry nr, the overflow
      // entry, is 0), the lanes' bitmaps cleared
      wave_sync();
      for (int i = lane; i <= nr; i += 4 * kWave) {
        int32_t v[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) v[t] = i + t * kWave < nr ? src[rb + i + t * kWave] : 0;
#pragma unroll
        for (int t = 0; t < 4; ++t)
          if (i + t * kWave <= nr) mdl[i + t * kWave] = v[t];
      }
      for (int w = 0; w < n_words; ++w) bm[w * kWave] = 0u;
      wave_sync();

      const uint32_t lim = uint32_t(nr);
      int run = 0, peak = 0;
      // A unit of 8 ids is taken in two halves: its ids and deltas (eight
      // LDS reads in flight at once), then its bits and running sum.  The
      // deltas of the next unit are read before the current one's bits and
      // sums, so the reads overlap that work (the bitmap and the deltas are
      // different words: the reads need not wait for the ORs).
      struct Fetched {
        uint32_t c[8];
        int32_t dl[8];
      };
      auto fetch = [&](const uint4 v, int lo, int hi, Fetched &f) {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const uint32_t w = q < 2 ? v.x : q < 4 ? v.y : q < 6 ? v.z : v.w;
          f.c[q] = min((q & 1) ? (w >> 16) : (w & 0xffffu), lim);
          f.dl[q] = q >= lo && q < hi ? mdl[f.c[q]] : 0;
        }
      };
      auto apply = [&](const Fetched &f, int lo, int hi) {
#pragma unroll
        for (int q = 0; q < 8; ++q)
          if (q >= lo && q < hi) {
            uint32_t wd;
            asm("v_lshrrev_b32 %0, 5, %1" : "=v"(wd) : "v"(f.c[q]));
            __hip_atomic_fetch_or(bm + wd * kWave, 1u << (f.c[q] & 31u), __ATOMIC_RELAXED,
                                  __HIP_MEMORY_SCOPE_WORKGROUP);
          }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          run += f.dl[q];
          if (q >= lo && q < hi) peak = max(peak, run);
        }
      };
      if (nr > 0) {
        const int u0 = rb >> 3, u1 = (re - 1) >> 3;   // first and last unit of 8 ids
        auto bounds = [&](int u, int &lo, int &hi) {
          lo = max(rb - 8 * u, 0);
          hi = min(re - 8 * u, 8);
        };
        // Rows are read 8 units (128 bytes) at a time, cooperatively: load i
        // brings rows 8i .. 8i+7, lane l reading unit (l & 7) of row
        // 8i + (l >> 3), so 8 lanes share each line; the units go through
        // the wave's staging area to the lane that owns the row.  A lane past
        // the end of the batch reads the last row; units past the section
        // are read (clamped to its last unit) but not processed.
        auto load_chunk = [&](int cu, uint4 (&r)[8]) {
          const uint32_t ub = uint32_t(min(cu + (lane & 7), u1)) * 16u;
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const uint32_t row = uint32_t(min(8 * i + (lane >> 3), n_live - 1));
            const auto x = __builtin_amdgcn_raw_buffer_load_b128(rows, row * row_bytes + ub, 0, 0);
            r[i] = make_uint4(uint32_t(x[0]), uint32_t(x[1]), uint32_t(x[2]), uint32_t(x[3]));
          }
        };
        const uint32_t put = uint32_t(((lane >> 3) * 8 + ((lane & 7) ^ ((lane >> 3) & 7))) * 16);
        uint4 nb[8];
        load_chunk(u0, nb);
        for (int cu = u0; cu <= u1; cu += 8) {
          // the staging area is written and read by this wave only: program
          // order of its LDS accesses is all it needs (no wait for the
          // global loads in flight)
          wave_lds_order();   // the previous chunk's reads are done
#pragma unroll
          for (int i = 0; i < 8; ++i) *reinterpret_cast<uint4 *>(stg + 1024u * i + put) = nb[i];
          wave_lds_order();
          uint4 b[8];
#pragma unroll
          for (int q = 0; q < 8; ++q)
            b[q] = *reinterpret_cast<const uint4 *>(stg + uint32_t((lane * 8 + (q ^ (lane & 7))) * 16));
          if (cu + 8 <= u1) load_chunk(cu + 8, nb);   // the next chunk, while this one runs
          {
            // (a chunk of eight units all inside the section takes the
            // variant without position bounds)
            auto run_chunk = [&](auto inner) {
              constexpr bool kInner = decltype(inner)::value;
              auto lim_of = [&](int u, int &lo, int &hi) {
                if constexpr (kInner) {
                  lo = 0;
                  hi = 8;
                } else {
                  bounds(u, lo, hi);
                }
              };
              Fetched fa, fb;
              int lo, hi;
              lim_of(cu, lo, hi);
              fetch(b[0], lo, hi, fa);
#pragma unroll
              for (int q = 0; q < 8; ++q) {
                if (!kInner && cu + q > u1) break;
                Fetched &cur = (q & 1) ? fb : fa;
                Fetched &nxt = (q & 1) ? fa : fb;
                if (q + 1 < 8 && (kInner || cu + q + 1 <= u1)) {
                  int l2, h2;
                  lim_of(cu + q + 1, l2, h2);
                  fetch(b[q + 1], l2, h2, nxt);
                }
                lim_of(cu + q, lo, hi);
                apply(cur, lo, hi);
              }
            };
            if (8 * cu >= rb && 8 * (cu + 8) <= re)
              run_chunk(std::integral_constant<bool, true>{});
            else
              run_chunk(std::integral_constant<bool, false>{});
          }
        }
      }
      uint32_t bits = 0;
      for (int w = 0; w < n_words; ++w) bits += uint32_t(__builtin_popcount(bm[w * kWave]));
      const bool ovf = (bm[(nr >> 5) * kWave] >> (nr & 31)) & 1u;
      const bool bad = ovf || bits != lim;
      const int cap_r = a.cap[r];
      const bool over = cap_r >= 0 && peak > cap_r;
      if (live) a.out_peak[cand * a.P + r] = peak;
      fl |= (bad ? 1u : 0u) | (over ? 2u : 0u);
    }
    if (fl) __hip_atomic_fetch_or(flg + lane, fl, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    __syncthreads();
    const uint32_t f = flg[lane];
    if (live && (f & 1u))
      for (int k = kb; k < ke; ++k) a.out_peak[cand * a.P + ranks[k]] = -1;
    if (wave == 0 && live) {
      a.out_flags[cand] = (f & 1u) ? uint8_t(DIP_FLAG_INVALID) : uint8_t((f & 2u) ? DIP_FLAG_CAP : 0u);
      if (f & 1u) {
        a.out_ms[cand] = -1;
        for (int q = 0; q < a.P; ++q) a.out_bub[cand * a.P + q] = -1;
      }
    }
    __syncthreads();   // the flag words are cleared for the next tile
  }
}

// -------------------------------------------------------------- order check
// An op whose predecessor runs on its own rank must come after it in the
// rank's order; if it comes first, the two wait for each other (the data edge
// one way, the order the other) and the candidate deadlocks: its makespan and
// bubbles are -1 and the deadlock flag is added.  One wave per (candidate,
// rank) section of the ranks that have such ops, a block per rank and chunk of
// candidates.  The main check has verified that a section is a permutation
// (candidates it found invalid are skipped), so the wave can write each id's
// position into a table, its inverse permutation, and then compare, for every
// op with an own-rank predecessor, the two positions: no test depends on the
// order in which the lanes take the ids.

__device__ __forceinline__ uint32_t id_of(const uint4 &v, int q) {
  const uint32_t w = q < 2 ? v.x : q < 4 ? v.y : q < 6 ? v.z : v.w;
  return (q & 1) ? (w >> 16) : (w & 0xffffu);
}

// steps of 64 units of a section held in registers between the two passes
// (longer sections read the rest again)
constexpr int kOrderRegSteps = 4;

__global__ __launch_bounds__(1024) void order_check_kernel(OrderCheckArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const uint32_t k = blockIdx.x >> 3;
  const int r = a.ranks[k % uint32_t(a.n_ranks)];
  const int64_t chunk = int64_t(k / uint32_t(a.n_ranks)) * 8 + (blockIdx.x & 7);
  if (chunk >= a.n_chunks) return;
  const int rb = a.rank_off[r], re = a.rank_off[r + 1];
  const int nr = re - rb;
  // the rank's predecessors (local id + 1, 0: none), entry nr 0; the wave's
  // positions table
  uint16_t *spl = reinterpret_cast<uint16_t *>(c_lds);
  uint16_t *pos = reinterpret_cast<uint16_t *>(c_lds + a.tab_bytes + wave * a.wave_bytes);
  {
    const int nt = a.wpb * kWave;
    for (int i = threadIdx.x; i <= nr; i += 4 * nt) {
      int32_t sp[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) sp[t] = i + t * nt < nr ? a.selfp[rb + i + t * nt] : 0;
#pragma unroll
      for (int t = 0; t < 4; ++t)
        if (i + t * nt <= nr) spl[i + t * nt] = uint16_t(sp[t]);
    }
  }
  __syncthreads();
  if (nr == 0) return;

  const int u0 = rb >> 3;
  const int u_last = (re - 1) >> 3;
  const int nu = u_last - u0 + 1;   // units of 8 ids touching the section
  const int ns = (nu + kWave - 1) / kWave;
  const int64_t c0 = chunk * int64_t(a.wpb) * a.per_wave + wave;
  for (int i = 0; i < a.per_wave; ++i) {
    const int64_t cand = c0 + int64_t(i) * a.wpb;
    if (cand >= a.n_cand) break;
    if (__builtin_amdgcn_readfirstlane(a.out_flags[cand]) & DIP_FLAG_INVALID) continue;
    const uint4 *row = reinterpret_cast<const uint4 *>(a.orders + cand * a.stride);
    auto unit_of = [&](int s) { return u0 + s * kWave + lane; };
    auto load = [&](int s) { return row[min(unit_of(s), u_last)]; };
    uint4 v[kOrderRegSteps];
#pragma unroll
    for (int s = 0; s < kOrderRegSteps; ++s)
      if (s < ns) v[s] = load(s);
    // positions (positions outside the section and ids out of range, which
    // a valid section has none of, go to entry nr)
    auto place = [&](const uint4 &w, int s) {
      const int u = unit_of(s);
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int p = 8 * u + q - rb;
        const bool in = p >= 0 && p < nr;
        pos[in ? min(id_of(w, q), uint32_t(nr)) : uint32_t(nr)] = uint16_t(p);
      }
    };
#pragma unroll
    for (int s = 0; s < kOrderRegSteps; ++s)
      if (s < ns) place(v[s], s);
    for (int s = kOrderRegSteps; s < ns; ++s) place(load(s), s);
    wave_lds_order();
    // (the units pass an empty asm statement, so that the second pass
    // decodes them again instead of keeping the first pass's 64 indices)
#pragma unroll
    for (int s = 0; s < kOrderRegSteps; ++s)
      asm volatile("" : "+v"(v[s].x), "+v"(v[s].y), "+v"(v[s].z), "+v"(v[s].w));
    bool late = false;
    auto test = [&](const uint4 &w, int s) {
      const int u = unit_of(s);
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int p = 8 * u + q - rb;
        const bool in = p >= 0 && p < nr;
        const uint32_t sp = spl[in ? min(id_of(w, q), uint32_t(nr)) : uint32_t(nr)];
        if (sp != 0u) late = late || int(pos[sp - 1u]) > p;
      }
    };
#pragma unroll
    for (int s = 0; s < kOrderRegSteps; ++s)
      if (s < ns) test(v[s], s);
    for (int s = kOrderRegSteps; s < ns; ++s) test(load(s), s);
    if (__builtin_amdgcn_ballot_w64(late) != 0ull) {
      if (lane == 0) {
        a.out_flags[cand] = uint8_t(a.out_flags[cand] | DIP_FLAG_DEADLOCK);
        a.out_ms[cand] = -1;
      }
      for (int q = lane; q < a.P; q += kWave) a.out_bub[cand * a.P + q] = -1;
    }
    wave_lds_order();   // this section's positions are read before the next one's are written
  }
}

}  // namespace

const void *check_kernel_ptr(int) { return reinterpret_cast<const void *>(check_kernel); }

hipError_t launch_check(int, int blocks, int wpb, size_t lds, hipStream_t s, const CheckArgs &a) {
  check_kernel<<<dim3(blocks), dim3(wpb * kWave), lds, s>>>(a);
  return hipGetLastError();
}

const void *tile_check_kernel_ptr() { return reinterpret_cast<const void *>(tile_check_kernel); }

hipError_t launch_tile_check(int blocks, int nw, size_t lds, hipStream_t s, const TileCheckArgs &a) {
  tile_check_kernel<<<dim3(blocks), dim3(nw * kWave), lds, s>>>(a);
  return hipGetLastError();
}

const void *order_check_kernel_ptr() { return reinterpret_cast<const void *>(order_check_kernel); }

hipError_t launch_order_check(int64_t blocks, int wpb, size_t lds, hipStream_t s,
                              const OrderCheckArgs &a) {
  order_check_kernel<<<dim3(uint32_t(blocks)), dim3(wpb * kWave), lds, s>>>(a);
  return hipGetLastError();
}

}  // namespace dipsim
