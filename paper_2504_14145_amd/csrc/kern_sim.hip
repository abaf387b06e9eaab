// kern_sim.hip -- timing simulation of candidate schedules, one wavefront
// holding 64 / PW candidates, lane r of a candidate's group playing rank r
// (the number of ranks P is a power of two, PW = P).
//
// What is simulated (Sec. 5.2 and 6.1): every rank runs its ops one at a
// time in its given order, each op as soon as the rank is free and the
// outputs of all of its predecessors have arrived,
//     start = max(free, max_p end(p) + comm(p, o)),   end = start + cost,
// and a candidate deadlocks when no op can ever start while ops remain.
//
// Rounds: every round each lane looks at the current op of its order.  End
// times travel between ranks as items: an op with consumers writes its end
// time, tagged with its rank-local id + 1, into a free slot of a pool of S
// slots owned by its rank, with a 4-bit count of the readers still to come
// (0 = free).  A consumer compares its predecessor's tag with the S tags of
// that rank's pool (one predecessor per round), folds end + comm into a
// running maximum and decrements the slot's count.  A producer whose pool is
// full waits (back-pressure).
//
// What is resident in LDS, and why:
//   * the op records, 8 bytes each and relative to the op (predecessor given
//     as a local-id and rank difference), so the records of model chunks
//     placed alike coincide; large tables are stored as pages of 16 records
//     with equal pages kept once and a page map per rank.  Every round's
//     record read is then an LDS read instead of a gather through the
//     vector-memory path;
//   * the pools of the candidates in flight (a few items per rank are live at
//     once, so a pool of 8 or 16 slots per rank suffices where a table of end
//     times by op would need 4 bytes per op);
//   * each lane's order ring: two 16-byte blocks of 8 ids of its rank's
//     section.  Every 4 rounds (the same rounds for all lanes, so that one
//     wait covers the loads) each lane that has moved into the later of its
//     two blocks loads the block after it from HBM into registers; 3 rounds
//     later the block is stored into the ring, over the one the lane left.
//     A lane fires at most one op per round and needs the id after its
//     current one, so the at most 6 rounds a block takes to arrive end before
//     the lane has used up the block it is in.
//
// Verdicts: a group is done when all of its lanes ran their whole order.  A
// round in which no lane of a group fired an op or read an item leaves its
// state unchanged for good: if no lane was held by back-pressure the orders
// deadlock; so they do if the lanes that wait for items wait on one another
// in a cycle (pools of any size would not free them); otherwise the bounded
// pools may be what stalls it, and the candidate goes to a retry list that a
// later pass re-simulates.  The permutation check and the memory scan ran
// before, in the check kernel, whose flags this kernel reads (invalid
// candidates are skipped) and extends.
#include "dip_sim.h"
#include "dev_util.h"
#include "internal.h"

namespace dipsim {
namespace {

extern __shared__ __align__(16) unsigned char s_lds[];

__device__ __forceinline__ uint32_t lds32(uint32_t a) {
  return *reinterpret_cast<const uint32_t *>(s_lds + a);
}
__device__ __forceinline__ uint2 lds64(uint32_t a) {
  return *reinterpret_cast<const uint2 *>(s_lds + a);
}
__device__ __forceinline__ void st32(uint32_t a, uint32_t v) {
  *reinterpret_cast<uint32_t *>(s_lds + a) = v;
}
__device__ __forceinline__ void st16(uint32_t a, uint32_t v) {
  *reinterpret_cast<uint16_t *>(s_lds + a) = uint16_t(v);
}
__device__ __forceinline__ void st64(uint32_t a, uint32_t x, uint32_t y) {
  *reinterpret_cast<uint2 *>(s_lds + a) = make_uint2(x, y);
}
__device__ __forceinline__ uint32_t *lds_word(uint32_t a) {
  return reinterpret_cast<uint32_t *>(__builtin_assume_aligned(s_lds + a, 4));
}
__device__ __forceinline__ void lds_add(uint32_t a, uint32_t v) {
  (void)__hip_atomic_fetch_add(lds_word(a), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
}
__device__ __forceinline__ void lds_sub(uint32_t a, uint32_t v) {
  (void)__hip_atomic_fetch_sub(lds_word(a), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
}
// LDS addresses as the hardware takes them (the dynamic array's own address
// added), for values computed outside the helpers above
typedef __attribute__((address_space(3))) unsigned char lds_byte_t;
__device__ __forceinline__ uint32_t lds_abs(uint32_t a) {
  return a + uint32_t(reinterpret_cast<uintptr_t>((lds_byte_t *)s_lds));
}
__device__ __forceinline__ uint32_t lds16_at(uint32_t abs_addr) {
  return *reinterpret_cast<const __attribute__((address_space(3))) uint16_t *>(uintptr_t(abs_addr));
}
// (x << s) + base in one instruction: written out, because the compiler
// turns (i & m) << s into (i << s) & (m << s) and then needs a separate add
template <int SH>
__device__ __forceinline__ uint32_t shl_add(uint32_t x, uint32_t base) {
  uint32_t d;
  asm("v_lshl_add_u32 %0, %1, %2, %3" : "=v"(d) : "v"(x), "i"(SH), "v"(base));
  return d;
}
__device__ __forceinline__ bool lane_in(uint64_t m) { return __builtin_amdgcn_inverse_ballot_w64(m); }
__device__ __forceinline__ uint64_t ballot(bool b) { return __builtin_amdgcn_ballot_w64(b); }

// A 16-byte order block of 8 ids (rows are padded to 8 ids, so a block of
// a row never reaches past it).
__device__ __forceinline__ uint4 load_block(const int16_t *row, uint32_t b) {
  return *reinterpret_cast<const uint4 *>(row + int64_t(b) * kSimBlockIds);
}
__device__ __forceinline__ void store_block(uint32_t at, const uint4 &v) {
  st64(at, v.x, v.y);
  st64(at + 8, v.z, v.w);
}

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// Which of a pool's S 16-bit tags (two to a word) equals `want`: with a
// weight of 16 + s for slot s, the sum over the slots whose tag differs,
// tag_miss_sum(S) - (16 + s) when slot s matches (tags are unique in a pool)
// and tag_miss_sum(S) when none does.  Per tag word: a packed XOR (equal
// halves become 0), a packed minimum with 1 (0 where equal, else 1) and a
// two-way dot product with the slots' weights.
template <int S>
__host__ __device__ constexpr uint32_t tag_miss_sum() {
  return uint32_t(S * (S - 1) / 2 + 16 * S);
}
template <int S>
__device__ __forceinline__ uint32_t tag_weighted_misses(const uint32_t (&tw)[S / 2], uint32_t want) {
  const uint32_t both = want * 0x10001u;
  uint32_t sum = 0;
#pragma unroll
  for (int i = 0; i < S / 2; ++i) {
    uint32_t y;
    asm("v_pk_min_u16 %0, %1, %2" : "=v"(y) : "v"(tw[i] ^ both), "s"(0x00010001u));
    const uint32_t w = (16u + 2u * i) | ((17u + 2u * i) << 16);
    sum = __builtin_amdgcn_udot2(__builtin_bit_cast(u16x2, y), __builtin_bit_cast(u16x2, w), sum,
                                 false);
  }
  return sum;
}

template <int PWL, int S, bool PAGED>
__global__ __launch_bounds__(1024) void sim_kernel(SimArgs a) {
  constexpr int PW = 1 << PWL;
  constexpr int G = kWave / PW;
  constexpr int kC = int(sim_count_words(S));
  constexpr uint32_t kPool = uint32_t(sim_pool_bytes(S));
  constexpr uint32_t kPools = uint32_t(sim_pool_offset(PW, S));
  constexpr uint32_t kTagRank = S == 4 ? 8u : 16u;   // a rank's tag bytes in one tag array
  constexpr uint32_t kEndAt = 4u * uint32_t(kC);      // end times after a pool's counts
  constexpr uint32_t kRing = uint32_t(sim_ring_offset(PW, S));
  constexpr uint32_t kGroup = uint32_t(sim_group_bytes(PW, S));
  static_assert(S == 4 || S == 8 || S == 16 || S == 32, "pool size");

  // the tables into LDS, once per block
  for (int i = threadIdx.x; i < a.tab_vec; i += blockDim.x)
    *reinterpret_cast<uint4 *>(s_lds + 16u * uint32_t(i)) = a.tab[i];
  __syncthreads();

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int grp = lane >> PWL;
  const int r = lane & (PW - 1);
  const bool on = r < a.P;
  const int gbit = grp << PWL;
  const int64_t n_slots = int64_t(gridDim.x) * a.wpb * G;
  const uint32_t gbase = a.state_base + uint32_t(wave * G + grp) * kGroup;
  const uint32_t rr = on ? uint32_t(r) : 0u;
  const uint32_t my_pool = gbase + kPools + rr * kPool;
  const uint32_t my_tags = gbase + rr * kTagRank;
  const uint32_t my_ring = gbase + kRing + rr * uint32_t(kSimRingBytes);
  int rb = 0, nr = 0, busy_r = 0, recb = 0;
  if (on) {
    const int4 li = reinterpret_cast<const int4 *>(a.lane_info)[r];
    rb = li.x;
    nr = li.y;
    busy_r = li.z;
    recb = li.w;
  }
  // absolute row positions: past this lane's section, its last block
  const uint32_t a_end = uint32_t(rb + nr);
  const uint32_t blk_last = uint32_t(rb + max(nr - 1, 0)) / uint32_t(kSimBlockIds);
  const uint32_t pmap_lane = lds_abs(a.off_pmap + 2u * uint32_t(recb));

  // the record of local id `id` of this lane's rank
  auto rec_of = [&](uint32_t id) -> uint2 {
    uint32_t first;   // record index of the page's first op, or of the rank's
    if constexpr (PAGED) {
      // (the page map holds multiples of 16: or-ing the offset in the page
      // adds it)
      first = lds16_at(shl_add<1>(id >> 4, pmap_lane)) | (id & 15u);
    } else {
      first = uint32_t(recb) + id;
    }
    return lds64(first << 3);
  };
  const uint32_t my_ring_abs = lds_abs(my_ring);
  auto ring_id = [&](uint32_t pos) { return lds16_at(shl_add<1>(pos & 15u, my_ring_abs)); };

  // candidates: positions k < n of the batch, or of the list in list mode
  const int64_t n_todo = a.list ? int64_t(*a.list_count) : a.n_cand;
  // slot of this group: block-major for a batch (a block's groups take
  // neighbouring candidates); in list mode, which carries few candidates,
  // block-minor, so that they spread over the CUs instead of sharing the
  // first few (either way a permutation of 0 .. n_slots - 1)
  int64_t k = a.list ? (int64_t(grp) * a.wpb + wave) * gridDim.x + blockIdx.x
                     : (int64_t(blockIdx.x) * a.wpb + wave) * G + grp;
  auto cand_at = [&](int64_t i) { return a.list ? a.list[i] : i; };

  // per-lane state
  int64_t cand = 0;
  bool has = false;        // the group holds a candidate
  uint8_t fl = 0;          // the check kernel's flags for it
  uint32_t cand_round = 0;
  uint32_t apos1 = 0;      // absolute row position of the op after the current one
  uint32_t tfree = 0, acc = 0;
  uint32_t lid1 = 0, cur0 = 0;  // current op: local id + 1, record word 0
  uint32_t ce = 0, xi = 0;      // its current edge word; index of its next extra edge
  uint32_t lb = 0;         // next absolute order block to load
  uint4 blk{};             // a loaded block waiting to be stored
  const int16_t *row = a.orders;

  // wave-uniform lane masks
  uint64_t m_live = 0;     // lanes running an op sequence
  uint64_t m_npend = 0;    // live lanes whose current op waits for no edge
  uint64_t m_blk = 0;      // lanes holding a loaded block for the ring

  auto set_current = [&](uint32_t id, uint2 c) {
    lid1 = id + 1u;
    cur0 = c.x;
    ce = c.y;
    xi = c.y + 1u;
    if (c.x >= (kSimHasPred | kSimMulti)) ce = lds32(a.off_extra + 4u * c.y);   // several predecessors
  };

  auto next_k = [&]() -> int64_t {
    const int64_t succ = k + n_slots;
    if (succ < a.static_end) return succ;
    uint32_t k = 0;
    if (r == 0) k = atomicAdd(a.retry_count + 1, 1u);
    k = uint32_t(__shfl(int(k), gbit, kWave));
    return a.static_end + int64_t(k);
  };

  // The lanes of one group call this together (a group without a candidate
  // keeps its lanes out of m_live, so its pool contents are never read).
  auto start_candidate = [&](uint32_t rnd) {
    // (candidates whose verdict the check kernel already settled: not a
    // permutation, or an op ordered before its own-rank predecessor)
    while (k < n_todo && (a.out_flags[cand_at(k)] & (DIP_FLAG_INVALID | DIP_FLAG_DEADLOCK)))
      k = next_k();
    has = k < n_todo;
    if (on) {   // empty pool: counts and tags zero
#pragma unroll
      for (int i = 0; i < kC; ++i) st32(my_pool + 4u * i, 0u);
#pragma unroll
      for (int i = 0; i < S / 2; ++i) st32(my_tags + 16u * PW * (i >> 2) + 4u * (i & 3), 0u);
    }
    if (!has) return;
    cand = cand_at(k);
    fl = a.out_flags[cand];
    cand_round = rnd;
    tfree = 0;
    acc = 0;
    if (!on || nr == 0) return;
    row = a.orders + cand * a.stride;
    // the first two blocks of the section into the ring
    const uint32_t b0 = uint32_t(rb) / uint32_t(kSimBlockIds);
    const uint32_t bn = min(b0 + 1u, blk_last);
    for (uint32_t b = b0; b <= bn; ++b) store_block(my_ring + (b & 1u) * 16u, load_block(row, b));
    lb = bn + 1u;
    apos1 = uint32_t(rb) + 1u;
    const uint32_t id0 = ring_id(uint32_t(rb));
    set_current(id0, rec_of(id0));
  };

  start_candidate(0);
  {
    const bool live = has && on && nr > 0;
    m_live = ballot(live);
    m_npend = m_live & ballot(int32_t(cur0) >= 0);
  }
  uint64_t g_has = any_in_group<PWL>(ballot(has));

  uint32_t rnd = 0;
  while (g_has) {
    // ---- order blocks: loaded every 4 rounds, stored 3 rounds later
    const uint32_t phase = rnd & 3u;
    if (phase == 3u && m_blk) {
      if (lane_in(m_blk)) {
        store_block(my_ring + (lb & 1u) * 16u, blk);
        ++lb;
      }
      m_blk = 0;
    }

    // ---- reads: the predecessor's pool, my counts, the next id
    // (the predecessor's rank: the rank difference sits in the edge word's
    // low bits, and P == PW)
    const uint32_t pr = (ce + rr) & uint32_t(PW - 1);
    const uint32_t pool = gbase + kPools + pr * kPool;
    const uint32_t p_tags = gbase + pr * kTagRank;
    const uint32_t want = lid1 + uint32_t(int32_t(ce << 12) >> 18);
    uint32_t tw[S / 2];
    if constexpr (S == 4) {
      const uint2 v = lds64(p_tags);
      tw[0] = v.x;
      tw[1] = v.y;
    } else {
#pragma unroll
      for (int i = 0; i < S / 8; ++i) {   // slots 8i .. 8i + 7 of every rank side by side
        const uint4 v = *reinterpret_cast<const uint4 *>(s_lds + p_tags + 16u * PW * i);
        tw[4 * i] = v.x;
        tw[4 * i + 1] = v.y;
        tw[4 * i + 2] = v.z;
        tw[4 * i + 3] = v.w;
      }
    }
    uint32_t cnt[kC];
#pragma unroll
    for (int i = 0; i < kC; ++i) cnt[i] = lds32(my_pool + 4u * i);
    const uint32_t idn = ring_id(apos1);
    // the next op's record, read ahead (used by the lanes that advance)
    const uint2 nrec = rec_of(idn);

    // the matching slot (tags are unique within a pool)
    const uint32_t wsum = tag_weighted_misses<S>(tw, want);
    const uint64_t m_found = ballot(wsum != tag_miss_sum<S>()) & m_live & ~m_npend;
    const uint32_t slot = (tag_miss_sum<S>() - 16u - wsum) & uint32_t(S - 1);
    const uint32_t hit_end = lds32(pool + kEndAt + 4u * slot);
    const bool found = lane_in(m_found);
    const uint32_t acc_n = found ? max(acc, hit_end + ((ce >> 20) & 0x7ffu)) : acc;
    // a free slot of my pool (reader count zero): the first one
    bool has_free = false;
    uint32_t sl = 0;
    uint32_t zfree = 0;   // (one count word) bit 4 s + 3 set for each free slot s
#pragma unroll
    for (int i = kC - 1; i >= 0; --i) {
      const uint32_t w = i * 8 + 8 <= S ? cnt[i] : (cnt[i] | (0xffffffffu << (4 * (S - i * 8))));
      const uint32_t z = ~(((w & 0x77777777u) + 0x77777777u) | w | 0x77777777u);   // 8 in zero nibbles
      if constexpr (kC == 1) {
        has_free = z != 0u;
        zfree = z;
      } else {
        sl = z ? 8u * uint32_t(i) + (uint32_t(__builtin_ctz(z)) >> 2) : sl;
        has_free = has_free || z != 0u;
      }
    }
    const uint32_t readers = (cur0 >> 20) & 15u;
    const uint64_t m_last = ballot(int32_t(ce) < 0);
    const uint64_t m_ready = (m_found & m_last) | m_npend;
    const uint64_t m_need = ballot(readers != 0u);
    const uint64_t m_fire = m_ready & (~m_need | ballot(has_free));
    const uint64_t m_held = m_ready & ~m_fire;
    const bool fire = lane_in(m_fire);
    const uint32_t en = max(tfree, acc_n) + (cur0 & kSimCostMax);

    // ---- writes: release what was read, publish what was produced
    if (found) {
      lds_sub(pool + (kC > 1 ? 4u * (slot >> 3) : 0u), 1u << (4u * (slot & 7u)));
    }
    if (lane_in(m_fire & m_need)) {
      if constexpr (kC == 1) {   // 4 x the first free slot (zfree is not 0 here)
        const uint32_t sl4 = uint32_t(__builtin_ctz(zfree)) - 3u;
        lds_add(my_pool, readers << sl4);
        st32(my_pool + kEndAt + sl4, en);
        st16(my_tags + (sl4 >> 1), lid1);
      } else {
        lds_add(my_pool + 4u * (sl >> 3), readers << (4u * (sl & 7u)));
        st32(my_pool + kEndAt + 4u * sl, en);
        st16(my_tags + 16u * PW * (sl >> 3) + 2u * (sl & 7u), lid1);
      }
    }

    // ---- register state
    const uint64_t m_fin = m_fire & ballot(apos1 == a_end);
    const uint64_t m_adv = m_fire & ~m_fin;
    const bool adv = lane_in(m_adv);
    const bool more = lane_in(m_found & ~m_fire & ~m_last);   // found, another edge to go
    if (fire) {
      tfree = en;
      acc = 0;
    } else if (found) {
      acc = acc_n;
    }
    if (more) {   // the op's next predecessor edge
      ce = lds32(a.off_extra + 4u * xi);
      ++xi;
    }
    if (adv) {   // the next op becomes current
      set_current(idn, nrec);
      ++apos1;
    }
    m_npend = ((m_npend & ~m_fire) | (m_found & m_last & ~m_fire) |
               (m_adv & ballot(int32_t(cur0) >= 0))) & ~m_fin;
    m_live &= ~m_fin;

    // ---- order blocks: every 4 rounds, a lane in the later of its two
    // blocks loads the one after it
    if (phase == 0u) {
      // (the current op is at apos1 - 1 >= 0: its block plus one is
      // (apos1 + 7) / 8)
      const uint32_t next_blk = (apos1 + uint32_t(kSimBlockIds) - 1u) / uint32_t(kSimBlockIds);
      const bool load = lane_in(m_live) && lb <= min(next_blk, blk_last);
      m_blk = ballot(load);
      if (load) blk = load_block(row, lb);
    }

    // ---- verdicts, every 8 rounds (a group that finished or stalled waits
    // for the next check; its state does not change meanwhile)
    ++rnd;
    if ((rnd & 7u) != 0u) continue;
    const uint64_t g_run = any_in_group<PWL>(m_live);
    const uint64_t g_done = g_has & ~g_run;   // every lane ran its whole order
    const uint64_t g_stall = g_run & ~any_in_group<PWL>(m_fire | m_found);
    const uint64_t g_over = g_run & ~g_stall &
                            any_in_group<PWL>(ballot(has && rnd - cand_round > a.round_limit));
    const uint64_t ev = g_done | g_stall | g_over;
    if (ev == 0) continue;

    // ---- some groups finished their candidate
    const uint64_t g_held = any_in_group<PWL>(m_held);
    // A stalled group with held lanes still deadlocks whatever the pool size
    // when the lanes that wait for an item wait on one another in a cycle:
    // a waiting lane's predecessor op has not run (its item would be in the
    // pool), so it waits on the predecessor's rank, and when that rank waits
    // too, on that rank's predecessor rank, and so on; a chain of PW steps
    // that meets no held or finished lane has closed a cycle of waiting
    // lanes, none of which can ever move.  Pointer doubling over the group's
    // lanes follows every chain PW steps.
    uint64_t g_cyc = 0;
    if (const uint64_t g_sh = g_stall & g_held) {
      const bool waiting = lane_in(m_live & ~m_npend & ~m_held);
      int x = waiting ? gbit + int((ce + rr) & uint32_t(PW - 1)) : -1;
#pragma unroll
      for (int s = 0; s < PWL; ++s) {
        const int y = __shfl(x, x < 0 ? lane : x, kWave);
        x = x < 0 ? -1 : y;
      }
      g_cyc = g_sh & any_in_group<PWL>(ballot(x >= 0));
    }
    const uint64_t m_ev = any_lane_of_group<PWL>(ev);
    if (lane_in(m_ev)) {
      const bool stalled = (g_stall >> gbit) & 1;
      const bool retry = (stalled && ((g_held >> gbit) & 1) && !((g_cyc >> gbit) & 1)) ||
                         ((g_over >> gbit) & 1);
      uint32_t T = on ? tfree : 0u;
#pragma unroll
      for (int off = 1; off < PW; off <<= 1) T = max(T, uint32_t(__shfl_xor(int(T), off, kWave)));
      if (has) {
        if (retry) {
          if (r == 0) {
            const uint32_t k = atomicAdd(a.retry_count, 1u);
            a.retry[k] = cand;
          }
        } else if (on) {
          a.out_bub[cand * a.P + r] = stalled ? -1 : int32_t(T) - busy_r;
          if (r == 0) {
            a.out_ms[cand] = stalled ? -1 : int32_t(T);
            if (stalled) a.out_flags[cand] = uint8_t(fl | DIP_FLAG_DEADLOCK);
          }
        }
      }
      k = next_k();
      start_candidate(rnd);
    }
    // the restarted groups' lanes: live and edge state from their new records
    const bool live_new = has && on && nr > 0;
    m_live = (m_live & ~m_ev) | (m_ev & ballot(live_new));
    m_npend = (m_npend & ~m_ev) | (m_ev & m_live & ballot(int32_t(cur0) >= 0));
    m_blk &= ~m_ev;
    g_has = any_in_group<PWL>(ballot(has));
  }
}

template <int S, bool PAGED>
const void *ptr_s(int pwl) {
  switch (pwl) {
    case 0: return reinterpret_cast<const void *>(sim_kernel<0, S, PAGED>);
    case 1: return reinterpret_cast<const void *>(sim_kernel<1, S, PAGED>);
    case 2: return reinterpret_cast<const void *>(sim_kernel<2, S, PAGED>);
    case 3: return reinterpret_cast<const void *>(sim_kernel<3, S, PAGED>);
    case 4: return reinterpret_cast<const void *>(sim_kernel<4, S, PAGED>);
    case 5: return reinterpret_cast<const void *>(sim_kernel<5, S, PAGED>);
    default: return reinterpret_cast<const void *>(sim_kernel<6, S, PAGED>);
  }
}

template <int S, bool PAGED>
void launch_s(int pwl, dim3 grid, dim3 block, size_t lds, hipStream_t s, const SimArgs &a) {
  switch (pwl) {
    case 0: sim_kernel<0, S, PAGED><<<grid, block, lds, s>>>(a); break;
    case 1: sim_kernel<1, S, PAGED><<<grid, block, lds, s>>>(a); break;
    case 2: sim_kernel<2, S, PAGED><<<grid, block, lds, s>>>(a); break;
    case 3: sim_kernel<3, S, PAGED><<<grid, block, lds, s>>>(a); break;
    case 4: sim_kernel<4, S, PAGED><<<grid, block, lds, s>>>(a); break;
    case 5: sim_kernel<5, S, PAGED><<<grid, block, lds, s>>>(a); break;
    default: sim_kernel<6, S, PAGED><<<grid, block, lds, s>>>(a); break;
  }
}

template <bool PAGED>
const void *ptr_p(int pwl, int slots) {
  switch (slots) {
    case 4: return ptr_s<4, PAGED>(pwl);
    case 16: return ptr_s<16, PAGED>(pwl);
    case 32: return ptr_s<32, PAGED>(pwl);
    default: return ptr_s<8, PAGED>(pwl);
  }
}

template <bool PAGED>
void launch_p(int pwl, int slots, dim3 grid, dim3 block, size_t lds, hipStream_t s,
              const SimArgs &a) {
  switch (slots) {
    case 4: launch_s<4, PAGED>(pwl, grid, block, lds, s, a); break;
    case 16: launch_s<16, PAGED>(pwl, grid, block, lds, s, a); break;
    case 32: launch_s<32, PAGED>(pwl, grid, block, lds, s, a); break;
    default: launch_s<8, PAGED>(pwl, grid, block, lds, s, a); break;
  }
}

}  // namespace

bool sim_slots_ok(int slots) { return slots == 4 || slots == 8 || slots == 16; }

const void *sim_kernel_ptr(int pwl, int slots, bool paged) {
  return paged ? ptr_p<true>(pwl, slots) : ptr_p<false>(pwl, slots);
}

hipError_t launch_sim(int pwl, int slots, bool paged, int blocks, int wpb, size_t lds,
                      hipStream_t s, const SimArgs &a) {
  const dim3 grid(blocks), block(wpb * kWave);
  if (paged)
    launch_p<true>(pwl, slots, grid, block, lds, s, a);
  else
    launch_p<false>(pwl, slots, grid, block, lds, s, a);
  return hipGetLastError();
}

}  // namespace dipsim
