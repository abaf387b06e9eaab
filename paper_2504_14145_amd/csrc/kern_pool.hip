// kern_pool.hip -- timing simulation with per-rank slot pools.
//
// What is simulated (Sec. 5.2 and 6.1): every rank runs its ops one at a time
// in its given order, each op as soon as the rank is free and the outputs of
// all of its predecessors have arrived,
//     start = max(free, max_p end(p) + comm(p, o)),   end = start + cost,
// and a candidate deadlocks when no op can ever start while ops remain.
//
// Layout of the work: one wavefront holds G = 64 / PW candidates (PW = the
// next power of two >= P); lane r of a group plays rank r.  Each round every
// lane looks at the next op of its order.  Ranks hand end times to each other
// through "items": the end time of an op that has consumers, tagged with the
// op's rank-local id + 1 (16 bits: the tag only has to be unique within its
// owner's pool).  An op's item lives in a small pool of S slots owned by the
// rank that ran the op: per slot a 4-bit count of the readers still to come
// (0 = free), a tag and an end time.  The pools of a candidate are laid out as
// arrays over its ranks (counts, then tags, then ends with an odd stride in
// words), so the lanes of a wave reading their own or a neighbour's pool hit
// distinct LDS banks.
//
// A consumer compares its predecessor's tag with the S tags of that rank's
// pool (one predecessor per round), reads the matching end, folds end + comm
// into a running maximum, and decrements the slot's reader count (an LDS
// atomic subtract on its nibble).  The owner reads its counts every round and
// writes each new item, with its number of readers, into a slot whose count
// is zero.  A rank whose op has consumers but whose pool is full waits:
// back-pressure.
//
// Only a few items are live at a time (an item dies once its consumers ran),
// so a candidate needs P pools of under 120 bytes, where a table of end times
// by op would need 4 bytes per op: many more candidates stay resident per CU,
// which is what hides the LDS and cache latencies of the round loop.
//
// Verdicts: a group is done when all of its lanes ran their whole order.  A
// round in which no lane of a group fired an op or read an item leaves its
// state unchanged for good: if no lane was held by back-pressure, the orders
// deadlock; otherwise the bounded pools may be what stalls it, and the
// candidate is appended to a retry list that the unbounded general kernel
// re-simulates.  The permutation check and the memory scan ran before, in the
// check kernel, whose flags this kernel reads (invalid candidates are skipped)
// and extends.
#include "dip_sim.h"
#include "dev_util.h"
#include "internal.h"

namespace dipsim {
namespace {

extern __shared__ __align__(16) unsigned char p_lds[];

// 4 ids (8 bytes) in global memory
typedef const __attribute__((address_space(1))) uint64_t *gblock_ptr;

__device__ __forceinline__ uint32_t ld32(uint32_t addr) {
  return *reinterpret_cast<const uint32_t *>(p_lds + addr);
}
__device__ __forceinline__ uint4 ld128(uint32_t addr) {
  return *reinterpret_cast<const uint4 *>(p_lds + addr);
}
__device__ __forceinline__ uint2 ld64(uint32_t addr) {
  return *reinterpret_cast<const uint2 *>(p_lds + addr);
}
__device__ __forceinline__ void st32(uint32_t addr, uint32_t v) {
  *reinterpret_cast<uint32_t *>(p_lds + addr) = v;
}
__device__ __forceinline__ void st16(uint32_t addr, uint32_t v) {
  *reinterpret_cast<uint16_t *>(p_lds + addr) = uint16_t(v);
}
__device__ __forceinline__ uint32_t *lds_word(uint32_t addr) {
  return reinterpret_cast<uint32_t *>(__builtin_assume_aligned(p_lds + addr, 4));
}
__device__ __forceinline__ void lds_add(uint32_t addr, uint32_t v) {
  (void)__hip_atomic_fetch_add(lds_word(addr), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
}
__device__ __forceinline__ void lds_sub(uint32_t addr, uint32_t v) {
  (void)__hip_atomic_fetch_sub(lds_word(addr), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
}

// TAB: the record and extra-edge tables are copied into the block's LDS (small
// topologies), ahead of the pools; otherwise they are read from global memory.
template <int PWL, int S, bool TAB>
__global__ __launch_bounds__(TAB ? 1024 : 256) void pool_kernel(PoolArgs a) {
  constexpr int PW = 1 << PWL;
  constexpr int G = kWave / PW;
  constexpr int kC = int(pool_count_words(S));   // count words per pool
  constexpr uint32_t kTags = uint32_t(pool_tags_offset(PW, S));
  constexpr uint32_t kEnds = uint32_t(pool_ends_offset(PW, S));
  constexpr uint32_t kEndStride = uint32_t(pool_end_stride(S));
  constexpr uint32_t kGroup = uint32_t(pool_group_bytes(PW, S));
  static_assert(S >= 4 && S <= 16 && (S & (S - 1)) == 0, "pool size");
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int grp = lane >> PWL;
  const int r = lane & (PW - 1);
  const bool on = r < a.P;
  const int gbit = grp << PWL;
  const int64_t n_slots = int64_t(gridDim.x) * a.wpb * G;
  const uint32_t gbase = a.pool_base + uint32_t(wave * G + grp) * kGroup;
  const uint32_t rr = uint32_t(on ? r : 0);
  const uint32_t my_cnt = gbase + rr * 4u * kC;
  // my tags and ends, from my counts' address and my rank (kept out of
  // registers: the compiler folds the constants)
  auto my_tag = [&]() { return gbase + kTags + rr * 2u * S; };
  auto my_end = [&]() { return gbase + kEnds + rr * kEndStride; };

  int rb = 0, nr = 0, busy_r = 0;
  if (on) {
    rb = a.rank_off[r];
    nr = a.rank_off[r + 1] - rb;
    busy_r = a.busy[r];
  }
  const int last = max(nr - 1, 0);
  const int rb2 = rb + 2, last_abs = rb + last;

  int64_t cand = (int64_t(blockIdx.x) * a.wpb + wave) * G + grp;
  uint32_t rnd = 0;          // rounds so far
  uint32_t cand_round = 0;   // round at which the group took its candidate
  bool has = false;   // the group holds a candidate
  uint8_t fl = 0;     // the check kernel's flags for the candidate
  int ptr = 0;
  uint32_t tfree = 0, acc = 0;
  // nothing (more) to wait for: a tag no item carries (items are tagged
  // rank-local id + 1 <= 32768 < kEdgeTagMask; free slots hold 0 or a dead
  // tag), marked as the last edge
  const int2 no_edge = make_int2(int(kNoEdgeWord), 0);
  const int2 dead_edge = make_int2(int(kDeadEdgeWord), 0);   // no op to run
  // record {cost, first edge's comm, first edge word | readers << 24,
  //         item tag (rank-local id + 1; 0: no consumers) | extra edges << 16}
  int4 cur = make_int4(0, 0, 0, 0);
  int2 ce = dead_edge;                    // current edge {pred edge word, comm}
  uint32_t ea = 0;                        // byte offset of the op's next extra edge
  // ids come from 8-byte blocks of the row (4 ids): blk holds the block with
  // the id at ptr + 2 (the order's last id past its end), nblk the block
  // after it, loaded when the lane entered blk
  int id2 = 0;                            // id at ptr + 2
  uint64_t blk = 0, nblk = 0;
  const int16_t *row0 = a.orders;         // this candidate's row
  // the block read by lanes that do not need one, kept in registers (a select
  // between two registers is one instruction), in the global address space
  // (a generic pointer would turn the load into a flat load, which every LDS
  // wait would then also wait for)
  gblock_ptr idle_b;
  {
    const uint64_t v = reinterpret_cast<uint64_t>(a.orders);
    uint32_t lo = uint32_t(v), hi = uint32_t(v >> 32);
    asm volatile("" : "+v"(lo), "+v"(hi));
    idle_b = reinterpret_cast<gblock_ptr>(uint64_t(lo) | (uint64_t(hi) << 32));
  }
  auto block_at = [&](uint32_t b) {   // block b of the candidate's row
    return reinterpret_cast<gblock_ptr>(reinterpret_cast<uint64_t>(row0)) + b;
  };
  // the id at absolute position pos, from the block holding it
  auto id_in = [](uint64_t bk, uint32_t pos) {
    return int(uint32_t(bk >> ((pos & 3u) * 16u)) & 0xffffu);
  };
  auto clamp_id = [&](int id) { return min(max(id, 0), last); };
  // records and edges through buffer descriptors: 32-bit byte offsets, and a
  // read past the end returns zeros instead of faulting
  const __amdgpu_buffer_rsrc_t rec_rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<int4 *>(a.rec), 0, a.rec_bytes, kBufferWord3);
  const __amdgpu_buffer_rsrc_t edge_rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<int2 *>(a.edge), 0, a.edge_bytes, kBufferWord3);
  if constexpr (TAB) {   // the tables into LDS, once per block
    for (uint32_t i = threadIdx.x; i < uint32_t(a.rec_bytes) / 16u; i += blockDim.x)
      *reinterpret_cast<int4 *>(p_lds + 16u * i) = a.rec[i];
    for (uint32_t i = threadIdx.x; i < uint32_t(a.edge_bytes) / 8u; i += blockDim.x)
      *reinterpret_cast<int2 *>(p_lds + a.tab_edges + 8u * i) = a.edge[i];
    __syncthreads();
  }
  auto rec_at_off = [&](uint32_t off) {   // byte offset
    if constexpr (TAB) {
      const uint4 v = ld128(off);
      return make_int4(int(v.x), int(v.y), int(v.z), int(v.w));
    } else {
      const auto v = __builtin_amdgcn_raw_buffer_load_b128(rec_rs, off, 0, 0);
      return make_int4(int(v[0]), int(v[1]), int(v[2]), int(v[3]));
    }
  };
  auto rec_at = [&](int g) { return rec_at_off(uint32_t(g) * 16u); };
  // the record of this lane's op with rank-local id `id` (the lane's part of
  // the table starts at its rank's first op)
  const unsigned char *rec_lane = p_lds + 16u * uint32_t(rb);
  const uint32_t rec_lane_off = 16u * uint32_t(rb);
  auto rec_of = [&](uint32_t id) {
    if constexpr (TAB) {
      const uint4 v = *reinterpret_cast<const uint4 *>(rec_lane + 16u * id);
      return make_int4(int(v.x), int(v.y), int(v.z), int(v.w));
    } else {
      return rec_at_off(rec_lane_off + 16u * id);
    }
  };
  auto edge_at = [&](uint32_t off) {   // byte offset
    if constexpr (TAB) {
      const uint2 v = ld64(a.tab_edges + off);
      return make_int2(int(v.x), int(v.y));
    } else {
      const auto v = __builtin_amdgcn_raw_buffer_load_b64(edge_rs, off, 0, 0);
      return make_int2(int(v[0]), int(v[1]));
    }
  };
  // the first edge of a record, and the byte offset of its extra edges
  auto first_edge = [](const int4 &rc) { return make_int2(rc.z, rc.y); };
  auto extra_off = [](const int4 &rc) { return (uint32_t(rc.w) >> 16) * 8u; };

  // Loads are staged, so that no round waits for a load it issued itself:
  // the next edge and a row block are fetched by every lane (lanes with none
  // to fetch read the table's first entry, resp. one shared block) and taken
  // at the top of the next round, resp. at its end; the record of the op at
  // ptr + 1 is fetched only by the lanes that advanced, into a register that
  // keeps its value otherwise, and first used by the next round's state
  // update (the order in which they are issued keeps each of those waits off
  // the younger loads).  (A block fetched under the lane mask would need a
  // second register and a wait for the load just issued.)
  int4 s0 = cur;       // record of the op at ptr + 1
  int2 se = no_edge;
  uint64_t sb = 0;     // a row block, for lanes that entered a new block
  bool take_edge = false, take_blk = false;

  // Candidates: group slot k (of n_slots) starts on candidate k and goes on
  // with its fixed successors k + n_slots, k + 2 n_slots, ...; with
  // a.next_cand, the candidates from a.static_end (a multiple of n_slots) are
  // handed out instead in the order groups ask for them, which evens out
  // slots that drew long candidates.  All lanes of the group call this
  // together.
  auto next_cand = [&]() -> int64_t {
    const int64_t succ = cand + n_slots;
    if (!a.next_cand || succ < a.static_end) return succ;
    uint32_t k = 0;
    if (r == 0) k = atomicAdd(a.next_cand, 1u);
    k = uint32_t(__shfl(int(k), gbit, kWave));
    return a.static_end + int64_t(k);
  };
  // All lanes of the group call this together.
  auto start_candidate = [&]() {
    while (cand < a.n_cand && (a.out_flags[cand] & (DIP_FLAG_INVALID | DIP_FLAG_DEADLOCK)))
      cand = next_cand();
    has = cand < a.n_cand;
    ce = dead_edge;
    ea = 0;   // (lanes on the dead edge fetch edges at ea)
    take_edge = false;
    take_blk = false;
    // counts and tags cleared (ends are read only under a tag), also by a
    // group left without a candidate: its lanes sit on the dead edge and
    // compare its tag with rank 0's, which must then hold no stale data
    if (on) {
#pragma unroll
      for (int i = 0; i < kC; ++i) st32(my_cnt + 4u * i, 0u);
      if constexpr (S == 4) {
        *reinterpret_cast<uint2 *>(p_lds + my_tag()) = make_uint2(0, 0);
      } else {
#pragma unroll
        for (int i = 0; i < S / 8; ++i)
          *reinterpret_cast<uint4 *>(p_lds + my_tag() + 16u * i) = make_uint4(0, 0, 0, 0);
      }
    }
    if (!has) return;
    fl = a.out_flags[cand];
    cand_round = rnd;
    ptr = 0;
    tfree = 0;
    acc = 0;
    if (on && nr > 0) {
      row0 = a.orders + cand * a.stride;
      const int16_t *row = row0 + rb;
      const int id0 = clamp_id(row[0]);
      const int id1 = clamp_id(row[min(1, last)]);
      const uint32_t pos2 = uint32_t(rb + min(2, last));
      blk = *block_at(pos2 >> 2);
      nblk = *block_at(min((pos2 >> 2) + 1u, uint32_t(last_abs) >> 2));
      id2 = id_in(blk, pos2);
      cur = rec_at(rb + id0);
      s0 = rec_at(rb + id1);
      ce = first_edge(cur);
      ea = extra_off(cur);
    }
  };

  start_candidate();
  uint64_t g_has = any_in_group<PWL>(__builtin_amdgcn_ballot_w64(has));

  while (g_has) {
    // ---- the edge fetched by the previous round
    if (take_edge) ce = se;
    asm volatile("" : "+v"(ce.x), "+v"(ce.y)::"memory");

    // ---- reads: the tags of the predecessor's pool, my reader counts
    const uint32_t want = uint32_t(ce.x) & kEdgeTagMask;
    const uint32_t rp = (uint32_t(ce.x) >> kEdgeRankShift) & 63u;   // the predecessor's rank
    const uint32_t p_cnt = gbase + rp * 4u * kC;
    const uint32_t p_end = gbase + kEnds + rp * kEndStride;
    uint32_t tw[S / 2];   // the S tags of its pool, two per word
    if constexpr (S == 4) {
      const uint2 v = ld64(gbase + kTags + rp * 2u * S);
      tw[0] = v.x;
      tw[1] = v.y;
    } else {
#pragma unroll
      for (int i = 0; i < S / 8; ++i) {
        const uint4 v = ld128(gbase + kTags + rp * 2u * S + 16u * i);
        tw[4 * i] = v.x;
        tw[4 * i + 1] = v.y;
        tw[4 * i + 2] = v.z;
        tw[4 * i + 3] = v.w;
      }
    }
    uint32_t cnt[kC];   // my reader counts, 8 nibbles per word
#pragma unroll
    for (int i = 0; i < kC; ++i) cnt[i] = ld32(my_cnt + 4u * i);
    // prefetch the op's next edge (taken if this round finds the current one;
    // lanes on their last edge read the table's first entry)
    const bool last_edge = ce.x < 0;   // kEdgeLast is the sign bit
    se = edge_at(!last_edge ? ea : 0u);

    // the matching slot, as index bits
    // (as wave masks: each compare's lanes, combined with scalar ops)
    uint64_t m_found = 0, mb0 = 0, mb1 = 0, mb2 = 0, mb3 = 0;
#pragma unroll
    for (int i = 0; i < S; ++i) {
      const uint32_t pair = tw[i / 2];
      const uint32_t t = (i & 1) ? (pair >> 16) : (pair & 0xffffu);
      const uint64_t m = __builtin_amdgcn_ballot_w64(t == want);
      m_found |= m;
      if (i & 1) mb0 |= m;
      if (i & 2) mb1 |= m;
      if (i & 4) mb2 |= m;
      if (i & 8) mb3 |= m;
    }
    const bool found = __builtin_amdgcn_inverse_ballot_w64(m_found);
    const uint32_t hit4 = (__builtin_amdgcn_inverse_ballot_w64(mb0) ? 4u : 0u) |
                          (__builtin_amdgcn_inverse_ballot_w64(mb1) ? 8u : 0u) |
                          (__builtin_amdgcn_inverse_ballot_w64(mb2) ? 16u : 0u) |
                          (__builtin_amdgcn_inverse_ballot_w64(mb3) ? 32u : 0u);   // 4 x slot
    const uint32_t hit = hit4 >> 2;
    const uint32_t hit_v = ld32(p_end + hit4);
    // a slot is free when its reader count is zero: the first such slot (sl,
    // meaningful when has_free)
    bool has_free = false;
    uint32_t sl = 0;
#pragma unroll
    for (int i = kC - 1; i >= 0; --i) {
      const uint32_t w = i * 8 + 8 <= S ? cnt[i] : (cnt[i] | (0xffffffffu << (4 * (S - i * 8))));
      const uint32_t z = ~(((w & 0x77777777u) + 0x77777777u) | w | 0x77777777u);   // 0x8 in zero nibbles
      if constexpr (kC == 1) {
        has_free = z != 0u;
        sl = uint32_t(__builtin_ctz(z)) >> 2;
      } else {
        sl = z ? 8u * uint32_t(i) + (uint32_t(__builtin_ctz(z)) >> 2) : sl;
        has_free = has_free || z != 0u;
      }
    }
    const uint32_t acc_n = found ? max(acc, hit_v + uint32_t(ce.y)) : acc;
    // ready: the last edge found now, or none left to find (no predecessors,
    // or the last one found in an earlier round)
    // (the decisions are taken on wave masks, one bit per lane, so that they
    // cost scalar instructions only; a lane with no op to run is on the dead
    // edge word, neither found nor last nor empty)
    const uint64_t m_last = __builtin_amdgcn_ballot_w64(last_edge);
    const uint64_t m_ready = (m_found & m_last) |
                             (~m_found & __builtin_amdgcn_ballot_w64(want == kEdgeTagMask));
    const uint64_t m_need = __builtin_amdgcn_ballot_w64((uint32_t(cur.w) & 0xffffu) != 0u);
    const uint64_t m_fire = m_ready & (~m_need | __builtin_amdgcn_ballot_w64(has_free));
    const bool fire = __builtin_amdgcn_inverse_ballot_w64(m_fire);
    const bool held = __builtin_amdgcn_inverse_ballot_w64(m_ready & ~m_fire);
    const uint32_t en = max(tfree, acc_n) + uint32_t(cur.x);

    // ---- writes: release what was read, publish what was produced
    // (with one count word, every slot index is below 8)
    if (found) lds_sub(p_cnt + (kC > 1 ? 4u * (hit >> 3) : 0u), 1u << (kC > 1 ? 4u * (hit & 7u) : hit4));
    if (__builtin_amdgcn_inverse_ballot_w64(m_fire & m_need)) {
      lds_add(my_cnt + (kC > 1 ? 4u * (sl >> 3) : 0u),
              ((uint32_t(cur.z) >> 24) & 15u) << (4u * (kC > 1 ? (sl & 7u) : sl)));   // readers
      st32(my_end() + 4u * sl, en);
      st16(my_tag() + 2u * sl, uint32_t(cur.w));
    }

    // ---- register state (fin: fired its last op; adv: fired another)
    const uint64_t m_fin = m_fire & __builtin_amdgcn_ballot_w64(ptr + 1 == nr);
    const bool fin = __builtin_amdgcn_inverse_ballot_w64(m_fin);
    const bool adv = __builtin_amdgcn_inverse_ballot_w64(m_fire & ~m_fin);
    take_edge = __builtin_amdgcn_inverse_ballot_w64(m_found & ~m_fire & ~m_last);
    if (fire) {
      // (s0 arrived a round ago at the latest; a lane that fired its last op
      // copies a record it never uses)
      tfree = en;
      acc = 0;
      ++ptr;
      cur = s0;
      ce = first_edge(s0);
      ea = extra_off(s0);
    } else if (found) {
      acc = acc_n;
      ea += 8u;   // (unused once the last edge is found)
      // found the last edge but held: nothing left to find (the comm is read
      // only with a found edge)
      if (last_edge) ce.x = no_edge.x;
    }
    if (fin) {
      ce.x = dead_edge.x;
      ea = 0;
    }
    // fetch, for an advance, the record of the op after the new current one
    // and the id after that
    {
      // the record of the op now at ptr + 1 (its id was at ptr + 2)
      if (adv) s0 = rec_of(uint32_t(id2));
      // the id now at ptr + 2; entering a new block, take the one fetched
      // ahead and fetch the block after it
      // the block fetched at the previous crossing, taken a full round after
      // its load (just before sb is reloaded)
      if (take_blk) nblk = sb;
      const uint32_t pos = uint32_t(min(rb2 + ptr, last_abs));
      // (past the order's end pos stays on its last id, and a crossing there
      // takes and fetches that last block again)
      const bool cross = adv && (pos & 3u) == 0u;
      if (cross) blk = nblk;
      id2 = id_in(blk, pos);   // (the same id again when the lane did not advance)
      take_blk = cross;
      const uint32_t nb = min((pos >> 2) + 1u, uint32_t(last_abs) >> 2);
      sb = *(cross ? block_at(nb) : idle_b);
    }

    ++rnd;
    const uint64_t b_fin = m_fin;
    const bool stall_check = (rnd & 7u) == 0u;
    if (!b_fin && !stall_check) continue;
    const uint64_t g_run = any_in_group<PWL>(__builtin_amdgcn_ballot_w64(has && ce.x != dead_edge.x));
    const uint64_t ev_done = g_has & ~g_run;
    uint64_t ev_stall = 0, ev_over = 0;
    if (stall_check) {
      ev_stall = g_run & ~any_in_group<PWL>(m_fire | m_found);
      // every round of a running group fires an op or reads an item, at most
      // N + E of them per candidate; a group past that bound is handed to the
      // general kernel rather than left running
      ev_over = g_run & ~ev_stall &
                any_in_group<PWL>(__builtin_amdgcn_ballot_w64(has && rnd - cand_round > a.round_limit));
    }
    const uint64_t ev = ev_done | ev_stall | ev_over;
    if (ev == 0) continue;

    // ---- some groups finished their candidate
    const uint64_t g_held = any_in_group<PWL>(__builtin_amdgcn_ballot_w64(held));   // (held as computed above)
    const bool mine_ev = (ev >> gbit) & 1;
    if (mine_ev) {
      const bool stalled = (ev_stall >> gbit) & 1;
      const bool retry = (stalled && ((g_held >> gbit) & 1)) || ((ev_over >> gbit) & 1);
      uint32_t T = on ? tfree : 0u;
#pragma unroll
      for (int off = 1; off < PW; off <<= 1) T = max(T, uint32_t(__shfl_xor(int(T), off, kWave)));
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
      cand = next_cand();
      start_candidate();
    }
    g_has = any_in_group<PWL>(__builtin_amdgcn_ballot_w64(has));
  }
}

template <int S, bool TAB>
const void *ptr_s(int pwl) {
  switch (pwl) {
    case 0: return reinterpret_cast<const void *>(pool_kernel<0, S, TAB>);
    case 1: return reinterpret_cast<const void *>(pool_kernel<1, S, TAB>);
    case 2: return reinterpret_cast<const void *>(pool_kernel<2, S, TAB>);
    case 3: return reinterpret_cast<const void *>(pool_kernel<3, S, TAB>);
    case 4: return reinterpret_cast<const void *>(pool_kernel<4, S, TAB>);
    case 5: return reinterpret_cast<const void *>(pool_kernel<5, S, TAB>);
    default: return reinterpret_cast<const void *>(pool_kernel<6, S, TAB>);
  }
}

template <int S, bool TAB>
void launch_s(int pwl, dim3 grid, dim3 block, size_t lds, hipStream_t s, const PoolArgs &a) {
  switch (pwl) {
    case 0: pool_kernel<0, S, TAB><<<grid, block, lds, s>>>(a); break;
    case 1: pool_kernel<1, S, TAB><<<grid, block, lds, s>>>(a); break;
    case 2: pool_kernel<2, S, TAB><<<grid, block, lds, s>>>(a); break;
    case 3: pool_kernel<3, S, TAB><<<grid, block, lds, s>>>(a); break;
    case 4: pool_kernel<4, S, TAB><<<grid, block, lds, s>>>(a); break;
    case 5: pool_kernel<5, S, TAB><<<grid, block, lds, s>>>(a); break;
    default: pool_kernel<6, S, TAB><<<grid, block, lds, s>>>(a); break;
  }
}

template <bool TAB>
const void *ptr_t(int pwl, int slots) {
  switch (slots) {
    case 4: return ptr_s<4, TAB>(pwl);
    case 16: return ptr_s<16, TAB>(pwl);
    default: return ptr_s<8, TAB>(pwl);
  }
}

template <bool TAB>
void launch_t(int pwl, int slots, dim3 grid, dim3 block, size_t lds, hipStream_t s, const PoolArgs &a) {
  switch (slots) {
    case 4: launch_s<4, TAB>(pwl, grid, block, lds, s, a); break;
    case 16: launch_s<16, TAB>(pwl, grid, block, lds, s, a); break;
    default: launch_s<8, TAB>(pwl, grid, block, lds, s, a); break;
  }
}

}  // namespace

bool pool_slots_ok(int slots) { return slots == 4 || slots == 8 || slots == 16; }

const void *pool_kernel_ptr(int pwl, int slots, bool tab) {
  return tab ? ptr_t<true>(pwl, slots) : ptr_t<false>(pwl, slots);
}

hipError_t launch_pool(int pwl, int slots, bool tab, int blocks, int wpb, size_t lds, hipStream_t s,
                       const PoolArgs &a) {
  const dim3 grid(blocks), block(wpb * kWave);
  if (tab)
    launch_t<true>(pwl, slots, grid, block, lds, s, a);
  else
    launch_t<false>(pwl, slots, grid, block, lds, s, a);
  return hipGetLastError();
}

}  // namespace dipsim
