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
// op's global index + 1 and with the number of consumers that still have to
// read it.  An op's item lives in a small pool of S slots owned by the rank
// that ran the op:
//
//     pool (16 + 8 S bytes):  freed mask | 12 bytes pad | S x {tag word, end}
//     tag word: bits 0-21 item tag, bits 22-31 readers left
//
// A consumer scans the S slots of its predecessor's pool for the tag (one
// predecessor per round), folds end + comm into a running maximum, and then
// either decrements the readers left or, as the last reader, releases the slot
// by setting its bit in the owner's freed mask (an LDS atomic OR).  The owner
// reads its freed mask every round, forgets released slots (clearing the bits
// it saw with an atomic AND) and writes each new item into a free slot.  A
// rank whose op has consumers but whose pool is full waits: back-pressure.
//
// Only a few items are live at a time (an item dies once its consumers ran),
// so a candidate needs P pools of a few hundred bytes, where a table of end
// times by op would need 4 bytes per op: many more candidates stay resident
// per CU, which is what hides the LDS and cache latencies of the round loop.
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

constexpr uint32_t kTagBits = 22;
constexpr uint32_t kTagMask = (1u << kTagBits) - 1u;
constexpr uint32_t kOneReader = 1u << kTagBits;
constexpr uint32_t kNoTag = kTagMask;  // never an item's tag: matches nothing

__device__ __forceinline__ uint32_t ld32(uint32_t addr) {
  return *reinterpret_cast<const uint32_t *>(p_lds + addr);
}
__device__ __forceinline__ uint4 ld128(uint32_t addr) {
  return *reinterpret_cast<const uint4 *>(p_lds + addr);
}
__device__ __forceinline__ void st32(uint32_t addr, uint32_t v) {
  *reinterpret_cast<uint32_t *>(p_lds + addr) = v;
}
__device__ __forceinline__ void st64(uint32_t addr, uint32_t lo, uint32_t hi) {
  *reinterpret_cast<uint2 *>(p_lds + addr) = make_uint2(lo, hi);
}
__device__ __forceinline__ uint32_t *lds_word(uint32_t addr) {
  return reinterpret_cast<uint32_t *>(__builtin_assume_aligned(p_lds + addr, 4));
}
__device__ __forceinline__ void lds_or(uint32_t addr, uint32_t v) {
  (void)__hip_atomic_fetch_or(lds_word(addr), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
}
__device__ __forceinline__ void lds_and(uint32_t addr, uint32_t v) {
  (void)__hip_atomic_fetch_and(lds_word(addr), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
}

template <int PWL, int S>
__global__ __launch_bounds__(256) void pool_kernel(PoolArgs a) {
  constexpr int PW = 1 << PWL;
  constexpr int G = kWave / PW;
  constexpr uint32_t kPool = 16u + 8u * S;
  constexpr uint32_t kFull = S == 32 ? 0xffffffffu : ((1u << S) - 1u);
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int grp = lane >> PWL;
  const int r = lane & (PW - 1);
  const bool on = r < a.P;
  const int gbit = grp << PWL;
  const int64_t n_slots = int64_t(gridDim.x) * a.wpb * G;
  const uint32_t gbase = uint32_t(wave * G + grp) * uint32_t(a.P) * kPool;
  const uint32_t my_pool = gbase + uint32_t(on ? r : 0) * kPool;

  int rb = 0, nr = 0, busy_r = 0;
  if (on) {
    rb = a.rank_off[r];
    nr = a.rank_off[r + 1] - rb;
    busy_r = a.busy[r];
  }
  const int last = max(nr - 1, 0);

  int64_t cand = (int64_t(blockIdx.x) * a.wpb + wave) * G + grp;
  bool has = false;   // the group holds a candidate
  bool act = false;   // this lane has an op to run
  uint8_t fl = 0;     // the check kernel's flags for the candidate
  int ptr = 0;
  uint32_t tfree = 0, acc = 0, mine = 0;
  int j = 0;
  int4 cur = make_int4(0, 0, 0, 0);               // {cost, item word, preds, first edge}
  int4 ce = make_int4(0, int(kNoTag), 0, 0);      // current edge {pred rank, tag, comm, 0}
  int4 n0 = cur, n1 = ce;                         // record of the op at ptr + 1
  int nid2 = 0;                                   // id at ptr + 2
  const int16_t *row = a.orders;

  auto load_rec = [&](int id, int4 &r0, int4 &r1) {
    const int4 *p = a.rec + 2 * int64_t(rb + id);
    r0 = p[0];
    r1 = p[1];
  };

  // All lanes of the group call this together.
  auto start_candidate = [&]() {
    while (cand < a.n_cand && (a.out_flags[cand] & DIP_FLAG_INVALID)) cand += n_slots;
    has = cand < a.n_cand;
    act = false;
    ce.y = int(kNoTag);
    if (!has) return;
    fl = a.out_flags[cand];
    if (on) {
      uint4 *p = reinterpret_cast<uint4 *>(p_lds + my_pool);
#pragma unroll
      for (int i = 0; i < int(kPool / 16); ++i) p[i] = make_uint4(0, 0, 0, 0);
    }
    ptr = 0;
    tfree = 0;
    acc = 0;
    mine = 0;
    j = 0;
    if (on && nr > 0) {
      row = a.orders + cand * a.stride + rb;
      const int id0 = min(max(int(row[0]), 0), last);
      const int id1 = min(max(int(row[min(1, last)]), 0), last);
      nid2 = min(max(int(row[min(2, last)]), 0), last);
      int4 c1;
      load_rec(id0, cur, c1);
      load_rec(id1, n0, n1);
      ce = cur.z > 0 ? c1 : make_int4(0, int(kNoTag), 0, 0);
      act = true;
    }
  };

  start_candidate();
  uint64_t g_has = any_in_group<PWL>(__builtin_amdgcn_ballot_w64(has));
  uint32_t round = 0;

  while (g_has) {
    // ---- reads: the predecessor's pool, my freed mask
    const uint32_t pa = gbase + uint32_t(ce.x) * kPool;
    uint4 q[S / 2];
#pragma unroll
    for (int i = 0; i < S / 2; ++i) q[i] = ld128(pa + 16u + 16u * i);
    const uint32_t fw = ld32(my_pool);
    lds_wait();

    const uint32_t want = uint32_t(ce.y);
    bool found = false;
    uint32_t hit_t = 0, hit_v = 0, hit = 0;
#pragma unroll
    for (int i = 0; i < S; ++i) {
      const uint32_t t = (i & 1) ? q[i / 2].z : q[i / 2].x;
      const uint32_t v = (i & 1) ? q[i / 2].w : q[i / 2].y;
      const bool m = (t & kTagMask) == want;
      found = found || m;
      hit_t = m ? t : hit_t;
      hit_v = m ? v : hit_v;
      hit = m ? uint32_t(i) : hit;
    }
    mine &= ~fw;
    const uint32_t free_m = ~mine & kFull;
    const uint32_t acc_n = found ? max(acc, hit_v + uint32_t(ce.z)) : acc;
    const int j_n = j + (found ? 1 : 0);
    const bool ready = act && j_n >= cur.z;
    const bool need_out = cur.y != 0;
    const bool fire = ready && (!need_out || free_m != 0u);
    const bool held = ready && !fire;
    const uint32_t en = max(tfree, acc_n) + uint32_t(cur.x);

    // ---- writes
    if (found) {
      if ((hit_t >> kTagBits) == 1u) lds_or(pa, 1u << hit);   // last reader frees
      else st32(pa + 16u + 8u * hit, hit_t - kOneReader);
    }
    if (on && fw != 0u) lds_and(my_pool, ~fw);
    if (fire && need_out) {
      const uint32_t s = uint32_t(__builtin_ctz(free_m));
      st64(my_pool + 16u + 8u * s, uint32_t(cur.y), en);
      mine |= 1u << s;
    }

    // ---- register state
    bool fin = false;
    if (fire) {
      tfree = en;
      acc = 0;
      j = 0;
      ++ptr;
      fin = ptr == nr;
      if (fin) {
        act = false;
        ce = make_int4(0, int(kNoTag), 0, 0);
      } else {
        cur = n0;
        ce = cur.z > 0 ? n1 : make_int4(0, int(kNoTag), 0, 0);
        load_rec(nid2, n0, n1);
        nid2 = min(max(int(row[min(ptr + 2, last)]), 0), last);
      }
    } else if (found) {
      acc = acc_n;
      j = j_n;
      ce = j_n < cur.z ? a.edge[cur.w + j_n] : make_int4(0, int(kNoTag), 0, 0);
    }

    ++round;
    const uint64_t b_fin = __builtin_amdgcn_ballot_w64(fin);
    const bool stall_check = (round & 7u) == 0u;
    if (!b_fin && !stall_check) continue;
    const uint64_t g_run = any_in_group<PWL>(__builtin_amdgcn_ballot_w64(act));
    const uint64_t ev_done = g_has & ~g_run;
    uint64_t ev_stall = 0;
    if (stall_check)
      ev_stall = g_run & ~any_in_group<PWL>(__builtin_amdgcn_ballot_w64(fire || found));
    const uint64_t ev = ev_done | ev_stall;
    if (ev == 0) continue;

    // ---- some groups finished their candidate
    const uint64_t g_held = any_in_group<PWL>(__builtin_amdgcn_ballot_w64(held));
    const bool mine_ev = (ev >> gbit) & 1;
    if (mine_ev) {
      const bool stalled = (ev_stall >> gbit) & 1;
      const bool retry = stalled && ((g_held >> gbit) & 1);
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
      cand += n_slots;
      start_candidate();
    }
    g_has = any_in_group<PWL>(__builtin_amdgcn_ballot_w64(has));
  }
}

template <int S>
const void *ptr_s(int pwl) {
  switch (pwl) {
    case 0: return reinterpret_cast<const void *>(pool_kernel<0, S>);
    case 1: return reinterpret_cast<const void *>(pool_kernel<1, S>);
    case 2: return reinterpret_cast<const void *>(pool_kernel<2, S>);
    case 3: return reinterpret_cast<const void *>(pool_kernel<3, S>);
    case 4: return reinterpret_cast<const void *>(pool_kernel<4, S>);
    case 5: return reinterpret_cast<const void *>(pool_kernel<5, S>);
    default: return reinterpret_cast<const void *>(pool_kernel<6, S>);
  }
}

template <int S>
void launch_s(int pwl, dim3 grid, dim3 block, size_t lds, hipStream_t s, const PoolArgs &a) {
  switch (pwl) {
    case 0: pool_kernel<0, S><<<grid, block, lds, s>>>(a); break;
    case 1: pool_kernel<1, S><<<grid, block, lds, s>>>(a); break;
    case 2: pool_kernel<2, S><<<grid, block, lds, s>>>(a); break;
    case 3: pool_kernel<3, S><<<grid, block, lds, s>>>(a); break;
    case 4: pool_kernel<4, S><<<grid, block, lds, s>>>(a); break;
    case 5: pool_kernel<5, S><<<grid, block, lds, s>>>(a); break;
    default: pool_kernel<6, S><<<grid, block, lds, s>>>(a); break;
  }
}

}  // namespace

bool pool_slots_ok(int slots) { return slots == 2 || slots == 4 || slots == 8 || slots == 16; }

const void *pool_kernel_ptr(int pwl, int slots) {
  switch (slots) {
    case 2: return ptr_s<2>(pwl);
    case 4: return ptr_s<4>(pwl);
    case 16: return ptr_s<16>(pwl);
    default: return ptr_s<8>(pwl);
  }
}

hipError_t launch_pool(int pwl, int slots, int blocks, int wpb, size_t lds, hipStream_t s,
                       const PoolArgs &a) {
  const dim3 grid(blocks), block(wpb * kWave);
  switch (slots) {
    case 2: launch_s<2>(pwl, grid, block, lds, s, a); break;
    case 4: launch_s<4>(pwl, grid, block, lds, s, a); break;
    case 16: launch_s<16>(pwl, grid, block, lds, s, a); break;
    default: launch_s<8>(pwl, grid, block, lds, s, a); break;
  }
  return hipGetLastError();
}

}  // namespace dipsim
