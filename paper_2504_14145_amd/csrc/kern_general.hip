// kern_general.hip -- simulation kernel for arbitrary DAGs (any number of
// predecessors per op, walked through the CSR).
//
// One wavefront simulates G candidates side by side: its 64 lanes split into
// G groups of PW lanes (PW = next power of two >= P), and lane r of a group
// plays physical rank r of that group's candidate, the rank that runs one
// pipeline stage at a time (Sec. 5.2).  Every lane walks its rank's order; in
// each round a lane fires its next op if all of the op's predecessors have
// ended, computing
//     start = max(free, max_p end(p) + comm(p)),  end = start + cost
// and publishing end(op) in its group's end-time table, where consumers on
// other lanes read it.  A wave ballot after each round tells every group
// whether any of its lanes fired; a round without progress while ops remain
// is a deadlock, because readiness never goes away once reached.  The memory
// scan (+act at a forward, -act at a backward, running max) rides along with
// each fire; ranks stalled by a deadlock finish their scan (and the
// permutation check) in a tail pass.  Makespan is a max-reduction over the
// group's lanes by cross-lane shuffles.
//
// Where the tables live is the variant:
//   1: op records + edges, order rows and end-time tables all in LDS;
//   2: op records/edges read through the caches, rows and end times in LDS;
//   3: only end times in LDS (rows read straight from HBM);
//   4: end times in device scratch (one region per resident wave).
//
// With a memory selection (Sec. 5.3) an op's cost and activation come from
// its stage pair's chosen candidate instead: the backward runs the
// candidate's extra time (its recomputation), and the pair holds the
// candidate's memory from its forward to its backward.
#include "dip_sim.h"
#include "internal.h"

namespace dipsim {
namespace {

using SimArgs = GeneralArgs;

enum : int { kOff = 0, kRun = 1, kDone = 2, kStall = 3 };

extern __shared__ __align__(16) unsigned char g_lds[];

template <int V>
__device__ __forceinline__ int4 load_rec(const SimArgs &a, int g) {
  if constexpr (V == 1) return reinterpret_cast<const int4 *>(g_lds)[g];
  else return a.rec[g];
}

template <int V>
__device__ __forceinline__ int2 load_edge(const SimArgs &a, int e) {
  if constexpr (V == 1)
    return reinterpret_cast<const int2 *>(g_lds + align16(int64_t(a.N) * 16))[e];
  else return a.edge[e];
}

template <int V>
__device__ __forceinline__ int load_order(const SimArgs &a, uint32_t ord_off, int grp,
                                          int64_t cand, int idx) {
  if constexpr (V <= 2)
    return reinterpret_cast<const int16_t *>(g_lds + ord_off)[int64_t(grp) * a.stride + idx];
  else return a.orders[cand * a.stride + idx];
}

template <int V>
__device__ __forceinline__ int load_end(const SimArgs &a, uint32_t end_off, int32_t *gbase,
                                        int g) {
  if constexpr (V <= 3) return reinterpret_cast<const int32_t *>(g_lds + end_off)[g];
  else return __hip_atomic_load(gbase + g, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

template <int V>
__device__ __forceinline__ void store_end(const SimArgs &a, uint32_t end_off, int32_t *gbase,
                                          int g, int v) {
  if constexpr (V <= 3) reinterpret_cast<int32_t *>(g_lds + end_off)[g] = v;
  else __hip_atomic_store(gbase + g, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Orders one round's end-time writes before the next round's reads: an
// LDS-only wait when the tables live in LDS (variants 1-3; the lanes of a
// group share a wavefront and its LDS operations execute in order), the
// workgroup release/acquire pair for tables in device scratch (variant 4).
template <int V>
__device__ __forceinline__ void round_fence() {
  if constexpr (V == 4) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  } else {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  }
}

// Cost and memory change of op g in candidate cand: its record's, or under a
// memory selection those of its pair's chosen candidate (the backward adds
// the candidate's time over the pair's fastest).  false for a choice beyond
// the pair's candidates.
__device__ __forceinline__ bool op_cost_mem(const SimArgs &a, const int4 &rc, int g, int64_t cand,
                                            int pair_base, int &cost, int &dmem) {
  cost = rc.x;
  dmem = rc.y;
  if (!a.choice) return true;
  const uint32_t w = uint32_t(a.lid_pair[g]);
  const int p = pair_base + int(w & 0x7fffffffu);
  const int c = a.choice[cand * a.n_pairs + p];
  if (c >= kMemoptMaxCands ||
      (c > 0 && a.cand_key[int64_t(p) * kMemoptMaxCands + c - 1] == kMemoptNoMove))
    return false;
  const int32_t m = a.cand_mem[int64_t(p) * kMemoptMaxCands + c];
  if (w >> 31) {
    cost += int(a.cand_time[int64_t(p) * kMemoptMaxCands + c] -
                a.cand_time[int64_t(p) * kMemoptMaxCands]);
    dmem = -m;
  } else {
    dmem = m;
  }
  return true;
}

__device__ __forceinline__ uint64_t group_bits(uint64_t ballot, int grp, int pwl) {
  if (pwl == 6) return ballot;
  const int pw = 1 << pwl;
  return (ballot >> (grp * pw)) & ((uint64_t(1) << pw) - 1);
}

template <int V>
__global__ __launch_bounds__(256) void sim_kernel(SimArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int pw = 1 << a.pwl;
  const int grp = lane >> a.pwl;
  const int r = lane & (pw - 1);
  const bool lane_on = grp < a.G && r < a.P;

  if constexpr (V == 1) {
    // op records and edges, shared by every wave of the block
    int4 *srec = reinterpret_cast<int4 *>(g_lds);
    int2 *sedge = reinterpret_cast<int2 *>(g_lds + align16(int64_t(a.N) * 16));
    for (int i = threadIdx.x; i < a.N; i += blockDim.x) srec[i] = a.rec[i];
    for (int i = threadIdx.x; i < a.E; i += blockDim.x) sedge[i] = a.edge[i];
    __syncthreads();
  }
  const uint32_t wave_off = a.tab_bytes + uint32_t(wave) * (a.ord_bytes + a.end_bytes);
  const uint32_t ord_off = wave_off;
  const uint32_t end_off = wave_off + a.ord_bytes + uint32_t(grp) * uint32_t(a.N) * 4u;
  const int64_t wslot = int64_t(blockIdx.x) * a.wpb + wave;
  int32_t *gbase = nullptr;
  if constexpr (V == 4) gbase = a.gends + (wslot * a.G + grp) * int64_t(a.N);

  int rb = 0, nr = 0, busy_r = 0, cap_r = -1, pair_base = 0;
  if (lane_on) {
    rb = a.rank_off[r];
    nr = a.rank_off[r + 1] - rb;
    busy_r = a.busy[r];
    cap_r = a.cap[r];
    if (a.choice) pair_base = a.pair_off[r];
  }

  const int64_t total_waves = int64_t(gridDim.x) * a.wpb;
  int64_t n_items = a.n_cand, n_groups = a.n_groups;
  if constexpr (V >= 3) {
    if (a.list) {
      n_items = int64_t(*a.list_count);
      n_groups = (n_items + a.G - 1) / a.G;
    }
  }
  for (int64_t cg = wslot; cg < n_groups; cg += total_waves) {
    const int64_t c0 = cg * a.G;
    const int64_t item = c0 + grp;
    const bool live = lane_on && item < n_items;
    int64_t cand = item;
    if constexpr (V >= 3) {
      if (a.list) cand = live ? a.list[item] : 0;
    }
    const int64_t n_here = min<int64_t>(a.G, n_items - c0);

    // ---- stage this wave's order rows (coalesced 16-byte loads) and reset
    //      the end-time tables to "not fired" (-1)
    if constexpr (V <= 2) {
      const int64_t n16 = n_here * a.stride * 2 / 16;
      const uint4 *src = reinterpret_cast<const uint4 *>(a.orders + c0 * a.stride);
      uint4 *dst = reinterpret_cast<uint4 *>(g_lds + ord_off);
      for (int64_t i = lane; i < n16; i += kWave) dst[i] = src[i];
    }
    if constexpr (V <= 3) {
      int32_t *tab = reinterpret_cast<int32_t *>(g_lds + wave_off + a.ord_bytes);
      const int n_words = a.G * a.N;
      for (int i = lane; i < n_words; i += kWave) tab[i] = -1;
    } else {
      if (live)  // the group's lanes share the reset of its table
        for (int i = r; i < a.N; i += a.P)
          __hip_atomic_store(gbase + i, -1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
    round_fence<V>();

    int ptr = 0, tfree = 0, mem = 0, peak = 0;
    int busy_run = 0;   // the rank's fired op time (its busy time under a selection)
    bool bad = false;
    int st = live ? (nr > 0 ? kRun : kDone) : kOff;

    // ---- rounds: every running lane tries to fire its next op
    for (;;) {
      bool fired = false;
      if (st == kRun) {
        const int o = load_order<V>(a, ord_off, grp, cand, rb + ptr);
        if (unsigned(o) >= unsigned(nr)) {
          bad = true;
        } else {
          const int g = rb + o;
          const int4 rc = load_rec<V>(a, g);
          int cost = 0, dmem = 0;
          if (load_end<V>(a, end_off, gbase, g) != -1) {
            bad = true;  // the id already fired: not a permutation
          } else if (!op_cost_mem(a, rc, g, cand, pair_base, cost, dmem)) {
            bad = true;  // a choice beyond the pair's candidates
          } else {
            int t = tfree;
            bool ready = true;
            for (int e = rc.z; e < rc.w; ++e) {
              const int2 ed = load_edge<V>(a, e);
              const int pe = load_end<V>(a, end_off, gbase, ed.x);
              ready = ready && pe >= 0;
              t = max(t, pe + ed.y);
            }
            if (ready) {
              const int en = t + cost;
              store_end<V>(a, end_off, gbase, g, en);
              tfree = en;
              busy_run += cost;
              mem += dmem;
              peak = max(peak, mem);
              fired = true;
              if (++ptr == nr) st = kDone;
            }
          }
        }
      }
      const uint64_t b_fire = __builtin_amdgcn_ballot_w64(fired);
      const uint64_t b_bad = __builtin_amdgcn_ballot_w64(bad);
      const uint64_t b_run = __builtin_amdgcn_ballot_w64(st == kRun);
      if (st == kRun) {
        if (group_bits(b_bad, grp, a.pwl)) st = kDone;          // reported invalid
        else if (!group_bits(b_fire, grp, a.pwl)) st = kStall;   // no progress: cycle
      }
      if (!b_run) break;
      round_fence<V>();
    }

    // ---- deadlocked groups: finish the order scan (memory, permutation)
    const uint64_t b_bad0 = __builtin_amdgcn_ballot_w64(bad);
    if (st == kStall && !group_bits(b_bad0, grp, a.pwl)) {
      for (int i = ptr; i < nr; ++i) {
        const int o = load_order<V>(a, ord_off, grp, cand, rb + i);
        if (unsigned(o) >= unsigned(nr)) { bad = true; break; }
        const int g = rb + o;
        if (load_end<V>(a, end_off, gbase, g) != -1) { bad = true; break; }
        store_end<V>(a, end_off, gbase, g, -2);
        int cost = 0, dmem = 0;
        if (!op_cost_mem(a, load_rec<V>(a, g), g, cand, pair_base, cost, dmem)) { bad = true; break; }
        mem += dmem;
        peak = max(peak, mem);
      }
    }

    // ---- group verdicts and outputs
    const uint64_t gb_bad = group_bits(__builtin_amdgcn_ballot_w64(bad), grp, a.pwl);
    const uint64_t gb_stall = group_bits(__builtin_amdgcn_ballot_w64(st == kStall), grp, a.pwl);
    const bool over = live && cap_r >= 0 && peak > cap_r;
    const uint64_t gb_cap = group_bits(__builtin_amdgcn_ballot_w64(over), grp, a.pwl);
    int T = live ? tfree : 0;
    for (int off = 1; off < pw; off <<= 1) T = max(T, __shfl_xor(T, off, kWave));
    if (live) {
      const int64_t o = cand * a.P + r;
      if (gb_bad) {
        a.out_bub[o] = -1;
        a.out_peak[o] = -1;
      } else {
        a.out_bub[o] = gb_stall ? -1 : T - (a.choice ? busy_run : busy_r);
        a.out_peak[o] = peak;
      }
      if (r == 0) {
        a.out_ms[cand] = (gb_bad || gb_stall) ? -1 : T;
        a.out_flags[cand] = gb_bad ? uint8_t(DIP_FLAG_INVALID)
                                   : uint8_t((gb_stall ? DIP_FLAG_DEADLOCK : 0u) |
                                             (gb_cap ? DIP_FLAG_CAP : 0u));
      }
    }
    round_fence<V>();  // this wave's LDS is reused by its next candidate group
  }
}

}  // namespace

const void *general_kernel_ptr(int v) {
  switch (v) {
    case 1: return reinterpret_cast<const void *>(sim_kernel<1>);
    case 2: return reinterpret_cast<const void *>(sim_kernel<2>);
    case 3: return reinterpret_cast<const void *>(sim_kernel<3>);
    default: return reinterpret_cast<const void *>(sim_kernel<4>);
  }
}

hipError_t launch_general(int v, int blocks, int wpb, size_t lds, hipStream_t s,
                          const GeneralArgs &a) {
  const dim3 grid(blocks), block(wpb * kWave);
  switch (v) {
    case 1: sim_kernel<1><<<grid, block, lds, s>>>(a); break;
    case 2: sim_kernel<2><<<grid, block, lds, s>>>(a); break;
    case 3: sim_kernel<3><<<grid, block, lds, s>>>(a); break;
    default: sim_kernel<4><<<grid, block, lds, s>>>(a); break;
  }
  return hipGetLastError();
}

}  // namespace dipsim
