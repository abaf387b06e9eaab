// kern_pipe.hip -- simulation kernel for pipeline-shaped instances: every op
// has at most one predecessor, or several predecessors that all run on one
// rank (the all-to-all joins between modality segments), and every time
// stays below 2^30.
//
// Lane mapping: one wavefront holds G = 64 / PW candidate groups of PW lanes
// (PW = next power of two >= P); lane r of a group is physical rank r of the
// group's current candidate, the rank that runs one pipeline stage at a time
// (Sec. 5.2).  Groups advance independently: when a group finishes a
// candidate it writes the outputs and starts its next one while the other
// groups of the wave keep simulating.
//
// A round, per running lane: read ONE end-time entry (the predecessor's, the
// join entry of a multi-predecessor op, or the group's zero cell) and the
// lane's own entry (a repeated id in the order shows up as already fired);
// if the predecessor has fired,
//     start = max(free, end(pred) + comm),   end = start + cost,
// publish end(op), add the op's activation delta to the running memory sum
// and its running max, and move on to the next op, whose record was loaded
// one op ahead.  Readiness never goes away once reached, so a group that
// fires nothing in a round while ops remain is deadlocked.
//
// Joins: an op o with k >= 2 predecessors owns a join block in the table
// {J, -, Amax, Acnt}.  Its predecessors (one rank, so one lane, in order)
// fold end + comm(p, o) into Amax and count in Acnt; the k-th arrival
// publishes J = max, which o polls as its single predecessor (comm 0), and
// clears Acnt.  So ready(o) = all k arrived and
// start(o) = max(free, max_p end(p) + comm(p, o)), as for any other op.
//
// End-time entries are (epoch << 30) | end.  Each group flips its epoch bit
// when it starts a candidate, which turns every entry of the previous
// candidate into "not fired" without clearing the table.  Invariant: a
// finished candidate leaves every op entry and join entry stamped with its
// epoch and every Acnt at 0 (fired; or stamped by the deadlock tail and the
// join reset; or by the full stamp of an invalid candidate).
//
// Order rows stream from HBM through a per-lane 64-bit window of four int16
// ids with the next four prefetched, so no order staging occupies LDS.
//
// Template parameters: PWL = log2(PW); GS = end-time tables in device scratch
// instead of LDS (for instances whose tables leave too few waves resident).
#include "dip_sim.h"
#include "internal.h"

namespace dipsim {
namespace {

extern __shared__ __align__(16) int32_t p_lds[];

enum : int { kOff = 0, kRun = 1, kDone = 2 };

// Mask with the lowest lane of every PW-lane group set.
template <int PWL>
constexpr uint64_t group_low_lanes() {
  uint64_t low = 1;
  for (int s = 1 << PWL; s < 64; s <<= 1) low |= low << s;
  return low;
}

// One bit per PW-lane group (at the group's lowest lane) for groups with any
// lane set in m.
template <int PWL>
__device__ __forceinline__ uint64_t group_any(uint64_t m) {
#pragma unroll
  for (int s = 1; s < (1 << PWL); s <<= 1) m |= m >> s;
  return m & group_low_lanes<PWL>();
}

template <bool GS>
__device__ __forceinline__ uint32_t tload(int32_t *tab, uint32_t byte_off) {
  int32_t *p = reinterpret_cast<int32_t *>(reinterpret_cast<char *>(tab) + byte_off);
  if constexpr (GS) return uint32_t(__hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP));
  else return uint32_t(*p);
}

template <bool GS>
__device__ __forceinline__ void tstore(int32_t *tab, uint32_t byte_off, uint32_t v) {
  int32_t *p = reinterpret_cast<int32_t *>(reinterpret_cast<char *>(tab) + byte_off);
  if constexpr (GS) __hip_atomic_store(p, int32_t(v), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  else *p = int32_t(v);
}

// Orders one round's table writes before the next round's reads.  Lanes of
// a group share a wavefront, so for LDS tables it is enough that the wave's
// LDS operations have completed (they execute in order); a workgroup fence
// would also drain every outstanding global load, including the prefetches.
// Device-scratch tables need the workgroup release/acquire.
template <bool GS>
__device__ __forceinline__ void round_fence() {
  if constexpr (GS) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  } else {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  }
}

struct OpRec {
  uint32_t cost;
  int32_t md;
  uint32_t poff;    // byte offset of the polled entry
  uint32_t pcomm;
  uint32_t jblk;    // byte offset of the join block this op feeds, 0 = none
  uint32_t jk;      // predecessors of that join
  uint32_t jcomm;   // latency of this op's edge into the join
  uint32_t g_off;   // byte offset of this op's own entry
};

template <int PWL, bool GS>
__global__ __launch_bounds__(256) void pipe_kernel(PipeArgs a) {
  constexpr int PW = 1 << PWL;
  constexpr int G = kWave / PW;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int grp = lane >> PWL;
  const int r = lane & (PW - 1);
  const bool on = r < a.P;
  const int64_t slot = (int64_t(blockIdx.x) * a.wpb + wave) * G + grp;
  const int64_t n_slots = int64_t(gridDim.x) * a.wpb * G;
  const uint32_t zero_off = uint32_t(a.N) * 4u;
  const int gbit = grp << PWL;

  int32_t *tab;
  uint32_t e;  // epoch bit of the group's table
  if constexpr (GS) {
    tab = a.gtab + slot * a.tab_stride;
    e = a.gepoch[slot] & 1u;
  } else {
    int32_t *wtab = p_lds + int64_t(wave) * G * a.tab_stride;
    const int n4 = G * a.tab_stride / 4;
    int4 *w4 = reinterpret_cast<int4 *>(wtab);
    for (int i = lane; i < n4; i += kWave) w4[i] = make_int4(0, 0, 0, 0);
    tab = wtab + grp * a.tab_stride;
    e = 0;
    round_fence<GS>();
  }

  int rb = 0, nr = 0, busy_r = 0, cap_r = -1;
  if (on) {
    rb = a.rank_off[r];
    nr = a.rank_off[r + 1] - rb;
    busy_r = a.busy[r];
    cap_r = a.cap[r];
  }
  const int sec_end = rb + nr;
  // last 4-aligned block of the section: window loads past it are clamped
  const int q_last = (sec_end - 1) & ~3;

  int64_t cand = slot;
  bool has = false;  // this group holds a candidate
  int st = kOff;
  bool bad = false;
  int ptr = 0;
  uint32_t tfree = 0;
  int mem = 0, peak = 0;
  uint32_t emask = 0;
  OpRec cur{}, nxt{};
  bool nxt_ok = true;  // the id behind 'nxt' was in range
  const uint64_t *row = nullptr;
  uint64_t win = 0, wnext = 0;
  int left = 0, wq = 0;

  auto pop = [&]() -> int {
    const int o = int(int16_t(uint16_t(win & 0xffffu)));
    win >>= 16;
    if (--left == 0) {
      win = wnext;
      left = 4;
      wnext = row[min(wq, q_last) >> 2];
      wq += 4;
    }
    return o;
  };
  // Load the record of the next id of the order (clamped into the section;
  // an out-of-range id is remembered and reported when it becomes current).
  auto load_next = [&]() {
    const int o = pop();
    nxt_ok = unsigned(o) < unsigned(nr);
    const int g = rb + (nxt_ok ? o : 0);
    const int4 *rp = a.rec + int64_t(g) * 2;
    const int4 q0 = rp[0];
    const int4 q1 = rp[1];
    nxt.cost = uint32_t(q0.x);
    nxt.md = q0.y;
    nxt.poff = uint32_t(q0.z);
    nxt.pcomm = uint32_t(q0.w);
    nxt.jblk = uint32_t(q1.x);
    nxt.jk = uint32_t(q1.y);
    nxt.jcomm = uint32_t(q1.z);
    nxt.g_off = uint32_t(g) * 4u;
  };
  auto start_candidate = [&]() {
    e ^= 1u;
    emask = e << kEpochShift;
    if (r == 0) tstore<GS>(tab, zero_off, emask);  // predecessor-less ops read 0 here
    ptr = 0; tfree = 0; mem = 0; peak = 0; bad = false;
    st = (on && nr > 0) ? kRun : (on ? kDone : kOff);
    if (st == kRun) {
      row = reinterpret_cast<const uint64_t *>(a.orders + cand * a.stride);
      const int q0 = rb & ~3;
      win = row[q0 >> 2];
      wnext = row[min(q0 + 4, q_last) >> 2];
      wq = q0 + 8;
      left = 4;
      for (int s = rb - q0; s > 0; --s) { win >>= 16; --left; }
      load_next();
      cur = nxt;
      bad = !nxt_ok;
      load_next();
    }
  };

  if (cand < a.n_cand) { has = true; start_candidate(); }
  uint64_t g_has = group_any<PWL>(__builtin_amdgcn_ballot_w64(has));

  while (g_has) {
    round_fence<GS>();
    bool fired = false;
    if (st == kRun && !bad) {
      const uint32_t y = tload<GS>(tab, cur.poff) ^ emask;
      const uint32_t own = tload<GS>(tab, cur.g_off) ^ emask;
      const bool dup = own < kValueLimit;  // this id already fired: not a permutation
      bad = dup;
      if (!dup && y < kValueLimit) {
        const uint32_t en = max(tfree, y + cur.pcomm) + cur.cost;
        tstore<GS>(tab, cur.g_off, en | emask);
        if (cur.jblk) {
          // fold into the join this op feeds; the last arrival publishes it
          const uint32_t v = en + cur.jcomm;
          const uint32_t amax = tload<GS>(tab, cur.jblk + 8);
          const uint32_t acnt = tload<GS>(tab, cur.jblk + 12);
          const uint32_t mx = acnt == 0 ? v : max(amax, v);
          if (acnt + 1 == cur.jk) {
            tstore<GS>(tab, cur.jblk, mx | emask);
            tstore<GS>(tab, cur.jblk + 12, 0u);
          } else {
            tstore<GS>(tab, cur.jblk + 8, mx);
            tstore<GS>(tab, cur.jblk + 12, acnt + 1);
          }
        }
        tfree = en;
        mem += cur.md;
        peak = max(peak, mem);
        fired = true;
        if (++ptr == nr) {
          st = kDone;
        } else {
          cur = nxt;
          bad = !nxt_ok;
          load_next();
        }
      }
    }
    const uint64_t b_fire = __builtin_amdgcn_ballot_w64(fired);
    const uint64_t b_run = __builtin_amdgcn_ballot_w64(st == kRun && !bad);
    const uint64_t b_bad = __builtin_amdgcn_ballot_w64(bad);
    const uint64_t g_run = group_any<PWL>(b_run);
    const uint64_t g_bad = b_bad ? group_any<PWL>(b_bad) : 0ull;
    const uint64_t ev_bad = g_has & g_bad;
    const uint64_t ev_stall = g_run & ~group_any<PWL>(b_fire) & ~g_bad;
    const uint64_t ev_done = g_has & ~g_run & ~g_bad;
    const uint64_t ev = ev_bad | ev_stall | ev_done;
    if (ev == 0) continue;

    // ---- some groups finished their candidate this round
    const bool mine = (ev >> gbit) & 1;
    const bool stalled = (ev_stall >> gbit) & 1;
    if (mine && stalled && st == kRun && !bad) {
      // deadlock tail: stamp the current and remaining ids of the order
      // (catching ids out of range or repeated) and finish the memory scan
      tstore<GS>(tab, cur.g_off, emask);
      mem += cur.md;
      peak = max(peak, mem);
      bool ok = nxt_ok;
      OpRec t = nxt;
      for (int i = ptr + 1; i < nr; ++i) {
        if (!ok || (tload<GS>(tab, t.g_off) ^ emask) < kValueLimit) { bad = true; break; }
        tstore<GS>(tab, t.g_off, emask);
        mem += t.md;
        peak = max(peak, mem);
        if (i + 1 < nr) {
          const int o = pop();
          ok = unsigned(o) < unsigned(nr);
          const int g = rb + (ok ? o : 0);
          t.g_off = uint32_t(g) * 4u;
          t.md = a.md[g];
        }
      }
    }
    const uint64_t g_bad2 = group_any<PWL>(__builtin_amdgcn_ballot_w64(bad));
    const bool over = on && cap_r >= 0 && peak > cap_r;
    const uint64_t g_cap = group_any<PWL>(__builtin_amdgcn_ballot_w64(over));
    if (mine) {
      const bool is_bad = (g_bad2 >> gbit) & 1;
      const bool is_cap = (g_cap >> gbit) & 1;
      uint32_t T = on ? tfree : 0u;
#pragma unroll
      for (int off = 1; off < PW; off <<= 1) T = max(T, uint32_t(__shfl_xor(int(T), off, kWave)));
      if (on) {
        const int64_t o = cand * a.P + r;
        if (is_bad) {
          a.out_bub[o] = -1;
          a.out_peak[o] = -1;
        } else {
          a.out_bub[o] = stalled ? -1 : int32_t(T) - busy_r;
          a.out_peak[o] = peak;
        }
        if (r == 0) {
          a.out_ms[cand] = (is_bad || stalled) ? -1 : int32_t(T);
          a.out_flags[cand] = is_bad ? uint8_t(DIP_FLAG_INVALID)
                                     : uint8_t((stalled ? DIP_FLAG_DEADLOCK : 0u) |
                                               (is_cap ? DIP_FLAG_CAP : 0u));
        }
      }
      if (is_bad) {
        // an invalid row may have left op entries unstamped: stamp them all
        for (int i = r; i < a.N; i += PW) tstore<GS>(tab, uint32_t(i) * 4u, emask);
      }
      if (is_bad || stalled) {
        // joins left incomplete: stamp their entries, clear their counts
        for (int j = r; j < a.n_joins; j += PW) {
          const uint32_t jb = a.join_base + uint32_t(j) * 16u;
          tstore<GS>(tab, jb, emask);
          tstore<GS>(tab, jb + 12, 0u);
        }
      }
      cand += n_slots;
      if (cand < a.n_cand) {
        start_candidate();
      } else {
        has = false;
        st = kOff;
      }
    }
    g_has = group_any<PWL>(__builtin_amdgcn_ballot_w64(has));
  }
  if constexpr (GS) {
    if (r == 0) a.gepoch[slot] = uint8_t(e);
  }
}

template <bool GS>
const void *ptr_for(int pwl) {
  switch (pwl) {
    case 0: return reinterpret_cast<const void *>(pipe_kernel<0, GS>);
    case 1: return reinterpret_cast<const void *>(pipe_kernel<1, GS>);
    case 2: return reinterpret_cast<const void *>(pipe_kernel<2, GS>);
    case 3: return reinterpret_cast<const void *>(pipe_kernel<3, GS>);
    case 4: return reinterpret_cast<const void *>(pipe_kernel<4, GS>);
    case 5: return reinterpret_cast<const void *>(pipe_kernel<5, GS>);
    default: return reinterpret_cast<const void *>(pipe_kernel<6, GS>);
  }
}

template <bool GS>
void launch_for(int pwl, dim3 grid, dim3 block, size_t lds, hipStream_t s, const PipeArgs &a) {
  switch (pwl) {
    case 0: pipe_kernel<0, GS><<<grid, block, lds, s>>>(a); break;
    case 1: pipe_kernel<1, GS><<<grid, block, lds, s>>>(a); break;
    case 2: pipe_kernel<2, GS><<<grid, block, lds, s>>>(a); break;
    case 3: pipe_kernel<3, GS><<<grid, block, lds, s>>>(a); break;
    case 4: pipe_kernel<4, GS><<<grid, block, lds, s>>>(a); break;
    case 5: pipe_kernel<5, GS><<<grid, block, lds, s>>>(a); break;
    default: pipe_kernel<6, GS><<<grid, block, lds, s>>>(a); break;
  }
}

}  // namespace

const void *pipe_kernel_ptr(int pwl, bool gs) {
  return gs ? ptr_for<true>(pwl) : ptr_for<false>(pwl);
}

hipError_t launch_pipe(int pwl, bool gs, int blocks, int wpb, size_t lds, hipStream_t s,
                       const PipeArgs &a) {
  const dim3 grid(blocks), block(wpb * kWave);
  if (gs) launch_for<true>(pwl, grid, block, lds, s, a);
  else launch_for<false>(pwl, grid, block, lds, s, a);
  return hipGetLastError();
}

}  // namespace dipsim
