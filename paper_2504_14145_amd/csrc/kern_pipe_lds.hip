// kern_pipe_lds.hip -- the pipeline kernel for instances whose per-candidate
// state fits in LDS: end-time tables, staged order rows and (optionally) the
// op records all live in LDS, so one round costs one LDS round trip.
//
// Same simulation as kern_pipe.hip (lanes = physical ranks, G candidate
// groups per wavefront advancing independently, one polled entry per op,
// join blocks for multi-predecessor ops, epoch-stamped end-time entries);
// see that file for the semantics.  What differs is the round's shape:
//
//   * every LDS read of a round is issued together -- the polled entry, the
//     op's own entry (duplicate check), the record of the next op of the
//     order and the id of the op after it -- and waited on once; firing then
//     advances with register moves, so no dependent access follows it;
//   * a group's row of candidate orders is copied into LDS when the group
//     starts the candidate (PW lanes, 16-byte coalesced copies);
//   * group verdicts are only computed when some lane finished or went bad
//     this round, or every 8th round for deadlocks (a deadlocked group never
//     fires again, so detecting it a few rounds late changes nothing).
//
// Records (16 bytes): {cost, memdelta, poll offset | comm << 16,
// join block offset | join comm << 16}; offsets are bytes into a group's
// table, which the host keeps under 64 KiB, and latencies stay below 2^16.
#include "dip_sim.h"
#include "internal.h"

namespace dipsim {
namespace {

extern __shared__ __align__(16) unsigned char q_lds[];

template <int PWL>
constexpr uint64_t low_lanes() {
  uint64_t low = 1;
  for (int s = 1 << PWL; s < 64; s <<= 1) low |= low << s;
  return low;
}

template <int PWL>
__device__ __forceinline__ uint64_t any_in_group(uint64_t m) {
#pragma unroll
  for (int s = 1; s < (1 << PWL); s <<= 1) m |= m >> s;
  return m & low_lanes<PWL>();
}

__device__ __forceinline__ uint32_t ld32(uint32_t addr) {
  return *reinterpret_cast<const uint32_t *>(q_lds + addr);
}
__device__ __forceinline__ void st32(uint32_t addr, uint32_t v) {
  *reinterpret_cast<uint32_t *>(q_lds + addr) = v;
}
__device__ __forceinline__ int ld_id(uint32_t addr) {
  return *reinterpret_cast<const int16_t *>(q_lds + addr);
}

__device__ __forceinline__ void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

template <int PWL, bool RL>
__global__ __launch_bounds__(256) void pipe_lds_kernel(PipeArgs a) {
  constexpr int PW = 1 << PWL;
  constexpr int G = kWave / PW;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int grp = lane >> PWL;
  const int r = lane & (PW - 1);
  const bool on = r < a.P;
  const int gbit = grp << PWL;
  const int64_t slot = (int64_t(blockIdx.x) * a.wpb + wave) * G + grp;
  const int64_t n_slots = int64_t(gridDim.x) * a.wpb * G;
  const uint32_t tab_bytes = uint32_t(a.tab_stride) * 4u;
  const uint32_t ord_bytes = uint32_t(a.stride) * 2u;
  const uint32_t rec_bytes = RL ? uint32_t(align16(int64_t(a.N) * 16)) : 0u;
  const uint32_t wave_base = rec_bytes + uint32_t(wave) * G * (tab_bytes + ord_bytes);
  const uint32_t tb = wave_base + uint32_t(grp) * tab_bytes;                   // my table
  const uint32_t ob = wave_base + G * tab_bytes + uint32_t(grp) * ord_bytes;  // my row
  const uint32_t zero_off = uint32_t(a.N) * 4u;
  const int last_pos = int(a.stride) - 1;

  // ---- block set-up: records, zeroed tables, the k of every join block
  if constexpr (RL) {
    int4 *rs = reinterpret_cast<int4 *>(q_lds);
    for (int i = threadIdx.x; i < a.N; i += blockDim.x) rs[i] = a.rec16[i];
  }
  {
    int4 *w4 = reinterpret_cast<int4 *>(q_lds + wave_base);
    const int n_tab4 = G * a.tab_stride / 4;
    for (int i = lane; i < n_tab4; i += kWave) w4[i] = make_int4(0, 0, 0, 0);  // G tables, contiguous
    lds_wait();
    for (int i = lane; i < G * a.n_joins; i += kWave) {
      const int gi = i / a.n_joins, j = i - gi * a.n_joins;
      st32(wave_base + uint32_t(gi) * tab_bytes + a.join_base + uint32_t(j) * 16u + 4u,
           uint32_t(a.jk[j]));
    }
  }
  if constexpr (RL) __syncthreads();
  else lds_wait();

  auto rec_at = [&](int g) -> int4 {
    if constexpr (RL) return reinterpret_cast<const int4 *>(q_lds)[g];
    else return a.rec16[g];
  };

  int rb = 0, nr = 0, busy_r = 0, cap_r = -1;
  if (on) {
    rb = a.rank_off[r];
    nr = a.rank_off[r + 1] - rb;
    busy_r = a.busy[r];
    cap_r = a.cap[r];
  }
  // A lane with nothing to fire (finished, invalid, idle) is parked: it polls
  // the never-ready cell, whose bit 31 no epoch mask can clear, so its poll
  // never succeeds and its own-entry check never trips.
  const uint32_t never_off = uint32_t(a.N + 1) * 4u;
  if (r == 0) st32(tb + never_off, 0x80000000u);

  int64_t cand = slot;
  bool has = false;
  int ptr = 0;
  uint32_t tfree = 0;
  int mem = 0, peak = 0;
  uint32_t e = 0, emask = 0;
  int4 cur = make_int4(0, 0, int32_t(never_off), 0);
  uint32_t cur_goff = never_off;
  int nid = 0;              // id at position ptr + 1 (possibly out of range)
  uint32_t oaddr = 0;       // LDS byte address of the id at position ptr + 2
  const uint32_t o_last = ob + uint32_t(last_pos) * 2u;
  bool pend_bad = false;    // set at start when the first id is out of range

  // Called by all PW lanes of a group together.
  auto start_candidate = [&]() {
    const uint4 *src = reinterpret_cast<const uint4 *>(a.orders + cand * a.stride);
    uint4 *dst = reinterpret_cast<uint4 *>(q_lds + ob);
    for (uint32_t i = uint32_t(r); i < ord_bytes / 16u; i += PW) dst[i] = src[i];
    lds_wait();
    e ^= 1u;
    emask = e << kEpochShift;
    if (r == 0) st32(tb + zero_off, emask);  // predecessor-less ops read 0 here
    ptr = 0; tfree = 0; mem = 0; peak = 0; pend_bad = false;
    cur.z = int32_t(never_off);
    cur_goff = never_off;
    if (on && nr > 0) {
      const int id0 = ld_id(ob + uint32_t(rb) * 2u);
      const bool ok0 = unsigned(id0) < unsigned(nr);
      if (ok0) {
        cur = rec_at(rb + id0);
        cur_goff = uint32_t(rb + id0) * 4u;
      }
      pend_bad = !ok0;
      nid = ld_id(ob + uint32_t(min(rb + 1, last_pos)) * 2u);
      oaddr = min(ob + uint32_t(rb + 2) * 2u, o_last);
    }
  };

  if (cand < a.n_cand) { has = true; start_candidate(); }
  uint64_t g_has = any_in_group<PWL>(__builtin_amdgcn_ballot_w64(has));
  uint32_t round = 0;

  while (g_has) {
    lds_wait();
    // ---- one round: all reads, one wait, then branch-free advance
    const uint32_t y_raw = ld32(tb + (uint32_t(cur.z) & 0xffffu));
    const uint32_t own_raw = ld32(tb + cur_goff);
    const bool nid_ok = unsigned(nid) < unsigned(nr);
    const int g1 = rb + (nid_ok ? nid : 0);
    const int4 nrec = rec_at(g1);
    const int id2 = ld_id(oaddr);
    asm volatile("" ::"v"(y_raw), "v"(own_raw), "v"(nrec.x), "v"(nrec.y), "v"(nrec.z),
                 "v"(nrec.w), "v"(id2));
    const uint32_t y = y_raw ^ emask;
    const bool dup = (own_raw ^ emask) < kValueLimit;  // already fired: not a permutation
    const bool fire = !dup && y < kValueLimit;
    const uint32_t en = max(tfree, y + (uint32_t(cur.z) >> 16)) + uint32_t(cur.x);
    if (fire) {
      st32(tb + cur_goff, en | emask);
      const uint32_t jb = uint32_t(cur.w) & 0xffffu;
      if (jb) {
        // fold into the join this op feeds; the last arrival publishes it
        const uint32_t v = en + (uint32_t(cur.w) >> 16);
        const uint32_t jk = ld32(tb + jb + 4u);
        const uint32_t amax = ld32(tb + jb + 8u);
        const uint32_t acnt = ld32(tb + jb + 12u);
        const uint32_t mx = acnt == 0 ? v : max(amax, v);
        if (acnt + 1u == jk) {
          st32(tb + jb, mx | emask);
          st32(tb + jb + 12u, 0u);
        } else {
          st32(tb + jb + 8u, mx);
          st32(tb + jb + 12u, acnt + 1u);
        }
      }
    }
    tfree = fire ? en : tfree;
    mem += fire ? cur.y : 0;
    peak = max(peak, mem);
    ptr += fire ? 1 : 0;
    const bool fin = fire && ptr == nr;
    const bool adv = fire && !fin;
    const bool bad = dup || pend_bad || (adv && !nid_ok);
    pend_bad = false;
    const bool park = fin || bad;
    cur.x = adv ? nrec.x : cur.x;
    cur.y = adv ? nrec.y : cur.y;
    cur.w = adv ? nrec.w : cur.w;
    cur.z = park ? int32_t(never_off) : (adv ? nrec.z : cur.z);
    cur_goff = park ? never_off : (adv ? uint32_t(g1) * 4u : cur_goff);
    nid = adv ? id2 : nid;
    oaddr = adv ? min(oaddr + 2u, o_last) : oaddr;

    ++round;
    const uint64_t b_bad = __builtin_amdgcn_ballot_w64(bad);
    const uint64_t b_fin = __builtin_amdgcn_ballot_w64(fin);
    const bool stall_check = (round & 7u) == 0u;
    if (!(b_bad | b_fin) && !stall_check) continue;
    const uint64_t b_run = __builtin_amdgcn_ballot_w64(cur_goff != never_off);
    const uint64_t g_run = any_in_group<PWL>(b_run);
    const uint64_t g_bad = any_in_group<PWL>(b_bad);
    const uint64_t ev_bad = g_has & g_bad;
    const uint64_t ev_done = g_has & ~g_run & ~g_bad;
    const uint64_t ev_stall =
        stall_check ? (g_run & ~any_in_group<PWL>(__builtin_amdgcn_ballot_w64(fire)) & ~g_bad)
                    : 0ull;
    const uint64_t ev = ev_bad | ev_done | ev_stall;
    if (ev == 0) continue;

    // ---- some groups finished their candidate
    const bool mine = (ev >> gbit) & 1;
    const bool stalled = (ev_stall >> gbit) & 1;
    bool tail_bad = false;
    if (mine && stalled && cur_goff != never_off) {
      // deadlock tail: stamp the current and remaining ids of the order
      // (catching ids out of range or repeated) and finish the memory scan
      st32(tb + cur_goff, emask);
      mem += cur.y;
      peak = max(peak, mem);
      for (int i = ptr + 1; i < nr; ++i) {
        const int o = ld_id(ob + uint32_t(rb + i) * 2u);
        if (unsigned(o) >= unsigned(nr)) { tail_bad = true; break; }
        const uint32_t off = uint32_t(rb + o) * 4u;
        if ((ld32(tb + off) ^ emask) < kValueLimit) { tail_bad = true; break; }
        st32(tb + off, emask);
        mem += rec_at(rb + o).y;
        peak = max(peak, mem);
      }
    }
    const uint64_t g_bad2 = any_in_group<PWL>(__builtin_amdgcn_ballot_w64(bad || tail_bad));
    const bool over = on && cap_r >= 0 && peak > cap_r;
    const uint64_t g_cap = any_in_group<PWL>(__builtin_amdgcn_ballot_w64(over));
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
        for (int i = r; i < a.N; i += PW) st32(tb + uint32_t(i) * 4u, emask);
      }
      if (is_bad || stalled) {
        for (int j = r; j < a.n_joins; j += PW) {
          const uint32_t jb = a.join_base + uint32_t(j) * 16u;
          st32(tb + jb, emask);
          st32(tb + jb + 12u, 0u);
        }
      }
      lds_wait();
      cand += n_slots;
      if (cand < a.n_cand) {
        start_candidate();
      } else {
        has = false;
        cur.z = int32_t(never_off);
        cur_goff = never_off;
      }
    }
    g_has = any_in_group<PWL>(__builtin_amdgcn_ballot_w64(has));
  }
}

template <bool RL>
const void *lds_ptr_for(int pwl) {
  switch (pwl) {
    case 0: return reinterpret_cast<const void *>(pipe_lds_kernel<0, RL>);
    case 1: return reinterpret_cast<const void *>(pipe_lds_kernel<1, RL>);
    case 2: return reinterpret_cast<const void *>(pipe_lds_kernel<2, RL>);
    case 3: return reinterpret_cast<const void *>(pipe_lds_kernel<3, RL>);
    case 4: return reinterpret_cast<const void *>(pipe_lds_kernel<4, RL>);
    case 5: return reinterpret_cast<const void *>(pipe_lds_kernel<5, RL>);
    default: return reinterpret_cast<const void *>(pipe_lds_kernel<6, RL>);
  }
}

template <bool RL>
void lds_launch_for(int pwl, dim3 grid, dim3 block, size_t lds, hipStream_t s,
                    const PipeArgs &a) {
  switch (pwl) {
    case 0: pipe_lds_kernel<0, RL><<<grid, block, lds, s>>>(a); break;
    case 1: pipe_lds_kernel<1, RL><<<grid, block, lds, s>>>(a); break;
    case 2: pipe_lds_kernel<2, RL><<<grid, block, lds, s>>>(a); break;
    case 3: pipe_lds_kernel<3, RL><<<grid, block, lds, s>>>(a); break;
    case 4: pipe_lds_kernel<4, RL><<<grid, block, lds, s>>>(a); break;
    case 5: pipe_lds_kernel<5, RL><<<grid, block, lds, s>>>(a); break;
    default: pipe_lds_kernel<6, RL><<<grid, block, lds, s>>>(a); break;
  }
}

}  // namespace

const void *pipe_lds_kernel_ptr(int pwl, bool rec_lds) {
  return rec_lds ? lds_ptr_for<true>(pwl) : lds_ptr_for<false>(pwl);
}

hipError_t launch_pipe_lds(int pwl, bool rec_lds, int blocks, int wpb, size_t lds,
                           hipStream_t s, const PipeArgs &a) {
  const dim3 grid(blocks), block(wpb * kWave);
  if (rec_lds) lds_launch_for<true>(pwl, grid, block, lds, s, a);
  else lds_launch_for<false>(pwl, grid, block, lds, s, a);
  return hipGetLastError();
}

}  // namespace dipsim
