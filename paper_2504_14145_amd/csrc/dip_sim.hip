// dip_sim.hip -- batched pipeline-schedule simulation for CDNA4 (gfx950).
//
// Implements the C ABI of include/dip_sim.h: host-side validation, device
// tables, kernel-variant choice and the two kernels (simulate, argmin).
//
// Simulation kernel layout.  One wavefront simulates G candidates side by
// side: its 64 lanes split into G groups of PW lanes (PW = next power of two
// >= P), and lane r of a group plays physical rank r of that group's
// candidate (the rank that runs one stage at a time, Sec. 5.2).  Every lane
// walks its rank's order; in each round a lane fires its next op if all of
// the op's predecessors have ended, computing
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
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <new>
#include <vector>

#include "dip_sim.h"

namespace {

thread_local hipError_t g_last_hip = hipSuccess;

constexpr int kWave = 64;
constexpr int kMaxRanks = 64;
constexpr int32_t kMaxOpsPerRank = 32768;
constexpr int64_t kScratchCap = int64_t(2) << 30;  // device scratch ceiling (variant 4)

#define DIP_HIP(expr)                      \
  do {                                     \
    hipError_t e_ = (expr);                \
    if (e_ != hipSuccess) {                \
      g_last_hip = e_;                     \
      return DIP_E_HIP;                    \
    }                                      \
  } while (0)

__host__ __device__ inline int64_t align16(int64_t x) { return (x + 15) & ~int64_t(15); }

// ---------------------------------------------------------------- kernels

struct SimArgs {
  const int16_t *orders;
  int64_t n_cand;
  int64_t stride;          // int16 elements per candidate row
  int64_t n_groups;        // ceil(n_cand / G)
  int32_t *out_ms;
  int32_t *out_bub;
  int32_t *out_peak;
  uint8_t *out_flags;
  const int4 *rec;         // [N] {cost, memdelta, pred_begin, pred_end}
  const int2 *edge;        // [E] {pred global index, comm}
  const int32_t *rank_off; // [P+1]
  const int32_t *busy;     // [P]
  const int32_t *cap;      // [P]
  int32_t *gends;          // variant 4: [resident waves][G][N]
  int32_t P, pwl, G, N, E, wpb;
  uint32_t tab_bytes;      // LDS bytes holding rec + edge (variant 1)
  uint32_t ord_bytes;      // LDS bytes of order rows per wave (variants 1, 2)
  uint32_t end_bytes;      // LDS bytes of end tables per wave (variants 1-3)
};

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

__device__ __forceinline__ void round_fence() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
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

  int rb = 0, nr = 0, busy_r = 0, cap_r = -1;
  if (lane_on) {
    rb = a.rank_off[r];
    nr = a.rank_off[r + 1] - rb;
    busy_r = a.busy[r];
    cap_r = a.cap[r];
  }

  const int64_t total_waves = int64_t(gridDim.x) * a.wpb;
  for (int64_t cg = wslot; cg < a.n_groups; cg += total_waves) {
    const int64_t c0 = cg * a.G;
    const int64_t cand = c0 + grp;
    const bool live = lane_on && cand < a.n_cand;
    const int64_t n_here = min<int64_t>(a.G, a.n_cand - c0);

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
    round_fence();

    int ptr = 0, tfree = 0, mem = 0, peak = 0;
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
          if (load_end<V>(a, end_off, gbase, g) != -1) {
            bad = true;  // the id already fired: not a permutation
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
              const int en = t + rc.x;
              store_end<V>(a, end_off, gbase, g, en);
              tfree = en;
              mem += rc.y;
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
      round_fence();
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
        mem += load_rec<V>(a, g).y;
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
        a.out_bub[o] = gb_stall ? -1 : T - busy_r;
        a.out_peak[o] = peak;
      }
      if (r == 0) {
        a.out_ms[cand] = (gb_bad || gb_stall) ? -1 : T;
        a.out_flags[cand] = gb_bad ? uint8_t(DIP_FLAG_INVALID)
                                   : uint8_t((gb_stall ? DIP_FLAG_DEADLOCK : 0u) |
                                             (gb_cap ? DIP_FLAG_CAP : 0u));
      }
    }
    round_fence();  // this wave's LDS is reused by its next candidate group
  }
}

// Argmin: packed key (makespan << 32 | index) per valid candidate; wave
// reduction with cross-lane shuffles, block reduction through LDS, then one
// 64-bit atomic min per block into the caller's running key.
__global__ __launch_bounds__(256) void argmin_kernel(const int32_t *ms, const uint8_t *flags,
                                                     int64_t n, uint64_t base,
                                                     unsigned long long *key) {
  __shared__ unsigned long long s_best[256 / kWave];
  unsigned long long best = ~0ull;
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) {
    if (flags[i] == 0) {
      const unsigned long long k =
          (static_cast<unsigned long long>(static_cast<uint32_t>(ms[i])) << 32) |
          static_cast<uint32_t>(base + uint64_t(i));
      best = k < best ? k : best;
    }
  }
  for (int off = kWave / 2; off > 0; off >>= 1) {
    const unsigned lo = __shfl_xor(static_cast<unsigned>(best), off, kWave);
    const unsigned hi = __shfl_xor(static_cast<unsigned>(best >> 32), off, kWave);
    const unsigned long long other = (static_cast<unsigned long long>(hi) << 32) | lo;
    best = other < best ? other : best;
  }
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  if (lane == 0) s_best[wave] = best;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long b = s_best[0];
    for (int w = 1; w < int(blockDim.x / kWave); ++w) b = s_best[w] < b ? s_best[w] : b;
    if (b != ~0ull) atomicMin(key, b);
  }
}

using KernelFn = void (*)(SimArgs);

KernelFn kernel_for(int v) {
  switch (v) {
    case 1: return sim_kernel<1>;
    case 2: return sim_kernel<2>;
    case 3: return sim_kernel<3>;
    default: return sim_kernel<4>;
  }
}

int ceil_pow2_log2(int p) {
  int l = 0;
  while ((1 << l) < p) ++l;
  return l;
}

}  // namespace

// ---------------------------------------------------------------- handle

struct dip_sim {
  int device = 0;
  int32_t P = 0, N = 0, E = 0, n_slots = 0;
  int64_t stride = 0;
  std::vector<int32_t> n_ops, rank_off, pred_ptr, pred_op, op_slot, cap;
  std::vector<uint8_t> kind;
  int32_t pwl = 0, G = 0;
  // device tables
  int4 *d_rec = nullptr;
  int2 *d_edge = nullptr;
  int32_t *d_rank_off = nullptr, *d_busy = nullptr, *d_cap = nullptr;
  int32_t *d_scratch = nullptr;
  int64_t scratch_bytes = 0;
  // pinned staging for cost uploads
  unsigned char *h_stage = nullptr;
  int64_t stage_bytes = 0;
  hipEvent_t stage_done = nullptr;
  bool stage_pending = false;
  bool costs_set = false;
  // launch configuration
  int variant = 0, wpb = 1;
  int64_t lds_bytes = 0;
  int max_blocks = 1;
  int n_cu = 1;
  int64_t lds_block_max = 65536, lds_cu = 65536;
  int forced_variant = 0, forced_wpb = 0;
};

namespace {

struct VariantBytes {
  int64_t tab, ord, end;
};

VariantBytes bytes_for(const dip_sim *h, int v) {
  VariantBytes b{0, 0, 0};
  const int64_t G = h->G;
  if (v == 1) b.tab = align16(int64_t(h->N) * 16) + align16(int64_t(h->E) * 8);
  if (v <= 2) b.ord = align16(G * h->stride * 2);
  if (v <= 3) b.end = align16(G * int64_t(h->N) * 4);
  return b;
}

int64_t lds_for(const dip_sim *h, int v, int wpb) {
  VariantBytes b = bytes_for(h, v);
  return b.tab + int64_t(wpb) * (b.ord + b.end);
}

// Resident blocks per CU for (variant, waves per block), from the occupancy
// calculator; 0 if the LDS does not fit.
int blocks_per_cu(dip_sim *h, int v, int wpb) {
  const int64_t lds = lds_for(h, v, wpb);
  if (lds > h->lds_block_max) return 0;
  KernelFn k = kernel_for(v);
  if (lds > 65536) {
    if (hipFuncSetAttribute(reinterpret_cast<const void *>(k),
                            hipFuncAttributeMaxDynamicSharedMemorySize,
                            int(lds)) != hipSuccess) {
      (void)hipGetLastError();
      return 0;
    }
  }
  int nb = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, reinterpret_cast<const void *>(k),
                                                   wpb * kWave, size_t(lds)) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  return nb;
}

int choose_config(dip_sim *h) {
  int best_v = 0, best_w = 0, best_waves = 0, best_nb = 0;
  const int v_lo = h->forced_variant ? h->forced_variant : 1;
  const int v_hi = h->forced_variant ? h->forced_variant : 4;
  for (int v = v_lo; v <= v_hi; ++v) {
    for (int w : {4, 2, 1}) {
      if (h->forced_wpb && w != h->forced_wpb) continue;
      const int nb = blocks_per_cu(h, v, w);
      if (nb <= 0) continue;
      const int waves = nb * w;
      // prefer the lower variant (less global traffic) unless a higher one
      // at least doubles the resident waves and the lower has fewer than 8
      if (best_v == 0 || (waves > best_waves && (v == best_v || (best_waves < 8 && waves >= 2 * best_waves)))) {
        best_v = v; best_w = w; best_waves = waves; best_nb = nb;
      }
    }
  }
  if (best_v == 0) return DIP_E_UNSUPPORTED;
  h->variant = best_v;
  h->wpb = best_w;
  h->lds_bytes = lds_for(h, best_v, best_w);
  h->max_blocks = best_nb * h->n_cu;
  if (best_v == 4) {
    const int64_t per_block = int64_t(best_w) * h->G * int64_t(h->N) * 4;
    const int64_t cap_blocks = std::max<int64_t>(1, kScratchCap / per_block);
    h->max_blocks = int(std::min<int64_t>(h->max_blocks, cap_blocks));
    const int64_t need = per_block * h->max_blocks;
    if (need > h->scratch_bytes) {
      if (h->d_scratch) { DIP_HIP(hipFree(h->d_scratch)); h->d_scratch = nullptr; }
      h->scratch_bytes = 0;
      if (hipMalloc(&h->d_scratch, size_t(need)) != hipSuccess) {
        (void)hipGetLastError();
        return DIP_E_NOMEM;
      }
      h->scratch_bytes = need;
    }
  }
  return DIP_OK;
}

int check_costs_against(int32_t P, const int32_t *n_ops, const int32_t *pred_ptr,
                        const int32_t *op_slot, const uint8_t *kind, int32_t n_slots,
                        const dip_costs *c) {
  if (!c || !c->op_cost || !c->slot_act) return DIP_E_INVAL;
  int64_t N = 0;
  for (int r = 0; r < P; ++r) N += n_ops[r];
  const int64_t E = pred_ptr[N];
  if (E > 0 && !c->edge_comm) return DIP_E_INVAL;
  int64_t total = 0;
  for (int64_t g = 0; g < N; ++g) {
    if (c->op_cost[g] < 0) return DIP_E_RANGE;
    total += c->op_cost[g];
  }
  for (int64_t e = 0; e < E; ++e) {
    if (c->edge_comm[e] < 0) return DIP_E_RANGE;
    total += c->edge_comm[e];
  }
  if (total > INT32_MAX) return DIP_E_RANGE;
  for (int32_t s = 0; s < n_slots; ++s)
    if (c->slot_act[s] < 0) return DIP_E_RANGE;
  // per rank: the running activation sum stays within int32 either way
  int64_t off = 0;
  for (int r = 0; r < P; ++r) {
    int64_t up = 0, down = 0;
    for (int64_t g = off; g < off + n_ops[r]; ++g) {
      const int64_t act = c->slot_act[op_slot[g]];
      if (kind[g] == 0) up += act; else down += act;
    }
    if (up > INT32_MAX || down > INT32_MAX) return DIP_E_RANGE;
    off += n_ops[r];
  }
  return DIP_OK;
}

int upload_costs(dip_sim *h, const dip_costs *c, hipStream_t stream) {
  int rc = check_costs_against(h->P, h->n_ops.data(), h->pred_ptr.data(), h->op_slot.data(),
                               h->kind.data(), h->n_slots, c);
  if (rc != DIP_OK) return rc;
  if (h->stage_pending) {
    DIP_HIP(hipEventSynchronize(h->stage_done));
    h->stage_pending = false;
  }
  int4 *rec = reinterpret_cast<int4 *>(h->h_stage);
  int2 *edge = reinterpret_cast<int2 *>(h->h_stage + align16(int64_t(h->N) * 16));
  int32_t *busy = reinterpret_cast<int32_t *>(h->h_stage + align16(int64_t(h->N) * 16) +
                                              align16(int64_t(std::max(h->E, 1)) * 8));
  for (int32_t g = 0; g < h->N; ++g) {
    const int32_t act = c->slot_act[h->op_slot[g]];
    rec[g] = make_int4(c->op_cost[g], h->kind[g] == 0 ? act : -act, h->pred_ptr[g],
                       h->pred_ptr[g + 1]);
  }
  for (int32_t e = 0; e < h->E; ++e) edge[e] = make_int2(h->pred_op[e], c->edge_comm[e]);
  for (int r = 0; r < h->P; ++r) {
    int64_t s = 0;
    for (int32_t g = h->rank_off[r]; g < h->rank_off[r + 1]; ++g) s += c->op_cost[g];
    busy[r] = int32_t(s);
  }
  DIP_HIP(hipMemcpyAsync(h->d_rec, rec, size_t(h->N) * 16, hipMemcpyHostToDevice, stream));
  if (h->E > 0)
    DIP_HIP(hipMemcpyAsync(h->d_edge, edge, size_t(h->E) * 8, hipMemcpyHostToDevice, stream));
  DIP_HIP(hipMemcpyAsync(h->d_busy, busy, size_t(h->P) * 4, hipMemcpyHostToDevice, stream));
  DIP_HIP(hipEventRecord(h->stage_done, stream));
  h->stage_pending = true;
  h->costs_set = true;
  return DIP_OK;
}

void release(dip_sim *h) {
  if (!h) return;
  (void)hipDeviceSynchronize();
  if (h->d_rec) (void)hipFree(h->d_rec);
  if (h->d_edge) (void)hipFree(h->d_edge);
  if (h->d_rank_off) (void)hipFree(h->d_rank_off);
  if (h->d_busy) (void)hipFree(h->d_busy);
  if (h->d_cap) (void)hipFree(h->d_cap);
  if (h->d_scratch) (void)hipFree(h->d_scratch);
  if (h->h_stage) (void)hipHostFree(h->h_stage);
  if (h->stage_done) (void)hipEventDestroy(h->stage_done);
  delete h;
}

}  // namespace

extern "C" {

int dip_sim_abi_version(void) { return DIP_SIM_ABI_VERSION; }

int dip_sim_check_topology(const dip_topology *t) {
  if (!t || !t->n_ops || !t->pred_ptr || !t->op_kind || !t->op_slot || !t->mem_cap)
    return DIP_E_INVAL;
  if (t->n_ranks <= 0) return DIP_E_INVAL;
  if (t->n_ranks > kMaxRanks) return DIP_E_UNSUPPORTED;
  int64_t N = 0;
  for (int r = 0; r < t->n_ranks; ++r) {
    if (t->n_ops[r] < 0 || t->n_ops[r] > kMaxOpsPerRank) return DIP_E_TOPO;
    N += t->n_ops[r];
  }
  if (N == 0 || N > INT32_MAX / 16) return DIP_E_TOPO;
  if (t->cand_stride < N || t->cand_stride % 8 != 0) return DIP_E_INVAL;
  if (t->n_slots < 0) return DIP_E_TOPO;
  if (t->pred_ptr[0] != 0) return DIP_E_TOPO;
  for (int64_t g = 0; g < N; ++g)
    if (t->pred_ptr[g + 1] < t->pred_ptr[g]) return DIP_E_TOPO;
  const int64_t E = t->pred_ptr[N];
  if (E > 0 && !t->pred_op) return DIP_E_INVAL;
  for (int64_t g = 0; g < N; ++g) {
    for (int32_t e = t->pred_ptr[g]; e < t->pred_ptr[g + 1]; ++e)
      if (t->pred_op[e] < 0 || t->pred_op[e] >= N || t->pred_op[e] == g) return DIP_E_TOPO;
    if (t->op_kind[g] > 1) return DIP_E_TOPO;
    if (t->op_slot[g] < 0 || t->op_slot[g] >= t->n_slots) return DIP_E_TOPO;
  }
  return DIP_OK;
}

int dip_sim_check_costs(const dip_topology *t, const dip_costs *c) {
  int rc = dip_sim_check_topology(t);
  if (rc != DIP_OK) return rc;
  return check_costs_against(t->n_ranks, t->n_ops, t->pred_ptr, t->op_slot, t->op_kind,
                             t->n_slots, c);
}

int dip_sim_create(const dip_topology *t, dip_sim **out) {
  if (!out) return DIP_E_INVAL;
  *out = nullptr;
  int rc = dip_sim_check_topology(t);
  if (rc != DIP_OK) return rc;
  dip_sim *h = new (std::nothrow) dip_sim();
  if (!h) return DIP_E_NOMEM;
  h->P = t->n_ranks;
  h->n_ops.assign(t->n_ops, t->n_ops + h->P);
  h->rank_off.assign(h->P + 1, 0);
  for (int r = 0; r < h->P; ++r) h->rank_off[r + 1] = h->rank_off[r] + t->n_ops[r];
  h->N = h->rank_off[h->P];
  h->E = t->pred_ptr[h->N];
  h->n_slots = t->n_slots;
  h->stride = t->cand_stride;
  h->pred_ptr.assign(t->pred_ptr, t->pred_ptr + h->N + 1);
  if (h->E > 0) h->pred_op.assign(t->pred_op, t->pred_op + h->E);
  h->kind.assign(t->op_kind, t->op_kind + h->N);
  h->op_slot.assign(t->op_slot, t->op_slot + h->N);
  h->cap.assign(t->mem_cap, t->mem_cap + h->P);
  h->pwl = ceil_pow2_log2(h->P);
  h->G = kWave >> h->pwl;

  auto fail = [&](int code) { release(h); return code; };
  auto hip_fail = [&](hipError_t e) { g_last_hip = e; release(h); return int(DIP_E_HIP); };
  hipError_t e;
  if ((e = hipGetDevice(&h->device)) != hipSuccess) return hip_fail(e);
  int v = 0;
  if ((e = hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, h->device)) != hipSuccess)
    return hip_fail(e);
  h->n_cu = std::max(1, v);
  if ((e = hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, h->device)) != hipSuccess)
    return hip_fail(e);
  h->lds_block_max = v;
  if (hipDeviceGetAttribute(&v, hipDeviceAttributeSharedMemPerBlockOptin, h->device) == hipSuccess && v > 0)
    h->lds_block_max = std::max<int64_t>(h->lds_block_max, v);
  (void)hipGetLastError();
  if ((e = hipMalloc(&h->d_rec, size_t(h->N) * 16)) != hipSuccess) return hip_fail(e);
  if ((e = hipMalloc(&h->d_edge, size_t(std::max(h->E, 1)) * 8)) != hipSuccess) return hip_fail(e);
  if ((e = hipMalloc(&h->d_rank_off, size_t(h->P + 1) * 4)) != hipSuccess) return hip_fail(e);
  if ((e = hipMalloc(&h->d_busy, size_t(h->P) * 4)) != hipSuccess) return hip_fail(e);
  if ((e = hipMalloc(&h->d_cap, size_t(h->P) * 4)) != hipSuccess) return hip_fail(e);
  if ((e = hipMemcpy(h->d_rank_off, h->rank_off.data(), size_t(h->P + 1) * 4,
                     hipMemcpyHostToDevice)) != hipSuccess)
    return hip_fail(e);
  if ((e = hipMemcpy(h->d_cap, h->cap.data(), size_t(h->P) * 4, hipMemcpyHostToDevice)) != hipSuccess)
    return hip_fail(e);
  h->stage_bytes = align16(int64_t(h->N) * 16) + align16(int64_t(std::max(h->E, 1)) * 8) +
                   align16(int64_t(h->P) * 4);
  if ((e = hipHostMalloc(reinterpret_cast<void **>(&h->h_stage), size_t(h->stage_bytes),
                         hipHostMallocDefault)) != hipSuccess)
    return hip_fail(e);
  if ((e = hipEventCreateWithFlags(&h->stage_done, hipEventDisableTiming)) != hipSuccess)
    return hip_fail(e);
  rc = choose_config(h);
  if (rc != DIP_OK) return fail(rc);
  *out = h;
  return DIP_OK;
}

int dip_sim_configure(dip_sim *h, int32_t variant, int32_t waves_per_block) {
  if (!h || variant < 0 || variant > 4) return DIP_E_INVAL;
  if (!(waves_per_block == 0 || waves_per_block == 1 || waves_per_block == 2 ||
        waves_per_block == 4))
    return DIP_E_INVAL;
  const int old_v = h->forced_variant, old_w = h->forced_wpb;
  h->forced_variant = variant;
  h->forced_wpb = waves_per_block;
  int rc = choose_config(h);
  if (rc != DIP_OK) {
    h->forced_variant = old_v;
    h->forced_wpb = old_w;
    (void)choose_config(h);
  }
  return rc;
}

int dip_sim_get_info(const dip_sim *h, dip_sim_info *info) {
  if (!h || !info) return DIP_E_INVAL;
  info->n_ranks = h->P;
  info->n_ops_total = h->N;
  info->n_edges = h->E;
  info->variant = h->variant;
  info->cand_stride = h->stride;
  info->lanes_per_group = 1 << h->pwl;
  info->groups_per_wave = h->G;
  info->waves_per_block = h->wpb;
  info->lds_bytes = int32_t(h->lds_bytes);
  info->max_blocks = h->max_blocks;
  info->scratch_bytes = h->scratch_bytes;
  return DIP_OK;
}

int dip_sim_evaluate(dip_sim *h, const dip_costs *costs, const int16_t *orders, int64_t n_cand,
                     int32_t *out_makespan, int32_t *out_bubble, int32_t *out_peakmem,
                     uint8_t *out_flags, void *stream_) {
  if (!h || n_cand < 0) return DIP_E_INVAL;
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  if (costs) {
    int rc = upload_costs(h, costs, stream);
    if (rc != DIP_OK) return rc;
  }
  if (!h->costs_set) return DIP_E_STATE;
  if (n_cand == 0) return DIP_OK;
  if (!orders || !out_makespan || !out_bubble || !out_peakmem || !out_flags) return DIP_E_INVAL;
  if ((reinterpret_cast<uintptr_t>(orders) & 15) != 0) return DIP_E_INVAL;
  if ((reinterpret_cast<uintptr_t>(out_makespan) | reinterpret_cast<uintptr_t>(out_bubble) |
       reinterpret_cast<uintptr_t>(out_peakmem)) & 3)
    return DIP_E_INVAL;
  SimArgs a{};
  a.orders = orders;
  a.n_cand = n_cand;
  a.stride = h->stride;
  a.n_groups = (n_cand + h->G - 1) / h->G;
  a.out_ms = out_makespan;
  a.out_bub = out_bubble;
  a.out_peak = out_peakmem;
  a.out_flags = out_flags;
  a.rec = h->d_rec;
  a.edge = h->d_edge;
  a.rank_off = h->d_rank_off;
  a.busy = h->d_busy;
  a.cap = h->d_cap;
  a.gends = h->d_scratch;
  a.P = h->P;
  a.pwl = h->pwl;
  a.G = h->G;
  a.N = h->N;
  a.E = h->E;
  a.wpb = h->wpb;
  const VariantBytes b = bytes_for(h, h->variant);
  a.tab_bytes = uint32_t(b.tab);
  a.ord_bytes = uint32_t(b.ord);
  a.end_bytes = uint32_t(b.end);
  const int64_t want_blocks = (a.n_groups + h->wpb - 1) / h->wpb;
  const int blocks = int(std::min<int64_t>(want_blocks, h->max_blocks));
  const dim3 grid(blocks), block(h->wpb * kWave);
  const size_t lds = size_t(h->lds_bytes);
  switch (h->variant) {
    case 1: sim_kernel<1><<<grid, block, lds, stream>>>(a); break;
    case 2: sim_kernel<2><<<grid, block, lds, stream>>>(a); break;
    case 3: sim_kernel<3><<<grid, block, lds, stream>>>(a); break;
    default: sim_kernel<4><<<grid, block, lds, stream>>>(a); break;
  }
  DIP_HIP(hipGetLastError());
  return DIP_OK;
}

int dip_sim_argmin(dip_sim *h, const int32_t *makespan, const uint8_t *flags, int64_t n_cand,
                   int64_t index_base, uint64_t *inout_best_key, void *stream_) {
  if (!h || n_cand < 0 || index_base < 0) return DIP_E_INVAL;
  if (index_base + n_cand > int64_t(UINT32_MAX)) return DIP_E_RANGE;
  if (n_cand == 0) return DIP_OK;
  if (!makespan || !flags || !inout_best_key) return DIP_E_INVAL;
  if ((reinterpret_cast<uintptr_t>(inout_best_key) & 7) || (reinterpret_cast<uintptr_t>(makespan) & 3))
    return DIP_E_INVAL;
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  const int threads = 256;
  const int64_t want = (n_cand + threads - 1) / threads;
  const int blocks = int(std::min<int64_t>(want, int64_t(h->n_cu) * 8));
  argmin_kernel<<<dim3(blocks), dim3(threads), 0, stream>>>(
      makespan, flags, n_cand, uint64_t(index_base),
      reinterpret_cast<unsigned long long *>(inout_best_key));
  DIP_HIP(hipGetLastError());
  return DIP_OK;
}

void dip_sim_destroy(dip_sim *h) { release(h); }

const char *dip_sim_strerror(int code) {
  switch (code) {
    case DIP_OK: return "ok";
    case DIP_E_INVAL: return "invalid argument (null pointer, negative count or misaligned buffer)";
    case DIP_E_TOPO: return "malformed topology";
    case DIP_E_RANGE: return "negative cost or totals that could overflow int32";
    case DIP_E_UNSUPPORTED: return "shape not supported by any kernel variant on this device";
    case DIP_E_NOMEM: return "out of memory";
    case DIP_E_HIP: return hipGetErrorString(g_last_hip);
    case DIP_E_STATE: return "no costs supplied yet";
    default: return "unknown error";
  }
}

}  // extern "C"
