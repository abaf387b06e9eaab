// internal.h -- shared between the host library and the kernel translation
// units of libdip_sim.  Not part of the public C ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace dipsim {

constexpr int kWave = 64;

__host__ __device__ inline int64_t align16(int64_t x) { return (x + 15) & ~int64_t(15); }

// ---------------------------------------------------------------- general
// General kernel: any DAG (predecessors walked through the CSR), tables
// placed per variant (1: all in LDS, 2: records in global, rows and end
// times in LDS, 3: only end times in LDS, 4: end times in device scratch).
struct GeneralArgs {
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
  // list mode (variants 3, 4 only): simulate candidates list[0 .. *list_count-1]
  const int64_t *list;
  const uint32_t *list_count;
  uint32_t tab_bytes;      // LDS bytes holding rec + edge (variant 1)
  uint32_t ord_bytes;      // LDS bytes of order rows per wave (variants 1, 2)
  uint32_t end_bytes;      // LDS bytes of end tables per wave (variants 1-3)
  // re-timing with a memory selection (choice != null): the backward of pair
  // p costs its op cost + cand_time[p][c] - cand_time[p][0] and the pair's
  // activation is cand_mem[p][c], c = choice[cand][p]
  const uint8_t *choice;   // [n_cand][n_pairs]
  int32_t n_pairs;
  const int32_t *lid_pair; // [N] pair index on its rank | kind << 31
  const int32_t *pair_off; // [P+1]
  const int64_t *cand_time;   // [pairs][kMemoptMaxCands]
  const int32_t *cand_mem;    // [pairs][kMemoptMaxCands]
  const uint32_t *cand_key;   // [pairs][kMemoptMaxCands] move keys: candidate c exists when
                              // c == 0 or key[c - 1] marks a move
};

const void *general_kernel_ptr(int variant);
hipError_t launch_general(int variant, int blocks, int wpb, size_t lds, hipStream_t s,
                          const GeneralArgs &a);

// Counters of one evaluate call, zeroed by its check kernel: per simulation
// pass (8, 16 and 32 slots) the count of its retry list and its on-demand
// candidate counter
constexpr int kRetryCounters = 8;

// ---------------------------------------------------------------- check
// Order-only verdict of each candidate: permutation check, per-rank peak
// memory, cap flag (one wavefront per candidate; an op-id bitmap in LDS).
struct CheckArgs {
  const int16_t *orders;
  int64_t n_cand;
  int64_t stride;
  int32_t *out_ms;
  int32_t *out_bub;
  int32_t *out_peak;
  uint8_t *out_flags;
  const int32_t *md;        // [N] +act at a forward, -act at a backward
  const int32_t *rank_off;  // [P+1]
  const int32_t *cap;       // [P]
  int32_t P, N, wpb;
  uint32_t *retry_count;    // [kRetryCounters] zeroed by the kernel when not
                            // null (retry counts and on-demand candidate
                            // counters of the simulation passes)
};

// bytes of one candidate's op-id bitmap
__host__ __device__ inline int64_t check_lds_per_group(int32_t N) { return int64_t(((N + 31) / 32 + 3) & ~3) * 4; }
const void *check_kernel_ptr(int pwl);
hipError_t launch_check(int pwl, int blocks, int wpb, size_t lds, hipStream_t s,
                        const CheckArgs &a);

// Order-only verdict by tiles of 64 consecutive candidates, lane = candidate:
// the waves of a block split the ranks between them (plan), and for each of
// its ranks a wave streams the rank's section of the 64 rows, with the rank's
// memory deltas and a per-lane op-id bitmap in the wave's LDS region.
struct TileCheckArgs {
  const int16_t *orders;
  int64_t n_cand;
  int64_t stride;
  int32_t *out_ms;
  int32_t *out_bub;
  int32_t *out_peak;
  uint8_t *out_flags;
  const int32_t *md;        // [N] +act at a forward, -act at a backward
  const int32_t *rank_off;  // [P+1]
  const int32_t *cap;       // [P]
  const int32_t *plan;      // [nw+1] offsets into the rank list, then the list [P]
  int32_t P, nw;
  int32_t md_bytes;         // bytes of a wave's delta area (16-aligned)
  int32_t region_bytes;     // bytes per wave: delta area + bitmap of 64 lanes
  uint32_t *retry_count;    // [kRetryCounters] zeroed by the kernel when not
                            // null (retry counts and on-demand candidate
                            // counters of the simulation passes)
};

// LDS of a tile-check block: the 64 candidates' flag words, then the waves'
// regions (deltas and bits of ids 0 .. max_nr, the last one the overflow
// entry; then the staging of 8 units of the 64 rows)
constexpr int kTileFlagBytes = 256;
// waves per tile-check block at most (12: LDS holds at most three waves per
// SIMD on the workloads that need many, and 168 registers per lane keep the
// staged units and the two units in flight out of scratch)
constexpr int kTileMaxWaves = 12;
constexpr int kTileStageBytes = 64 * 8 * 16;
__host__ __device__ inline int32_t tile_md_bytes(int32_t max_nr) { return ((max_nr + 1) * 4 + 15) & ~15; }
__host__ __device__ inline int32_t tile_region_bytes(int32_t max_nr) {
  return tile_md_bytes(max_nr) + ((max_nr + 32) / 32) * 64 * 4 + kTileStageBytes;
}
const void *tile_check_kernel_ptr();
hipError_t launch_tile_check(int blocks, int nw, size_t lds, hipStream_t s, const TileCheckArgs &a);

// Own-rank order of the ranks whose ops wait on an op of their own rank: one
// wave per (candidate, rank) section, a block per rank and chunk of
// candidates, with the rank's own-rank predecessors in LDS and a table of the
// section's positions per wave.  Runs after the tile check: skips candidates
// flagged invalid; adds the deadlock flag and -1 makespan and bubbles.
struct OrderCheckArgs {
  const int16_t *orders;
  int64_t n_cand;
  int64_t stride;
  int32_t *out_ms;
  int32_t *out_bub;
  uint8_t *out_flags;
  const int32_t *selfp;     // [N] local id + 1 of the op's own-rank predecessor (0: none)
  const int32_t *rank_off;  // [P+1]
  const int32_t *ranks;     // [n_ranks] the ranks checked
  int64_t n_chunks;         // chunks of wpb * per_wave candidates
  int32_t P, n_ranks, wpb, per_wave;
  int32_t tab_bytes;        // LDS: predecessors [max_nr + 1] uint16 (16-aligned)
  int32_t wave_bytes;       // per wave: positions [max_nr + 1] uint16 (16-aligned)
};
__host__ __device__ inline int32_t order_table_bytes(int32_t max_nr) { return int32_t(align16(int64_t(max_nr + 1) * 2)); }
// blocks of a launch over n_chunks chunks of n_ranks ranks: chunk j's blocks
// are 8 apart, so they share j % 8 and with it the XCD the dispatcher sends
// them to
__host__ __device__ inline int64_t order_blocks(int64_t n_chunks, int32_t n_ranks) {
  return 8 * int64_t(n_ranks) * ((n_chunks + 7) / 8);
}
const void *order_check_kernel_ptr();
hipError_t launch_order_check(int64_t blocks, int wpb, size_t lds, hipStream_t s,
                              const OrderCheckArgs &a);

// ---------------------------------------------------------------- pool
// Timing simulation with per-rank slot pools holding the end times still to
// be read (see kern_pool.hip).
struct PoolArgs {
  const int16_t *orders;
  int64_t n_cand;
  int64_t stride;
  int32_t *out_ms;
  int32_t *out_bub;
  uint8_t *out_flags;       // the check kernel's verdicts, extended here
  const int4 *rec;          // [N] {cost, first edge's comm,
                            //      first edge word | readers << 24,
                            //      item tag (rank-local id + 1) or 0 | extra edges << 16}
  const int2 *edge;         // extra edges (an op's second to last), {edge word, comm}
  const int32_t *rank_off;  // [P+1]
  const int32_t *busy;      // [P]
  int32_t P, wpb;
  int64_t *retry;           // [n_cand] candidates the pools could not hold
  uint32_t *retry_count;
  int32_t rec_bytes, edge_bytes;  // sizes of rec and edge (buffer descriptors)
  uint32_t round_limit;           // rounds a candidate may take (N + E + 16)
  uint32_t tab_edges;             // tables in LDS: byte offset of the extra edges
  uint32_t pool_base;             // byte offset of the pools in LDS
  uint32_t *next_cand;            // null: slot k takes k, k + n_slots, ...; else a
                                  // counter of those handed out on demand
  int64_t static_end;             // with next_cand: candidates below it (a multiple of
                                  // n_slots) go to fixed successors, the rest on demand
};

// dword 3 of a raw buffer descriptor on CDNA
constexpr int kBufferWord3 = 0x00020000;

// edge word: predecessor tag (its rank-local id + 1) | its rank << 16 |
// kEdgeLast (the sign bit) on an op's last predecessor edge; an op without
// predecessors starts on kNoEdgeWord (a tag no item carries, marked last).
// In a pool record the word also carries the op's reader count in bits 24-27.
constexpr uint32_t kEdgeTagMask = 0xffffu;
constexpr uint32_t kEdgeRankShift = 16;
constexpr uint32_t kEdgeLast = 1u << 31;
constexpr uint32_t kNoEdgeWord = kEdgeTagMask | kEdgeLast;
// the edge word of a lane with no op to run: a tag no item carries, not last
// (so the lane is never ready)
constexpr uint32_t kDeadEdgeWord = kEdgeTagMask - 1;

// The pools of one candidate (a group of PW lanes, P <= PW ranks) in LDS, as
// arrays over the ranks so that lanes reading their own or a neighbour's pool
// fall in distinct banks:
//   counts [PW][C] words, C = ceil(S / 8): a 4-bit reader count per slot
//                          (0 = free slot)
//   tags   [PW][S] 16-bit, 16-byte aligned
//   ends   [PW][S + 1] words (the extra word makes the stride odd in words)
// padded so that the group's size in words is congruent to PW modulo the 32
// banks: the count words of consecutive groups then tile the banks.
__host__ __device__ constexpr int64_t pool_count_words(int slots) { return (slots + 7) / 8; }
__host__ __device__ constexpr int64_t pool_tags_offset(int pw, int slots) {
  return (int64_t(pw) * 4 * pool_count_words(slots) + 15) / 16 * 16;
}
__host__ __device__ constexpr int64_t pool_ends_offset(int pw, int slots) {
  return pool_tags_offset(pw, slots) + int64_t(pw) * 2 * slots;
}
__host__ __device__ constexpr int64_t pool_end_stride(int slots) { return 4 * int64_t(slots) + 4; }
__host__ __device__ constexpr int64_t pool_group_bytes(int pw, int slots) {
  const int64_t raw = pool_ends_offset(pw, slots) + int64_t(pw) * pool_end_stride(slots);
  const int64_t want = pw >= 32 ? 0 : 4 * (pw < 4 ? 4 : pw);   // residue modulo 128 bytes
  int64_t x = (raw + 15) / 16 * 16;
  while (x % 128 != want) x += 16;
  return x;
}
bool pool_slots_ok(int slots);
// tables in LDS when they take at most this many bytes
constexpr int64_t kPoolTabMax = 16384;
const void *pool_kernel_ptr(int pwl, int slots, bool tab);
hipError_t launch_pool(int pwl, int slots, bool tab, int blocks, int wpb, size_t lds, hipStream_t s,
                       const PoolArgs &a);

// ---------------------------------------------------------------- sim
// Timing simulation with LDS-resident compact op records and per-lane order
// rings (see kern_sim.hip).
//
// Record (8 bytes) of an op, relative to the op itself so that ops of
// identically placed model chunks share records:
//   w0 = cost (bits 0-19) | consumers (20-23) | several predecessors (30) |
//        has predecessors (31) (the top bits, so that each test is one
//        compare: w0 < 0 as a signed word, and w0 >= both flags)
//   w1 = the edge word of its only predecessor, or, with several, the index
//        of its first edge word in the extra-edge table (the rest follow, the
//        last one marked)
// Edge word: (pred rank - own rank) mod P (bits 0-5) | pred local id - own
//   local id (6-19, two's complement) | latency (20-30) | last (31).
constexpr uint32_t kSimCostBits = 20;
constexpr uint32_t kSimCostMax = (1u << kSimCostBits) - 1;
constexpr uint32_t kSimCommMax = 2047;
constexpr int32_t kSimDeltaMax = 8191;          // |pred local id - own local id|
constexpr uint32_t kSimMulti = 1u << 30;
constexpr uint32_t kSimHasPred = 1u << 31;
constexpr uint32_t kSimLast = 1u << 31;
// ops per record page (paged tables: a rank's records come in pages of 16
// consecutive local ids, equal pages stored once); the page map holds each
// page's first record index (page number x 16), so at most kSimMaxPages pages
constexpr int kSimPage = 16;
constexpr int kSimMaxPages = 4096;

// Per-candidate LDS state of the simulation kernel, for a group of PW lanes
// (one per rank; the kernel requires P == PW):
//   tags   [S / 8][PW][8] 16-bit (local id + 1 of the op whose end time a pool
//          slot holds; slots 8h .. 8h + 7 of all ranks together, 16 bytes per
//          rank, so that a group's 16-byte tag reads tile the banks; with
//          S = 4, [PW][4])
//   pools  [PW] sim_pool_bytes(S) each: C = ceil(S / 8) count words (4-bit
//          reader count per slot), then S end-time words; padded to an odd
//          number of words so that different ranks' pools start in different
//          banks
//   rings  [PW] order rings of kSimRingBytes: two 16-byte blocks of 8 ids
//          (and an 8-byte pad)
constexpr int64_t kSimBlockIds = 8;
constexpr int64_t kSimRingBytes = 40;
__host__ __device__ constexpr int64_t sim_count_words(int slots) { return (slots + 7) / 8; }
__host__ __device__ constexpr int64_t sim_tag_bytes(int pw, int slots) { return int64_t(pw) * 2 * slots; }
__host__ __device__ constexpr int64_t sim_pool_bytes(int slots) {
  const int64_t words = sim_count_words(slots) + slots;
  return 4 * (words % 2 == 0 ? words + 1 : words);
}
__host__ __device__ constexpr int64_t sim_pool_offset(int pw, int slots) {
  return (sim_tag_bytes(pw, slots) + 15) / 16 * 16;
}
__host__ __device__ constexpr int64_t sim_ring_offset(int pw, int slots) {
  return (sim_pool_offset(pw, slots) + int64_t(pw) * sim_pool_bytes(slots) + 15) / 16 * 16;
}
// padded so that the group's size in words is congruent to PW modulo the 32
// banks (4 words below 4 lanes): the same word of consecutive groups then
// falls in different banks
__host__ __device__ constexpr int64_t sim_group_bytes(int pw, int slots) {
  const int64_t raw = sim_ring_offset(pw, slots) + int64_t(pw) * kSimRingBytes;
  const int64_t want = pw >= 32 ? 0 : 4 * (pw < 4 ? 4 : pw);   // residue modulo 128 bytes
  int64_t x = (raw + 15) / 16 * 16;
  while (x % 128 != want) x += 16;
  return x;
}

struct SimArgs {
  const int16_t *orders;
  int64_t n_cand;
  int64_t stride;
  int32_t *out_ms;
  int32_t *out_bub;
  uint8_t *out_flags;        // the check kernel's verdicts, extended here
  const uint4 *tab;          // LDS image of the tables: records, page map, extra edges
  int32_t tab_vec;           // its size in 16-byte units
  uint32_t off_pmap;         // byte offset of the page map (paged records)
  uint32_t off_extra;        // byte offset of the extra edges
  const int32_t *lane_info;  // [P][4] {first global op, ops, busy time, record base}
                             // record base: first record (direct) or first page-map entry
  uint32_t state_base;       // byte offset of the first group's state
  int32_t P, wpb;
  int64_t *retry;            // candidates the pools could not hold
  uint32_t *retry_count;     // [2] their count, candidates handed out on demand
  // list mode (list != null): simulate list[0 .. *list_count - 1] instead of
  // 0 .. n_cand - 1 (a second pass, with larger pools, over the first pass's
  // retry list); candidates are then taken by fixed successors only
  const int64_t *list;
  const uint32_t *list_count;
  int64_t static_end;        // candidates below it (a multiple of the resident groups)
                             // go to fixed successors, the rest are handed out on
                             // demand through retry_count[1]; INT64_MAX: none
  uint32_t round_limit;      // rounds one candidate may take
};
bool sim_slots_ok(int slots);
const void *sim_kernel_ptr(int pwl, int slots, bool paged);
hipError_t launch_sim(int pwl, int slots, bool paged, int blocks, int wpb, size_t lds,
                      hipStream_t s, const SimArgs &a);

// ---------------------------------------------------------------- greedy
// Dual-queue stage interleaving (see kern_greedy.hip).  Groups are numbered
// internally forward groups first, then backward ones, each in the caller's
// order; "position" is a group's rank among the groups of its kind under the
// candidate's priorities.
struct GreedyArgs {
  const int32_t *prio;      // [n_cand][G] caller-indexed priorities
  int64_t n_cand;
  int16_t *out_orders;      // [n_cand][stride] or null
  int64_t stride;
  int32_t *out_ms;
  int32_t *out_bub;
  int32_t *out_peak;
  uint8_t *out_flags;
  const int4 *rec;          // [G][P][2] per (internal group, rank):
                            //   {cost, act, local id | successors << 16 (0xffff: no stage),
                            //    index of the second successor in succ},
                            //   {first successor: word, comm, join or -1, join's predecessors}
  const int4 *succ;         // further successors, same form as the second half of rec
  const int32_t *caller;    // [G] caller index of each internal group
  const int32_t *src;       // [P+1] offsets, then the internal groups of each rank's sources
  const int32_t *rank_off;  // [P+1]
  const int32_t *busy;      // [P]
  const int32_t *cap;       // [P]
  int32_t P, G, GF, J, K, wpb;
  int32_t n_rounds;         // N: every round schedules one stage of every candidate
  int32_t has_cap;          // some rank has a cap
  int32_t meta_bytes;       // block-shared LDS: caller index of each group (u16)
  int32_t cand_bytes;       // LDS per candidate, 16-aligned
  int32_t off_gpos, off_ord, off_grk, off_pend, off_npend, off_join;  // within a candidate
  const int64_t *list;      // list mode: candidates list[0 .. *list_count-1]
  const uint32_t *list_count;
  int64_t *retry;           // candidates whose inbox overflowed
  uint32_t *retry_count;
  uint64_t *gring;          // device-memory inboxes: P * (2K + 1) entries per resident
                            // candidate slot, slot = (block * wpb + wave) * (64 >> pwl) + group
};
// successor word: internal group | kind << 16 | rank << 17
constexpr uint32_t kGreedyNoStage = 0xffffu;
// nw: bitmap words per kind (1, 2, 4, 8, 16, 32); gring: inboxes in device
// memory (GreedyArgs::gring) rather than LDS
// Zeroes n (<= 64) words: a kernel instead of a memset node, so that code a
// caller captures into a HIP graph holds no memset.
hipError_t launch_zero_words(uint32_t *p, int n, hipStream_t s);
const void *greedy_kernel_ptr(int pwl, int nw, bool gring);
hipError_t launch_greedy(int pwl, int nw, bool gring, int blocks, int wpb, size_t lds, hipStream_t s,
                         const GreedyArgs &a);

// ---------------------------------------------------------------- rollouts
// Random completions of a class prefix (MCTS rollouts) turned into priority
// vectors (see kern_rollout.hip).
struct RolloutArgs {
  int64_t n;                 // rollouts (rows), all leaves
  int64_t per_leaf;          // rows per leaf: leaf l has rows l * per_leaf ...
  int32_t *out_prio;         // [n][G] caller-indexed group priorities
  const int32_t *seqs;       // [leaves][n_classes]: the leaf's prefix, then the other classes ascending
  const int32_t *depths;     // [leaves] prefix lengths
  const int32_t *group_class;// [G] caller-indexed
  uint64_t seed, draw;       // leaf l draws with draw + l
  int32_t n_classes, G;
};
hipError_t launch_rollout_prio(hipStream_t s, const RolloutArgs &a);

// ---------------------------------------------------------------- memory optimisation
// Per (candidate schedule, rank): one memory candidate per stage pair (see
// kern_memopt.hip).
constexpr int kMemoptMaxCands = 8;
// A move takes a pair from its candidate j to j + 1.  Its key orders the moves
// of one rank as the greedy compares them: the dense rank of the added time
// per freed unit (dt / dm, compared exactly) above kMemoptPairBits bits of
// pair index, so the least key is the least ratio, lowest pair on ties.
constexpr int kMemoptPairBits = 14;
constexpr uint32_t kMemoptNoMove = 0xffffffffu;
struct MemoptArgs {
  const int16_t *orders;
  int64_t n_cand;
  int64_t stride;
  int64_t *out_time;          // [n][P]
  int32_t *out_peak;          // [n][P]
  uint8_t *out_status;        // [n][P] 1 within the cap (5 % gap proven), 3 within the cap
                              // (not proven), 0 not reachable, 2 order not a permutation
  uint8_t *out_choice;        // [n][n_pairs] chosen candidate of every pair, or null
  const int32_t *rank_off;    // [P+1] ops
  const int32_t *pair_off;    // [P+1] pairs of each rank (slot order)
  const int32_t *lid_pair;    // [N] pair index on its rank | kind << 31 (by global op)
  const int64_t *cand_time;   // [pairs][kMemoptMaxCands], time ascending
  const int32_t *cand_mem;    // [pairs][kMemoptMaxCands]
  const uint32_t *move_key;   // [pairs][kMemoptMaxCands] move j -> j + 1; kMemoptNoMove past the last
  const int32_t *move_dm;     // [pairs][kMemoptMaxCands] memory it frees; 0 past the last
  const int32_t *cap;         // [P]
  int32_t P, max_pairs;
  int32_t n_pairs;            // pairs of all ranks
  int32_t bb_nodes;           // placements the branch and bound may examine
  int32_t bytes_per_thread;   // LDS per thread: 9 bytes per pair
};
hipError_t launch_memopt(int threads_per_block, hipStream_t s, const MemoptArgs &a);
// a wave per (schedule, rank), waves_per_block schedules of one rank per block,
// up to 64 * ppl pairs per rank (ppl 1, 2, 4, 8); LDS per block:
// (68 + 7 * waves_per_block) bytes per pair
hipError_t launch_memopt_wave(int ppl, int waves_per_block, hipStream_t s, const MemoptArgs &a);
size_t memopt_wave_lds(int32_t max_pairs, int waves_per_block);

// ---------------------------------------------------------------- argmin
// Least (makespan << 32 | base + index) over unflagged rows into *key, per
// segment of seg_len rows (index counted within the segment; key[s] for
// segment s); one segment: seg_len = n.
hipError_t launch_argmin(int blocks, hipStream_t s, const int32_t *ms, const uint8_t *flags,
                         int64_t n, int64_t seg_len, int n_seg, uint64_t base,
                         unsigned long long *key);

}  // namespace dipsim
