/*
 * Seeded candidate-order generator (input generation only).
 *
 * A candidate is one action order per physical rank: a permutation of the
 * rank's ops (the per-worker action list of the paper's execution plans,
 * Sec. 6.3).  This file produces such orders deterministically from
 * (seed, workload id, candidate index), independent of how the candidate
 * range is split into chunks or threads.  It computes no times: every
 * decision below counts ops, never microseconds.
 *
 * Recipes
 *   MODE_1F1B  one segment, one lane per rank: the textbook one-forward-
 *              one-backward order per stage (warm-up of min(S-s-1, M)
 *              forwards, steady 1F1B, cool-down backwards).
 *   MODE_LIST  a random linear extension of the data-edge DAG built by
 *              sweeps: in every sweep each rank takes at most one op that was
 *              ready before the sweep began.  Among ready ops a rank prefers
 *              the microbatch with the best random priority (a random
 *              microbatch permutation per candidate, the role MCTS plays in
 *              Sec. 5.1) and alternates forward/backward when both are ready,
 *              while capping in-flight forwards the way 1F1B does (Sec. 5.2's
 *              dual queues, with op counts in place of times).  Because the
 *              per-rank orders are projections of one topological order they
 *              never deadlock.
 *   swaps      afterwards k ~ U{0..max_swaps} adjacent transpositions at a
 *              uniform (rank, position); these may create deadlocks.
 *   pool       MODE_LIST bases generated once per pool slot; a candidate
 *              copies a uniformly drawn base and applies its swaps.
 *
 * Random numbers: SplitMix64 (Steele, Lea and Flood, OOPSLA 2014) used as a
 * counter-based stream keyed by (seed, workload id, purpose, index).
 */
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define MODE_1F1B 0
#define MODE_LIST 1

#define PURPOSE_CAND 2
#define PURPOSE_POOL 3

static inline uint64_t sm_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

typedef struct { uint64_t s; } rng_t;

static inline uint64_t rng_next(rng_t *r) {
  r->s += 0x9E3779B97F4A7C15ULL;
  return sm_mix(r->s);
}

/* uniform integer in [0, n) by the multiply-shift reduction of a 32-bit draw */
static inline uint32_t rng_below(rng_t *r, uint32_t n) {
  return (uint32_t)(((rng_next(r) >> 32) * (uint64_t)n) >> 32);
}

static rng_t rng_for(uint64_t seed, uint64_t cid, uint64_t purpose, uint64_t index) {
  rng_t r;
  uint64_t k = sm_mix(seed + 0x9E3779B97F4A7C15ULL);
  k = sm_mix(k ^ (cid * 0xD1B54A32D192ED03ULL));
  k = sm_mix(k ^ (purpose * 0x8CB92BA72F3D8DD7ULL));
  k = sm_mix(k ^ index);
  r.s = k;
  return r;
}

uint64_t dipgen_draw(uint64_t seed, uint64_t cid, uint64_t purpose, uint64_t index,
                     int64_t k) {
  /* the k-th raw draw of a stream, exposed for determinism tests */
  rng_t r = rng_for(seed, cid, purpose, index);
  uint64_t x = 0;
  for (int64_t i = 0; i <= k; ++i) x = rng_next(&r);
  return x;
}

typedef struct {
  int32_t n_ranks;
  int32_t n_mb;             /* microbatches (priority classes) */
  int32_t n_lanes;
  const int64_t *rank_off;  /* [P+1] */
  const int32_t *pred_ptr;  /* [N+1] */
  const int32_t *succ_ptr;  /* [N+1] */
  const int32_t *succ_op;   /* [E] */
  const uint8_t *op_kind;   /* [N] */
  const int32_t *op_mb;     /* [N] */
  const int32_t *op_rank;   /* [N] */
  const int32_t *rank_first_lane; /* [P] */
} dipgen_topo;

typedef struct {
  int32_t mode, max_swaps, pool, limit_jitter;
  uint64_t seed, cid;
  const int16_t *pool_orders; /* [pool][stride] for pool mode */
  int64_t stride;
} dipgen_recipe;

/* ---- binary min-heap of 64-bit keys ------------------------------------ */
typedef struct { uint64_t *a; int32_t n; } heap_t;

static void heap_push(heap_t *h, uint64_t k) {
  int32_t i = h->n++;
  while (i > 0) {
    int32_t p = (i - 1) >> 1;
    if (h->a[p] <= k) break;
    h->a[i] = h->a[p];
    i = p;
  }
  h->a[i] = k;
}

static uint64_t heap_pop(heap_t *h) {
  uint64_t top = h->a[0];
  uint64_t k = h->a[--h->n];
  int32_t i = 0;
  for (;;) {
    int32_t c = 2 * i + 1;
    if (c >= h->n) break;
    if (c + 1 < h->n && h->a[c + 1] < h->a[c]) ++c;
    if (h->a[c] >= k) break;
    h->a[i] = h->a[c];
    i = c;
  }
  if (h->n > 0) h->a[i] = k;
  return top;
}

typedef struct {
  int32_t *cnt;      /* [N] unresolved predecessors */
  int32_t *prio;     /* [M] microbatch priority */
  int32_t *just;     /* [P] ops emitted in the current sweep */
  int32_t *fill;     /* [P] */
  int32_t *inflight; /* [P] */
  int32_t *limit;    /* [P] */
  uint8_t *last;     /* [P] */
  heap_t *hf, *hb;   /* [P] */
  uint64_t *heap_mem;
} work_t;

static int work_init(work_t *w, const dipgen_topo *t) {
  int32_t P = t->n_ranks;
  int64_t N = t->rank_off[P];
  memset(w, 0, sizeof(*w));
  w->cnt = (int32_t *)malloc(sizeof(int32_t) * (N + 1));
  w->prio = (int32_t *)malloc(sizeof(int32_t) * (t->n_mb + 1));
  w->just = (int32_t *)malloc(sizeof(int32_t) * P);
  w->fill = (int32_t *)malloc(sizeof(int32_t) * P);
  w->inflight = (int32_t *)malloc(sizeof(int32_t) * P);
  w->limit = (int32_t *)malloc(sizeof(int32_t) * P);
  w->last = (uint8_t *)malloc(P);
  w->hf = (heap_t *)malloc(sizeof(heap_t) * P);
  w->hb = (heap_t *)malloc(sizeof(heap_t) * P);
  w->heap_mem = (uint64_t *)malloc(sizeof(uint64_t) * (2 * N + 2));
  if (!w->cnt || !w->prio || !w->just || !w->fill || !w->inflight || !w->limit ||
      !w->last || !w->hf || !w->hb || !w->heap_mem)
    return -1;
  /* each rank's two heaps get disjoint slices sized by the rank's op count */
  int64_t off = 0;
  for (int32_t r = 0; r < P; ++r) {
    int64_t nr = t->rank_off[r + 1] - t->rank_off[r];
    w->hf[r].a = w->heap_mem + off; off += nr;
    w->hb[r].a = w->heap_mem + off; off += nr;
  }
  return 0;
}

static void work_free(work_t *w) {
  free(w->cnt); free(w->prio); free(w->just); free(w->fill); free(w->inflight);
  free(w->limit); free(w->last); free(w->hf); free(w->hb); free(w->heap_mem);
}

static void order_1f1b(const dipgen_topo *t, int16_t *out) {
  int32_t S = t->n_ranks;
  for (int32_t s = 0; s < S; ++s) {
    int32_t M = (int32_t)((t->rank_off[s + 1] - t->rank_off[s]) / 2);
    int16_t *o = out + t->rank_off[s];
    int32_t w = S - s - 1 < M ? S - s - 1 : M, k = 0;
    for (int32_t m = 0; m < w; ++m) o[k++] = (int16_t)(2 * m);
    for (int32_t i = 0; i < M - w; ++i) {
      o[k++] = (int16_t)(2 * (w + i));
      o[k++] = (int16_t)(2 * i + 1);
    }
    for (int32_t m = M - w; m < M; ++m) o[k++] = (int16_t)(2 * m + 1);
  }
}

static int order_list(const dipgen_topo *t, work_t *w, rng_t *rng, int32_t jitter,
                      int16_t *out) {
  int32_t P = t->n_ranks, M = t->n_mb;
  int64_t N = t->rank_off[P];
  /* random microbatch priority: a uniform permutation (Fisher-Yates) */
  for (int32_t j = 0; j < M; ++j) w->prio[j] = j;
  for (int32_t j = M - 1; j > 0; --j) {
    int32_t k = (int32_t)rng_below(rng, (uint32_t)(j + 1));
    int32_t tmp = w->prio[j]; w->prio[j] = w->prio[k]; w->prio[k] = tmp;
  }
  for (int32_t r = 0; r < P; ++r) {
    w->hf[r].n = w->hb[r].n = 0;
    w->fill[r] = 0;
    w->inflight[r] = 0;
    w->last[r] = 1;
    w->limit[r] = t->n_lanes - t->rank_first_lane[r] +
                  (jitter > 0 ? (int32_t)rng_below(rng, (uint32_t)jitter + 1) : 0);
  }
  for (int64_t g = 0; g < N; ++g) {
    w->cnt[g] = t->pred_ptr[g + 1] - t->pred_ptr[g];
    if (w->cnt[g] == 0) {
      int32_t r = t->op_rank[g];
      uint64_t key = ((uint64_t)w->prio[t->op_mb[g]] << 32) | (uint64_t)g;
      heap_push(t->op_kind[g] ? &w->hb[r] : &w->hf[r], key);
    }
  }
  int64_t emitted = 0;
  while (emitted < N) {
    int32_t any = 0;
    /* second attempt lifts the in-flight caps: with interleaved lanes every
       rank can sit at its cap while the op that would free one waits behind
       another rank's cap */
    for (int32_t attempt = 0; attempt < 2 && !any; ++attempt) {
      for (int32_t r = 0; r < P; ++r) {
        int32_t canF = w->hf[r].n > 0 && (attempt == 1 || w->inflight[r] < w->limit[r]);
        int32_t canB = w->hb[r].n > 0;
        int32_t takeB;
        if (canF && canB) takeB = (w->last[r] == 0);
        else if (canB) takeB = 1;
        else if (canF) takeB = 0;
        else { w->just[r] = -1; continue; }
        uint64_t key = heap_pop(takeB ? &w->hb[r] : &w->hf[r]);
        int32_t g = (int32_t)(key & 0xffffffffu);
        out[t->rank_off[r] + w->fill[r]++] = (int16_t)(g - t->rank_off[r]);
        w->inflight[r] += takeB ? -1 : 1;
        w->last[r] = (uint8_t)takeB;
        w->just[r] = g;
        any = 1;
      }
    }
    if (!any) return -1; /* impossible for an acyclic data graph */
    for (int32_t r = 0; r < P; ++r) {
      int32_t g = w->just[r];
      if (g < 0) continue;
      ++emitted;
      for (int32_t e = t->succ_ptr[g]; e < t->succ_ptr[g + 1]; ++e) {
        int32_t s = t->succ_op[e];
        if (--w->cnt[s] == 0) {
          int32_t rs = t->op_rank[s];
          uint64_t k2 = ((uint64_t)w->prio[t->op_mb[s]] << 32) | (uint64_t)s;
          heap_push(t->op_kind[s] ? &w->hb[rs] : &w->hf[rs], k2);
        }
      }
    }
  }
  return 0;
}

static void apply_swaps(const dipgen_topo *t, rng_t *rng, int32_t max_swaps,
                        int16_t *out) {
  if (max_swaps <= 0) return;
  int32_t k = (int32_t)rng_below(rng, (uint32_t)max_swaps + 1);
  for (int32_t i = 0; i < k; ++i) {
    int32_t r = (int32_t)rng_below(rng, (uint32_t)t->n_ranks);
    int64_t nr = t->rank_off[r + 1] - t->rank_off[r];
    if (nr < 2) { (void)rng_below(rng, 1); continue; }
    int64_t p = rng_below(rng, (uint32_t)(nr - 1));
    int16_t *o = out + t->rank_off[r];
    int16_t tmp = o[p]; o[p] = o[p + 1]; o[p + 1] = tmp;
  }
}

static int gen_one(const dipgen_topo *t, const dipgen_recipe *rc, work_t *w,
                   int64_t idx, uint64_t purpose, int16_t *out) {
  int64_t N = t->rank_off[t->n_ranks];
  rng_t rng = rng_for(rc->seed, rc->cid, purpose, (uint64_t)idx);
  if (rc->mode == MODE_1F1B) {
    order_1f1b(t, out);
  } else if (rc->pool > 0 && purpose == PURPOSE_CAND) {
    uint32_t b = rng_below(&rng, (uint32_t)rc->pool);
    memcpy(out, rc->pool_orders + (int64_t)b * rc->stride, sizeof(int16_t) * N);
  } else {
    if (order_list(t, w, &rng, rc->limit_jitter, out) != 0) return -1;
  }
  if (purpose == PURPOSE_CAND) apply_swaps(t, &rng, rc->max_swaps, out);
  for (int64_t i = N; i < rc->stride; ++i) out[i] = 0;
  return 0;
}

typedef struct {
  const dipgen_topo *t;
  const dipgen_recipe *rc;
  int64_t i0, i1, base;
  uint64_t purpose;
  int16_t *out;
  int rc_out;
} job_t;

static void *run_job(void *arg) {
  job_t *j = (job_t *)arg;
  work_t w;
  if (work_init(&w, j->t) != 0) { j->rc_out = -2; work_free(&w); return NULL; }
  for (int64_t i = j->i0; i < j->i1; ++i) {
    if (gen_one(j->t, j->rc, &w, j->base + i, j->purpose,
                j->out + i * j->rc->stride) != 0) {
      j->rc_out = -1;
      break;
    }
  }
  work_free(&w);
  return NULL;
}

/* Generate candidates [first, first+n) (or pool bases when purpose == POOL)
 * into out[n][stride].  Returns 0, -1 on a cyclic data graph, -2 on OOM. */
int dipgen_orders(const dipgen_topo *t, const dipgen_recipe *rc, int32_t purpose,
                  int64_t first, int64_t n, int16_t *out, int32_t n_threads) {
  if (n <= 0) return 0;
  if (n_threads < 1) n_threads = 1;
  if (n_threads > 256) n_threads = 256;
  if (n < n_threads) n_threads = (int32_t)n;
  pthread_t th[256];
  int created[256];
  job_t jobs[256];
  int64_t per = (n + n_threads - 1) / n_threads;
  for (int32_t k = 0; k < n_threads; ++k) {
    jobs[k].t = t; jobs[k].rc = rc; jobs[k].base = first;
    jobs[k].i0 = k * per < n ? k * per : n;
    jobs[k].i1 = (k + 1) * per < n ? (k + 1) * per : n;
    jobs[k].purpose = (uint64_t)purpose; jobs[k].out = out; jobs[k].rc_out = 0;
    created[k] = 0;
    if (jobs[k].i0 >= jobs[k].i1) continue;
    if (n_threads > 1 && pthread_create(&th[k], NULL, run_job, &jobs[k]) == 0)
      created[k] = 1;
    else
      run_job(&jobs[k]);
  }
  int ret = 0;
  for (int32_t k = 0; k < n_threads; ++k)
    if (created[k]) pthread_join(th[k], NULL);
  for (int32_t k = 0; k < n_threads; ++k)
    if (jobs[k].rc_out != 0) ret = jobs[k].rc_out;
  return ret;
}
