/*
 * dip_oracle.c -- CPU oracle for batched pipeline-schedule simulation.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load or call this file.  It shares no code,
 * header, table or helper with the GPU library, and the GPU library never
 * calls it.
 *
 * What it computes (DIP, arXiv 2504.14145), for each candidate schedule of one
 * instance:
 *
 *   Instance: ops (pipeline stages, Sec. 5.2) placed on physical ranks, each
 *   with an integer cost; data edges p -> o with an integer transfer latency
 *   (asynchronous point-to-point, Sec. 6.3); a memory slot per op whose
 *   activation is held from the forward's start to the matching backward's
 *   end (the liveness of a stage pair in Sec. 5.3's memory constraint).
 *
 *   Candidate: one order per rank (the worker's action list, Sec. 6.3).
 *
 *   Timing: a rank runs one op at a time, in its order, each op as soon as
 *   the rank is free and every predecessor's output has arrived -- the
 *   t_last / t_start rule of Sec. 5.2, with timestamps populated in
 *   topological order as Sec. 6.1's simulator does.  So
 *       start(o) = max(free(rank(o)), max_p end(p) + comm(p, o)),
 *       end(o)   = start(o) + cost(o).
 *   If no op can ever start while ops remain, the orders deadlock.
 *
 *   Outputs: makespan T = latest end; bubble_r = T - (sum of rank r's costs),
 *   the idle time of rank r over [0, T]; peak_r = the largest prefix sum of
 *   +act (at each F) / -act (at each B) along rank r's order, starting from 0;
 *   flag bits: 1 deadlock, 2 some peak_r > cap_r (cap_r >= 0), 4 a rank's
 *   section is not a permutation of its op ids.  Deadlocked candidates report
 *   T = bubble = -1 and keep their peaks; invalid ones report -1 everywhere.
 *
 * Method: a discrete-event simulation.  Completion events sit in a min-heap
 * ordered by (time, rank).  When an op completes, its rank advances and tries
 * to launch its next op; a rank whose next op still has an unfinished
 * predecessor parks on that predecessor and is retried when it completes.
 * An empty heap with ops left over is a deadlock.
 *
 * All arithmetic is integer; intermediate times are carried in 64 bits and
 * the entry points return -3 if any result would not fit in int32.
 */
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define FLAG_DEADLOCK 1u
#define FLAG_CAP 2u
#define FLAG_INVALID 4u

typedef struct {
  int32_t n_ranks;
  const int64_t *rank_off;   /* [P+1] global op offset of each rank */
  const int32_t *pred_ptr;   /* [N+1] */
  const int32_t *pred_op;    /* [E] global index of the predecessor */
  const uint8_t *op_kind;    /* [N] 0 = F, 1 = B */
  const int32_t *op_slot;    /* [N] */
  int32_t n_slots;
  const int32_t *mem_cap;    /* [P] */
  const int32_t *op_cost;    /* [N] */
  const int32_t *edge_comm;  /* [E] */
  const int32_t *slot_act;   /* [n_slots] */
} dor_instance;

typedef struct {
  int64_t *end;        /* [N] end time, valid once done */
  int64_t *start;      /* [N] */
  uint8_t *done;       /* [N] */
  int32_t *park_head;  /* [N] first rank parked on this op, -1 none */
  int32_t *park_next;  /* [P] */
  int64_t *ptr;        /* [P] position in the rank's order */
  int64_t *free_at;    /* [P] end of the rank's last op */
  uint8_t *seen;       /* [max n_r] permutation check */
  uint64_t *heap;      /* [P] events (time << 32 | rank) */
  int32_t heap_n;
} dor_work;

static int work_alloc(dor_work *w, const dor_instance *I) {
  int64_t N = I->rank_off[I->n_ranks];
  int64_t maxr = 1;
  for (int32_t r = 0; r < I->n_ranks; ++r) {
    int64_t nr = I->rank_off[r + 1] - I->rank_off[r];
    if (nr > maxr) maxr = nr;
  }
  memset(w, 0, sizeof(*w));
  w->end = (int64_t *)malloc(sizeof(int64_t) * (N + 1));
  w->start = (int64_t *)malloc(sizeof(int64_t) * (N + 1));
  w->done = (uint8_t *)malloc(N + 1);
  w->park_head = (int32_t *)malloc(sizeof(int32_t) * (N + 1));
  w->park_next = (int32_t *)malloc(sizeof(int32_t) * (I->n_ranks + 1));
  w->ptr = (int64_t *)malloc(sizeof(int64_t) * (I->n_ranks + 1));
  w->free_at = (int64_t *)malloc(sizeof(int64_t) * (I->n_ranks + 1));
  w->seen = (uint8_t *)malloc(maxr + 1);
  w->heap = (uint64_t *)malloc(sizeof(uint64_t) * (I->n_ranks + 1));
  if (!w->end || !w->start || !w->done || !w->park_head || !w->park_next || !w->ptr ||
      !w->free_at || !w->seen || !w->heap)
    return -2;
  return 0;
}

static void work_release(dor_work *w) {
  free(w->end); free(w->start); free(w->done); free(w->park_head); free(w->park_next);
  free(w->ptr); free(w->free_at); free(w->seen); free(w->heap);
}

static void ev_push(dor_work *w, uint64_t k) {
  int32_t i = w->heap_n++;
  while (i > 0) {
    int32_t p = (i - 1) / 2;
    if (w->heap[p] <= k) break;
    w->heap[i] = w->heap[p];
    i = p;
  }
  w->heap[i] = k;
}

static uint64_t ev_pop(dor_work *w) {
  uint64_t top = w->heap[0];
  uint64_t k = w->heap[--w->heap_n];
  int32_t i = 0;
  for (;;) {
    int32_t c = 2 * i + 1;
    if (c >= w->heap_n) break;
    if (c + 1 < w->heap_n && w->heap[c + 1] < w->heap[c]) ++c;
    if (w->heap[c] >= k) break;
    w->heap[i] = w->heap[c];
    i = c;
  }
  if (w->heap_n > 0) w->heap[i] = k;
  return top;
}

/* Try to start rank r's next op.  Returns -3 on int32 overflow, else 0. */
static int try_launch(const dor_instance *I, dor_work *w, const int16_t *order, int32_t r) {
  int64_t base = I->rank_off[r];
  int64_t nr = I->rank_off[r + 1] - base;
  if (w->ptr[r] >= nr) return 0;
  int64_t g = base + order[base + w->ptr[r]];
  int64_t ready_at = w->free_at[r];
  for (int32_t e = I->pred_ptr[g]; e < I->pred_ptr[g + 1]; ++e) {
    int32_t p = I->pred_op[e];
    if (!w->done[p]) {               /* park on the unfinished predecessor */
      w->park_next[r] = w->park_head[p];
      w->park_head[p] = r;
      return 0;
    }
    int64_t arrive = w->end[p] + I->edge_comm[e];
    if (arrive > ready_at) ready_at = arrive;
  }
  w->start[g] = ready_at;
  w->end[g] = ready_at + I->op_cost[g];
  if (w->end[g] > INT32_MAX) return -3;
  w->free_at[r] = w->end[g];
  ev_push(w, ((uint64_t)w->end[g] << 32) | (uint64_t)r);
  return 0;
}

/* Simulate one candidate.  start/end may be NULL; when given they receive
 * per-op times (-1 for ops that never ran). */
static int eval_one(const dor_instance *I, dor_work *w, const int16_t *order,
                    int32_t *makespan, int32_t *bubble, int32_t *peak, uint8_t *flags,
                    int32_t *start_out, int32_t *end_out) {
  int32_t P = I->n_ranks;
  int64_t N = I->rank_off[P];
  uint8_t f = 0;

  /* 1. each rank's section must be a permutation of 0 .. n_r - 1 */
  for (int32_t r = 0; r < P; ++r) {
    int64_t base = I->rank_off[r], nr = I->rank_off[r + 1] - base;
    memset(w->seen, 0, (size_t)nr + 1);
    for (int64_t i = 0; i < nr; ++i) {
      int32_t id = order[base + i];
      if (id < 0 || id >= nr || w->seen[id]) { f |= FLAG_INVALID; break; }
      w->seen[id] = 1;
    }
  }
  if (f & FLAG_INVALID) {
    *makespan = -1;
    for (int32_t r = 0; r < P; ++r) { bubble[r] = -1; peak[r] = -1; }
    *flags = f;
    if (start_out) for (int64_t g = 0; g < N; ++g) { start_out[g] = -1; end_out[g] = -1; }
    return 0;
  }

  /* 2. memory: prefix sums of +act / -act along each rank's order */
  for (int32_t r = 0; r < P; ++r) {
    int64_t base = I->rank_off[r], nr = I->rank_off[r + 1] - base;
    int64_t mem = 0, pk = 0;
    for (int64_t i = 0; i < nr; ++i) {
      int64_t g = base + order[base + i];
      int64_t a = I->slot_act[I->op_slot[g]];
      if (I->op_kind[g] == 0) {
        mem += a;
        if (mem > pk) pk = mem;
      } else {
        mem -= a;
      }
    }
    if (pk > INT32_MAX) return -3;
    peak[r] = (int32_t)pk;
    if (I->mem_cap[r] >= 0 && pk > I->mem_cap[r]) f |= FLAG_CAP;
  }

  /* 3. event loop */
  for (int64_t g = 0; g < N; ++g) { w->done[g] = 0; w->park_head[g] = -1; w->end[g] = -1; w->start[g] = -1; }
  for (int32_t r = 0; r < P; ++r) { w->ptr[r] = 0; w->free_at[r] = 0; w->park_next[r] = -1; }
  w->heap_n = 0;
  for (int32_t r = 0; r < P; ++r)
    if (try_launch(I, w, order, r) != 0) return -3;
  int64_t n_done = 0;
  while (w->heap_n > 0) {
    uint64_t ev = ev_pop(w);
    int32_t r = (int32_t)(ev & 0xffffffffu);
    int64_t base = I->rank_off[r];
    int64_t g = base + order[base + w->ptr[r]];
    w->done[g] = 1;
    ++n_done;
    w->ptr[r] += 1;
    if (try_launch(I, w, order, r) != 0) return -3;
    int32_t q = w->park_head[g];
    w->park_head[g] = -1;
    while (q >= 0) {
      int32_t nxt = w->park_next[q];
      w->park_next[q] = -1;
      if (try_launch(I, w, order, q) != 0) return -3;
      q = nxt;
    }
  }

  if (start_out) {
    for (int64_t g = 0; g < N; ++g) {
      start_out[g] = w->done[g] ? (int32_t)w->start[g] : -1;
      end_out[g] = w->done[g] ? (int32_t)w->end[g] : -1;
    }
  }
  if (n_done < N) {           /* 4. stalled with ops left: deadlock */
    f |= FLAG_DEADLOCK;
    *makespan = -1;
    for (int32_t r = 0; r < P; ++r) bubble[r] = -1;
    *flags = f;
    return 0;
  }
  /* 5. makespan and per-rank idle time */
  int64_t T = 0;
  for (int32_t r = 0; r < P; ++r) if (w->free_at[r] > T) T = w->free_at[r];
  *makespan = (int32_t)T;
  for (int32_t r = 0; r < P; ++r) {
    int64_t busy = 0;
    for (int64_t g = I->rank_off[r]; g < I->rank_off[r + 1]; ++g) busy += I->op_cost[g];
    bubble[r] = (int32_t)(T - busy);
  }
  *flags = f;
  return 0;
}

typedef struct {
  const dor_instance *I;
  const int16_t *orders;
  int64_t stride, i0, i1;
  int32_t *makespan, *bubble, *peak;
  uint8_t *flags;
  int rc;
} dor_job;

static void *dor_run(void *arg) {
  dor_job *j = (dor_job *)arg;
  dor_work w;
  int32_t P = j->I->n_ranks;
  if (work_alloc(&w, j->I) != 0) { j->rc = -2; work_release(&w); return NULL; }
  for (int64_t i = j->i0; i < j->i1; ++i) {
    int rc = eval_one(j->I, &w, j->orders + i * j->stride, &j->makespan[i],
                      &j->bubble[i * P], &j->peak[i * P], &j->flags[i], NULL, NULL);
    if (rc != 0) { j->rc = rc; break; }
  }
  work_release(&w);
  return NULL;
}

/* Evaluate n_cand candidates; candidates are independent, so n_threads
 * threads take contiguous ranges (the per-candidate simulation itself is
 * single-threaded).  Returns 0, -2 (out of memory) or -3 (int32 overflow). */
int dor_eval(const dor_instance *I, const int16_t *orders, int64_t n_cand, int64_t stride,
             int32_t *makespan, int32_t *bubble, int32_t *peak, uint8_t *flags,
             int32_t n_threads) {
  if (n_cand <= 0) return 0;
  if (n_threads < 1) n_threads = 1;
  if (n_threads > 256) n_threads = 256;
  if (n_cand < n_threads) n_threads = (int32_t)n_cand;
  pthread_t th[256];
  int created[256];
  dor_job jobs[256];
  int64_t per = (n_cand + n_threads - 1) / n_threads;
  for (int32_t k = 0; k < n_threads; ++k) {
    dor_job *j = &jobs[k];
    j->I = I; j->orders = orders; j->stride = stride;
    j->i0 = k * per < n_cand ? k * per : n_cand;
    j->i1 = (k + 1) * per < n_cand ? (k + 1) * per : n_cand;
    j->makespan = makespan; j->bubble = bubble; j->peak = peak; j->flags = flags;
    j->rc = 0;
    created[k] = 0;
    if (j->i0 >= j->i1) continue;
    if (n_threads > 1 && pthread_create(&th[k], NULL, dor_run, j) == 0) created[k] = 1;
    else dor_run(j);
  }
  int rc = 0;
  for (int32_t k = 0; k < n_threads; ++k) {
    if (created[k]) pthread_join(th[k], NULL);
    if (jobs[k].rc != 0) rc = jobs[k].rc;
  }
  return rc;
}

/* One candidate with its full timeline: start/end per global op. */
int dor_timeline(const dor_instance *I, const int16_t *order, int32_t *makespan,
                 int32_t *bubble, int32_t *peak, uint8_t *flags, int32_t *start,
                 int32_t *end) {
  dor_work w;
  if (work_alloc(&w, I) != 0) { work_release(&w); return -2; }
  int rc = eval_one(I, &w, order, makespan, bubble, peak, flags, start, end);
  work_release(&w);
  return rc;
}

/* Lexicographically smallest (makespan, index) over candidates whose flags
 * are all clear.  Returns the global index (index_base + i) or -1. */
int64_t dor_argmin(const int32_t *makespan, const uint8_t *flags, int64_t n,
                   int64_t index_base, int32_t *best_makespan) {
  int64_t best = -1;
  int32_t bm = 0;
  for (int64_t i = 0; i < n; ++i) {
    if (flags[i] != 0) continue;
    if (best < 0 || makespan[i] < bm) { best = i; bm = makespan[i]; }
  }
  if (best_makespan) *best_makespan = best < 0 ? -1 : bm;
  return best < 0 ? -1 : index_base + best;
}
