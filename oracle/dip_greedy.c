/*
 * dip_greedy.c -- CPU oracle for DIP's dual-queue stage interleaving.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load or call this file.  It shares no code,
 * header, table or helper with the GPU library, and the GPU library never
 * calls it.
 *
 * What it computes (DIP, arXiv 2504.14145, Sec. 5.2), for each candidate
 * priority vector of one instance (the instance layout of dip_oracle.c):
 *
 *   Priorities.  Every op (pipeline stage) belongs to a priority group -- a
 *   pipeline segment of Sec. 5.1, one sub-microbatch's forward or backward
 *   through a run of model chunks -- and a candidate gives one integer
 *   priority per group, larger first.  Equal priorities are ordered by group
 *   index (the fixed order Sec. 5.1 imposes between equal-priority
 *   segments), and stages of one group on one rank by rank-local id.
 *
 *   State (Sec. 5.2, "Initialization").  Per rank: t_last, the end of its last
 *   scheduled stage (0 at first), the kind of that stage, and its queued
 *   forward and backward stages.  Per stage: t_start, the earliest time its
 *   inputs are all present: 0 for a stage without predecessors; otherwise
 *   unknown (+inf, not queued) until every predecessor is scheduled, then
 *   max over predecessors p of end(p) + comm(p, o).  A stage is queued on its
 *   rank from that moment until it is scheduled.
 *
 *   One step (Sec. 5.2, "Iterative Scheduling"), repeated until every stage
 *   is scheduled.  For every rank, with t_fw / t_bw the smallest t_start in
 *   its forward / backward queue:
 *     t_min = max(t_last, min(t_fw, t_bw)), the earliest time the rank can
 *             start a queued stage;
 *     if t_fw < t_last and t_bw < t_last: the kind opposite to the last
 *             scheduled one (the 1F1B alternation), and among queued stages
 *             of that kind with t_start <= t_last the highest priority;
 *     otherwise: among all queued stages with t_start <= t_min (each starts
 *             at t_min, so none adds idle time) the highest priority.
 *   Memory (Sec. 5.2, "Memory Constraints"): the rank's live activation is
 *   the sum of act over its scheduled forwards whose backward is not yet
 *   scheduled.  If the choice is a forward that would take the live
 *   activation above the rank's cap (cap >= 0), the forward queue is disabled
 *   for this step and the rank decides again from its backward queue alone
 *   (t_fw = +inf).  The rank with the smallest t_min (lowest index on ties)
 *   schedules its choice: start = t_min, end = start + cost, t_last = end,
 *   successors' t_start updated.  If no rank can choose while stages remain
 *   -- every queued stage is a forward held back by the cap -- the cap is
 *   lifted for that one step (the schedule will then exceed it, and the
 *   outputs flag it).
 *
 *   Outputs: each rank's order (rank-local ids in scheduling order, the
 *   layout the simulator consumes) and the greedy's own timeline: makespan
 *   T = latest end, bubble_r = T - sum of rank r's costs, peak_r = largest
 *   live activation, flag 2 if some peak_r > cap_r (cap_r >= 0).  Because a
 *   stage is scheduled only after all its predecessors, with start =
 *   max(t_last, t_start), these are exactly what the simulator computes for
 *   the emitted orders.
 *
 * The steps follow the paper's order; nothing is batched or reordered.  Per
 * rank the queued stages sit in an unordered list that is scanned at every
 * step (slow and plain on purpose).  Integer arithmetic throughout; times in
 * 64 bits, -3 if a result does not fit int32.
 */
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define G_FLAG_CAP 2u
#define G_INF INT64_MAX

typedef struct {
  int32_t n_ranks;
  const int64_t *rank_off;
  const int32_t *pred_ptr;
  const int32_t *pred_op;
  const uint8_t *op_kind;
  const int32_t *op_slot;
  int32_t n_slots;
  const int32_t *mem_cap;
  const int32_t *op_cost;
  const int32_t *edge_comm;
  const int32_t *slot_act;
} dgr_instance;   /* same field order as the simulator oracle's instance */

typedef struct {
  int64_t N;
  int32_t *succ_ptr;   /* [N+1] */
  int32_t *succ_op;    /* [E] */
  int32_t *succ_edge;  /* [E] index into pred_op / edge_comm */
  int32_t *op_rank;    /* [N] */
} dgr_graph;

typedef struct {
  int64_t *acc;        /* [N] running max of end(p) + comm over scheduled preds */
  int64_t *tstart;     /* [N] valid while queued */
  int64_t *start, *end;/* [N] */
  int32_t *left;       /* [N] predecessors not yet scheduled */
  int32_t *qpos;       /* [N] position in its rank's queue, -1 if not queued */
  int32_t *queue;      /* [N] per-rank queues, rank r at rank_off[r] */
  int32_t *qn;         /* [P] */
  int64_t *t_last, *live, *peak;  /* [P] */
  int32_t *last_kind;  /* [P] -1 none, 0 F, 1 B */
  int32_t *emitted;    /* [P] */
} dgr_work;

static int graph_build(const dgr_instance *I, dgr_graph *g) {
  int32_t P = I->n_ranks;
  int64_t N = I->rank_off[P];
  int32_t E = I->pred_ptr[N];
  memset(g, 0, sizeof(*g));
  g->N = N;
  g->succ_ptr = (int32_t *)calloc((size_t)N + 1, sizeof(int32_t));
  g->succ_op = (int32_t *)malloc(sizeof(int32_t) * ((size_t)E + 1));
  g->succ_edge = (int32_t *)malloc(sizeof(int32_t) * ((size_t)E + 1));
  g->op_rank = (int32_t *)malloc(sizeof(int32_t) * ((size_t)N + 1));
  int32_t *fill = (int32_t *)calloc((size_t)N + 1, sizeof(int32_t));
  if (!g->succ_ptr || !g->succ_op || !g->succ_edge || !g->op_rank || !fill) {
    free(fill);
    return -2;
  }
  for (int32_t r = 0; r < P; ++r)
    for (int64_t o = I->rank_off[r]; o < I->rank_off[r + 1]; ++o) g->op_rank[o] = r;
  for (int32_t e = 0; e < E; ++e) g->succ_ptr[I->pred_op[e] + 1] += 1;
  for (int64_t o = 0; o < N; ++o) g->succ_ptr[o + 1] += g->succ_ptr[o];
  for (int64_t o = 0; o < N; ++o)
    for (int32_t e = I->pred_ptr[o]; e < I->pred_ptr[o + 1]; ++e) {
      int32_t p = I->pred_op[e];
      int32_t k = g->succ_ptr[p] + fill[p]++;
      g->succ_op[k] = (int32_t)o;
      g->succ_edge[k] = e;
    }
  free(fill);
  return 0;
}

static void graph_release(dgr_graph *g) {
  free(g->succ_ptr); free(g->succ_op); free(g->succ_edge); free(g->op_rank);
}

static int work_alloc(dgr_work *w, int64_t N, int32_t P) {
  memset(w, 0, sizeof(*w));
  size_t n = (size_t)N + 1, p = (size_t)P + 1;
  w->acc = (int64_t *)malloc(sizeof(int64_t) * n);
  w->tstart = (int64_t *)malloc(sizeof(int64_t) * n);
  w->start = (int64_t *)malloc(sizeof(int64_t) * n);
  w->end = (int64_t *)malloc(sizeof(int64_t) * n);
  w->left = (int32_t *)malloc(sizeof(int32_t) * n);
  w->qpos = (int32_t *)malloc(sizeof(int32_t) * n);
  w->queue = (int32_t *)malloc(sizeof(int32_t) * n);
  w->qn = (int32_t *)malloc(sizeof(int32_t) * p);
  w->t_last = (int64_t *)malloc(sizeof(int64_t) * p);
  w->live = (int64_t *)malloc(sizeof(int64_t) * p);
  w->peak = (int64_t *)malloc(sizeof(int64_t) * p);
  w->last_kind = (int32_t *)malloc(sizeof(int32_t) * p);
  w->emitted = (int32_t *)malloc(sizeof(int32_t) * p);
  if (!w->acc || !w->tstart || !w->start || !w->end || !w->left || !w->qpos || !w->queue ||
      !w->qn || !w->t_last || !w->live || !w->peak || !w->last_kind || !w->emitted)
    return -2;
  return 0;
}

static void work_release(dgr_work *w) {
  free(w->acc); free(w->tstart); free(w->start); free(w->end); free(w->left); free(w->qpos);
  free(w->queue); free(w->qn); free(w->t_last); free(w->live); free(w->peak);
  free(w->last_kind); free(w->emitted);
}

static void enqueue(const dgr_instance *I, const dgr_graph *G, dgr_work *w, int32_t o,
                    int64_t t) {
  int32_t r = G->op_rank[o];
  w->tstart[o] = t;
  w->qpos[o] = w->qn[r];
  w->queue[I->rank_off[r] + w->qn[r]] = o;
  w->qn[r] += 1;
}

static void dequeue(const dgr_instance *I, const dgr_graph *G, dgr_work *w, int32_t o) {
  int32_t r = G->op_rank[o];
  int64_t base = I->rank_off[r];
  int32_t i = w->qpos[o], last = w->queue[base + w->qn[r] - 1];
  w->queue[base + i] = last;
  w->qpos[last] = i;
  w->qn[r] -= 1;
  w->qpos[o] = -1;
}

/* a outranks b: larger priority, then smaller group index, then smaller op
 * index (op indices of one rank follow its rank-local ids) */
static int outranks(const int32_t *op_group, const int32_t *prio, int32_t a, int32_t b) {
  int32_t pa = prio[op_group[a]], pb = prio[op_group[b]];
  if (pa != pb) return pa > pb;
  if (op_group[a] != op_group[b]) return op_group[a] < op_group[b];
  return a < b;
}

/* Rank r's choice for this step: returns the op (or -1) and its t_min. */
static int32_t rank_choice(const dgr_instance *I, const dgr_work *w, const int32_t *op_group,
                           const int32_t *prio, int32_t r, int use_cap, int64_t *t_min_out) {
  int64_t base = I->rank_off[r];
  int64_t t_last = w->t_last[r];
  for (int fw_on = 1; fw_on >= 0; --fw_on) {
    int64_t t_fw = G_INF, t_bw = G_INF;
    for (int32_t i = 0; i < w->qn[r]; ++i) {
      int32_t o = w->queue[base + i];
      if (I->op_kind[o] == 0) {
        if (fw_on && w->tstart[o] < t_fw) t_fw = w->tstart[o];
      } else if (w->tstart[o] < t_bw) {
        t_bw = w->tstart[o];
      }
    }
    if (t_fw == G_INF && t_bw == G_INF) return -1;
    int64_t t_min = t_fw < t_bw ? t_fw : t_bw;
    if (t_min < t_last) t_min = t_last;
    int alternate = t_fw < t_last && t_bw < t_last;
    int want = w->last_kind[r] == 0 ? 1 : 0;   /* 1F1B: the other kind */
    int32_t best = -1;
    for (int32_t i = 0; i < w->qn[r]; ++i) {
      int32_t o = w->queue[base + i];
      int kind = I->op_kind[o];
      if (kind == 0 && !fw_on) continue;
      if (alternate ? (kind != want || w->tstart[o] > t_last) : w->tstart[o] > t_min) continue;
      if (best < 0 || outranks(op_group, prio, o, best)) best = o;
    }
    if (use_cap && fw_on && I->op_kind[best] == 0 && I->mem_cap[r] >= 0 &&
        w->live[r] + I->slot_act[I->op_slot[best]] > I->mem_cap[r])
      continue;                                 /* forward queue disabled */
    *t_min_out = t_min;
    return best;
  }
  return -1;
}

static int greedy_one(const dgr_instance *I, const dgr_graph *G, dgr_work *w,
                      const int32_t *op_group, const int32_t *prio, int16_t *order,
                      int32_t *makespan, int32_t *bubble, int32_t *peak, uint8_t *flags,
                      int32_t *start_out, int32_t *end_out) {
  int32_t P = I->n_ranks;
  int64_t N = G->N;
  for (int32_t r = 0; r < P; ++r) {
    w->qn[r] = 0; w->t_last[r] = 0; w->live[r] = 0; w->peak[r] = 0;
    w->last_kind[r] = -1; w->emitted[r] = 0;
  }
  for (int64_t o = 0; o < N; ++o) {
    w->acc[o] = 0;
    w->qpos[o] = -1;
    w->start[o] = w->end[o] = -1;
    w->left[o] = I->pred_ptr[o + 1] - I->pred_ptr[o];
  }
  for (int64_t o = 0; o < N; ++o)
    if (w->left[o] == 0) enqueue(I, G, w, (int32_t)o, 0);

  for (int64_t step = 0; step < N; ++step) {
    int32_t pick = -1, pick_r = -1;
    int64_t pick_t = 0;
    for (int use_cap = 1; use_cap >= 0 && pick < 0; --use_cap) {
      for (int32_t r = 0; r < P; ++r) {
        int64_t t;
        int32_t o = rank_choice(I, w, op_group, prio, r, use_cap, &t);
        if (o >= 0 && (pick < 0 || t < pick_t)) { pick = o; pick_r = r; pick_t = t; }
      }
    }
    if (pick < 0) return -4;                    /* cyclic data graph */
    int32_t r = pick_r, o = pick;
    dequeue(I, G, w, o);
    w->start[o] = pick_t;
    w->end[o] = pick_t + I->op_cost[o];
    if (w->end[o] > INT32_MAX) return -3;
    w->t_last[r] = w->end[o];
    w->last_kind[r] = I->op_kind[o];
    int64_t a = I->slot_act[I->op_slot[o]];
    if (I->op_kind[o] == 0) {
      w->live[r] += a;
      if (w->live[r] > w->peak[r]) w->peak[r] = w->live[r];
    } else {
      w->live[r] -= a;
    }
    order[I->rank_off[r] + w->emitted[r]] = (int16_t)(o - I->rank_off[r]);
    w->emitted[r] += 1;
    for (int32_t k = G->succ_ptr[o]; k < G->succ_ptr[o + 1]; ++k) {
      int32_t s = G->succ_op[k];
      int64_t t = w->end[o] + I->edge_comm[G->succ_edge[k]];
      if (t > w->acc[s]) w->acc[s] = t;
      if (--w->left[s] == 0) enqueue(I, G, w, s, w->acc[s]);
    }
  }

  int64_t T = 0;
  uint8_t f = 0;
  for (int64_t o = 0; o < N; ++o) if (w->end[o] > T) T = w->end[o];
  *makespan = (int32_t)T;
  for (int32_t r = 0; r < P; ++r) {
    int64_t busy = 0;
    for (int64_t o = I->rank_off[r]; o < I->rank_off[r + 1]; ++o) busy += I->op_cost[o];
    bubble[r] = (int32_t)(T - busy);
    if (w->peak[r] > INT32_MAX) return -3;
    peak[r] = (int32_t)w->peak[r];
    if (I->mem_cap[r] >= 0 && w->peak[r] > I->mem_cap[r]) f |= G_FLAG_CAP;
  }
  *flags = f;
  if (start_out)
    for (int64_t o = 0; o < N; ++o) { start_out[o] = (int32_t)w->start[o]; end_out[o] = (int32_t)w->end[o]; }
  return 0;
}

typedef struct {
  const dgr_instance *I;
  const dgr_graph *G;
  const int32_t *op_group, *prio;
  int32_t n_groups;
  int64_t stride, i0, i1;
  int16_t *orders;
  int32_t *makespan, *bubble, *peak;
  uint8_t *flags;
  int rc;
} dgr_job;

static void *dgr_run(void *arg) {
  dgr_job *j = (dgr_job *)arg;
  dgr_work w;
  int32_t P = j->I->n_ranks;
  if (work_alloc(&w, j->G->N, P) != 0) { j->rc = -2; work_release(&w); return NULL; }
  for (int64_t i = j->i0; i < j->i1; ++i) {
    int rc = greedy_one(j->I, j->G, &w, j->op_group, j->prio + i * j->n_groups,
                        j->orders + i * j->stride, &j->makespan[i], &j->bubble[i * P],
                        &j->peak[i * P], &j->flags[i], NULL, NULL);
    if (rc != 0) { j->rc = rc; break; }
  }
  work_release(&w);
  return NULL;
}

/* Interleave n_cand candidates (prio: [n_cand][n_groups]); candidate i's orders
 * go to orders[i * stride ...] (entries past N untouched).  Candidates are
 * independent, so n_threads threads take contiguous ranges.  Returns 0, -2
 * (out of memory), -3 (int32 overflow) or -4 (the data edges form a cycle). */
int dgr_greedy(const dgr_instance *I, const int32_t *op_group, int32_t n_groups,
               const int32_t *prio, int64_t n_cand, int64_t stride, int16_t *orders,
               int32_t *makespan, int32_t *bubble, int32_t *peak, uint8_t *flags,
               int32_t n_threads) {
  if (n_cand <= 0) return 0;
  dgr_graph G;
  if (graph_build(I, &G) != 0) { graph_release(&G); return -2; }
  if (n_threads < 1) n_threads = 1;
  if (n_threads > 256) n_threads = 256;
  if (n_cand < n_threads) n_threads = (int32_t)n_cand;
  pthread_t th[256];
  int created[256];
  dgr_job jobs[256];
  int64_t per = (n_cand + n_threads - 1) / n_threads;
  for (int32_t k = 0; k < n_threads; ++k) {
    dgr_job *j = &jobs[k];
    j->I = I; j->G = &G; j->op_group = op_group; j->prio = prio; j->n_groups = n_groups;
    j->stride = stride; j->orders = orders;
    j->i0 = k * per < n_cand ? k * per : n_cand;
    j->i1 = (k + 1) * per < n_cand ? (k + 1) * per : n_cand;
    j->makespan = makespan; j->bubble = bubble; j->peak = peak; j->flags = flags;
    j->rc = 0;
    created[k] = 0;
    if (j->i0 >= j->i1) continue;
    if (n_threads > 1 && pthread_create(&th[k], NULL, dgr_run, j) == 0) created[k] = 1;
    else dgr_run(j);
  }
  int rc = 0;
  for (int32_t k = 0; k < n_threads; ++k) {
    if (created[k]) pthread_join(th[k], NULL);
    if (jobs[k].rc != 0) rc = jobs[k].rc;
  }
  graph_release(&G);
  return rc;
}

/* One candidate with the greedy's own per-op start and end times. */
int dgr_greedy_timeline(const dgr_instance *I, const int32_t *op_group, const int32_t *prio,
                        int16_t *order, int32_t *makespan, int32_t *bubble, int32_t *peak,
                        uint8_t *flags, int32_t *start, int32_t *end) {
  dgr_graph G;
  dgr_work w;
  if (graph_build(I, &G) != 0) { graph_release(&G); return -2; }
  int rc = work_alloc(&w, G.N, I->n_ranks);
  if (rc == 0)
    rc = greedy_one(I, &G, &w, op_group, prio, order, makespan, bubble, peak, flags, start, end);
  work_release(&w);
  graph_release(&G);
  return rc;
}
