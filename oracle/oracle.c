/*
 * CPU oracle for the batched dataflow replay -- TEST INFRASTRUCTURE ONLY.
 * Only the tests and the benchmark's CPU-baseline leg load this library.
 *
 * It is a direct discrete-event simulation of the paper's simulation module
 * (Sec. 2, "Dataflow based simulation"), one scenario at a time, with no
 * blocking, fusion or reordering beyond what that loop states.  The global
 * ready list is a binary min-heap of ops whose dependency counters reached
 * zero, keyed by (ready time, priority, op id).  Popping it in key order
 * serves every device's queue first-in-first-out by ready time: an op that
 * becomes ready when its last predecessor finishes at time t is pushed with
 * key t, strictly later than the key just popped because durations are at
 * least 1 ns, so pops come out in nondecreasing key order, and everything
 * that finishes at t is on the heap before the first op keyed t is popped.
 * A popped op starts when both it is ready and its device has finished the
 * previous op (the device's "finish time"), and the iteration time is the
 * largest finish time of any device.
 *
 * The critical path (longest path, devices ignored) is a plain topological
 * sweep; it is the iteration time with unlimited devices (Sec. 1: finding the
 * performance bottleneck).
 */
#include "oracle.h"

#include <pthread.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int32_t n, nres;
  const int64_t *sp;
  const int32_t *si;
  const int32_t *res;
  const int32_t *prio;
  int32_t *indeg; /* number of incoming edge occurrences */
} graph_t;

/* Kahn's algorithm on the edge multiset: returns 1 if every op is ordered. */
static int topo_order(const graph_t *g, int32_t *order) {
  int32_t *cnt = (int32_t *)malloc(sizeof(int32_t) * (size_t)(g->n ? g->n : 1));
  if (!cnt) return -1;
  memcpy(cnt, g->indeg, sizeof(int32_t) * (size_t)g->n);
  int32_t head = 0, tail = 0;
  for (int32_t v = 0; v < g->n; ++v)
    if (cnt[v] == 0) order[tail++] = v;
  while (head < tail) {
    int32_t v = order[head++];
    for (int64_t e = g->sp[v]; e < g->sp[v + 1]; ++e)
      if (--cnt[g->si[e]] == 0) order[tail++] = g->si[e];
  }
  free(cnt);
  return tail == g->n;
}

static int check_graph(graph_t *g, int need_res) {
  if (g->n < 0 || (g->n > 0 && (!g->sp || (need_res && (!g->res || g->nres < 1)))))
    return ORC_E_INVAL;
  if (g->n == 0) return ORC_OK;
  if (g->sp[0] != 0) return ORC_E_INVAL;
  for (int32_t v = 0; v < g->n; ++v)
    if (g->sp[v + 1] < g->sp[v]) return ORC_E_INVAL;
  if (g->sp[g->n] > 0 && !g->si) return ORC_E_INVAL;
  for (int64_t e = 0; e < g->sp[g->n]; ++e)
    if (g->si[e] < 0 || g->si[e] >= g->n) return ORC_E_RANGE;
  if (need_res)
    for (int32_t v = 0; v < g->n; ++v)
      if (g->res[v] < 0 || g->res[v] >= g->nres) return ORC_E_RANGE;
  return ORC_OK;
}

static int build_indeg(graph_t *g) {
  g->indeg = (int32_t *)calloc((size_t)(g->n ? g->n : 1), sizeof(int32_t));
  if (!g->indeg) return ORC_E_NOMEM;
  for (int64_t e = 0; e < (g->n ? g->sp[g->n] : 0); ++e) g->indeg[g->si[e]]++;
  return ORC_OK;
}

/* ---------------------------------------------------------------- replay */

typedef struct {
  int64_t *ready; /* [n] ready time of each op (max finish of its predecessors) */
  int32_t *cnt;   /* [n] predecessors not yet finished */
  int64_t *fin;   /* [n] finish time */
  int64_t *rfree; /* [nres] time each device finishes its last op */
  int32_t *heap;  /* [n] the ready list */
  int32_t hsize;
  int32_t *prev;  /* [n] or NULL: the op that ran before each op on its device (-1: none) */
  int32_t *last;  /* [nres] with prev: the last op each device ran */
  int32_t *nrun;  /* [nres] with gaps: ops each device has run */
} sim_ws;

/* key order of the ready list: ready time, then priority, then op id */
static int key_less(const graph_t *g, const sim_ws *w, int32_t a, int32_t b) {
  if (w->ready[a] != w->ready[b]) return w->ready[a] < w->ready[b];
  int32_t pa = g->prio ? g->prio[a] : a, pb = g->prio ? g->prio[b] : b;
  if (pa != pb) return pa < pb;
  return a < b;
}

static void heap_push(const graph_t *g, sim_ws *w, int32_t v) {
  int32_t i = w->hsize++;
  w->heap[i] = v;
  while (i > 0) {
    int32_t p = (i - 1) / 2;
    if (!key_less(g, w, w->heap[i], w->heap[p])) break;
    int32_t t = w->heap[i];
    w->heap[i] = w->heap[p];
    w->heap[p] = t;
    i = p;
  }
}

static int32_t heap_pop(const graph_t *g, sim_ws *w) {
  int32_t top = w->heap[0];
  w->heap[0] = w->heap[--w->hsize];
  int32_t i = 0;
  for (;;) {
    int32_t l = 2 * i + 1, r = l + 1, m = i;
    if (l < w->hsize && key_less(g, w, w->heap[l], w->heap[m])) m = l;
    if (r < w->hsize && key_less(g, w, w->heap[r], w->heap[m])) m = r;
    if (m == i) break;
    int32_t t = w->heap[i];
    w->heap[i] = w->heap[m];
    w->heap[m] = t;
    i = m;
  }
  return top;
}

typedef struct {
  const graph_t *g;
  int64_t s0, s1;
  const int32_t *dur;
  int64_t ld_dur;
  const uint16_t *place;
  int64_t ld_place;
  int32_t *makespan, *finish, *status;
  int64_t ld_fin;
  int rc;
  const int32_t *gap; /* [nres] or NULL: a device's idle time between consecutive ops */
  const int32_t *delay; /* [nres] or NULL: time after an op finishes until its outputs reach its successors */
} run_job;

static void replay_one(const run_job *J, sim_ws *w, int64_t s) {
  const graph_t *g = J->g;
  int32_t st = 0;
  /* per-scenario input checks */
  for (int32_t v = 0; v < g->n; ++v) {
    if (J->dur[(int64_t)v * J->ld_dur + s] < 1) st |= ORC_ST_BAD_DUR;
    if (J->place && J->place[(int64_t)v * J->ld_place + s] >= (uint32_t)g->nres) st |= ORC_ST_BAD_RES;
  }
  int64_t span = 0;
  if (!st) {
    for (int32_t v = 0; v < g->n; ++v) {
      w->ready[v] = 0;
      w->cnt[v] = g->indeg[v];
    }
    for (int32_t r = 0; r < g->nres; ++r) w->rfree[r] = 0;
    if (w->prev)
      for (int32_t r = 0; r < g->nres; ++r) w->last[r] = -1;
    if (J->gap)
      for (int32_t r = 0; r < g->nres; ++r) w->nrun[r] = 0;
    w->hsize = 0;
    /* (1) every op with no predecessors is ready at t = 0 */
    for (int32_t v = 0; v < g->n; ++v)
      if (w->cnt[v] == 0) heap_push(g, w, v);
    while (w->hsize > 0) {
      int32_t v = heap_pop(g, w);
      int32_t r = J->place ? (int32_t)J->place[(int64_t)v * J->ld_place + s] : g->res[v];
      /* the device can start again when its last op has finished and, with
       * gaps, its gap after that op has passed */
      int64_t avail = w->rfree[r];
      if (J->gap && w->nrun[r] > 0) avail += J->gap[r];
      int64_t start = w->ready[v] > avail ? w->ready[v] : avail;
      int64_t f = start + J->dur[(int64_t)v * J->ld_dur + s];
      if (f > INT32_MAX) {
        st |= ORC_ST_OVERFLOW;
        break;
      }
      w->fin[v] = f;
      w->rfree[r] = f;
      if (J->gap) w->nrun[r]++;
      if (w->prev) {
        w->prev[v] = w->last[r];
        w->last[r] = v;
      }
      /* (2) the finished op updates its successors' dependency counters; its
       * outputs reach them at f, or with delays f + delay[r] */
      const int64_t out = J->delay ? f + J->delay[r] : f;
      for (int64_t e = g->sp[v]; e < g->sp[v + 1]; ++e) {
        int32_t x = g->si[e];
        if (out > w->ready[x]) w->ready[x] = out;
        if (--w->cnt[x] == 0) heap_push(g, w, x);
      }
    }
    if (!st) /* the finish time of the last device */
      for (int32_t r = 0; r < g->nres; ++r)
        if (w->rfree[r] > span) span = w->rfree[r];
  }
  if (J->status) J->status[s] = st;
  J->makespan[s] = st ? -1 : (int32_t)span;
  if (J->finish && !st)
    for (int32_t v = 0; v < g->n; ++v) J->finish[(int64_t)v * J->ld_fin + s] = (int32_t)w->fin[v];
}

static void *run_range(void *arg) {
  run_job *J = (run_job *)arg;
  const graph_t *g = J->g;
  size_t n = (size_t)(g->n ? g->n : 1), R = (size_t)g->nres;
  sim_ws w;
  w.ready = (int64_t *)malloc(n * sizeof(int64_t));
  w.cnt = (int32_t *)malloc(n * sizeof(int32_t));
  w.fin = (int64_t *)malloc(n * sizeof(int64_t));
  w.rfree = (int64_t *)malloc((R ? R : 1) * sizeof(int64_t));
  w.heap = (int32_t *)malloc(n * sizeof(int32_t));
  w.prev = w.last = NULL;
  w.nrun = (int32_t *)malloc((R ? R : 1) * sizeof(int32_t));
  if (!w.ready || !w.cnt || !w.fin || !w.rfree || !w.heap || !w.nrun) {
    J->rc = ORC_E_NOMEM;
  } else {
    for (int64_t s = J->s0; s < J->s1; ++s) replay_one(J, &w, s);
  }
  free(w.ready);
  free(w.cnt);
  free(w.fin);
  free(w.rfree);
  free(w.heap);
  free(w.nrun);
  return NULL;
}

static int run_threads(void *(*fn)(void *), void *jobs, size_t job_size, int64_t n_scen,
                       int32_t n_threads, void (*set_range)(void *, int64_t, int64_t)) {
  if (n_threads < 1) n_threads = 1;
  if (n_scen < n_threads) n_threads = (int32_t)(n_scen > 0 ? n_scen : 1);
  pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)n_threads);
  if (!th) return ORC_E_NOMEM;
  for (int32_t t = 0; t < n_threads; ++t) {
    void *job = (char *)jobs + job_size * (size_t)t;
    set_range(job, n_scen * t / n_threads, n_scen * (t + 1) / n_threads);
  }
  int32_t started = 0;
  for (int32_t t = 1; t < n_threads; ++t) {
    if (pthread_create(&th[t], NULL, fn, (char *)jobs + job_size * (size_t)t) != 0) break;
    started = t;
  }
  fn(jobs);
  for (int32_t t = 1; t <= started; ++t) pthread_join(th[t], NULL);
  /* threads that could not be started run here */
  for (int32_t t = started + 1; t < n_threads; ++t) fn((char *)jobs + job_size * (size_t)t);
  free(th);
  return ORC_OK;
}

static void set_run_range(void *p, int64_t a, int64_t b) {
  ((run_job *)p)->s0 = a;
  ((run_job *)p)->s1 = b;
}

int oracle_run_batch(int32_t n_ops, int32_t n_res, const int64_t *succ_ptr,
                     const int32_t *succ_idx, const int32_t *op_res, const int32_t *prio,
                     int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                     const uint16_t *place, int64_t ld_place, int32_t *makespan,
                     int32_t *finish, int64_t ld_fin, int32_t *status, int32_t n_threads) {
  return oracle_run_batch_dev(n_ops, n_res, succ_ptr, succ_idx, op_res, prio, NULL, NULL, n_scen, dur,
                              ld_dur, place, ld_place, makespan, finish, ld_fin, status, n_threads);
}

int oracle_run_batch_gap(int32_t n_ops, int32_t n_res, const int64_t *succ_ptr,
                         const int32_t *succ_idx, const int32_t *op_res, const int32_t *prio,
                         const int32_t *gap, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                         const uint16_t *place, int64_t ld_place, int32_t *makespan,
                         int32_t *finish, int64_t ld_fin, int32_t *status, int32_t n_threads) {
  return oracle_run_batch_dev(n_ops, n_res, succ_ptr, succ_idx, op_res, prio, gap, NULL, n_scen, dur,
                              ld_dur, place, ld_place, makespan, finish, ld_fin, status, n_threads);
}

int oracle_run_batch_dev(int32_t n_ops, int32_t n_res, const int64_t *succ_ptr,
                         const int32_t *succ_idx, const int32_t *op_res, const int32_t *prio,
                         const int32_t *gap, const int32_t *delay, int64_t n_scen, const int32_t *dur,
                         int64_t ld_dur, const uint16_t *place, int64_t ld_place, int32_t *makespan,
                         int32_t *finish, int64_t ld_fin, int32_t *status, int32_t n_threads) {
  graph_t g = {n_ops, n_res, succ_ptr, succ_idx, op_res, prio, NULL};
  int rc = check_graph(&g, 1);
  if (rc) return rc;
  for (int32_t r = 0; r < n_res; ++r)
    if ((gap && gap[r] < 0) || (delay && delay[r] < 0)) return ORC_E_INVAL;
  if (n_scen < 0 || (n_scen > 0 && !makespan)) return ORC_E_INVAL;
  if (n_scen > 0 && n_ops > 0) {
    if (!dur || ld_dur < n_scen) return ORC_E_INVAL;
    if (place && ld_place < n_scen) return ORC_E_INVAL;
    if (finish && ld_fin < n_scen) return ORC_E_INVAL;
  }
  if ((rc = build_indeg(&g))) return rc;
  int32_t *order = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n_ops ? n_ops : 1));
  if (!order) {
    free(g.indeg);
    return ORC_E_NOMEM;
  }
  int acyclic = topo_order(&g, order);
  free(order);
  if (acyclic != 1) {
    free(g.indeg);
    return acyclic < 0 ? ORC_E_NOMEM : ORC_E_CYCLE;
  }
  if (n_threads < 1) n_threads = 1;
  run_job *jobs = (run_job *)calloc((size_t)n_threads, sizeof(run_job));
  if (!jobs) {
    free(g.indeg);
    return ORC_E_NOMEM;
  }
  for (int32_t t = 0; t < n_threads; ++t) {
    run_job J = {&g, 0, 0, dur, ld_dur, place, ld_place, makespan, finish, status, ld_fin, 0, gap, delay};
    jobs[t] = J;
  }
  rc = run_threads(run_range, jobs, sizeof(run_job), n_scen, n_threads, set_run_range);
  for (int32_t t = 0; t < n_threads && !rc; ++t) rc = jobs[t].rc;
  free(jobs);
  free(g.indeg);
  return rc;
}

/* ------------------------------------------------- bandwidth sharing */

typedef struct {
  const graph_t *g;
  int64_t s0, s1;
  const int32_t *dur;
  int64_t ld_dur;
  int32_t *makespan, *finish, *status;
  int64_t ld_fin;
  int rc;
  const uint8_t *share;
} share_job;

/* one shared device: the service units each active op has received since
 * time 0 (vt, as of time tl), and its active ops with the units at which
 * each is done */
typedef struct {
  uint64_t vt;
  int64_t tl;
  int32_t k;
  int32_t op[ORC_SHARE_MAX];
  uint64_t need[ORC_SHARE_MAX];
} link_t;

/* bring the device's service count to time t (k constant since tl) */
static void link_advance(link_t *L, int64_t t) {
  if (L->k > 0) L->vt += (uint64_t)(t - L->tl) * (ORC_SHARE_UNIT / (uint64_t)L->k);
  L->tl = t;
}

/* the first integer ns at which the device's next op is done (k > 0) */
static int64_t link_next(const link_t *L) {
  uint64_t m = L->need[0];
  for (int32_t i = 1; i < L->k; ++i)
    if (L->need[i] < m) m = L->need[i];
  const uint64_t per_ns = ORC_SHARE_UNIT / (uint64_t)L->k;
  return L->tl + (int64_t)((m - L->vt + per_ns - 1) / per_ns);
}

static void release_succ(const graph_t *g, sim_ws *w, int32_t v, int64_t t) {
  for (int64_t e = g->sp[v]; e < g->sp[v + 1]; ++e) {
    int32_t x = g->si[e];
    if (t > w->ready[x]) w->ready[x] = t;
    w->cnt[x] -= 1;
    if (w->cnt[x] == 0) heap_push(g, w, x);
  }
}

static void share_one(share_job *J, sim_ws *w, link_t *links, int64_t s) {
  const graph_t *g = J->g;
  int32_t st = 0;
  for (int32_t v = 0; v < g->n; ++v) {
    const int32_t dv = J->dur[(int64_t)v * J->ld_dur + s];
    if (dv < 1) st |= ORC_ST_BAD_DUR;
  }
  int64_t span = 0;
  if (!st) {
    for (int32_t v = 0; v < g->n; ++v) {
      w->ready[v] = 0;
      w->cnt[v] = g->indeg[v];
    }
    for (int32_t r = 0; r < g->nres; ++r) {
      w->rfree[r] = 0;
      links[r].vt = links[r].tl = 0;
      links[r].k = 0;
    }
    w->hsize = 0;
    for (int32_t v = 0; v < g->n; ++v)
      if (w->cnt[v] == 0) heap_push(g, w, v);
    for (;;) {
      /* the earliest finish on a shared device (lowest device on ties) */
      int32_t lr = -1;
      int64_t lt = 0;
      for (int32_t r = 0; r < g->nres; ++r)
        if (J->share[r] && links[r].k > 0) {
          int64_t t = link_next(&links[r]);
          if (lr < 0 || t < lt) {
            lr = r;
            lt = t;
          }
        }
      if (lr >= 0 && (w->hsize == 0 || lt <= w->ready[w->heap[0]])) {
        if (lt > INT32_MAX) {
          st |= ORC_ST_OVERFLOW;
          break;
        }
        link_t *L = &links[lr];
        link_advance(L, lt);
        /* every active op that has its units leaves at lt */
        for (int32_t i = 0; i < L->k;) {
          if (L->need[i] <= L->vt) {
            int32_t v = L->op[i];
            w->fin[v] = lt;
            if (lt > span) span = lt;
            L->op[i] = L->op[L->k - 1];
            L->need[i] = L->need[L->k - 1];
            L->k--;
            release_succ(g, w, v, lt);
          } else {
            ++i;
          }
        }
        continue;
      }
      if (w->hsize == 0) break;
      int32_t v = heap_pop(g, w);
      int32_t r = g->res[v];
      int64_t d = J->dur[(int64_t)v * J->ld_dur + s];
      if (J->share[r]) {
        /* joins the device's active ops at its ready time */
        link_t *L = &links[r];
        if (L->k == ORC_SHARE_MAX) {
          st |= ORC_ST_SHARE_LIMIT;
          break;
        }
        link_advance(L, w->ready[v]);
        L->op[L->k] = v;
        L->need[L->k] = L->vt + (uint64_t)d * ORC_SHARE_UNIT;
        L->k++;
        continue;
      }
      int64_t start = w->ready[v] > w->rfree[r] ? w->ready[v] : w->rfree[r];
      int64_t f = start + d;
      if (f > (int64_t)INT32_MAX) {
        st |= ORC_ST_OVERFLOW;
        break;
      }
      w->fin[v] = f;
      w->rfree[r] = f;
      if (f > span) span = f;
      release_succ(g, w, v, f);
    }
  }
  if (J->status) J->status[s] = st;
  J->makespan[s] = st ? -1 : (int32_t)span;
  if (J->finish && !st)
    for (int32_t v = 0; v < g->n; ++v) J->finish[(int64_t)v * J->ld_fin + s] = (int32_t)w->fin[v];
}

static void *share_range(void *arg) {
  share_job *J = (share_job *)arg;
  const graph_t *g = J->g;
  size_t n = (size_t)(g->n ? g->n : 1), R = (size_t)(g->nres ? g->nres : 1);
  sim_ws w;
  memset(&w, 0, sizeof(w));
  w.ready = (int64_t *)malloc(n * sizeof(int64_t));
  w.cnt = (int32_t *)malloc(n * sizeof(int32_t));
  w.fin = (int64_t *)malloc(n * sizeof(int64_t));
  w.rfree = (int64_t *)malloc(R * sizeof(int64_t));
  w.heap = (int32_t *)malloc(n * sizeof(int32_t));
  link_t *links = (link_t *)malloc(R * sizeof(link_t));
  if (!w.ready || !w.cnt || !w.fin || !w.rfree || !w.heap || !links) {
    J->rc = ORC_E_NOMEM;
  } else {
    for (int64_t s = J->s0; s < J->s1; ++s) share_one(J, &w, links, s);
  }
  free(w.ready);
  free(w.cnt);
  free(w.fin);
  free(w.rfree);
  free(w.heap);
  free(links);
  return NULL;
}

static void set_share_range(void *p, int64_t a, int64_t b) {
  ((share_job *)p)->s0 = a;
  ((share_job *)p)->s1 = b;
}

int oracle_run_batch_share(int32_t n_ops, int32_t n_res, const int64_t *succ_ptr,
                           const int32_t *succ_idx, const int32_t *op_res, const int32_t *prio,
                           const uint8_t *share, int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                           int32_t *makespan, int32_t *finish, int64_t ld_fin, int32_t *status,
                           int32_t n_threads) {
  graph_t g = {n_ops, n_res, succ_ptr, succ_idx, op_res, prio, NULL};
  int rc = check_graph(&g, 1);
  if (rc) return rc;
  if (n_scen < 0 || (n_scen > 0 && !makespan)) return ORC_E_INVAL;
  if (n_scen > 0 && n_ops > 0) {
    if (!dur || ld_dur < n_scen) return ORC_E_INVAL;
    if (finish && ld_fin < n_scen) return ORC_E_INVAL;
  }
  uint8_t *sh = (uint8_t *)calloc((size_t)(n_res > 0 ? n_res : 1), 1);
  if (!sh) return ORC_E_NOMEM;
  for (int32_t r = 0; r < n_res; ++r) sh[r] = share ? share[r] != 0 : 0;
  if ((rc = build_indeg(&g))) {
    free(sh);
    return rc;
  }
  int32_t *order = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n_ops ? n_ops : 1));
  int acyclic = order ? topo_order(&g, order) : -1;
  free(order);
  if (acyclic != 1) {
    free(g.indeg);
    free(sh);
    return acyclic < 0 ? ORC_E_NOMEM : ORC_E_CYCLE;
  }
  if (n_threads < 1) n_threads = 1;
  share_job *jobs = (share_job *)calloc((size_t)n_threads, sizeof(share_job));
  if (!jobs) {
    free(g.indeg);
    free(sh);
    return ORC_E_NOMEM;
  }
  for (int32_t t = 0; t < n_threads; ++t) {
    share_job J = {&g, 0, 0, dur, ld_dur, makespan, finish, status, ld_fin, 0, sh};
    jobs[t] = J;
  }
  rc = run_threads(share_range, jobs, sizeof(share_job), n_scen, n_threads, set_share_range);
  for (int32_t t = 0; t < n_threads && !rc; ++t) rc = jobs[t].rc;
  free(jobs);
  free(g.indeg);
  free(sh);
  return rc;
}

/* --------------------------------------------------------- critical path */

typedef struct {
  const graph_t *g;
  const int32_t *order;
  int64_t s0, s1;
  const int32_t *dur;
  int64_t ld_dur;
  int32_t *cp_len;
  int rc;
} cp_job;

/* dist(v) = d(v) + max over predecessors of dist, in topological order.
 * Returns 0 on success, 1 on a bad duration or a path above INT32_MAX. */
static int longest_paths(const graph_t *g, const int32_t *order, const int32_t *dur,
                         int64_t ld_dur, int64_t s, int64_t *best, int64_t *dist) {
  for (int32_t v = 0; v < g->n; ++v) best[v] = 0;
  for (int32_t k = 0; k < g->n; ++k) {
    int32_t v = order[k];
    int32_t d = dur[(int64_t)v * ld_dur + s];
    if (d < 1) return 1;
    dist[v] = best[v] + d;
    if (dist[v] > INT32_MAX) return 1;
    for (int64_t e = g->sp[v]; e < g->sp[v + 1]; ++e)
      if (dist[v] > best[g->si[e]]) best[g->si[e]] = dist[v];
  }
  return 0;
}

static void *cp_range(void *arg) {
  cp_job *J = (cp_job *)arg;
  size_t n = (size_t)(J->g->n ? J->g->n : 1);
  int64_t *best = (int64_t *)malloc(n * sizeof(int64_t));
  int64_t *dist = (int64_t *)malloc(n * sizeof(int64_t));
  if (!best || !dist) {
    J->rc = ORC_E_NOMEM;
  } else {
    for (int64_t s = J->s0; s < J->s1; ++s) {
      if (longest_paths(J->g, J->order, J->dur, J->ld_dur, s, best, dist)) {
        J->cp_len[s] = -1;
        continue;
      }
      int64_t m = 0;
      for (int32_t v = 0; v < J->g->n; ++v)
        if (dist[v] > m) m = dist[v];
      J->cp_len[s] = (int32_t)m;
    }
  }
  free(best);
  free(dist);
  return NULL;
}

static void set_cp_range(void *p, int64_t a, int64_t b) {
  ((cp_job *)p)->s0 = a;
  ((cp_job *)p)->s1 = b;
}

int oracle_critical_path(int32_t n_ops, const int64_t *succ_ptr, const int32_t *succ_idx,
                         int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                         int32_t *cp_len, int64_t path_scen, int32_t *path_ops,
                         int32_t path_cap, int32_t *path_len, int32_t n_threads) {
  graph_t g = {n_ops, 1, succ_ptr, succ_idx, NULL, NULL, NULL};
  int rc = check_graph(&g, 0);
  if (rc) return rc;
  if (n_scen < 0 || (n_scen > 0 && !cp_len)) return ORC_E_INVAL;
  if (n_scen > 0 && n_ops > 0 && (!dur || ld_dur < n_scen)) return ORC_E_INVAL;
  if (path_scen >= n_scen || (path_scen >= 0 && (!path_len || (path_cap > 0 && !path_ops))))
    return ORC_E_INVAL;
  if ((rc = build_indeg(&g))) return rc;
  int32_t *order = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n_ops ? n_ops : 1));
  if (!order) {
    free(g.indeg);
    return ORC_E_NOMEM;
  }
  int acyclic = topo_order(&g, order);
  if (acyclic != 1) {
    free(order);
    free(g.indeg);
    return acyclic < 0 ? ORC_E_NOMEM : ORC_E_CYCLE;
  }
  if (n_threads < 1) n_threads = 1;
  cp_job *jobs = (cp_job *)calloc((size_t)n_threads, sizeof(cp_job));
  if (!jobs) rc = ORC_E_NOMEM;
  for (int32_t t = 0; t < n_threads && !rc; ++t) {
    cp_job J = {&g, order, 0, 0, dur, ld_dur, cp_len, 0};
    jobs[t] = J;
  }
  if (!rc) rc = run_threads(cp_range, jobs, sizeof(cp_job), n_scen, n_threads, set_cp_range);
  for (int32_t t = 0; t < n_threads && !rc; ++t) rc = jobs[t].rc;
  free(jobs);

  if (!rc && path_scen >= 0) {
    size_t n = (size_t)(n_ops ? n_ops : 1);
    int64_t *best = (int64_t *)malloc(n * sizeof(int64_t));
    int64_t *dist = (int64_t *)malloc(n * sizeof(int64_t));
    int32_t *pred_ptr = (int32_t *)calloc(n + 1, sizeof(int32_t));
    int32_t *pred_idx = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n_ops ? succ_ptr[n_ops] + 1 : 1));
    int32_t *rev = (int32_t *)malloc(n * sizeof(int32_t));
    if (!best || !dist || !pred_ptr || !pred_idx || !rev) {
      rc = ORC_E_NOMEM;
    } else if (n_ops == 0 || longest_paths(&g, order, dur, ld_dur, path_scen, best, dist)) {
      *path_len = 0;
    } else {
      /* predecessor lists, for stepping back */
      for (int32_t v = 0; v < n_ops; ++v) pred_ptr[v + 1] = g.indeg[v];
      for (int32_t v = 0; v < n_ops; ++v) pred_ptr[v + 1] += pred_ptr[v];
      int32_t *fill = rev; /* reuse as a cursor array first */
      for (int32_t v = 0; v < n_ops; ++v) fill[v] = pred_ptr[v];
      for (int32_t u = 0; u < n_ops; ++u)
        for (int64_t e = succ_ptr[u]; e < succ_ptr[u + 1]; ++e) pred_idx[fill[succ_idx[e]]++] = u;
      int32_t v = 0;
      for (int32_t x = 1; x < n_ops; ++x)
        if (dist[x] > dist[v]) v = x;
      int32_t len = 0;
      for (;;) {
        rev[len++] = v;
        int64_t want = dist[v] - dur[(int64_t)v * ld_dur + path_scen];
        if (want == 0) break;
        int32_t nxt = -1;
        for (int32_t k = pred_ptr[v]; k < pred_ptr[v + 1]; ++k) {
          int32_t p = pred_idx[k];
          if (dist[p] == want && (nxt < 0 || p < nxt)) nxt = p;
        }
        v = nxt;
        if (v < 0) break; /* cannot happen: some predecessor lies on a longest path */
      }
      *path_len = len;
      for (int32_t k = 0; k < len && k < path_cap; ++k) path_ops[k] = rev[len - 1 - k];
    }
    free(best);
    free(dist);
    free(pred_ptr);
    free(pred_idx);
    free(rev);
  }
  free(order);
  free(g.indeg);
  return rc;
}

/* ------------------------------------------------- static-order replay */

/*
 * Each device runs its ops in one fixed order: the order in which they appear
 * in a given permutation of all ops (Sec. 2 describes each device's queue;
 * here the queue order is fixed in advance instead of by arrival).  An op
 * starts when every predecessor and the op before it on its device have
 * finished, so finish(v) = d(v) + max(finish of predecessors, finish of the
 * previous op on the device).  The ops are visited in a topological order of
 * the DAG together with the device-order edges.
 */
typedef struct {
  const graph_t *g;
  const int32_t *topo, *next_on_dev;
  int64_t s0, s1;
  const int32_t *dur;
  int64_t ld_dur;
  int32_t *makespan, *finish, *status;
  int64_t ld_fin;
  int rc;
} st_job;

static void static_one(const st_job *J, int64_t *ready, int64_t *fin, int64_t s) {
  const graph_t *g = J->g;
  int32_t st = 0;
  for (int32_t v = 0; v < g->n; ++v)
    if (J->dur[(int64_t)v * J->ld_dur + s] < 1) st = ORC_ST_BAD_DUR;
  int64_t span = 0;
  if (!st) {
    for (int32_t v = 0; v < g->n; ++v) ready[v] = 0;
    for (int32_t k = 0; k < g->n; ++k) {
      int32_t v = J->topo[k];
      fin[v] = ready[v] + J->dur[(int64_t)v * J->ld_dur + s];
      if (fin[v] > INT32_MAX) {
        st = ORC_ST_OVERFLOW;
        break;
      }
      if (fin[v] > span) span = fin[v];
      for (int64_t e = g->sp[v]; e < g->sp[v + 1]; ++e)
        if (fin[v] > ready[g->si[e]]) ready[g->si[e]] = fin[v];
      int32_t nx = J->next_on_dev[v];
      if (nx >= 0 && fin[v] > ready[nx]) ready[nx] = fin[v];
    }
  }
  if (J->status) J->status[s] = st;
  J->makespan[s] = st ? -1 : (int32_t)span;
  if (J->finish && !st)
    for (int32_t v = 0; v < g->n; ++v) J->finish[(int64_t)v * J->ld_fin + s] = (int32_t)fin[v];
}

static void *static_range(void *arg) {
  st_job *J = (st_job *)arg;
  size_t n = (size_t)(J->g->n ? J->g->n : 1);
  int64_t *ready = (int64_t *)malloc(n * sizeof(int64_t));
  int64_t *fin = (int64_t *)malloc(n * sizeof(int64_t));
  if (!ready || !fin)
    J->rc = ORC_E_NOMEM;
  else
    for (int64_t s = J->s0; s < J->s1; ++s) static_one(J, ready, fin, s);
  free(ready);
  free(fin);
  return NULL;
}

static void set_static_range(void *p, int64_t a, int64_t b) {
  ((st_job *)p)->s0 = a;
  ((st_job *)p)->s1 = b;
}

int oracle_static_run(int32_t n_ops, int32_t n_res, const int64_t *succ_ptr,
                      const int32_t *succ_idx, const int32_t *op_res, const int32_t *order,
                      int64_t n_scen, const int32_t *dur, int64_t ld_dur, int32_t *makespan,
                      int32_t *finish, int64_t ld_fin, int32_t *status, int32_t n_threads) {
  graph_t g = {n_ops, n_res, succ_ptr, succ_idx, op_res, NULL, NULL};
  int rc = check_graph(&g, 1);
  if (rc) return rc;
  if (n_ops > 0 && !order) return ORC_E_INVAL;
  if (n_scen < 0 || (n_scen > 0 && !makespan)) return ORC_E_INVAL;
  if (n_scen > 0 && n_ops > 0 && (!dur || ld_dur < n_scen || (finish && ld_fin < n_scen)))
    return ORC_E_INVAL;
  size_t n = (size_t)(n_ops ? n_ops : 1);
  int32_t *seen = (int32_t *)calloc(n, sizeof(int32_t));
  int32_t *next_on_dev = (int32_t *)malloc(n * sizeof(int32_t));
  int32_t *last_on_dev = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n_res > 0 ? n_res : 1));
  int32_t *cnt = (int32_t *)calloc(n, sizeof(int32_t));
  int32_t *topo = (int32_t *)malloc(n * sizeof(int32_t));
  if (!seen || !next_on_dev || !last_on_dev || !cnt || !topo) rc = ORC_E_NOMEM;
  /* the order must name every op exactly once */
  for (int32_t k = 0; k < n_ops && !rc; ++k) {
    int32_t v = order[k];
    if (v < 0 || v >= n_ops || seen[v]) rc = ORC_E_INVAL;
    else seen[v] = 1;
  }
  if (!rc) {
    /* device-order edges: each op to the next op on its device */
    for (int32_t r = 0; r < n_res; ++r) last_on_dev[r] = -1;
    for (int32_t v = 0; v < n_ops; ++v) next_on_dev[v] = -1;
    for (int32_t k = 0; k < n_ops; ++k) {
      int32_t v = order[k], r = op_res[v];
      if (last_on_dev[r] >= 0) next_on_dev[last_on_dev[r]] = v;
      last_on_dev[r] = v;
    }
    /* Kahn over DAG edges (with repeats) plus device-order edges */
    for (int32_t u = 0; u < n_ops; ++u) {
      for (int64_t e = succ_ptr[u]; e < succ_ptr[u + 1]; ++e) cnt[succ_idx[e]]++;
      if (next_on_dev[u] >= 0) cnt[next_on_dev[u]]++;
    }
    int32_t head = 0, tail = 0;
    for (int32_t v = 0; v < n_ops; ++v)
      if (cnt[v] == 0) topo[tail++] = v;
    while (head < tail) {
      int32_t v = topo[head++];
      for (int64_t e = succ_ptr[v]; e < succ_ptr[v + 1]; ++e)
        if (--cnt[succ_idx[e]] == 0) topo[tail++] = succ_idx[e];
      if (next_on_dev[v] >= 0 && --cnt[next_on_dev[v]] == 0) topo[tail++] = next_on_dev[v];
    }
    if (tail != n_ops) rc = ORC_E_CYCLE; /* the device orders contradict the dependencies */
  }
  if (!rc && n_scen > 0) {
    if (n_threads < 1) n_threads = 1;
    st_job *jobs = (st_job *)calloc((size_t)n_threads, sizeof(st_job));
    if (!jobs) {
      rc = ORC_E_NOMEM;
    } else {
      for (int32_t t = 0; t < n_threads; ++t) {
        st_job J = {&g, topo, next_on_dev, 0, 0, dur, ld_dur, makespan, finish, status, ld_fin, 0};
        jobs[t] = J;
      }
      rc = run_threads(static_range, jobs, sizeof(st_job), n_scen, n_threads, set_static_range);
      for (int32_t t = 0; t < n_threads && !rc; ++t) rc = jobs[t].rc;
      free(jobs);
    }
  }
  free(seen);
  free(next_on_dev);
  free(last_on_dev);
  free(cnt);
  free(topo);
  return rc;
}


/* ------------------------------------------------ bottleneck attribution */

/*
 * Where the iteration time goes (Sec. 1: finding the performance
 * bottleneck).  After the replay of a scenario, the binding chain starts at
 * the op that finishes last (lowest id among equals) and walks back: an op
 * that starts at t > 0 started then either because a predecessor finished at
 * t (the chain steps to the lowest-id such predecessor) or because its device
 * finished the op before it at t (the chain steps to that op); it ends at an
 * op that starts at 0.  The chain has no gaps, so its durations sum to the
 * makespan; chain[r] is the part spent on device r.  busy[r] is the total
 * duration of the ops device r ran.
 */
typedef struct {
  run_job run;
  const int32_t *pred_ptr, *pred_idx;
  int32_t *busy, *chain, *chain_ops;
  int64_t ld_res, path_scen;
  int32_t *path_ops, path_cap, *path_len;
} at_job;

static int32_t device_of(const run_job *J, int32_t v, int64_t s) {
  return J->place ? (int32_t)J->place[(int64_t)v * J->ld_place + s] : J->g->res[v];
}

static void attribute_one(const at_job *A, sim_ws *w, int32_t *rev, int64_t s) {
  const run_job *J = &A->run;
  const graph_t *g = J->g;
  replay_one(J, w, s);
  int32_t st = J->status[s];
  for (int32_t r = 0; r < g->nres; ++r) {
    A->busy[(int64_t)r * A->ld_res + s] = 0;
    A->chain[(int64_t)r * A->ld_res + s] = 0;
  }
  A->chain_ops[s] = -1;
  if (s == A->path_scen) *A->path_len = 0;
  if (st || g->n == 0) {
    if (!st) A->chain_ops[s] = 0;
    return;
  }
  int64_t busy_r, chain_r;
  int32_t last = 0;
  for (int32_t v = 0; v < g->n; ++v) {
    int32_t r = device_of(J, v, s);
    busy_r = A->busy[(int64_t)r * A->ld_res + s] + J->dur[(int64_t)v * J->ld_dur + s];
    A->busy[(int64_t)r * A->ld_res + s] = (int32_t)busy_r;
    if (w->fin[v] > w->fin[last]) last = v;
  }
  int32_t len = 0, v = last;
  for (;;) {
    int32_t r = device_of(J, v, s);
    int64_t d = J->dur[(int64_t)v * J->ld_dur + s];
    chain_r = A->chain[(int64_t)r * A->ld_res + s] + d;
    A->chain[(int64_t)r * A->ld_res + s] = (int32_t)chain_r;
    rev[len++] = v;
    int64_t start = w->fin[v] - d;
    if (start == 0) break;
    int32_t nxt = -1;
    for (int32_t k = A->pred_ptr[v]; k < A->pred_ptr[v + 1]; ++k) {
      int32_t p = A->pred_idx[k];
      if (w->fin[p] == start && (nxt < 0 || p < nxt)) nxt = p;
    }
    v = nxt >= 0 ? nxt : w->prev[v];
    if (v < 0) break; /* cannot happen after a correct replay: the device finished an op at start */
  }
  A->chain_ops[s] = len;
  if (s == A->path_scen) {
    *A->path_len = len;
    for (int32_t k = 0; k < len && k < A->path_cap; ++k) A->path_ops[k] = rev[len - 1 - k];
  }
}

static void *attribute_range(void *arg) {
  at_job *A = (at_job *)arg;
  const graph_t *g = A->run.g;
  size_t n = (size_t)(g->n ? g->n : 1), R = (size_t)g->nres;
  sim_ws w;
  w.ready = (int64_t *)malloc(n * sizeof(int64_t));
  w.cnt = (int32_t *)malloc(n * sizeof(int32_t));
  w.fin = (int64_t *)malloc(n * sizeof(int64_t));
  w.rfree = (int64_t *)malloc((R ? R : 1) * sizeof(int64_t));
  w.heap = (int32_t *)malloc(n * sizeof(int32_t));
  w.prev = (int32_t *)malloc(n * sizeof(int32_t));
  w.last = (int32_t *)malloc((R ? R : 1) * sizeof(int32_t));
  w.nrun = NULL;
  int32_t *rev = (int32_t *)malloc(n * sizeof(int32_t));
  if (!w.ready || !w.cnt || !w.fin || !w.rfree || !w.heap || !w.prev || !w.last || !rev)
    A->run.rc = ORC_E_NOMEM;
  else
    for (int64_t s = A->run.s0; s < A->run.s1; ++s) attribute_one(A, &w, rev, s);
  free(w.ready);
  free(w.cnt);
  free(w.fin);
  free(w.rfree);
  free(w.heap);
  free(w.prev);
  free(w.last);
  free(rev);
  return NULL;
}

static void set_attribute_range(void *p, int64_t a, int64_t b) {
  ((at_job *)p)->run.s0 = a;
  ((at_job *)p)->run.s1 = b;
}

int oracle_attribute(int32_t n_ops, int32_t n_res, const int64_t *succ_ptr,
                     const int32_t *succ_idx, const int32_t *op_res, const int32_t *prio,
                     int64_t n_scen, const int32_t *dur, int64_t ld_dur,
                     const uint16_t *place, int64_t ld_place, int32_t *makespan,
                     int32_t *status, int32_t *busy, int32_t *chain, int64_t ld_res,
                     int32_t *chain_ops, int64_t path_scen, int32_t *path_ops,
                     int32_t path_cap, int32_t *path_len, int32_t n_threads) {
  graph_t g = {n_ops, n_res, succ_ptr, succ_idx, op_res, prio, NULL};
  int rc = check_graph(&g, 1);
  if (rc) return rc;
  if (n_scen < 0 || (n_scen > 0 && (!makespan || !status || !busy || !chain || !chain_ops)))
    return ORC_E_INVAL;
  if (n_scen > 0 && (ld_res < n_scen || (n_ops > 0 && (!dur || ld_dur < n_scen))))
    return ORC_E_INVAL;
  if (n_scen > 0 && n_ops > 0 && place && ld_place < n_scen) return ORC_E_INVAL;
  if (path_scen >= n_scen || (path_scen >= 0 && (!path_len || (path_cap > 0 && !path_ops))))
    return ORC_E_INVAL;
  if ((rc = build_indeg(&g))) return rc;
  size_t n = (size_t)(n_ops ? n_ops : 1);
  int32_t *order = (int32_t *)malloc(n * sizeof(int32_t));
  int32_t *pred_ptr = (int32_t *)calloc(n + 1, sizeof(int32_t));
  int32_t *pred_idx = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n_ops ? succ_ptr[n_ops] + 1 : 1));
  int32_t *fill = (int32_t *)malloc(n * sizeof(int32_t));
  if (!order || !pred_ptr || !pred_idx || !fill) rc = ORC_E_NOMEM;
  if (!rc) {
    int acyclic = topo_order(&g, order);
    if (acyclic != 1) rc = acyclic < 0 ? ORC_E_NOMEM : ORC_E_CYCLE;
  }
  if (!rc) { /* predecessor lists */
    for (int32_t v = 0; v < n_ops; ++v) pred_ptr[v + 1] = pred_ptr[v] + g.indeg[v];
    for (int32_t v = 0; v < n_ops; ++v) fill[v] = pred_ptr[v];
    for (int32_t u = 0; u < n_ops; ++u)
      for (int64_t e = succ_ptr[u]; e < succ_ptr[u + 1]; ++e) pred_idx[fill[succ_idx[e]]++] = u;
  }
  if (!rc && n_scen > 0) {
    if (n_threads < 1) n_threads = 1;
    at_job *jobs = (at_job *)calloc((size_t)n_threads, sizeof(at_job));
    if (!jobs) {
      rc = ORC_E_NOMEM;
    } else {
      for (int32_t t = 0; t < n_threads; ++t) {
        at_job A = {{&g, 0, 0, dur, ld_dur, place, ld_place, makespan, NULL, status, 0, 0, NULL, NULL},
                    pred_ptr, pred_idx, busy, chain, chain_ops, ld_res, path_scen, path_ops,
                    path_cap, path_len};
        jobs[t] = A;
      }
      rc = run_threads(attribute_range, jobs, sizeof(at_job), n_scen, n_threads, set_attribute_range);
      for (int32_t t = 0; t < n_threads && !rc; ++t) rc = jobs[t].run.rc;
      free(jobs);
    }
  }
  free(order);
  free(pred_ptr);
  free(pred_idx);
  free(fill);
  free(g.indeg);
  return rc;
}

/* ------------------------------------------------- scenario generation */
/*
 * Philox4x32-10 and Philox4x64-10, the counter-based generators of Salmon,
 * Moraes, Dror and Shaw ("Parallel random numbers: as easy as 1, 2, 3",
 * SC'11), written from that definition: ten rounds; a round multiplies
 * words 0 and 2 by the two round multipliers, and the new words are
 * (hi(M1*x2) ^ x1 ^ k0, lo(M1*x2), hi(M0*x0) ^ x3 ^ k1, lo(M0*x0)); the key
 * words grow by the Weyl constants (golden ratio, sqrt(3) - 1) after every
 * round.
 */
void oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int r = 0; r < 10; ++r) {
    uint64_t p0 = (uint64_t)0xD2511F53u * x0;
    uint64_t p1 = (uint64_t)0xCD9E8D57u * x2;
    uint32_t y0 = (uint32_t)(p1 >> 32) ^ x1 ^ k0;
    uint32_t y1 = (uint32_t)p1;
    uint32_t y2 = (uint32_t)(p0 >> 32) ^ x3 ^ k1;
    uint32_t y3 = (uint32_t)p0;
    x0 = y0, x1 = y1, x2 = y2, x3 = y3;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  out[0] = x0, out[1] = x1, out[2] = x2, out[3] = x3;
}

void oracle_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]) {
  uint64_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  uint64_t k0 = key[0], k1 = key[1];
  for (int r = 0; r < 10; ++r) {
    unsigned __int128 p0 = (unsigned __int128)0xD2E7470EE14C6C93ull * x0;
    unsigned __int128 p1 = (unsigned __int128)0xCA5A826395121157ull * x2;
    uint64_t y0 = (uint64_t)(p1 >> 64) ^ x1 ^ k0;
    uint64_t y1 = (uint64_t)p1;
    uint64_t y2 = (uint64_t)(p0 >> 64) ^ x3 ^ k1;
    uint64_t y3 = (uint64_t)p0;
    x0 = y0, x1 = y1, x2 = y2, x3 = y3;
    k0 += 0x9E3779B97F4A7C15ull;
    k1 += 0xBB67AE8584CAA73Bull;
  }
  out[0] = x0, out[1] = x1, out[2] = x2, out[3] = x3;
}

/*
 * One generated duration (the scenario generator's definition):
 *   S = scen0 + s (global scenario index), k = (S / knob_block) mod n_knobs,
 *   b = base[k][v];
 *   (x0..x3) = Philox4x32-10(counter (lo32(S), hi32(S), v, 0),
 *                            key (lo32(seed), hi32(seed)));
 *   U = sum of the eight 16-bit halves of x0..x3 (an Irwin-Hall sum of 8
 *       uniforms on 0..65535), t = 2U - 524280 (zero mean, |t| <= 524280);
 *   d = b + floor((b * t * noise + 2^39) / 2^40), exact in int64.
 * A base outside [1, 2^24] gives d = 0 (an invalid duration).
 */
static int32_t gen_one(const int32_t *base, int32_t n_ops, int32_t n_knobs, int64_t knob_block,
                       uint32_t noise, uint64_t seed, int64_t S, int32_t v) {
  int64_t k = (S / knob_block) % n_knobs;
  int64_t b = base[k * (int64_t)n_ops + v];
  if (b < 1 || b > ((int64_t)1 << 24)) return 0;
  uint32_t ctr[4] = {(uint32_t)S, (uint32_t)((uint64_t)S >> 32), (uint32_t)v, 0};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t x[4];
  oracle_philox4x32_10(ctr, key, x);
  int64_t U = 0;
  for (int i = 0; i < 4; ++i) U += (int64_t)(x[i] & 0xFFFFu) + (int64_t)(x[i] >> 16);
  int64_t t = 2 * U - 524280;
  int64_t q = b * t * (int64_t)noise; /* |q| < 2^24 * 2^19 * 2^20 = 2^63 */
  int64_t adj = (q + ((int64_t)1 << 39)) >> 40; /* arithmetic shift: floor */
  return (int32_t)(b + adj);
}

typedef struct {
  int32_t n;
  const int32_t *base;
  int32_t n_knobs;
  int64_t knob_block;
  uint32_t noise;
  uint64_t seed;
  int64_t scen0;
  int32_t *dur;
  int64_t ld;
  int64_t s0, s1;
} gen_job;

static void *gen_range(void *arg) {
  gen_job *J = (gen_job *)arg;
  for (int32_t v = 0; v < J->n; ++v)
    for (int64_t s = J->s0; s < J->s1; ++s)
      J->dur[v * J->ld + s] =
          gen_one(J->base, J->n, J->n_knobs, J->knob_block, J->noise, J->seed, J->scen0 + s, v);
  return NULL;
}

static void set_gen_range(void *p, int64_t a, int64_t b) {
  ((gen_job *)p)->s0 = a;
  ((gen_job *)p)->s1 = b;
}

int oracle_generate(int32_t n_ops, int64_t n_scen, const int32_t *base, int32_t n_knobs,
                    int64_t knob_block, uint32_t noise, uint64_t seed, int64_t scen0,
                    int32_t *dur, int64_t ld_dur, int32_t n_threads) {
  if (n_ops < 0 || n_scen < 0 || n_knobs < 1 || knob_block < 1 || scen0 < 0 ||
      noise >= (1u << 20) || ld_dur < n_scen || n_scen > INT64_MAX - scen0)
    return ORC_E_INVAL;
  if (n_ops == 0 || n_scen == 0) return ORC_OK;
  if (!base || !dur) return ORC_E_INVAL;
  if (n_threads < 1) n_threads = 1;
  gen_job *jobs = (gen_job *)calloc((size_t)n_threads, sizeof(gen_job));
  if (!jobs) return ORC_E_NOMEM;
  for (int32_t t = 0; t < n_threads; ++t)
    jobs[t] = (gen_job){n_ops, base, n_knobs, knob_block, noise, seed, scen0, dur, ld_dur, 0, 0};
  int rc = run_threads(gen_range, jobs, sizeof(gen_job), n_scen, n_threads, set_gen_range);
  free(jobs);
  return rc;
}
