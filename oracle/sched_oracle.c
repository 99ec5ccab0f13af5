/*
 * sched_oracle.c -- plain, slow, obviously correct CPU oracle of A_max, A_min
 * and H-SF (arXiv 2508.14544).
 *
 * TEST INFRASTRUCTURE ONLY: used by tests/, the smoke check and the benchmark's
 * CPU-baseline leg.  It shares no code with the HIP path.
 *
 * What it follows:
 *   - Section 2 (problem setting): one worker, KV cache of M tokens; a request
 *     started at p with true output o holds s + (tau - p) tokens at step tau,
 *     for tau in [p, p + o]; its latency is p + o (minus its arrival).
 *   - Equation (2) (future-feasibility constraint) for admissions.
 *   - Algorithm 1 (A_max): every output is taken to be u.
 *   - Algorithm 2 / Algorithm 4 (A_min, per-request lower bounds): plan with
 *     the running lower bound o~, evict in ascending o~ on projected overflow
 *     at t+1 and raise o~ to the tokens already generated.
 *   - Algorithm 3 (H-SF): plan with the true output o, shortest first.
 *   - Algorithm 5 (A_l, the promote-l policy of Section 5.1): plan a new run
 *     with o~ = l; a run that reaches l generated tokens unfinished is removed,
 *     its o~ becomes u, and it rejoins the queue behind every fresh request
 *     (promoted requests keep their promotion order); it may restart at once.
 *   - The adaptive switch of Section 5.1 between A_min and A_l at
 *     alpha* = (3 - sqrt 5)/2, from Theorems 5.1 and 5.2.
 *   - The auxiliary A_random (Appendix, proof of Theorem 3.1): plan with the
 *     true o and add waiting requests in a given random order while equation
 *     (2) holds (the order arrives as per-request priorities).
 *   - Equation (3) (total end-to-end latency).
 * Readings where the paper is silent (each listed in the design notes):
 *   memory of a run counts at both its start and its completion step; a
 *   request completing at t still occupies s+o at t; the admitted set is the
 *   longest feasible prefix of the waiting requests in key order; ties break by
 *   the caller's tie key if one is given, then by ascending request index (the
 *   paper breaks them uniformly at random; a random tie key is such an order);
 *   an evicted request waits and may restart from
 *   t+1; o~ <- max(o~, tokens generated); online arrivals join the waiting set
 *   at their arrival step and latency is measured from arrival.
 */
#include "sched_oracle.h"

#include <stdlib.h>
#include <string.h>

enum { NOT_ARRIVED = 0, WAITING = 1, RUNNING = 2, DONE = 3 };

/* ---------------------------------------------------------------------------
 * Waiting set: binary min-heap of request indices ordered by (key, tie, index),
 * where key is the planning length (A_max, A_min, H-SF), the queue position
 * (A_l) or the priority (A_random), and tie the caller's tie key (if any).
 * Only "peek the smallest" and "remove the smallest" are needed, because the
 * admission walk stops at the first request that does not fit.
 * ------------------------------------------------------------------------- */
typedef struct {
  int32_t* idx;
  int64_t size;
  const int64_t* key;
  const int32_t* tie; /* tie-break before the index; NULL = index only */
} heap_t;

static int key_less(const heap_t* h, int32_t x, int32_t y) {
  if (h->key[x] != h->key[y]) return h->key[x] < h->key[y];
  if (h->tie && h->tie[x] != h->tie[y]) return h->tie[x] < h->tie[y];
  return x < y;
}

static void heap_push(heap_t* h, int32_t r) {
  int64_t i = h->size++;
  h->idx[i] = r;
  while (i > 0) {
    int64_t parent = (i - 1) / 2;
    if (!key_less(h, h->idx[i], h->idx[parent])) break;
    int32_t tmp = h->idx[i];
    h->idx[i] = h->idx[parent];
    h->idx[parent] = tmp;
    i = parent;
  }
}

static void heap_pop(heap_t* h) {
  h->idx[0] = h->idx[--h->size];
  int64_t i = 0;
  for (;;) {
    int64_t lft = 2 * i + 1, rgt = lft + 1, m = i;
    if (lft < h->size && key_less(h, h->idx[lft], h->idx[m])) m = lft;
    if (rgt < h->size && key_less(h, h->idx[rgt], h->idx[m])) m = rgt;
    if (m == i) break;
    int32_t tmp = h->idx[i];
    h->idx[i] = h->idx[m];
    h->idx[m] = tmp;
    i = m;
  }
}

/* ---------------------------------------------------------------------------
 * Equation (2), evaluated at the planned end of every member.
 * A planned set is a list of runs (start p, prompt s, planned end E).  A run is
 * present at step c iff c <= E and then holds s + c - p tokens.  Between two
 * consecutive planned ends the set of present runs is fixed and the total only
 * grows with c, so the constraint for all t' in [t, max E] holds iff it holds
 * at every planned end.  This is the literal double loop.
 * ------------------------------------------------------------------------- */
static int feasible(int64_t nq, const int64_t* qp, const int64_t* qs, const int64_t* qe,
                    int64_t M) {
  for (int64_t ci = 0; ci < nq; ci++) {
    int64_t c = qe[ci];
    int64_t mem = 0;
    for (int64_t k = 0; k < nq; k++)
      if (qe[k] >= c) mem += qs[k] + c - qp[k];
    if (mem > M) return 0;
  }
  return 1;
}

/* Sort record: the eviction order (o~, tie, index) of A_min, A_l's fresh-queue
 * order (arrival, tie, index) and its same-step promotion order (queue
 * position) all sort (key, tie, i) triples. */
typedef struct {
  int32_t i;
  int32_t tie;
  int64_t key_est;
} evict_key_t;

static int cmp_evict(const void* x, const void* y) {
  const evict_key_t* a = (const evict_key_t*)x;
  const evict_key_t* b = (const evict_key_t*)y;
  if (a->key_est != b->key_est) return a->key_est < b->key_est ? -1 : 1;
  if (a->tie != b->tie) return a->tie < b->tie ? -1 : 1;
  return a->i < b->i ? -1 : (a->i > b->i);
}

int64_t orc_default_step_cap(int32_t n, const int32_t* a, const int32_t* o) {
  int64_t max_a = 0, sum = 0;
  for (int32_t i = 0; i < n; i++) {
    if (a && a[i] > max_a) max_a = a[i];
    sum += (int64_t)o[i] + 1;
  }
  int64_t cap = 4 * (max_a + sum) + 64;
  if (cap > ((int64_t)1 << 30)) cap = (int64_t)1 << 30;
  return cap;
}

static void log_event(orc_event_t* ev, int64_t cap, int64_t* cnt, int64_t t, int32_t kind,
                      int32_t req) {
  if (ev && *cnt < cap) {
    ev[*cnt].t = t;
    ev[*cnt].kind = kind;
    ev[*cnt].req = req;
  }
  (*cnt)++;
}

/* Per-instance validation, in priority order: arrivals, request data, size. */
static int validate(int32_t n, const int32_t* a, const int32_t* s, const int32_t* o,
                    const int32_t* l, const int32_t* u, int32_t algo, int64_t M) {
  for (int32_t i = 0; i < n; i++) {
    int64_t ai = a ? a[i] : 0;
    if (ai < 0) return ORC_E_ARRIVAL;
    if (i > 0 && a && a[i] < a[i - 1]) return ORC_E_ARRIVAL;
  }
  const int need_l = algo == ORC_AMIN || algo == ORC_AELL;
  const int need_u = algo == ORC_AMAX || algo == ORC_AELL;
  for (int32_t i = 0; i < n; i++) {
    if (o[i] < 1 || s[i] < 0) return ORC_E_INTERVAL;
    if (need_l && (l[i] < 1 || l[i] > o[i])) return ORC_E_INTERVAL;
    if (need_u && u[i] < o[i]) return ORC_E_INTERVAL;
  }
  for (int32_t i = 0; i < n; i++) {
    if ((int64_t)s[i] + o[i] > M) return ORC_E_TOO_BIG;
    if (need_u && (int64_t)s[i] + u[i] > M) return ORC_E_TOO_BIG;
  }
  return ORC_OK;
}

int32_t orc_adaptive_choice(int32_t n, const int32_t* l, const int32_t* u) {
  int64_t L = 0, U = 0;
  for (int32_t i = 0; i < n; i++) {
    L += l[i];
    U += u[i];
  }
  /* alpha = L/U < (3 - sqrt 5)/2  <=>  sqrt(5) U < 3U - 2L  <=>  5 U^2 < (3U - 2L)^2 */
  if (n == 0 || 3 * U - 2 * L <= 0) return ORC_AMIN;
  const unsigned __int128 d = (unsigned __int128)(3 * U - 2 * L);
  const unsigned __int128 uu = (unsigned __int128)U;
  return d * d > 5 * uu * uu ? ORC_AELL : ORC_AMIN;
}

int orc_simulate(int32_t n, const int32_t* a, const int32_t* s, const int32_t* o,
                 const int32_t* l, const int32_t* u, const int32_t* prio, const int32_t* tie,
                 int32_t algo, int64_t M,
                 int64_t step_cap, int32_t* completion, int32_t* evictions,
                 int64_t* tel, int64_t* makespan, int64_t* request_steps,
                 int64_t* total_evictions, int64_t* stats, orc_event_t* events,
                 int64_t events_cap, int64_t* n_events) {
  int64_t nev = 0;
  if (stats) memset(stats, 0, sizeof(int64_t) * ORC_STAT_COUNT);
  *tel = 0;
  *makespan = 0;
  *request_steps = 0;
  *total_evictions = 0;
  if (n_events) *n_events = 0;
  if (n < 0 || M <= 0 || (n > 0 && (!s || !o || !completion))) return ORC_E_INVAL;
  if (algo < ORC_AMAX || algo > ORC_ARANDOM) return ORC_E_INVAL;
  if (n > 0 && algo == ORC_ARANDOM && !prio) return ORC_E_INVAL;
  if (n > 0 && (algo == ORC_AMIN || algo == ORC_AELL || algo == ORC_ADAPTIVE) && !l) return ORC_E_INVAL;
  if (n > 0 && (algo == ORC_AMAX || algo == ORC_AELL || algo == ORC_ADAPTIVE) && !u) return ORC_E_INVAL;
  if (algo == ORC_ADAPTIVE) algo = orc_adaptive_choice(n, l, u);
  for (int32_t i = 0; i < n; i++) {
    completion[i] = -1;
    if (evictions) evictions[i] = 0;
  }
  int st = validate(n, a, s, o, l, u, algo, M);
  if (st != ORC_OK || n == 0) return st;
  if (step_cap <= 0) step_cap = orc_default_step_cap(n, a, o);

  int32_t* state = (int32_t*)calloc(n, sizeof(int32_t));
  int64_t* p = (int64_t*)calloc(n, sizeof(int64_t));       /* last start step       */
  int64_t* est = (int64_t*)calloc(n, sizeof(int64_t));     /* planning length       */
  int32_t* running = (int32_t*)malloc(sizeof(int32_t) * n);
  int32_t* done_now = (int32_t*)malloc(sizeof(int32_t) * n);
  int32_t* deferred = (int32_t*)malloc(sizeof(int32_t) * n); /* evicted last step  */
  int32_t* heap_mem = (int32_t*)malloc(sizeof(int32_t) * n);
  int64_t* qp = (int64_t*)malloc(sizeof(int64_t) * (n + 1));
  int64_t* qs = (int64_t*)malloc(sizeof(int64_t) * (n + 1));
  int64_t* qe = (int64_t*)malloc(sizeof(int64_t) * (n + 1));
  evict_key_t* ek = (evict_key_t*)malloc(sizeof(evict_key_t) * n);
  int32_t* evc = (int32_t*)calloc(n, sizeof(int32_t));
  /* queue position (A_l): fresh requests by index, promoted ones after every
   * fresh one, in promotion order */
  int64_t* qpos = (int64_t*)malloc(sizeof(int64_t) * n);
  int32_t* promoted = (int32_t*)malloc(sizeof(int32_t) * n);
  int64_t n_promotions = 0;
  heap_t waiting = {heap_mem, 0, algo == ORC_AELL || algo == ORC_ARANDOM ? qpos : est, tie};

  /* Planning length: u (A_max, Alg. 1), o (H-SF, Alg. 3), o~ initialised to l
   * (A_min, Alg. 2 and Alg. 4; A_l, Alg. 5). */
  for (int32_t i = 0; i < n; i++) {
    est[i] = (algo == ORC_AMAX) ? u[i] : (algo == ORC_HSF || algo == ORC_ARANDOM) ? o[i] : l[i];
    qpos[i] = algo == ORC_ARANDOM ? prio[i] : i;
  }
  /* A_l's fresh queue: by arrival, equal arrivals by (tie, index) */
  if (algo == ORC_AELL && tie) {
    for (int32_t i = 0; i < n; i++) {
      ek[i].i = i;
      ek[i].tie = tie[i];
      ek[i].key_est = a ? a[i] : 0;
    }
    qsort(ek, n, sizeof(evict_key_t), cmp_evict);
    for (int32_t r = 0; r < n; r++) qpos[ek[r].i] = r;
  }

  int32_t n_running = 0, n_deferred = 0, n_done = 0, next_arrival = 0;
  int32_t n_evicted_waiting = 0;
  int64_t t = 0;
  for (;; t++) {
    if (t > step_cap) {
      st = ORC_E_STEP_CAP;
      break;
    }
    /* 1. arrivals, and requests evicted at the previous step become eligible */
    while (next_arrival < n && (a ? a[next_arrival] : 0) <= t) {
      state[next_arrival] = WAITING;
      heap_push(&waiting, next_arrival);
      next_arrival++;
    }
    for (int32_t k = 0; k < n_deferred; k++) heap_push(&waiting, deferred[k]);
    n_deferred = 0;

    /* 2. completions: a run started at p with true length o ends at p + o */
    int32_t n_done_now = 0, kept = 0;
    for (int32_t k = 0; k < n_running; k++) {
      int32_t i = running[k];
      if (p[i] + o[i] == t) {
        state[i] = DONE;
        completion[i] = (int32_t)t;
        done_now[n_done_now++] = i;
        n_done++;
        log_event(events, events_cap, &nev, t, ORC_EV_COMPLETE, i);
      } else {
        running[kept++] = i;
      }
    }
    n_running = kept;

    /* 3. stop once every request has finished */
    if (n_done == n) break;

    /* 4. A_min: if the running set's projected memory at t+1 exceeds M, remove
     *    runs in ascending (o~, index) until it fits; each removed request's
     *    lower bound becomes the number of tokens it had generated (kept
     *    monotone), and it waits again from t+1 (Alg. 2 / Alg. 4). */
    if (algo == ORC_AMIN) {
      int64_t P = 0;
      for (int32_t k = 0; k < n_running; k++) {
        int32_t i = running[k];
        P += s[i] + (t + 1) - p[i];
      }
      if (P > M) {
        for (int32_t k = 0; k < n_running; k++) {
          ek[k].i = running[k];
          ek[k].tie = tie ? tie[running[k]] : 0;
          ek[k].key_est = est[running[k]];
        }
        qsort(ek, n_running, sizeof(evict_key_t), cmp_evict);
        if (stats) {
          int64_t lg = 0;
          while ((INT64_C(1) << lg) < n_running) lg++;
          stats[ORC_STAT_WORK] += (int64_t)n_running * lg;
        }
        int32_t n_removed = 0;
        for (int32_t k = 0; k < n_running && P > M; k++) {
          int32_t i = ek[k].i;
          P -= s[i] + (t + 1) - p[i];
          int64_t generated = t - p[i];
          if (generated > est[i]) est[i] = generated;
          evc[i]++;
          state[i] = WAITING;
          deferred[n_deferred++] = i;
          n_evicted_waiting++;
          n_removed++;
          log_event(events, events_cap, &nev, t, ORC_EV_EVICT, i);
        }
        kept = 0;
        for (int32_t k = 0; k < n_running; k++)
          if (state[running[k]] == RUNNING) running[kept++] = running[k];
        n_running = kept;
        if (stats) stats[ORC_STAT_EVICT_EVENTS]++;
        (void)n_removed;
      }
    }

    /* 4'. A_l: a run that has generated o~ = l tokens without finishing has
     *     o > l; it leaves the running set, plans with u from now on and joins
     *     the back of the queue (same-step promotions in the order of their
     *     fresh-queue positions: index order without tie keys), where it may
     *     be admitted again at this step (Alg. 5). */
    if (algo == ORC_AELL) {
      int32_t n_prom = 0;
      kept = 0;
      for (int32_t k = 0; k < n_running; k++) {
        int32_t i = running[k];
        if (p[i] + est[i] == t) promoted[n_prom++] = i;
        else running[kept++] = i;
      }
      if (n_prom > 0) {
        if (stats) {
          stats[ORC_STAT_EVICT_EVENTS]++;
          stats[ORC_STAT_WORK] += n_running;
        }
        n_running = kept;
        /* a request is promoted at most once, so qpos still holds its fresh position */
        for (int32_t x = 0; x < n_prom; x++) {
          ek[x].i = promoted[x];
          ek[x].tie = 0;
          ek[x].key_est = qpos[promoted[x]];
        }
        qsort(ek, n_prom, sizeof(evict_key_t), cmp_evict);
        for (int32_t x = 0; x < n_prom; x++) {
          int32_t i = ek[x].i;
          est[i] = u[i];
          qpos[i] = (int64_t)n + n_promotions++;
          evc[i]++;
          state[i] = WAITING;
          n_evicted_waiting++;
          heap_push(&waiting, i);
          log_event(events, events_cap, &nev, t, ORC_EV_EVICT, i);
        }
      }
    }

    /* 5. admission: the planned set holds the runs completing now (present
     *    only at c = t) and the running ones (planned end p + est, but at least
     *    t+1 since they are known to be present then).  Walk the eligible
     *    waiting requests in (est, index) order and add each one whose
     *    addition keeps equation (2); stop at the first that does not fit. */
    int64_t nq = 0;
    for (int32_t k = 0; k < n_done_now; k++) {
      int32_t i = done_now[k];
      qp[nq] = p[i];
      qs[nq] = s[i];
      qe[nq] = t;
      nq++;
    }
    for (int32_t k = 0; k < n_running; k++) {
      int32_t i = running[k];
      int64_t e = p[i] + est[i];
      if (e < t + 1) e = t + 1;
      qp[nq] = p[i];
      qs[nq] = s[i];
      qe[nq] = e;
      nq++;
    }
    while (waiting.size > 0) {
      int32_t w = waiting.idx[0];
      qp[nq] = t;
      qs[nq] = s[w];
      qe[nq] = t + est[w];
      if (stats) {
        stats[ORC_STAT_TESTS]++;
        stats[ORC_STAT_WORK] += nq + 1;
      }
      if (!feasible(nq + 1, qp, qs, qe, M)) break;
      nq++;
      heap_pop(&waiting);
      if (evc[w] > 0) n_evicted_waiting--;
      state[w] = RUNNING;
      p[w] = t;
      running[n_running++] = w;
      log_event(events, events_cap, &nev, t, ORC_EV_START, w);
    }

    /* 6. this step processes every running request once */
    *request_steps += n_running;
    if (stats) {
      stats[ORC_STAT_WORK] += (int64_t)n_running * (algo == ORC_AMIN ? 2 : 1);
      if (n_running > stats[ORC_STAT_MAX_RUNNING]) stats[ORC_STAT_MAX_RUNNING] = n_running;
      if (n_evicted_waiting > stats[ORC_STAT_MAX_EVICTED_WAIT])
        stats[ORC_STAT_MAX_EVICTED_WAIT] = n_evicted_waiting;
      if (waiting.size + n_deferred > stats[ORC_STAT_MAX_WAITING])
        stats[ORC_STAT_MAX_WAITING] = waiting.size + n_deferred;
    }
  }
  if (stats) stats[ORC_STAT_STEPS] = t;

  /* Equation (3), with latency measured from arrival. */
  for (int32_t i = 0; i < n; i++) {
    if (evictions) evictions[i] = evc[i];
    *total_evictions += evc[i];
    if (completion[i] >= 0) {
      *tel += (int64_t)completion[i] - (a ? a[i] : 0);
      if (completion[i] > *makespan) *makespan = completion[i];
    }
  }
  if (n_events) *n_events = nev;

  free(state);
  free(p);
  free(est);
  free(running);
  free(done_now);
  free(deferred);
  free(heap_mem);
  free(qp);
  free(qs);
  free(qe);
  free(ek);
  free(evc);
  free(qpos);
  free(promoted);
  return st;
}
