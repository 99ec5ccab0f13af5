/*
 * sched_oracle.h -- plain CPU oracle of the memory-constrained LLM-inference
 * schedulers A_max, A_min and H-SF (arXiv 2508.14544).
 *
 * TEST INFRASTRUCTURE ONLY.  This oracle exists so that tests, the smoke check
 * and the benchmark's CPU-baseline leg can check the HIP path against a slow,
 * obviously correct implementation.  Nothing in the product path may include,
 * link or call it.  It shares no code with the HIP library.
 */
#ifndef SCHED_ORACLE_H
#define SCHED_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ORC_AELL: the promote-l policy A_l (Section 5.1, Algorithm 5);
 * ORC_ADAPTIVE: per instance, A_l when the ratio alpha = (sum l)/(sum u) is
 * below alpha* = (3 - sqrt 5)/2 (where Theorem 5.2's bound for A_l is below
 * Theorem 5.1's for A_min, Section 5.1), A_min otherwise. */
/* ORC_ARANDOM: the auxiliary policy A_random (Appendix, used in the proof of
 * Theorem 3.1): plan with the true o and walk the waiting requests in a random
 * order given by the caller as per-request priorities (ascending, ties by
 * index). */
enum { ORC_AMAX = 0, ORC_AMIN = 1, ORC_HSF = 2, ORC_AELL = 3, ORC_ADAPTIVE = 4, ORC_ARANDOM = 5 };

enum {
  ORC_OK = 0,
  ORC_E_INVAL = -1,     /* bad call arguments                                 */
  ORC_E_INTERVAL = -2,  /* o<1, s<0, or the interval the algorithm needs is bad */
  ORC_E_TOO_BIG = -3,   /* a request can never fit: s+o>M (A_max: s+u>M)      */
  ORC_E_STEP_CAP = -4,  /* step cap reached with unfinished requests          */
  ORC_E_ARRIVAL = -7    /* arrival < 0 or arrivals not non-decreasing         */
};

/* Event kinds written to the optional event log. */
enum { ORC_EV_START = 0, ORC_EV_EVICT = 1, ORC_EV_COMPLETE = 2 };

typedef struct {
  int64_t t;
  int32_t kind;
  int32_t req;
} orc_event_t;

/* Statistics slots (stats[ORC_STAT_*]). */
enum {
  ORC_STAT_MAX_RUNNING = 0,     /* max |running set| after admission          */
  ORC_STAT_MAX_EVICTED_WAIT = 1,/* max number of evicted requests waiting      */
  ORC_STAT_MAX_WAITING = 2,     /* max number of waiting requests              */
  ORC_STAT_STEPS = 3,           /* number of steps simulated                   */
  ORC_STAT_TESTS = 4,           /* feasibility tests evaluated                 */
  ORC_STAT_EVICT_EVENTS = 5,    /* steps at which at least one eviction happened */
  ORC_STAT_WORK = 6,            /* algorithmic work count: per step |S_t| (twice for A_min:
                                   projection), per feasibility test |Q| (planned set with the
                                   candidate), per eviction event |S_t| ceil(log2 |S_t|) (a sort) */
  ORC_STAT_COUNT = 8
};

/*
 * Simulate one instance of n requests.
 *   a, s, o : arrival step, prompt size, true output length (length n).
 *   l, u    : predicted interval bounds; l is needed for A_min, u for A_max,
 *             both for A_l and the adaptive choice (either may be NULL when the
 *             algorithm does not read it).
 *   prio    : per-request priorities (the random order of A_random); needed
 *             only for ORC_ARANDOM (NULL otherwise).
 *   tie     : per-request tie keys, or NULL.  The paper breaks ties among
 *             equal planning lengths uniformly at random (Algorithm 2's
 *             eviction and admission sorts, Algorithm 1's random sample); the
 *             oracle orders equal keys by (tie, index), so a random tie key is
 *             such a random order and NULL means index order.  A_l's fresh
 *             queue is ordered by (arrival, tie, index), and its same-step
 *             promotions by their fresh-queue positions.
 *   algo    : ORC_AMAX, ORC_AMIN, ORC_HSF, ORC_AELL, ORC_ADAPTIVE (which
 *             simulates orc_adaptive_choice's algorithm) or ORC_ARANDOM.
 *   M       : KV-cache budget in tokens (> 0).
 *   step_cap: last step index that may be simulated; <= 0 selects the default
 *             min(2^30, 4*(max a + sum(o+1)) + 64).
 * Outputs: completion[i] (-1 if unfinished), evictions[i] (may be NULL),
 *   *tel = sum over completed of (C_i - a_i), *makespan = max C_i (0 if none),
 *   *request_steps = sum over steps of the running-set size,
 *   *total_evictions, stats[ORC_STAT_COUNT] (may be NULL),
 *   events (may be NULL; at most events_cap are written, *n_events counts all).
 * Returns the instance status (ORC_OK or a negative code).
 */
int orc_simulate(int32_t n, const int32_t* a, const int32_t* s, const int32_t* o,
                 const int32_t* l, const int32_t* u, const int32_t* prio, const int32_t* tie,
                 int32_t algo, int64_t M,
                 int64_t step_cap, int32_t* completion, int32_t* evictions,
                 int64_t* tel, int64_t* makespan, int64_t* request_steps,
                 int64_t* total_evictions, int64_t* stats, orc_event_t* events,
                 int64_t events_cap, int64_t* n_events);

/* The adaptive choice for one instance: ORC_AELL iff (sum l)/(sum u) <
 * (3 - sqrt 5)/2, decided exactly as (3U - 2L)^2 > 5U^2; ORC_AMIN otherwise
 * (also for n = 0). */
int32_t orc_adaptive_choice(int32_t n, const int32_t* l, const int32_t* u);

/* The default step cap for an instance (same formula as above). */
int64_t orc_default_step_cap(int32_t n, const int32_t* a, const int32_t* o);

#ifdef __cplusplus
}
#endif
#endif
