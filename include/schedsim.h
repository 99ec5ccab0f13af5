/*
 * schedsim.h -- C ABI of the MI355X (gfx950) simulator of the memory-constrained
 * LLM-inference schedulers A_max, A_min, H-SF and A_l (arXiv 2508.14544).
 *
 * Problem (Section 2): one worker with a KV cache of M tokens serves n
 * requests; request i has prompt size s_i, true output length o_i (revealed
 * only by running it) and a predicted interval [l_i, u_i] containing o_i.
 * Time is discrete.  A request started at step p holds s_i + (tau - p) tokens
 * at every step tau in [p, p + o_i] and completes at C_i = p + o_i.  Memory in
 * use may never exceed M (equation (1)).  A running request may be cancelled;
 * it then loses its generated tokens and waits again (Section 2, cancellation).
 * The metric is the total end-to-end latency, equation (3): sum of C_i - a_i.
 *
 * Policies (one per call):
 *   SCHED_AMAX  Algorithm 1: plan every request with length u_i; admit while
 *               equation (2) holds.  Never cancels.
 *   SCHED_AMIN  Algorithms 2 and 4: plan with a lower bound o~_i (initially
 *               l_i); when the running set's memory at t+1 would exceed M,
 *               cancel runs in ascending (o~_i, i) until it fits and raise each
 *               cancelled request's o~_i to the tokens it had generated.
 *   SCHED_HSF   Algorithm 3 (hindsight shortest-first): plan with the true o_i.
 *   SCHED_AELL  Algorithm 5, the promote-l policy A_l of Section 5.1: plan a
 *               new run with l_i; a run that has generated l_i tokens without
 *               finishing (so o_i > l_i) is cancelled, plans with u_i from then
 *               on, and waits behind every fresh request (cancelled requests in
 *               the order they were cancelled, same step by index); it may
 *               restart in the step it was cancelled.
 *   SCHED_ADAPTIVE  The switch of Section 5.1: per instance, SCHED_AELL when
 *               (sum l_i)/(sum u_i) < (3 - sqrt 5)/2 (below this ratio the
 *               competitive-ratio bound of Theorem 5.2 for A_l is the smaller
 *               one; Theorem 5.1 bounds A_min), SCHED_AMIN otherwise.  The
 *               comparison is exact: (3U - 2L)^2 > 5U^2.
 *   SCHED_ARANDOM  The auxiliary A_random (Appendix, in the proof of Theorem
 *               3.1): plan with the true o_i like H-SF, but walk the waiting
 *               requests in a random order, given as per-request priorities
 *               (ascending; ties by index) drawn by the caller.
 * Each step, waiting requests are tried in ascending (planning length, index)
 * order (A_l: the queue order above) and the longest prefix that keeps
 * equation (2) is started.  Ties break by ascending request index, or by an
 * optional per-request tie key first (the paper breaks ties uniformly at
 * random, Algorithms 1, 2 and 4; a random tie key is such a random order).
 * Requests arriving at step a_i join the waiting set at that step (the paper
 * has every a_i = 0).
 *
 * All pointers in sched_instances_t and sched_results_t are DEVICE pointers
 * (e.g. torch tensors on the GPU), allocated and owned by the caller; the
 * library keeps none of them after the work queued on the stream completes.
 * Calls are asynchronous on `stream` (a hipStream_t; NULL = default stream).
 */
#ifndef SCHEDSIM_H
#define SCHEDSIM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SCHED_AMAX = 0,
  SCHED_AMIN = 1,
  SCHED_HSF = 2,
  SCHED_AELL = 3,
  SCHED_ADAPTIVE = 4,
  SCHED_ARANDOM = 5
} sched_algo_t;

/* Return codes of the calls (synchronous) and per-instance status values
 * (written to results.status, valid once the stream has reached the call). */
enum {
  SCHED_OK = 0,
  SCHED_E_INVAL = -1,       /* call: NULL/inconsistent arguments, M <= 0 or M >= 2^30.
                               status: offsets out of range or n_k > max_requests */
  SCHED_E_INTERVAL = -2,    /* status: o < 1, s < 0, or l < 1 or l > o (A_min, A_l, adaptive),
                               or u < o (A_max, A_l, adaptive)                                   */
  SCHED_E_TOO_BIG = -3,     /* status: s + o > M, or s + u > M (A_max, and A_l also when the
                               adaptive policy picks it): can never run                         */
  SCHED_E_STEP_CAP = -4,    /* status: unfinished requests when the step cap was passed        */
  SCHED_E_HIP = -5,         /* call: a HIP runtime call failed                                  */
  SCHED_E_UNSUPPORTED = -6, /* call: capacity request beyond what the kernels hold.
                               status: o, u or l >= 2^15, s >= 2^16, n >= 2^17, a priority
                               outside [0, 2^15), or more than 8192 requests (4096 where eight
                               waves' bitmaps do not fit the LDS; or more than a forced
                               running_capacity) would run at once                              */
  SCHED_E_ARRIVAL = -7,     /* status: an arrival < 0 or arrivals not non-decreasing in index  */
  SCHED_E_SCRATCH = -8      /* call (sched_simulate_noalloc): the call needs more workspace than
                               SCHED_NOALLOC_SCRATCH_BYTES                                       */
};

/* Size of the per-device workspace of sched_simulate_noalloc (96 MiB). */
#define SCHED_NOALLOC_SCRATCH_BYTES (96u << 20)

/* A batch of K independent instances in CSR layout.  Instance k owns requests
 * [offsets[k], offsets[k+1]); request fields are int32 arrays of length N. */
typedef struct {
  int32_t num_instances;    /* K >= 0                                                  */
  int32_t max_requests;     /* upper bound on every n_k; sizes on-chip state (< 2^17)  */
  int64_t total_requests;   /* N = offsets[K]                                          */
  const int64_t* offsets;   /* [K+1], offsets[0] = 0, non-decreasing                    */
  const int32_t* arrival;   /* [N] arrival step a_i, non-decreasing per instance; NULL = all 0 */
  const int32_t* prompt;    /* [N] prompt size s_i                                      */
  const int32_t* output;    /* [N] true output length o_i (the simulated world)         */
  const int32_t* lower;     /* [N] l_i; required for SCHED_AMIN, SCHED_AELL, SCHED_ADAPTIVE */
  const int32_t* upper;     /* [N] u_i; required for SCHED_AMAX, SCHED_AELL, SCHED_ADAPTIVE */
  const int32_t* priority;  /* [N] A_random's order (ascending, ties by index); required for
                               SCHED_ARANDOM, unused otherwise                              */
  const int32_t* tie_key;   /* [N] or NULL.  Order among requests whose planning keys are
                               equal: by (tie_key, index) instead of index, in every policy's
                               admission order and in A_min's cancellation order (A_random:
                               equal priorities).  A_l's queue of fresh requests is ordered by
                               (arrival, tie_key, index) and its same-step cancellations by
                               that queue order.  Any int32 values; equal tie keys fall back
                               to the index.  The library sorts them once per call (8 bytes of
                               workspace and 8 of staging per request).                    */
} sched_instances_t;

/* Outputs.  Per request: completion step C_i (-1 if it never completed) and
 * the number of times it was cancelled.  Per instance: total latency
 * sum(C_i - a_i) over completed requests (equation (3)), makespan max C_i,
 * request-steps (sum over steps of the number of running requests, wasted
 * work included), total cancellations (A_l: promotions) and status, and the
 * policy the instance was simulated with (the requested one, or SCHED_AMIN /
 * SCHED_AELL under SCHED_ADAPTIVE).  Instances whose status is not SCHED_OK
 * and not SCHED_E_STEP_CAP report C_i = -1 and zero counters. */
typedef struct {
  int32_t* completion;      /* [N] required     */
  int32_t* evictions;       /* [N] or NULL      */
  int64_t* total_latency;   /* [K] required     */
  int32_t* makespan;        /* [K] or NULL      */
  int64_t* request_steps;   /* [K] or NULL      */
  int64_t* total_evictions; /* [K] or NULL      */
  int32_t* status;          /* [K] required     */
  int32_t* algo_used;       /* [K] or NULL      */
} sched_results_t;

/* Capacities.  Outputs never depend on any of the sizes below, nor on which
 * other instances share a batch: an instance whose running set or cancelled
 * set outgrows the room of one launch is simulated again from step 0 by a
 * later launch with more room.  One wave holds up to 1024 concurrently running
 * requests; an instance that needs more is simulated again by a workgroup of 4
 * waves (4096 runs), then of 8 waves (8192 runs; for A_max and A_l only when
 * n_max is below about 96000, where the LDS holds eight copies of the waiting
 * set's bitmaps and the completion lists).  Only an instance that needs more,
 * or more than a forced running_capacity, ends with SCHED_E_UNSUPPORTED. */
typedef struct {
  int64_t step_cap;         /* last simulated step; <= 0: per instance
                               min(2^30, 4*(max a + sum(o+1)) + 64)                       */
  int32_t running_capacity; /* > 0 (<= 1024): hold at most this many concurrently running
                               requests per instance, rounded up to 64, 128, 256, 320, 384,
                               512 or 1024, on one wave; an instance that needs more gets
                               SCHED_E_UNSUPPORTED.  0: as many as it needs (one wave's
                               register rows follow the running set, 128 to 640 runs, then
                               1024 in a retry launch; beyond that, workgroups as above)    */
  int32_t evicted_capacity; /* LDS slots of A_min's cancelled set in the first launch; 0:
                               default (min(n_max, 16384) for batches of at most 64 instances,
                               else, for n_max <= 1024, min(n_max, the slots that a wave's
                               share of a CU's LDS leaves beside its bitmaps and staged
                               completion steps, at least 512 and at most 1024), and
                               min(n_max, 1024) above; clipped to what a workgroup's LDS
                               holds).  An instance
                               that outgrows them is simulated again with as many slots as the
                               LDS holds, and one that outgrows those with a set of n slots in
                               global memory (8 bytes of workspace per request when n_max
                               exceeds the LDS room).  A_l's queue of promoted requests is
                               always an array of n entries in global memory (8 bytes of
                               workspace per request).                                      */
  void* event_before;       /* hipEvent_t recorded just before the simulation kernel, or NULL */
  void* event_after;        /* hipEvent_t recorded just after it, or NULL                  */
  int32_t evicted_lds_limit;/* > 0: at most this many LDS slots for the cancelled set in any
                               launch (beyond them the global-memory set); 0: as many as fit.
                               For tests of the global-memory set on small instances.      */
  int32_t workgroup_waves;  /* 0 or 1: one wave per instance first (the default).  2 or 4:
                               every instance is simulated by a workgroup of that many waves
                               from the start, each wave holding 1/W of the running set in
                               1024/(64 W) register rows (SCHED_AMAX, SCHED_AMIN, SCHED_HSF
                               only; other values or policies give SCHED_E_INVAL).  The waves
                               agree on each step's decisions through LDS and a barrier; the
                               outputs are the same.  A_min's cancelled set then lives in
                               global memory (n entries per wave) unless two waves' copies
                               fit the LDS.                                                  */
} sched_options_t;

/* Simulate every instance with the given policy (algo: a sched_algo_t value,
 * passed as int32_t so that any value is well defined; others give
 * SCHED_E_INVAL) and budget M (0 < M < 2^30).
 * Returns SCHED_OK once the work is queued, or a call-level error code (then
 * nothing was queued).  Per-instance problems are reported in results.status;
 * other instances still run.  Scratch memory is allocated stream-ordered on
 * `stream` and released after the kernels (stream-ordered).  SCHED_ADAPTIVE
 * runs its A_l instances on a second stream that the library creates once per
 * device (default priority, kept until the process ends) and joins back into
 * `stream` with events, so all of the call's work is ordered before whatever
 * the caller queues on `stream` next. */
int sched_simulate(const sched_instances_t* instances, int32_t algo, int64_t M,
                   const sched_results_t* results, void* stream);

/* Same, with options (opts may be NULL = all defaults). */
int sched_simulate_opts(const sched_instances_t* instances, int32_t algo, int64_t M,
                        const sched_results_t* results, void* stream,
                        const sched_options_t* opts);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same as
 * sched_simulate_opts, but the workspace is a fixed array of
 * SCHED_NOALLOC_SCRATCH_BYTES in device memory that the library holds on each
 * device it runs on until the process ends, and nothing is allocated (no
 * hipMalloc, no stream or event creation: SCHED_ADAPTIVE runs both of its
 * policies on `stream`).  The workspace needs 20 bytes per request plus 8 per
 * instance (12 for A_min with upper bounds and the adaptive policy, 16 for A_min
 * batches of more than 16 instances per CU, plus 256 bytes), 16 more
 * per request with tie keys, and 8 more per request for
 * A_l and the adaptive policy or when n_max exceeds the LDS room of A_min's
 * cancelled set, and, for A_min when n_max exceeds 1024 (workgroup launches
 * whose waves keep cancelled sets in global memory), up to 64 MiB more
 * (8 * W * n_max bytes per workgroup of W waves, for at most as many
 * workgroups as fit in 64 MiB); a call that needs more returns
 * SCHED_E_SCRATCH before queueing anything (e.g. at most about 5.0 million
 * requests without tie keys).  Every call on a device shares that device's
 * array: calls whose work overlaps on one device (other streams, other host
 * threads) race and must be serialised by the caller.  Outputs, statuses and
 * the caller's pointers are as for sched_simulate_opts. */
int sched_simulate_noalloc(const sched_instances_t* instances, int32_t algo, int64_t M,
                           const sched_results_t* results, void* stream, const sched_options_t* opts);

/* Validation only: writes to status[K] (device) the per-instance status that
 * sched_simulate would give each instance before simulating it (SCHED_OK,
 * SCHED_E_INVAL for bad offsets, SCHED_E_ARRIVAL, SCHED_E_INTERVAL,
 * SCHED_E_TOO_BIG or SCHED_E_UNSUPPORTED for field values beyond the
 * kernels' widths), reading the same request fields as sched_simulate with
 * `algo` (the adaptive policy validates with the policy it picks).  No
 * workspace; asynchronous on `stream`.  Returns a call-level code like
 * sched_simulate (SCHED_E_INVAL for NULL pointers or M outside (0, 2^30)). */
int sched_validate(const sched_instances_t* instances, int32_t algo, int64_t M, int32_t* status,
                   void* stream);

/* The hindsight optimum of tiny instances (n_k <= 8): the minimum total
 * latency (equation (3)) over every non-preemptive schedule that knows the
 * true outputs and keeps equation (1) (the OPT of the competitive analysis,
 * Section 2), by exhaustive branch and bound on the GPU: a first launch gives
 * every instance one wave (its 64 lanes test 64 start steps of a request at
 * once) and min(node_cap, 2^17) nodes; the instances not finished by then are
 * searched again by a second launch of as many 16-wave workgroups as the
 * device holds at once, whose waves claim the pieces below the starts of an
 * instance's first two requests one at a time from any unfinished instance
 * (the first launch's best is the starting bound; best totals are shared in
 * global memory at every claim and in LDS within a workgroup), each wave with
 * at most node_cap nodes per instance it works on.  The second launch takes a
 * stream-ordered workspace of 16 bytes per instance (hipMallocAsync).  Reads
 * offsets, arrival (NULL = all 0), prompt and output of `instances`
 * (device pointers; lower, upper and priority are ignored).  upper_bound
 * (device, [K] or NULL) may give, per instance, the total latency of a known
 * feasible schedule (e.g. a policy's), which only speeds the search up
 * (values <= 0 are ignored; a bound that is not achievable gives a wrong
 * answer, since the search looks only for strictly better schedules).  Writes, per
 * instance, total_latency[K] and status[K] (SCHED_OK, SCHED_E_ARRIVAL,
 * SCHED_E_INTERVAL for o < 1 or s < 0, SCHED_E_TOO_BIG for s + o > M,
 * SCHED_E_INVAL for bad offsets, SCHED_E_UNSUPPORTED when max a + sum(o + 1)
 * reaches 2^27, SCHED_E_STEP_CAP when a wave's search exceeded node_cap nodes
 * (total_latency then holds the best schedule found, an upper bound)), and,
 * if nodes is not NULL, nodes[K] searched (start steps tested, both launches).
 * node_cap <= 0 selects 2^26; larger
 * budgets are clamped to 2^31 - 1.  Returns SCHED_E_UNSUPPORTED if max_requests > 8 (nothing
 * queued), SCHED_E_INVAL for NULL pointers or M outside (0, 2^30). */
int sched_optimum(const sched_instances_t* instances, int64_t M, const int64_t* upper_bound,
                  int64_t* total_latency, int32_t* status, int64_t* nodes, int64_t node_cap, void* stream);

/* Human-readable text for a return or status code (static storage). */
const char* sched_strerror(int code);

/* Library ABI version (major * 100 + minor). */
int sched_version(void);

#ifdef __cplusplus
}
#endif
#endif /* SCHEDSIM_H */
