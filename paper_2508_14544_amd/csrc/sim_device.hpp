// sim_device.hpp -- gfx950 kernels of the scheduler simulator (device code).
//
// One wave64 simulates one instance from t = 0 to its last completion (or a
// workgroup of W waves, see group_exchange); nothing returns to the host
// between steps.
//
// k_prepare (per instance): validates the requests, computes the default step
//   cap, initialises the per-request outputs, and ranks the requests by
//   (initial planning length, tie key, index) with a stable LSD radix sort
//   (8-bit digits, LDS histogram, ballot-based stable scatter).  The ranked
//   records (key, s | o << 16) go to a workspace slice of the instance.
//
// k_simulate_ladder / k_simulate_ladder_wide / k_simulate / k_simulate_group
// (per instance), one body per policy (A_max, A_min, H-SF, A_l, A_random; the
// adaptive policy runs the A_min and the A_l bodies, each on its own
// instances), state:
//   running set R    -- ROWS x 64 register slots, row r lane j holds one run:
//                       planned end Rend = p + est, x = s - p + t_r, completion
//                       C = p + o, key = est << 17 | rank, and h = f(Rend) +
//                       Rend - t_r, where f(c) is the planned memory at step c of
//                       all runs whose planned end is >= c (equation (2) summed
//                       over the planned set).  t_r is a base step that keeps the
//                       int32 values small (rebased every 2^16 steps).  A wave
//                       moves, state and all, along a ladder of bodies with 2, 3,
//                       5, 8, 10 (then 12, 16) rows as its running set grows and
//                       shrinks; instances beyond 1024 runs go to workgroups.
//                       Scans cover every row of the current body.
//   fresh waiting F  -- two-level bitmap over key ranks in LDS; the smallest
//                       waiting key is the first set bit.  Its word is cached in
//                       scalar registers until it empties.
//   cancelled V      -- A_min: a register row U of recent cancellations in
//                       front of an unsorted (key, s | o << 16) array in LDS
//                       (or global memory), the smallest key found by a wave
//                       min-reduction; A_l: an append-only queue of promoted
//                       requests in global memory read through a register
//                       window.
// Per step: arrivals set bits of F; runs with C == t complete (A_l: runs still
// present at their planned end are promoted to the back of the queue); for
// A_min the projected memory P at t+1 is compared with M and runs are
// cancelled in ascending key while P > M; then candidates (smallest key of F,
// U and V; A_l: F first) are admitted while equation (2) holds.  The admission
// test needs only O(1) wave reductions because the planned set before the test
// is always feasible (every checkpoint after the candidate's planned end was
// verified when its runs were admitted), so it checks: step t (runs completing
// now hold s+o), step t+1 when a run is already past its planned end, every
// existing planned end <= the candidate's via max h, and the candidate's own
// planned end.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <mutex>
#include <type_traits>

#include "schedsim.h"
#include "wave.hpp"

namespace sk {

// global-memory (address space 1) views of device arrays
typedef __attribute__((address_space(1))) int32_t g_i32;
typedef __attribute__((address_space(1))) uint64_t g_u64;

constexpr int kIdxBits = 17;
constexpr uint32_t kIdxMask = (1u << kIdxBits) - 1u;
constexpr int32_t kEstLimit = 1 << 15;
constexpr int32_t kPromptLimit = 1 << 16;
constexpr int32_t kRebase = 1 << 16;
constexpr int64_t kCapLimit = int64_t(1) << 30;

struct Params {
  int32_t K;
  int32_t max_requests;
  int64_t N;
  const int64_t* offsets;
  const int32_t* arrival;
  const int32_t* prompt;
  const int32_t* output;
  const int32_t* lower;
  const int32_t* upper;
  const int32_t* priority;
  const int32_t* tie_key;   // NULL: equal keys by index; else by (tie key, index)
  int32_t* completion;
  int32_t* evictions;
  int64_t* total_latency;
  int32_t* makespan;
  int64_t* request_steps;
  int64_t* total_evictions;
  int32_t* status;
  int32_t* algo_used;    // optional output: the policy each instance ran
  int32_t M;
  int64_t step_cap;      // > 0: user cap for every instance
  // workspace
  uint32_t* sort_a;
  uint32_t* sort_b;
  uint2* rec;
  int32_t* rank_of;
  int32_t* u_of_rank;    // A_l: u of the request at each rank (the workspace of the second sort buffer)
  int32_t* cap;
  int32_t* algo_of;      // adaptive runs: the policy each instance runs (else NULL)
  // with tie keys: each request's rank in tie order (its identity inside the
  // kernels, in place of the index), the inverse map, and staging arrays of
  // the per-request outputs indexed by that rank (copied out in index order
  // at the end)
  int32_t* tr_of;
  int32_t* idx_of;
  int32_t* comp_st;
  int32_t* ev_st;
  // cancelled set in global memory (the last retry pass): n entries per instance
  uint64_t* vglob;
  // LDS layout of k_simulate
  int32_t nw_max;        // 64-bit words of the level-0 bitmap
  int32_t nw1_max;       // 64-bit words of the level-1 bitmap
  int32_t cap_v;         // evicted-set capacity (LDS passes)
  int32_t retry_status;  // status for an outgrown running set: a later pass (kRetryRows) or SCHED_E_UNSUPPORTED
  int32_t retry_v_status;// status for an outgrown evicted set: a later pass (kRetryV) or SCHED_E_UNSUPPORTED
  int32_t run_mask;      // retry passes: bit 0 runs kRetryRows instances, bit 1 kRetryV ones
  int32_t run_cap;       // retry passes: most runs at once (a caller's forced capacity), else INT32_MAX
  // completion steps staged in LDS after the cancelled set (n_max slots) and
  // written out coalesced at the end of an instance
  int32_t stage_comp;
  // workgroup passes with global cancelled sets: n_max entries per wave of
  // each workgroup of the launch
  uint64_t* vgroup;
  // A_min with upper bounds (alone or in the adaptive policy): each instance's
  // issue-priority class (0-2 by the width of its intervals; 3: none), or -1
  // when all instances share a class
  int32_t* pclass;
  // A_min batches served in several rounds of waves: the order in which the
  // first launch takes the instances (longest expected first), built from a
  // key per instance and kOrderBuckets counters (then the buckets' cursors)
  int32_t* order;
  int32_t* okey;
  int32_t* obucket;
  // k_prepare: nonzero when its key sort runs in two LDS buffers of
  // max_requests entries (dynamic LDS) instead of sort_a / sort_b
  int32_t pre_lds;
};

// buckets of the launch-order key
constexpr int kOrderBuckets = 64;

// Internal statuses of an instance handed to a later pass: its running set
// outgrew the register rows, or its cancelled set outgrew its slots.  The
// later pass simulates it again from step 0 with more room.
constexpr int kRetryRows = -100;
constexpr int kRetryV = -101;

// ---------------------------------------------------------------------------
// k_prepare
// ---------------------------------------------------------------------------
// One stable LSD radix pass of a wave over the n elements src[0..n) -> dst,
// by the 8-bit digit dig(element): LDS histogram, wave scan of the bucket
// starts, and a stable scatter that ranks equal digits inside each 64-element
// chunk with 8 ballots.
template <typename DigitFn>
__device__ __forceinline__ void radix_pass(uint32_t* hist, const uint32_t* src, uint32_t* dst, int n, DigitFn dig) {
  const int lane = threadIdx.x;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int j = lane; j < 256; j += 64) hist[j] = 0;
  __syncthreads();
  for (int c = 0; c < n; c += 64) {
    const int i = c + lane;
    if (i < n) atomicAdd(&hist[dig(src[i])], 1u);
  }
  __syncthreads();
  {
    uint32_t h0 = hist[4 * lane], h1 = hist[4 * lane + 1], h2 = hist[4 * lane + 2], h3 = hist[4 * lane + 3];
    int32_t tot = static_cast<int32_t>(h0 + h1 + h2 + h3);
    int32_t ex = wave::inclusive_scan_i32(tot) - tot;
    __syncthreads();
    hist[4 * lane] = ex;
    hist[4 * lane + 1] = ex + h0;
    hist[4 * lane + 2] = ex + h0 + h1;
    hist[4 * lane + 3] = ex + h0 + h1 + h2;
  }
  __syncthreads();
  for (int c = 0; c < n; c += 64) {
    const int i = c + lane;
    const bool act = i < n;
    const uint32_t key = act ? src[i] : 0u;
    const uint32_t d = act ? dig(key) : 0u;
    uint64_t eq = wave::ballot(act);
    for (int bit = 0; bit < 8; ++bit) {
      const uint64_t bal = wave::ballot(act && ((d >> bit) & 1u));
      eq &= ((d >> bit) & 1u) ? bal : ~bal;
    }
    const int rank = __builtin_popcountll(eq & lt_mask);
    const uint32_t base = act ? hist[d] : 0u;
    __syncthreads();
    if (act) {
      dst[base + rank] = key;
      if (rank == 0) hist[d] = base + static_cast<uint32_t>(__builtin_popcountll(eq));
    }
    __syncthreads();
  }
  __syncthreads();
}

// Stable sort of the request indices 0..n-1 by the 32-bit key key(i) (four
// radix passes; a byte on which every key agrees is skipped).  Returns the
// buffer holding the sorted indices (a or b).
template <typename KeyFn>
__device__ __forceinline__ uint32_t* sort_indices_by(uint32_t* hist, uint32_t* a, uint32_t* b, int n, KeyFn key,
                                                     bool init) {
  const int lane = threadIdx.x;
  uint32_t kand = 0xFFFFFFFFu, kor = 0u;
  for (int c = 0; c < n; c += 64) {
    const int i = c + lane;
    if (i < n) {
      if (init) a[i] = static_cast<uint32_t>(i);
      const uint32_t k = key(static_cast<uint32_t>(i));
      kand &= k;
      kor |= k;
    }
  }
  for (int off = 32; off >= 1; off >>= 1) {
    kand &= static_cast<uint32_t>(__shfl_xor(static_cast<int>(kand), off, 64));
    kor |= static_cast<uint32_t>(__shfl_xor(static_cast<int>(kor), off, 64));
  }
  const uint32_t varies = kand ^ kor;
  __syncthreads();
  for (int pass = 0; pass < 4; ++pass) {
    const int sh = 8 * pass;
    if (((varies >> sh) & 0xFFu) == 0u) continue;
    radix_pass(hist, a, b, n, [&](uint32_t e) { return (key(e) >> sh) & 0xFFu; });
    uint32_t* t = a;
    a = b;
    b = t;
  }
  return a;
}

// Per-instance validation (shared by k_prepare and k_validate): the status
// and, through *algo_out, the policy the instance runs (the adaptive choice);
// also the default step cap.
template <int ALGO>
__device__ __forceinline__ int validate_instance(const Params& P, int k, int* algo_out, int64_t* cap_out) {
  const int lane = threadIdx.x;
  const int64_t b = P.offsets[k];
  const int64_t e = P.offsets[k + 1];
  int status = SCHED_OK;
  if (b < 0 || e < b || e > P.N || e - b > P.max_requests) status = SCHED_E_INVAL;
  const int n = (status == SCHED_OK) ? static_cast<int>(e - b) : 0;

  // l is read by A_min and A_l, u by A_max and A_l; the adaptive policy reads
  // both (their sums pick the policy) and validates with the one it picks
  constexpr bool kReadL = ALGO == SCHED_AMIN || ALGO == SCHED_AELL || ALGO == SCHED_ADAPTIVE;
  constexpr bool kReadU = ALGO == SCHED_AMAX || ALGO == SCHED_AELL || ALGO == SCHED_ADAPTIVE;
  constexpr bool kReadP = ALGO == SCHED_ARANDOM;
  bool arr_bad = false, int_bad = false, big_bad = false, unsup = (n >= (1 << kIdxBits));
  bool bad_l = false, unsup_l = false, bad_u = false, big_u = false, unsup_u = false;
  int64_t max_a = 0, sum_o = 0, sum_l = 0, sum_u = 0;
  int32_t prev_last = 0;
  for (int c = 0; c < n; c += 64) {
    const int i = c + lane;
    const bool act = i < n;
    int32_t a = 0, s = 0, o = 1, lo = 1, up = 1, pr = 0;
    if (act) {
      a = P.arrival ? P.arrival[b + i] : 0;
      s = P.prompt[b + i];
      o = P.output[b + i];
      if (kReadL) lo = P.lower[b + i];
      if (kReadU) up = P.upper[b + i];
      if (kReadP) pr = P.priority[b + i];
    }
    int32_t ap = __shfl_up(a, 1, 64);
    if (lane == 0) ap = prev_last;
    prev_last = __shfl(a, 63, 64);
    if (act) {
      if (a < 0 || (i > 0 && a < ap)) arr_bad = true;
      if (o < 1 || s < 0) int_bad = true;
      if (lo < 1 || lo > o) bad_l = true;
      if (up < o) bad_u = true;
      if (static_cast<int64_t>(s) + o > P.M) big_bad = true;
      if (static_cast<int64_t>(s) + up > P.M) big_u = true;
      if (o >= kEstLimit || s >= kPromptLimit || pr < 0 || pr >= kEstLimit) unsup = true;
      if (lo >= kEstLimit) unsup_l = true;
      if (up >= kEstLimit) unsup_u = true;
      max_a = a > max_a ? a : max_a;
      sum_o += static_cast<int64_t>(o) + 1;
      sum_l += lo;
      sum_u += up;
    }
  }
  // the policy this instance runs; the adaptive one takes A_l when
  // L/U < (3 - sqrt 5)/2, i.e. sqrt(5) U < 3U - 2L, i.e. 5U^2 < (3U - 2L)^2
  int algo = ALGO;
  if (ALGO == SCHED_ADAPTIVE) {
    const int64_t L = wave::sum_i64(sum_l), U = wave::sum_i64(sum_u);
    const int64_t d = 3 * U - 2 * L;
    algo = SCHED_AMIN;
    if (n > 0 && d > 0) {
      const unsigned __int128 dd = static_cast<unsigned __int128>(d) * static_cast<unsigned __int128>(d);
      const unsigned __int128 uu = static_cast<unsigned __int128>(U) * static_cast<unsigned __int128>(U);
      if (dd > 5 * uu) algo = SCHED_AELL;
    }
  }
  const bool use_l = algo == SCHED_AMIN || algo == SCHED_AELL;
  const bool use_u = algo == SCHED_AMAX || algo == SCHED_AELL;
  int_bad = int_bad || (use_l && bad_l) || (use_u && bad_u);
  big_bad = big_bad || (use_u && big_u);
  unsup = unsup || (use_l && unsup_l) || (use_u && unsup_u);
  if (status == SCHED_OK) {
    if (wave::ballot(arr_bad)) status = SCHED_E_ARRIVAL;
    else if (wave::ballot(int_bad)) status = SCHED_E_INTERVAL;
    else if (wave::ballot(big_bad)) status = SCHED_E_TOO_BIG;
    else if (wave::ballot(unsup)) status = SCHED_E_UNSUPPORTED;
  }
  const int64_t max_a_all = wave::max_i64(max_a);
  const int64_t sum_o_all = wave::sum_i64(sum_o);
  int64_t cap = P.step_cap > 0 ? P.step_cap : 4 * (max_a_all + sum_o_all) + 64;
  if (cap > kCapLimit) cap = kCapLimit;
  *algo_out = algo;
  *cap_out = cap;
  return status;
}

// Validation only (sched_validate): status per instance.
template <int ALGO>
__global__ __launch_bounds__(64) void k_validate(Params P) {
  const int k = blockIdx.x;
  int algo = ALGO;
  int64_t cap = 0;
  const int status = validate_instance<ALGO>(P, k, &algo, &cap);
  if (threadIdx.x == 0) {
    P.status[k] = status;
    if (P.algo_used) P.algo_used[k] = algo;
  }
}

template <int ALGO>
__global__ __launch_bounds__(64) void k_prepare(Params P) {
  __shared__ uint32_t hist[256];
  const int k = blockIdx.x;
  const int lane = threadIdx.x;
  int algo = ALGO;
  int64_t cap = 0;
  const int status = validate_instance<ALGO>(P, k, &algo, &cap);
  const int64_t b = P.offsets[k];
  const int n = (status == SCHED_OK) ? static_cast<int>(P.offsets[k + 1] - b) : 0;
  const bool tie = P.tie_key != nullptr;

  // per-request outputs start as "not completed, never cancelled" (with tie
  // keys, the staging arrays the kernels write too)
  const int64_t e = P.offsets[k + 1];
  const int n_init = (b >= 0 && e > b && e <= P.N && e - b <= P.max_requests) ? static_cast<int>(e - b) : 0;
  for (int c = 0; c < n_init; c += 64) {
    const int i = c + lane;
    if (i < n_init) {
      P.completion[b + i] = -1;
      if (P.evictions) P.evictions[b + i] = 0;
      if (tie) {
        P.comp_st[b + i] = -1;
        if (P.evictions) P.ev_st[b + i] = 0;
      }
    }
  }
  if (lane == 0) {
    P.status[k] = status;
    P.cap[k] = static_cast<int32_t>(cap);
    if (P.algo_of) P.algo_of[k] = algo;
    if (P.algo_used) P.algo_used[k] = algo;
    if (P.pclass) P.pclass[k] = 3;
    if (P.okey && (status != SCHED_OK || n == 0)) {
      P.okey[k] = 0;
      atomicAdd(&P.obucket[0], 1);
    }
  }
  if (status != SCHED_OK || n == 0) return;
  if (P.pclass && algo == SCHED_AMIN) {
    // wide intervals mean more cancellations, so longer simulations: the
    // class by sum(u - l) / sum(l) (< 0.3, < 0.75, above)
    int64_t w = 0, l = 0;
    for (int c = 0; c < n; c += 64) {
      const int i = c + lane;
      if (i < n) {
        w += P.upper[b + i] - P.lower[b + i];
        l += P.lower[b + i];
      }
    }
    w = wave::sum_i64(w);
    l = wave::sum_i64(l);
    if (lane == 0) P.pclass[k] = 4 * w >= 3 * l ? 2 : 10 * w >= 3 * l ? 1 : 0;
  }
  if (P.okey) {
    // A_min cancels until its lower bounds have grown to the true lengths, so
    // the instances whose lower bounds fall furthest below them run longest:
    // the key is 16 * sum(o - l) / sum(l), at most kOrderBuckets - 1
    int64_t w = 0, l = 0;
    for (int c = 0; c < n; c += 64) {
      const int i = c + lane;
      if (i < n) {
        w += P.output[b + i] - P.lower[b + i];
        l += P.lower[b + i];
      }
    }
    w = wave::sum_i64(w);
    l = wave::sum_i64(l);
    if (lane == 0) {
      const int64_t q = l > 0 ? (16 * w) / l : 0;
      const int key = q < kOrderBuckets - 1 ? static_cast<int>(q) : kOrderBuckets - 1;
      P.okey[k] = key;
      atomicAdd(&P.obucket[key], 1);
    }
  }

  // ---- tie keys: each request's rank in the order (tie key, index) (A_l:
  // (arrival, tie key, index), its fresh-queue order) is its identity in the
  // keys below; tr_of maps index -> rank, idx_of rank -> index
  if (tie) {
    const int32_t* tk = P.tie_key + b;
    uint32_t* S = sort_indices_by(hist, P.sort_a + b, P.sort_b + b, n,
                                  [&](uint32_t i) { return static_cast<uint32_t>(tk[i]) ^ 0x80000000u; }, true);
    if (algo == SCHED_AELL && P.arrival) {
      const int32_t* ar = P.arrival + b;
      uint32_t* other = S == P.sort_a + b ? P.sort_b + b : P.sort_a + b;
      S = sort_indices_by(hist, S, other, n, [&](uint32_t i) { return static_cast<uint32_t>(ar[i]); }, false);
    }
    for (int c = 0; c < n; c += 64) {
      const int r = c + lane;
      if (r < n) {
        const uint32_t i = S[r];
        P.tr_of[b + i] = r;
        P.idx_of[b + r] = static_cast<int32_t>(i);
      }
    }
    __syncthreads();
  }

  // ---- keys (k0 << 17 | id), k0 = u (A_max), l (A_min, A_l), o (H-SF), the
  // priority (A_random, which plans with o); id = the index, or the tie rank,
  // placed at position id so that the stable sort below keeps id order.  The
  // two sort buffers are in LDS when the launch gave them room (P.pre_lds)
  extern __shared__ uint32_t pre_buf[];
  uint32_t* const ka = P.pre_lds ? pre_buf : P.sort_a + b;
  uint32_t* const kb = P.pre_lds ? pre_buf + P.max_requests : P.sort_b + b;
  for (int c = 0; c < n; c += 64) {
    const int i = c + lane;
    if (i < n) {
      int32_t est = (algo == SCHED_AMAX)   ? P.upper[b + i]
                    : (algo == SCHED_HSF)  ? P.output[b + i]
                    : (algo == SCHED_ARANDOM) ? P.priority[b + i]
                                           : P.lower[b + i];
      const uint32_t id = tie ? static_cast<uint32_t>(P.tr_of[b + i]) : static_cast<uint32_t>(i);
      ka[id] = (static_cast<uint32_t>(est) << kIdxBits) | id;
    }
  }
  __syncthreads();
  // ---- stable LSD radix sort on bits 17..24 then 25..31 (A_l's queue is in
  // id order: its ranks are the ids, no sort)
  for (int pass = 0; pass < (algo == SCHED_AELL ? 0 : 2); ++pass) {
    const uint32_t* src = pass == 0 ? ka : kb;
    uint32_t* dst = pass == 0 ? kb : ka;
    const int shift = kIdxBits + 8 * pass;
    radix_pass(hist, src, dst, n, [&](uint32_t key) { return (key >> shift) & 0xFFu; });
  }
  // ---- ranked records and inverse ranks (rank_of is indexed by request index)
  for (int c = 0; c < n; c += 64) {
    const int r = c + lane;
    if (r < n) {
      const uint32_t key = ka[r];
      const uint32_t id = key & kIdxMask;
      const uint32_t idx = tie ? static_cast<uint32_t>(P.idx_of[b + id]) : id;
      const uint32_t s = static_cast<uint32_t>(P.prompt[b + idx]);
      const uint32_t o = static_cast<uint32_t>(P.output[b + idx]);
      P.rec[b + r] = make_uint2(key, s | (o << 16));
      P.rank_of[b + idx] = r;
      if (algo == SCHED_AELL) P.u_of_rank[b + r] = P.upper[b + idx];
    }
  }
}

// ---------------------------------------------------------------------------
// k_simulate
// ---------------------------------------------------------------------------
// r_end of an empty slot of the running set (below every planned end)
constexpr int32_t kEmpty = INT32_MIN;
// r_c of an empty slot (after every step)
constexpr int32_t kNever = 0x7FFFFFFF;

__device__ __forceinline__ uint64_t uniform_u64(uint64_t v) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v >> 32));
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ __forceinline__ uint32_t uniform_u32(uint32_t v) {
  return static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int32_t>(v)));
}

// The loop-carried state of one instance's simulation, handed from one body
// to another with a different number of register rows (the row ladder: 2, 3,
// 5, 8, 10 rows).  A body grows at an admission that finds no free slot (the
// next body's extra rows start empty) and shrinks, at the start of a step's
// admissions, once the running set fits a smaller body with room to spare (it
// first moves the runs of its upper rows into free slots of the lower ones).
// The LDS sets stay where they are.  `resume`: continue with the admissions of
// step t (false: start step t from its arrivals).
template <int SR>
struct SimStateT {
  static constexpr int kRows = SR;
  int32_t r_end[SR], r_x[SR], r_c[SR], r_h[SR], r_u[SR];
  uint32_t r_key[SR];
  int fr_row;
  uint64_t fr_mask;
  int32_t N, X, t_r, next_c, aw_base, aw_a, aw_rank, arr_ptr, next_a, f_rank, fw_base, f_u, fw_u;
  uint32_t f_key, f_so, fw_key, fw_so, v_key, v_so;
  uint64_t f_word;
  int32_t nV, nVe, v_pos, v_head, v_u, n_done, retry_at, t, DT;
  int64_t rsteps, tot_ev;
  uint32_t u_key, u_so, u_gate;   // A_min: the register row of recent cancellations (per lane)
  uint64_t u_used;
  uint32_t uh_key, uh_so;
  int32_t uh_lane;
  int32_t next_rows;
  bool resume;
  uint32_t vw_lo, vw_hi;          // A_l: register window of the promoted queue (per lane)
  int32_t vw_base;
};
// the narrow ladder (up to 10 rows, four waves a SIMD) and the wide one (up
// to 16 rows, for few large instances and for instances that outgrow the
// narrow one)
using SimState = SimStateT<10>;
using SimStateWide = SimStateT<16>;
// Status of a body that handed its state over (TO_STATE) instead of ending.
constexpr int kResume = -102;

// The row ladders: the body above each rung (0: none).  The narrow ladder
// is 2, 3, 5, 8, 10; the wide one continues with 12 and 16.
__host__ __device__ constexpr int ladder_up(int rows, int top) {
  return rows >= top ? 0
         : rows == 2 ? 3 : rows == 3 ? 5 : rows == 5 ? 8 : rows == 8 ? 10 : rows == 10 ? 12 : rows == 12 ? 16 : 0;
}
// A body shrinks to the smallest rung that holds its runs with this many
// slots to spare (hysteresis: a shrink is never followed at once by a grow).
constexpr int kShrinkSpare = 16;
// A_min: at the start of a step, a register row of recent cancellations that
// holds more than this many entries goes to the LDS set
constexpr int kURowFlush = 48;

// The state of an instance at step 0 (what a body starting fresh holds).
template <typename ST>
__device__ __forceinline__ void fresh_state(ST& st) {
#pragma unroll
  for (int r = 0; r < ST::kRows; ++r) {
    st.r_end[r] = INT32_MIN; st.r_x[r] = 0; st.r_c[r] = 0x7FFFFFFF; st.r_h[r] = 0; st.r_key[r] = 0xFFFFFFFFu;
    st.r_u[r] = 0;
  }
  st.fr_row = 0; st.fr_mask = ~0ull; st.N = 0; st.X = 0; st.t_r = 0; st.next_c = 0x7FFFFFFF;
  st.aw_base = -64; st.aw_a = 0x7FFFFFFF; st.aw_rank = 0; st.arr_ptr = 0; st.next_a = 0;
  st.f_rank = -1; st.fw_base = -1; st.f_word = 0ull; st.f_key = 0xFFFFFFFFu; st.f_so = 0; st.fw_key = 0xFFFFFFFFu;
  st.fw_so = 0; st.f_u = 0; st.fw_u = 0; st.nV = 0; st.nVe = 0; st.v_pos = -1; st.v_head = 0;
  st.v_key = 0xFFFFFFFFu; st.v_so = 0; st.v_u = 0; st.n_done = 0; st.retry_at = 0; st.t = 0; st.DT = 0;
  st.rsteps = 0; st.tot_ev = 0; st.next_rows = 2; st.resume = false;
  st.u_key = 0xFFFFFFFFu; st.u_so = 0; st.u_gate = 0; st.u_used = 0ull;
  st.uh_key = 0xFFFFFFFFu; st.uh_so = 0; st.uh_lane = -1;
  st.vw_lo = 0; st.vw_hi = 0; st.vw_base = -(1 << 30);
}

// ---------------------------------------------------------------------------
// A workgroup of W > 1 waves simulating one instance.  Every wave holds its
// own ROWS register rows of the running set (W x 64 x ROWS slots) and its own
// copy of the rest of the state (the bitmaps and the cancelled set in an LDS
// block of its own, the scalars, the register row of recent cancellations),
// which it updates exactly as the other waves do.  What depends on the whole
// running set is agreed at exchanges: each wave writes its partial results
// (a wave reduction over its rows), a barrier, and lane j < W of every wave
// reads wave j's partials, which one fold inside a 16-lane row combines.  A
// branch around an exchange depends only on state that every wave holds
// alike, so every wave reaches the same exchanges in the same order.  A new
// run goes to the wave that holds the fewest (counts kept alike in every
// wave: lane j holds wave j's).
// ---------------------------------------------------------------------------
// 64-bit LDS words before the waves' blocks: two alternating exchange buffers
// of W x 8 32-bit words, and for the policies whose runs may complete before
// their planned end (A_max, A_l) a list of each wave's completions at a step
// (W x 64 x ROWS entries).
__host__ __device__ constexpr int group_pre_words(int algo, int w, int rows) {
  return 8 * w + ((algo == SCHED_AMAX || algo == SCHED_AELL) ? w * 64 * rows : 0);
}

// A workgroup barrier that orders LDS accesses only (pending global stores
// are not waited for).
__device__ __forceinline__ void group_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// One exchange of four 32-bit words per wave (two with `b`): lane j < W gets
// wave j's words; lanes >= W get their own wave's.  The two buffers alternate,
// so a wave can be at most one exchange ahead of another while it writes.
template <int W>
__device__ __forceinline__ uint4 group_exchange(uint4* red, int& par, int wv, int lane, uint4 a, uint4* b = nullptr) {
  uint4* buf = red + par * 2 * W;
  if (lane == 0) {
    buf[wv] = a;
    if (b) buf[W + wv] = *b;
  }
  group_barrier();
  par ^= 1;
  const int j = lane < W ? lane : wv;
  if (b) *b = buf[W + j];
  return buf[j];
}

// Folds over the lanes of the first 16-lane row (lanes >= W hold neutral values).
__device__ __forceinline__ uint32_t lanes_min_u32(uint32_t v) {
  return uniform_u32(wave::fold_in_row(v, wave::OpMinU32{}));
}
__device__ __forceinline__ int32_t lanes_max_i32(int32_t v) {
  return wave::uniform(static_cast<int32_t>(wave::fold_in_row(static_cast<uint32_t>(v), wave::OpMaxI32{})));
}
__device__ __forceinline__ int32_t lanes_sum_i32(int32_t v) {
  return wave::uniform(static_cast<int32_t>(wave::fold_in_row(static_cast<uint32_t>(v), wave::OpAddU32{})));
}

// Simulates instance k (whose validation status is st0) with ROWS register
// rows and writes its outputs.  A running set that outgrows the rows ends the
// simulation with `retry_status` (the per-request outputs are then reset), or,
// with TO_STATE, saves the state to *st and returns kResume at once.  With
// FROM_STATE the body continues from *st instead of starting at step 0.  A
// cancelled set that outgrows its P.cap_v LDS slots ends it with
// P.retry_v_status; with VGLOBAL the set lives in global memory (n slots, the
// most it can hold).  CAPPED holds the running set to P.run_cap runs.  W > 1:
// a workgroup of W waves simulates the instance (see group_exchange).
template <int ALGO, int ROWS, bool FROM_STATE = false, bool TO_STATE = false, bool VGLOBAL = false,
          bool CAPPED = false, typename ST = SimState, int W = 1, bool CLS = true, bool PRIO = true>
__device__ __forceinline__ int sim_instance(const Params& P, const int k, const int st0, const int retry_status,
                                           ST* st = nullptr) {
  constexpr int kStateRows = ST::kRows;
  static_assert(!(FROM_STATE || TO_STATE) || ROWS <= kStateRows, "state holds at most kStateRows rows");
  static_assert(W == 1 || (W <= 16 && !FROM_STATE && !TO_STATE && !CAPPED), "a workgroup runs fixed rows");
  // only A_min and A_l have cancelled (or promoted) requests waiting: for the
  // other policies every head is fresh, and the code of the cancelled set is
  // left out of their kernels
  constexpr bool kHasV = ALGO == SCHED_AMIN || ALGO == SCHED_AELL;
  extern __shared__ uint64_t lds64[];
  const int lane = W > 1 ? static_cast<int>(threadIdx.x & 63u) : static_cast<int>(threadIdx.x);
  const int wv = W > 1 ? wave::uniform(static_cast<int32_t>(threadIdx.x >> 6)) : 0;
  const int64_t b = P.offsets[k];
  // a body that hands its state over only ever runs valid, non-empty instances
  const int n = (TO_STATE || st0 == SCHED_OK) ? static_cast<int>(P.offsets[k + 1] - b) : 0;
  const int32_t M = P.M;

  int status = st0;
  int handoff = 0;  // TO_STATE: rows of the body that continues (status kResume)
  // counters live in vector registers (see wave::in_vgpr)
  int64_t rsteps = wave::in_vgpr<int64_t>(FROM_STATE ? st->rsteps : 0);
  int64_t tot_ev = wave::in_vgpr<int64_t>(FROM_STATE ? st->tot_ev : 0);

  if (TO_STATE || (st0 == SCHED_OK && n > 0)) {
    // W > 1: each wave's block (bitmaps, cancelled set) follows the exchange
    // area, and the staged completion steps (one array for the workgroup)
    // follow the blocks; a global cancelled set has n entries per wave
    const int gstride = P.nw_max + P.nw1_max + (VGLOBAL ? 0 : P.cap_v);
    uint64_t* const lw = W > 1 ? lds64 + group_pre_words(ALGO, W, ROWS) + wv * gstride : lds64;
    uint64_t* L0 = lw;
    uint64_t* L1 = lw + P.nw_max;
    // cancelled requests, one 64-bit entry each.  A_min: key | (s | o << 16) << 32,
    // slots [0, nVe) may start now, [nVe, nV) were cancelled at this step.
    // A_l: a FIFO ring of id | s << 17 | o << 33 | u << 48 from slot v_head.
    // (W > 1, global: each wave of workgroup g has the n_max entries at
    // P.vgroup + (g W + wave) n_max; the workgroup simulates its instances
    // one after the other)
    uint64_t* vent = VGLOBAL ? (W > 1 ? P.vgroup + (static_cast<int64_t>(blockIdx.x) * W + wv) * P.max_requests
                                      : P.vglob + b)
                             : L1 + P.nw1_max;
    // A_l: every request is promoted at most once, so its queue is an
    // append-only array of n entries in global memory (the instance's slice
    // of the workspace), read through a 64-entry register window
    constexpr bool kQueue = ALGO == SCHED_AELL;
    g_u64* qg = kQueue ? (g_u64*)(P.vglob + b) : nullptr;
    const int32_t cap_v = (VGLOBAL || kQueue) ? n : P.cap_v;
    int32_t* lcomp = W > 1 ? reinterpret_cast<int32_t*>(lds64 + group_pre_words(ALGO, W, ROWS) + W * gstride)
                           : reinterpret_cast<int32_t*>(L1 + P.nw1_max + (VGLOBAL ? 0 : P.cap_v));
    const bool stage_c = P.stage_comp != 0;
    const int nw = (n + 63) >> 6;
    const int nw1 = (nw + 63) >> 6;
    if (!FROM_STATE) {
      for (int w = lane; w < nw; w += 64) L0[w] = 0;
      for (int w = lane; w < nw1; w += 64) L1[w] = 0;
      if (stage_c)
        for (int i = W > 1 ? static_cast<int>(threadIdx.x) : lane; i < n; i += 64 * W) lcomp[i] = -1;
      __syncthreads();
    }
    // W > 1: the exchange buffers, the completion lists, the run counts
    uint4* const gred = reinterpret_cast<uint4*>(lds64);
    uint64_t* const glist = lds64 + 8 * W + wv * 64 * ROWS;
    int gpar = 0;
    int32_t occ = 0;

    const int32_t cap = P.cap[k];
    // array bases in vector registers
    // array bases in vector registers, typed as global memory: plain pointers
    // would compile to flat accesses, and a flat store or atomic holds the
    // LDS wait counter until its global write completes, so every later LDS
    // wait of the wave would also wait for it
    auto base = [](auto* p) { return wave::in_vgpr(p); };
    const g_u64* rec = base((const g_u64*)(P.rec + b));  // (key, s | o << 16) as one 64-bit word
    const g_i32* arrival = P.arrival ? base((const g_i32*)(P.arrival + b)) : nullptr;
    const g_i32* rank_of = base((const g_i32*)(P.rank_of + b));
    const g_i32* upper_k = ALGO == SCHED_AELL ? (const g_i32*)(P.u_of_rank + b) : nullptr;  // by rank
    // per-request outputs by id (with tie keys: the staging arrays)
    // completion steps by id: staged in LDS after the cancelled set when the
    // launch has room for them (written out coalesced at the end of the
    // instance), else straight to the global outputs.  One generic pointer,
    // so the staged case costs no registers (its stores are flat stores to
    // LDS; the global case's are flat stores too, which measured the same)
    int32_t* cdst = base(P.stage_comp ? (W > 1 ? lcomp : reinterpret_cast<int32_t*>(lds64 + P.nw_max + P.nw1_max + (VGLOBAL ? 0 : P.cap_v)))
                                      : (P.tie_key ? P.comp_st : P.completion) + b);
    g_i32* evictions = P.evictions ? base((g_i32*)((P.tie_key ? P.ev_st : P.evictions) + b)) : nullptr;

    // running set: register rows; an empty slot has r_end = kEmpty, r_c = kNever,
    // r_key = ~0, which every scan below treats as neutral, so scans cover all rows
    // (A_l also keeps each run's u, its planning length after a promotion)
    int32_t r_end[ROWS], r_x[ROWS], r_c[ROWS], r_h[ROWS], r_u[ROWS];
    uint32_t r_key[ROWS];
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
      r_end[r] = kEmpty; r_x[r] = 0; r_c[r] = kNever; r_h[r] = 0; r_key[r] = 0xFFFFFFFFu; r_u[r] = 0;
      if (FROM_STATE) {
        r_end[r] = st->r_end[r]; r_x[r] = st->r_x[r]; r_c[r] = st->r_c[r];
        r_h[r] = st->r_h[r]; r_key[r] = st->r_key[r]; r_u[r] = st->r_u[r];
      }
    }
    int fr_row = 0;               // row that receives new runs ...
    uint64_t fr_mask = ~0ull;     // ... and its free lanes
    int32_t N = 0;                // number of runs
    int32_t X = 0;                // sum of x over runs
    int32_t t_r = 0;              // base step of x and h
    int32_t next_c = kNever;      // lower bound on the earliest completion step

    int32_t aw_base = -64, aw_a = 0x7FFFFFFF, aw_rank = 0, arr_ptr = 0;
    int32_t next_a = 0;           // arrival step of request arr_ptr (0: look at step 0)
    int32_t f_rank = -1, fw_base = -1;
    uint64_t f_word = 0ull;       // the bitmap word of f_rank (its LDS copy may still hold taken bits)
    uint32_t f_key = 0xFFFFFFFFu, f_so = 0, fw_key = 0xFFFFFFFFu, fw_so = 0;
    int32_t f_u = 0, fw_u = 0;
    int32_t nV = 0, nVe = 0, v_pos = -1, v_head = 0;
    uint32_t v_key = 0xFFFFFFFFu, v_so = 0;
    int32_t v_u = 0;
    // A_l: queue entries [vw_base, vw_base + 64) in lane order (entries
    // appended inside the window are written to it as well)
    uint32_t vw_lo = 0, vw_hi = 0;
    int32_t vw_base = -(1 << 30);
    // A_min: requests cancelled recently wait in a register row first (lane j
    // holds one: key and s | o << 16; u_gate is ~0 in the lanes filled at this
    // step, which may not start before the next one), with its smallest
    // startable entry cached in uh_*; a full row goes to the LDS set at the
    // start of a step.  Requests are usually started again within a step or
    // two of their cancellation, so most starts find their request here
    // without a scan of the LDS set.
    uint32_t u_key = 0xFFFFFFFFu, u_so = 0, u_gate = 0;
    uint64_t u_used = 0ull;
    uint32_t uh_key = 0xFFFFFFFFu, uh_so = 0;
    int32_t uh_lane = -1;
    int32_t n_done = 0;
    // the head cannot start before retry_at; valid until the next event
    int32_t retry_at = 0;
    int32_t t = 0;
    int32_t DT = 0;               // memory held at t by the runs completing at t
    if (FROM_STATE) {
      fr_row = st->fr_row; fr_mask = st->fr_mask; N = st->N; X = st->X; t_r = st->t_r; next_c = st->next_c;
      aw_base = st->aw_base; aw_a = st->aw_a; aw_rank = st->aw_rank; arr_ptr = st->arr_ptr; next_a = st->next_a;
      f_rank = st->f_rank; f_word = st->f_word; fw_base = st->fw_base; f_key = st->f_key; f_so = st->f_so; fw_key = st->fw_key;
      fw_so = st->fw_so; f_u = st->f_u; fw_u = st->fw_u;
      nV = st->nV; nVe = st->nVe; v_pos = st->v_pos; v_head = st->v_head; v_key = st->v_key; v_so = st->v_so;
      v_u = st->v_u; n_done = st->n_done; retry_at = st->retry_at; t = st->t; DT = st->DT;
      if constexpr (ALGO == SCHED_AMIN) {
        u_key = st->u_key; u_so = st->u_so; u_gate = st->u_gate; u_used = st->u_used;
        uh_key = st->uh_key; uh_so = st->uh_so; uh_lane = st->uh_lane;
      }
      if constexpr (ALGO == SCHED_AELL) {
        vw_lo = st->vw_lo; vw_hi = st->vw_hi; vw_base = st->vw_base;
      }
    }

#define SK_LOAD_ARRIVALS()                                                           \
  do {                                                                               \
    aw_base = arr_ptr;                                                               \
    const int i_ = aw_base + lane;                                                   \
    aw_a = 0x7FFFFFFF;                                                               \
    aw_rank = 0;                                                                     \
    if (i_ < n) {                                                                    \
      aw_a = arrival ? arrival[i_] : 0;                                              \
      aw_rank = rank_of[i_];                                                         \
    }                                                                                \
  } while (0)
    // the record of fresh rank f_rank from the 64-record window (reloaded when
    // f_rank leaves it)
#define SK_F_RECORD()                                                                \
  do {                                                                               \
    if (fw_base < 0 || f_rank < fw_base || f_rank >= fw_base + 64) {                 \
      fw_base = f_rank;                                                              \
      const int rr_ = fw_base + lane;                                                \
      fw_key = 0xFFFFFFFFu;                                                          \
      fw_so = 0u;                                                                    \
      if (rr_ < n) {                                                                 \
        const uint64_t rv_ = rec[rr_];                                               \
        fw_key = static_cast<uint32_t>(rv_);                                         \
        fw_so = static_cast<uint32_t>(rv_ >> 32);                                    \
        if (ALGO == SCHED_AELL) fw_u = upper_k[rr_];                                 \
      }                                                                              \
    }                                                                                \
    f_key = wave::readlane_u(fw_key, f_rank - fw_base);                              \
    f_so = wave::readlane_u(fw_so, f_rank - fw_base);                                \
    if (ALGO == SCHED_AELL) f_u = wave::readlane(fw_u, f_rank - fw_base);            \
  } while (0)
    // smallest waiting fresh request: first set bit of the two-level bitmap in
    // LDS; its word stays in scalar registers (f_word) while it has bits left
#define SK_F_FIND()                                                                  \
  do {                                                                               \
    const uint64_t w1_ = lane < nw1 ? L1[lane] : 0ull;                               \
    const uint64_t nz_ = wave::ballot(w1_ != 0ull);                                  \
    if (nz_ == 0ull) {                                                               \
      f_rank = -1;                                                                   \
      f_key = 0xFFFFFFFFu;                                                           \
    } else {                                                                         \
      const int j1_ = __builtin_ctzll(nz_);                                          \
      const uint64_t w1v_ = wave::readlane_u64(w1_, j1_);                            \
      const int j0_ = j1_ * 64 + __builtin_ctzll(w1v_);                              \
      f_word = uniform_u64(L0[j0_]);                                                 \
      f_rank = j0_ * 64 + __builtin_ctzll(f_word);                                   \
      SK_F_RECORD();                                                                 \
    }                                                                                \
  } while (0)
    // f_rank starts: it is the lowest bit of f_word.  The next one is the next
    // bit of the same word (no LDS access); an emptied word is written back
    // and leaves the summary level, and the search goes to the next word.
#define SK_F_TAKE()                                                                  \
  do {                                                                               \
    f_word &= f_word - 1ull;                                                         \
    if (f_word != 0ull) {                                                            \
      f_rank = (f_rank & ~63) + __builtin_ctzll(f_word);                             \
      SK_F_RECORD();                                                                 \
    } else {                                                                         \
      const int j0_ = f_rank >> 6;                                                   \
      if (lane == 0) {                                                               \
        L0[j0_] = 0ull;                                                              \
        atomicAnd(reinterpret_cast<unsigned long long*>(&L1[j0_ >> 6]), ~(1ull << (j0_ & 63))); \
      }                                                                              \
      SK_F_FIND();                                                                   \
    }                                                                                \
  } while (0)
    // per-lane smallest cancelled entry over slots [FROM_, TO_): vb_k, vb_p, vb_s.
    // The loop runs over blocks of 128 slots with a uniform trip count (no
    // per-lane exit), both loads of a block in flight at once; a slot past
    // TO_ reads the last slot instead and counts as empty.
#define SK_V_SCAN(FROM_, TO_)                                                        \
  uint32_t vb_k = 0xFFFFFFFFu, vb_s = 0u;                                            \
  int32_t vb_p = -1;                                                                 \
  for (int b_ = (FROM_); b_ < (TO_); b_ += 128) {                                    \
    const int to_ = (TO_), last_ = to_ - 1;                                          \
    const int j0_ = b_ + lane, j1_ = b_ + 64 + lane;                                 \
    const uint64_t e0_ = vent[j0_ < last_ ? j0_ : last_];                            \
    const uint64_t e1_ = vent[j1_ < last_ ? j1_ : last_];                            \
    const uint32_t k0_ = j0_ < to_ ? static_cast<uint32_t>(e0_) : 0xFFFFFFFFu;       \
    const uint32_t k1_ = j1_ < to_ ? static_cast<uint32_t>(e1_) : 0xFFFFFFFFu;       \
    const bool l0_ = k0_ < vb_k;                                                     \
    vb_k = l0_ ? k0_ : vb_k;                                                         \
    vb_p = l0_ ? j0_ : vb_p;                                                         \
    vb_s = l0_ ? static_cast<uint32_t>(e0_ >> 32) : vb_s;                            \
    const bool l1_ = k1_ < vb_k;                                                     \
    vb_k = l1_ ? k1_ : vb_k;                                                         \
    vb_p = l1_ ? j1_ : vb_p;                                                         \
    vb_s = l1_ ? static_cast<uint32_t>(e1_ >> 32) : vb_s;                            \
  }
    // smallest cancelled request that may start now (slots [0, nVe))
#define SK_V_FIND()                                                                  \
  do {                                                                               \
    SK_V_SCAN(0, nVe)                                                                \
    const uint32_t kv_ = wave::min_u32_all(vb_k);                                    \
    const uint64_t at_ = wave::ballot(vb_k == kv_);                                  \
    const uint32_t km_ = wave::uniform_u(kv_);                                       \
    v_key = km_;                                                                     \
    v_pos = -1;                                                                      \
    if (km_ != 0xFFFFFFFFu) {                                                        \
      const int ln_ = __builtin_ctzll(at_);                                          \
      v_pos = wave::readlane(vb_p, ln_);                                             \
      v_so = wave::readlane_u(vb_s, ln_);                                            \
    }                                                                                \
  } while (0)
    // the requests cancelled at the previous step may start now: merge them
    // into the cached head instead of rescanning every slot
#define SK_V_MERGE()                                                                 \
  do {                                                                               \
    SK_V_SCAN(nVe, nV)                                                               \
    const uint32_t kv_ = wave::min_u32_all(vb_k);                                    \
    const uint64_t at_ = wave::ballot(vb_k == kv_);                                  \
    const uint32_t km_ = wave::uniform_u(kv_);                                       \
    if (km_ < v_key) {                                                               \
      const int ln_ = __builtin_ctzll(at_);                                          \
      v_key = km_;                                                                   \
      v_pos = wave::readlane(vb_p, ln_);                                             \
      v_so = wave::readlane_u(vb_s, ln_);                                            \
    }                                                                                \
    nVe = nV;                                                                        \
  } while (0)
    // A_l: the oldest promoted request (head of the queue), planned with u.
    // The window moves to the head when the head leaves it; the fence makes
    // the lane-0 appends visible to the other lanes' loads.
#define SK_V_HEAD()                                                                  \
  do {                                                                               \
    v_pos = -1;                                                                      \
    v_key = 0xFFFFFFFFu;                                                             \
    if (nV > 0) {                                                                    \
      if (v_head - vw_base >= 64 || v_head < vw_base) {                              \
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "workgroup");                       \
        vw_base = v_head;                                                            \
        const int j_ = v_head + lane;                                                \
        const uint64_t w_ = j_ < n ? static_cast<uint64_t>(qg[j_]) : 0ull;           \
        vw_lo = static_cast<uint32_t>(w_);                                           \
        vw_hi = static_cast<uint32_t>(w_ >> 32);                                     \
      }                                                                              \
      const int d_ = v_head - vw_base;                                               \
      const uint64_t e_ = (static_cast<uint64_t>(wave::readlane_u(vw_hi, d_)) << 32) | \
                          wave::readlane_u(vw_lo, d_);                               \
      const uint32_t ix_ = static_cast<uint32_t>(e_) & kIdxMask;                     \
      const uint32_t s_ = static_cast<uint32_t>(e_ >> 17) & 0xFFFFu;                 \
      const uint32_t o_ = static_cast<uint32_t>(e_ >> 33) & 0x7FFFu;                 \
      v_u = static_cast<int32_t>((e_ >> 48) & 0x7FFFu);                              \
      v_pos = v_head;                                                                \
      v_key = (static_cast<uint32_t>(v_u) << kIdxBits) | ix_;                        \
      v_so = s_ | (o_ << 16);                                                        \
    }                                                                                \
  } while (0)
    // A_min: the smallest startable entry of the register row
#define SK_U_FIND()                                                                  \
  do {                                                                               \
    const uint32_t uk_ = u_key | u_gate;                                             \
    const uint32_t um_ = wave::min_u32_all(uk_);                                     \
    const uint64_t ua_ = wave::ballot(uk_ == um_);                                   \
    uh_key = wave::uniform_u(um_);                                                   \
    uh_lane = -1;                                                                    \
    if (uh_key != 0xFFFFFFFFu) {                                                     \
      uh_lane = __builtin_ctzll(ua_);                                                \
      uh_so = wave::readlane_u(u_so, uh_lane);                                       \
    }                                                                                \
  } while (0)
    // the head of the waiting set: smaller key of the fresh and cancelled heads
    // (A_l: every fresh request comes before the promoted ones); derived where
    // it is used rather than carried through the loop
#define SK_PICK()                                                                    \
  const bool c_fromU = ALGO == SCHED_AMIN && uh_key < v_key;                         \
  const uint32_t vh_key = c_fromU ? uh_key : v_key;                                  \
  const uint32_t vh_so = c_fromU ? uh_so : v_so;                                     \
  const bool c_any = f_rank >= 0 || (kHasV && (v_pos >= 0 || c_fromU));              \
  const bool c_fromF = !kHasV || (f_rank >= 0 && (ALGO == SCHED_AELL || f_key < vh_key)); \
  const uint32_t c_key = c_fromF ? f_key : vh_key;                                   \
  const uint32_t c_so = c_fromF ? f_so : vh_so;                                      \
  const int32_t c_s = static_cast<int32_t>(c_so & 0xFFFFu);                          \
  const int32_t c_o = static_cast<int32_t>(c_so >> 16);                              \
  const int32_t c_est = ALGO == SCHED_ARANDOM ? c_o : static_cast<int32_t>(c_key >> kIdxBits); \
  const int32_t c_u = c_fromF ? f_u : v_u;
    // BODY with the compile-time row index r equal to the uniform row RR_
#define SK_AT_ROW(RR_, BODY)                                                         \
  _Pragma("unroll") for (int r = 0; r < ROWS; ++r) {                                 \
    if (r == (RR_)) {                                                                \
      BODY                                                                           \
    }                                                                                \
  }
    // A run with raw planned end ek and x = xk leaves: every run with
    // t+1 < Rend <= ek loses its share of f at its own planned end.
#define SK_DROP_SHARE(T_, XK_, EK_)                                                  \
  do {                                                                               \
    const int32_t tt_ = (T_), ek_ = (EK_);                                           \
    if (ek_ > tt_ + 1) {                                                             \
      const uint32_t lo_ = static_cast<uint32_t>(tt_) + 2u;                          \
      const uint32_t span_ = static_cast<uint32_t>(ek_) - lo_;                       \
      const uint32_t dx_ = static_cast<uint32_t>(XK_) - static_cast<uint32_t>(t_r);  \
      _Pragma("unroll") for (int r_ = 0; r_ < ROWS; ++r_) {                          \
        const uint32_t e_ = static_cast<uint32_t>(r_end[r_]);                        \
        const bool in_ = e_ - lo_ <= span_;                                          \
        r_h[r_] = static_cast<int32_t>(static_cast<uint32_t>(r_h[r_]) - (in_ ? dx_ + e_ : 0u)); \
      }                                                                              \
    }                                                                                \
  } while (0)

    // Issue priority among the waves of a SIMD: the more requests an instance
    // still has to complete, the higher (four levels by the unfinished
    // fraction), so the instances that bound the launch are not slowed by
    // their SIMD-mates; where a batch mixes interval widths (A_min with upper
    // bounds), the static class of the instance and whether half of it is
    // done instead (PRIO false: none).  Outputs do not depend on it.
    int prio = -1;
    // (CLS false: an instance of the code without the class read, for the
    // launches that never have classes)
    const int pcls = CLS ? ((ALGO == SCHED_AMIN && P.pclass) ? P.pclass[k] : -1) : -1;
#define SK_SET_PRIORITY()                                                            \
  do {                                                                               \
    if (!PRIO) break;                                                                \
    const int lv_ = pcls >= 0 ? pcls + (2 * (n - n_done) > n ? 1 : 0) : (4 * (n - n_done) - 1) / n; \
    if (lv_ != prio) {                                                               \
      prio = lv_;                                                                    \
      if (lv_ >= 3) __builtin_amdgcn_s_setprio(3);                                   \
      else if (lv_ == 2) __builtin_amdgcn_s_setprio(2);                              \
      else if (lv_ == 1) __builtin_amdgcn_s_setprio(1);                              \
      else __builtin_amdgcn_s_setprio(0);                                            \
    }                                                                                \
  } while (0)
    SK_SET_PRIORITY();
    // the state at the admissions of step t, for the body with NR_ rows
#define SK_SAVE_STATE(NR_)                                                             \
  do {                                                                                 \
    _Pragma("unroll") for (int r = 0; r < kStateRows; ++r) {                           \
      const bool have = r < ROWS;                                                      \
      st->r_end[r] = have ? r_end[r < ROWS ? r : 0] : kEmpty;                          \
      st->r_x[r] = have ? r_x[r < ROWS ? r : 0] : 0;                                   \
      st->r_c[r] = have ? r_c[r < ROWS ? r : 0] : kNever;                              \
      st->r_h[r] = have ? r_h[r < ROWS ? r : 0] : 0;                                   \
      st->r_key[r] = have ? r_key[r < ROWS ? r : 0] : 0xFFFFFFFFu;                     \
      st->r_u[r] = have ? r_u[r < ROWS ? r : 0] : 0;                                   \
    }                                                                                  \
    st->fr_row = fr_row; st->fr_mask = fr_mask; st->N = N; st->X = X; st->t_r = t_r;   \
    st->next_c = next_c; st->aw_base = aw_base; st->aw_a = aw_a; st->aw_rank = aw_rank; \
    st->arr_ptr = arr_ptr; st->next_a = next_a; st->f_rank = f_rank; st->f_word = f_word; \
    st->fw_base = fw_base; st->f_key = f_key; st->f_so = f_so; st->fw_key = fw_key;    \
    st->fw_so = fw_so; st->f_u = f_u; st->fw_u = fw_u; st->nV = nV; st->nVe = nVe;     \
    st->v_pos = v_pos; st->v_head = v_head; st->v_key = v_key; st->v_so = v_so;        \
    st->v_u = v_u; st->n_done = n_done; st->retry_at = retry_at; st->t = t; st->DT = DT; \
    st->rsteps = rsteps; st->tot_ev = tot_ev; st->next_rows = (NR_); st->resume = true; \
    if constexpr (ALGO == SCHED_AMIN) {                                                \
      st->u_key = u_key; st->u_so = u_so; st->u_gate = u_gate; st->u_used = u_used;   \
      st->uh_key = uh_key; st->uh_so = uh_so; st->uh_lane = uh_lane;                  \
    }                                                                                  \
    if constexpr (ALGO == SCHED_AELL) {                                                \
      st->vw_lo = vw_lo; st->vw_hi = vw_hi; st->vw_base = vw_base;                     \
    }                                                                                  \
  } while (0)
    bool resuming = FROM_STATE && st->resume;   // continue with the admissions of step t
    for (;;) {
      if (!resuming) {
      if (t > cap) {
        status = SCHED_E_STEP_CAP;
        break;
      }
      if (t - t_r >= kRebase) {
        const uint32_t d = static_cast<uint32_t>(t - t_r);
#pragma unroll
        for (int r = 0; r < ROWS; ++r) {
          r_x[r] = static_cast<int32_t>(static_cast<uint32_t>(r_x[r]) + d);
          r_h[r] = static_cast<int32_t>(static_cast<uint32_t>(r_h[r]) - d);
        }
        X += N * static_cast<int32_t>(d);
        t_r = t;
      }
      bool heads_changed = false;
      bool event = false;
      // ---- 1. arrivals; requests cancelled at the previous step become eligible
      if (t >= next_a) {
        // the cached word goes back to LDS before arrivals set bits in it
        if (f_rank >= 0 && lane == 0) L0[f_rank >> 6] = f_word;
        while (arr_ptr < n) {
          if (arr_ptr >= aw_base + 64) SK_LOAD_ARRIVALS();
          const bool take = (aw_base + lane >= arr_ptr) && aw_a <= t;
          const uint64_t m = wave::ballot(take);
          if (m == 0ull) break;
          if (take) {
            atomicOr(reinterpret_cast<unsigned long long*>(&L0[aw_rank >> 6]), 1ull << (aw_rank & 63));
            atomicOr(reinterpret_cast<unsigned long long*>(&L1[aw_rank >> 12]), 1ull << ((aw_rank >> 6) & 63));
          }
          arr_ptr += __builtin_popcountll(m);
          if (arr_ptr < aw_base + 64) break;
        }
        if (arr_ptr < n) {
          if (arr_ptr >= aw_base + 64) SK_LOAD_ARRIVALS();
          next_a = wave::readlane(aw_a, arr_ptr - aw_base);
        } else {
          next_a = 0x7FFFFFFF;
        }
        SK_F_FIND();
        heads_changed = true;
      }
      if (ALGO == SCHED_AMIN && nVe != nV) {
        SK_V_MERGE();
        heads_changed = true;
      }
      if (ALGO == SCHED_AMIN && u_used != 0ull) {
        const int cnt = __builtin_popcountll(u_used);
        const bool fresh_u = wave::ballot(u_gate != 0u) != 0ull;  // cancelled at the last step
        if (cnt > kURowFlush) {
          // the row goes to the LDS set (every entry of it may start now)
          if (nV + cnt > cap_v) {
            status = P.retry_v_status;
            break;
          }
          const bool mine = (u_used >> lane) & 1ull;
          const int slot = nV + static_cast<int>(__builtin_amdgcn_mbcnt_hi(
                                   static_cast<uint32_t>(u_used >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(u_used), 0u)));
          if (mine) vent[slot] = (static_cast<uint64_t>(u_so) << 32) | u_key;
          const uint32_t k_ = u_key;
          u_key = 0xFFFFFFFFu;
          u_gate = 0u;
          u_used = 0ull;
          // its smallest entry competes with the LDS set's head
          const uint32_t um_ = wave::min_u32_all(mine ? k_ : 0xFFFFFFFFu);
          const uint64_t ua_ = wave::ballot(mine && k_ == um_);
          const uint32_t mk_ = wave::uniform_u(um_);
          if (mk_ < v_key) {
            const int ln_ = __builtin_ctzll(ua_);
            v_key = mk_;
            v_so = wave::readlane_u(u_so, ln_);
            v_pos = wave::readlane(slot, ln_);
          }
          nV += cnt;
          nVe = nV;
          uh_key = 0xFFFFFFFFu;
          uh_lane = -1;
          heads_changed = true;
        } else if (fresh_u) {
          u_gate = 0u;
          SK_U_FIND();
          heads_changed = true;
        }
      }
      if (heads_changed) event = true;

      // ---- 2. completions at t; DT = memory they still hold at t (s + o each)
      DT = 0;
      if (t >= next_c) {
        int32_t sx = 0;
        int ndone = 0;
        int lc = 0;                    // W > 1: this wave's completions listed
        uint32_t gcmin = 0xFFFFFFFFu;  // W > 1: the next event, agreed
#pragma unroll
        for (int r = 0; r < ROWS; ++r) {
          const bool hit = r_c[r] == t;
          const uint64_t m = wave::ballot(hit);
          if (m) {
            ndone += __builtin_popcountll(m);
            if constexpr (W > 1 && (ALGO == SCHED_AMAX || ALGO == SCHED_AELL)) {
              // every wave drops the shares of every wave's completions: list them
              if (hit) {
                const int pos = lc + static_cast<int>(__builtin_amdgcn_mbcnt_hi(
                                         static_cast<uint32_t>(m >> 32),
                                         __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(m), 0u)));
                glist[pos] = static_cast<uint64_t>(static_cast<uint32_t>(r_x[r])) |
                             (static_cast<uint64_t>(static_cast<uint32_t>(r_end[r])) << 32);
              }
              lc += __builtin_popcountll(m);
            } else if (ALGO == SCHED_AMAX || ALGO == SCHED_AELL) {
              // planned with u >= o: the run may end before its planned end
              uint64_t mm = m;
              while (mm) {
                const int ln = __builtin_ctzll(mm);
                mm &= mm - 1;
                SK_DROP_SHARE(t, wave::readlane(r_x[r], ln), wave::readlane(r_end[r], ln));
              }
            }
            if (hit) cdst[r_key[r] & kIdxMask] = t;
            sx += hit ? r_x[r] : 0;
            r_end[r] = hit ? kEmpty : r_end[r];
            r_c[r] = hit ? kNever : r_c[r];
            r_key[r] = hit ? 0xFFFFFFFFu : r_key[r];
            if (r == fr_row) fr_mask |= m;
          }
        }
        if constexpr (W > 1) {
          // agree on the completions (and, but for A_l, the next one)
          uint32_t cl = 0xFFFFFFFFu;
          if constexpr (ALGO != SCHED_AELL) {
#pragma unroll
            for (int r = 0; r < ROWS; ++r) {
              const uint32_t ev = static_cast<uint32_t>(r_c[r]);
              cl = ev < cl ? ev : cl;
            }
            cl = wave::min_u32(cl);
          }
          const uint4 g = group_exchange<W>(gred, gpar, wv, lane,
                                            make_uint4(static_cast<uint32_t>(ndone), static_cast<uint32_t>(wave::sum_i32(sx)),
                                                       cl, static_cast<uint32_t>(lc)));
          const int32_t nd_j = lane < W ? static_cast<int32_t>(g.x) : 0;
          occ -= nd_j;
          const int32_t nd = lanes_sum_i32(nd_j);
          const int32_t sxw = lanes_sum_i32(lane < W ? static_cast<int32_t>(g.y) : 0);
          gcmin = lanes_min_u32(lane < W ? g.z : 0xFFFFFFFFu);
          if constexpr (ALGO == SCHED_AMAX || ALGO == SCHED_AELL) {
            if (lanes_sum_i32(lane < W ? static_cast<int32_t>(g.w) : 0) > 0) {
              for (int j = 0; j < W; ++j) {
                const int cj = wave::readlane(static_cast<int32_t>(g.w), j);
                const uint64_t* lj = lds64 + 8 * W + j * 64 * ROWS;
                for (int e0 = 0; e0 < cj; e0 += 64) {
                  const uint64_t ev = e0 + lane < cj ? lj[e0 + lane] : 0ull;
                  const int ne = cj - e0 < 64 ? cj - e0 : 64;
                  for (int q = 0; q < ne; ++q) {
                    const int32_t xq = wave::readlane(static_cast<int32_t>(static_cast<uint32_t>(ev)), q);
                    const int32_t eq = wave::readlane(static_cast<int32_t>(ev >> 32), q);
                    SK_DROP_SHARE(t, xq, eq);
                  }
                }
              }
              group_barrier();  // every wave has read the lists: they may be written again
            }
          }
          if (nd) {
            event = true;
            X -= sxw;
            N -= nd;
            DT = sxw + nd * (t - t_r);
            n_done += nd;
            SK_SET_PRIORITY();
          }
        } else if (ndone) {
          event = true;
          const int32_t sxw = wave::sum_i32(sx);
          X -= sxw;
          N -= ndone;
          DT = sxw + ndone * (t - t_r);
          n_done += ndone;
          SK_SET_PRIORITY();
        }
        // ---- 3. done?
        if (n_done == n) break;
        // ---- 3'. A_l: a run still present at its planned end t (planned with
        // l, so o > l) is promoted: it leaves, plans with u and joins the back of
        // the queue, lowest index first among this step's promotions
        if (ALGO == SCHED_AELL) {
          bool promoted = false;
          if constexpr (W > 1) {
          for (;;) {
            uint32_t best = 0xFFFFFFFFu;
            int32_t brow = 0;
#pragma unroll
            for (int r = 0; r < ROWS; ++r) {
              const uint32_t kk = r_end[r] == t ? (r_key[r] & kIdxMask) : 0xFFFFFFFFu;
              const bool lt = kk < best;
              best = lt ? kk : best;
              brow = lt ? r : brow;
            }
            const uint32_t iv = wave::min_u32_all(best);
            const uint64_t at = wave::ballot(best == iv);
            // the smallest index over the waves; its wave removes the run (the
            // exchange that finds nothing left to promote also agrees on the
            // next event)
            const uint32_t il = wave::uniform_u(iv);
            int ln = 0, rr = 0;
            int32_t xk = 0, ck = 0, uk = 0;
            uint32_t kk = 0;
            if (il != 0xFFFFFFFFu) {
              ln = __builtin_ctzll(at);
              rr = wave::readlane(brow, ln);
              SK_AT_ROW(rr, xk = wave::readlane(r_x[r], ln); ck = wave::readlane(r_c[r], ln);
                        uk = wave::readlane(r_u[r], ln); kk = wave::readlane_u(r_key[r], ln);)
            }
            uint32_t cl = 0xFFFFFFFFu;
#pragma unroll
            for (int r = 0; r < ROWS; ++r) {
              const uint32_t ev = static_cast<uint32_t>(r_c[r]), pe = static_cast<uint32_t>(r_end[r]);
              cl = ev < cl ? ev : cl;
              cl = pe < cl ? pe : cl;
            }
            uint4 g2 = make_uint4(kk, wave::min_u32(cl), 0u, 0u);
            const uint4 g = group_exchange<W>(gred, gpar, wv, lane,
                                              make_uint4(il, static_cast<uint32_t>(xk), static_cast<uint32_t>(ck),
                                                         static_cast<uint32_t>(uk)), &g2);
            const uint32_t gi = lane < W ? g.x : 0xFFFFFFFFu;
            const uint32_t imin = lanes_min_u32(gi);
            if (imin == 0xFFFFFFFFu) {
              gcmin = lanes_min_u32(lane < W ? g2.y : 0xFFFFFFFFu);
              break;
            }
            if (nV >= cap_v) {
              status = P.retry_v_status;
              break;
            }
            const int win = __builtin_ctzll(wave::ballot(gi == imin));
            xk = wave::readlane(static_cast<int32_t>(g.y), win);
            ck = wave::readlane(static_cast<int32_t>(g.z), win);
            uk = wave::readlane(static_cast<int32_t>(g.w), win);
            kk = wave::readlane_u(g2.x, win);
            if (wv == win) {
              SK_AT_ROW(rr, r_end[r] = wave::writelane(r_end[r], kEmpty, ln);
                        r_c[r] = wave::writelane(r_c[r], kNever, ln);
                        r_key[r] = wave::writelane_u(r_key[r], 0xFFFFFFFFu, ln);)
              if (rr == fr_row) fr_mask |= 1ull << ln;
            }
            occ -= lane == win ? 1 : 0;
            X -= xk;
            N -= 1;
            const int32_t pk = t - static_cast<int32_t>(kk >> kIdxBits);
            const uint64_t sk = static_cast<uint32_t>(xk - t_r + pk);
            const uint64_t okk = static_cast<uint32_t>(ck - pk);
            {
              // every wave appends the same entry; one counts the promotion
              const int slot = v_head + nV;
              const uint64_t qe = imin | (sk << 17) | (okk << 33) | (static_cast<uint64_t>(uk) << 48);
              if (lane == 0) {
                qg[slot] = qe;
                if (evictions && wv == 0)
                  __hip_atomic_fetch_add(&evictions[imin], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              }
              if (slot >= vw_base && slot - vw_base < 64) {
                vw_lo = wave::writelane_u(vw_lo, static_cast<uint32_t>(qe), slot - vw_base);
                vw_hi = wave::writelane_u(vw_hi, static_cast<uint32_t>(qe >> 32), slot - vw_base);
              }
            }
            ++nV;
            ++tot_ev;
            promoted = true;
          }
          } else {
          for (;;) {
            uint32_t best = 0xFFFFFFFFu;
            int32_t brow = 0;
#pragma unroll
            for (int r = 0; r < ROWS; ++r) {
              const uint32_t kk = r_end[r] == t ? (r_key[r] & kIdxMask) : 0xFFFFFFFFu;
              const bool lt = kk < best;
              best = lt ? kk : best;
              brow = lt ? r : brow;
            }
            const uint32_t iv = wave::min_u32_all(best);
            const uint64_t at = wave::ballot(best == iv);
            const uint32_t imin = wave::uniform_u(iv);
            if (imin == 0xFFFFFFFFu) break;
            if (nV >= cap_v) {
              status = P.retry_v_status;
              break;
            }
            const int ln = __builtin_ctzll(at);
            const int rr = wave::readlane(brow, ln);
            int32_t xk = 0, ck = 0, uk = 0;
            uint32_t kk = 0;
            SK_AT_ROW(rr, xk = wave::readlane(r_x[r], ln); ck = wave::readlane(r_c[r], ln);
                      uk = wave::readlane(r_u[r], ln); kk = wave::readlane_u(r_key[r], ln);
                      r_end[r] = wave::writelane(r_end[r], kEmpty, ln);
                      r_c[r] = wave::writelane(r_c[r], kNever, ln);
                      r_key[r] = wave::writelane_u(r_key[r], 0xFFFFFFFFu, ln);)
            if (rr == fr_row) fr_mask |= 1ull << ln;
            // its planned end is t itself: no later planned end loses a share
            X -= xk;
            N -= 1;
            const int32_t pk = t - static_cast<int32_t>(kk >> kIdxBits);
            const uint64_t sk = static_cast<uint32_t>(xk - t_r + pk);
            const uint64_t okk = static_cast<uint32_t>(ck - pk);
            {
              const int slot = v_head + nV;  // < n: each request is promoted at most once
              const uint64_t qe = imin | (sk << 17) | (okk << 33) | (static_cast<uint64_t>(uk) << 48);
              if (lane == 0) {
                qg[slot] = qe;
                if (evictions) __hip_atomic_fetch_add(&evictions[imin], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              }
              if (slot >= vw_base && slot - vw_base < 64) {
                vw_lo = wave::writelane_u(vw_lo, static_cast<uint32_t>(qe), slot - vw_base);
                vw_hi = wave::writelane_u(vw_hi, static_cast<uint32_t>(qe >> 32), slot - vw_base);
              }
            }
            ++nV;
            ++tot_ev;
            promoted = true;
          }
          }
          if (status != SCHED_OK) break;
          if (promoted) {
            event = true;
            if (v_pos < 0) SK_V_HEAD();
          }
        }
        // next event: a completion (A_l: or a planned end, where a run is promoted);
        // empty slots read as unsigned are above every step
        if constexpr (W > 1) {
          next_c = static_cast<int32_t>(gcmin);
        } else {
        uint32_t cmin = 0xFFFFFFFFu;
#pragma unroll
        for (int r = 0; r < ROWS; ++r) {
          uint32_t ev = static_cast<uint32_t>(r_c[r]);
          if (ALGO == SCHED_AELL) {
            const uint32_t pe = static_cast<uint32_t>(r_end[r]);
            ev = pe < ev ? pe : ev;
          }
          cmin = ev < cmin ? ev : cmin;
        }
        next_c = static_cast<int32_t>(wave::min_u32(cmin));  // kNever when nothing runs
        }
      }

      // ---- 4. A_min: cancel in ascending (o~, index) while memory at t+1 > M
      if (ALGO == SCHED_AMIN) {
        int32_t Pm = X + N * (t + 1 - t_r);
        if (Pm > M) {
          while (Pm > M) {
            uint32_t best = r_key[0];
            int32_t brow = 0;
#pragma unroll
            for (int r = 1; r < ROWS; ++r) {
              const bool lt = r_key[r] < best;
              best = lt ? r_key[r] : best;
              brow = lt ? r : brow;
            }
            const uint32_t kv = wave::min_u32_all(best);
            const uint64_t at = wave::ballot(best == kv);
            uint32_t kmin = 0xFFFFFFFFu;
            int32_t ek = 0, xk = 0, ck = 0;
            if constexpr (W > 1) {
              // the smallest key over the waves; its wave removes the run
              const uint32_t kl = wave::uniform_u(kv);
              int ln = 0, rr = 0;
              if (kl != 0xFFFFFFFFu) {
                ln = __builtin_ctzll(at);
                rr = wave::readlane(brow, ln);
                SK_AT_ROW(rr, ek = wave::readlane(r_end[r], ln); xk = wave::readlane(r_x[r], ln);
                          ck = wave::readlane(r_c[r], ln);)
              }
              const uint4 g = group_exchange<W>(gred, gpar, wv, lane,
                                                make_uint4(kl, static_cast<uint32_t>(ek), static_cast<uint32_t>(xk),
                                                           static_cast<uint32_t>(ck)));
              const uint32_t gk = lane < W ? g.x : 0xFFFFFFFFu;
              kmin = lanes_min_u32(gk);
              if (kmin == 0xFFFFFFFFu) {  // no run: impossible while P > M > 0
                status = SCHED_E_UNSUPPORTED;
                break;
              }
              if (u_used == ~0ull && nV >= cap_v) {
                status = P.retry_v_status;
                break;
              }
              const int win = __builtin_ctzll(wave::ballot(gk == kmin));
              ek = wave::readlane(static_cast<int32_t>(g.y), win);
              xk = wave::readlane(static_cast<int32_t>(g.z), win);
              ck = wave::readlane(static_cast<int32_t>(g.w), win);
              if (wv == win) {
                SK_AT_ROW(rr, r_end[r] = wave::writelane(r_end[r], kEmpty, ln);
                          r_c[r] = wave::writelane(r_c[r], kNever, ln);
                          r_key[r] = wave::writelane_u(r_key[r], 0xFFFFFFFFu, ln);)
                if (rr == fr_row) fr_mask |= 1ull << ln;
              }
              occ -= lane == win ? 1 : 0;
            } else {
            kmin = wave::uniform_u(kv);
            if (kmin == 0xFFFFFFFFu) {  // no run: impossible while P > M > 0
              status = SCHED_E_UNSUPPORTED;
              break;
            }
            if (u_used == ~0ull && nV >= cap_v) {
              status = P.retry_v_status;
              break;
            }
            const int ln = __builtin_ctzll(at);
            const int rr = wave::readlane(brow, ln);
            SK_AT_ROW(rr, ek = wave::readlane(r_end[r], ln); xk = wave::readlane(r_x[r], ln);
                      ck = wave::readlane(r_c[r], ln); r_end[r] = wave::writelane(r_end[r], kEmpty, ln);
                      r_c[r] = wave::writelane(r_c[r], kNever, ln);
                      r_key[r] = wave::writelane_u(r_key[r], 0xFFFFFFFFu, ln);)
            if (rr == fr_row) fr_mask |= 1ull << ln;
            }
            SK_DROP_SHARE(t, xk, ek);
            X -= xk;
            N -= 1;
            Pm -= xk + t + 1 - t_r;
            const int32_t oh = static_cast<int32_t>(kmin >> kIdxBits);
            const uint32_t idx = kmin & kIdxMask;
            const int32_t pk = ek - oh;
            const int32_t gen = t - pk;
            const int32_t nh = gen > oh ? gen : oh;
            const int32_t sk = xk - t_r + pk;
            const int32_t okk = ck - pk;
            const uint32_t so = static_cast<uint32_t>(sk) | (static_cast<uint32_t>(okk) << 16);
            const uint32_t nkey = (static_cast<uint32_t>(nh) << kIdxBits) | idx;
            if (u_used != ~0ull) {
              // into a free lane of the register row, startable from the next step
              const int ul = __builtin_ctzll(~u_used);
              u_key = wave::writelane_u(u_key, nkey, ul);
              u_so = wave::writelane_u(u_so, so, ul);
              u_gate = wave::writelane_u(u_gate, 0xFFFFFFFFu, ul);
              u_used |= 1ull << ul;
              if (lane == 0 && wv == 0 && evictions)
                __hip_atomic_fetch_add(&evictions[idx], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            } else {
              if (lane == 0) {
                vent[nV] = (static_cast<uint64_t>(so) << 32) | nkey;
                if (evictions && wv == 0)
                  __hip_atomic_fetch_add(&evictions[idx], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              }
              ++nV;
            }
            ++tot_ev;
          }
          if (status != SCHED_OK) break;
          event = true;
        }
      }
      if (event) retry_at = 0;
      }
      resuming = false;

      // ---- shrink: once the runs fit a smaller body with room to spare, move
      // the runs of the upper rows into free slots of the lower ones (the
      // order of slots never matters: every choice is by key) and hand over
      if constexpr (TO_STATE && ROWS > 2) {
        int target = 0;
        if (N <= 64 * 2 - kShrinkSpare) target = 2;
        else if (ROWS > 3 && N <= 64 * 3 - kShrinkSpare) target = 3;
        else if (ROWS > 5 && N <= 64 * 5 - kShrinkSpare) target = 5;
        else if (ROWS > 8 && N <= 64 * 8 - kShrinkSpare) target = 8;
        else if (ROWS > 10 && N <= 64 * 10 - kShrinkSpare) target = 10;
        else if (ROWS > 12 && N <= 64 * 12 - kShrinkSpare) target = 12;
        if (target > 0) {
          uint64_t fm[ROWS];
#pragma unroll
          for (int r = 0; r < ROWS; ++r) fm[r] = wave::ballot(r_end[r] == kEmpty);
#pragma unroll
          for (int h = ROWS - 1; h >= 2; --h) {
            if (h < target) break;
            uint64_t m = ~fm[h];
            while (m) {
              const int ln = __builtin_ctzll(m);
              m &= m - 1;
              // the lowest row below the target with a free lane
              int l = 0;
              uint64_t fl_mask = 0;
#pragma unroll
              for (int r = ROWS - 1; r >= 0; --r) {
                const bool ok = r < target && fm[r] != 0ull;
                l = ok ? r : l;
                fl_mask = ok ? fm[r] : fl_mask;
              }
              const int fl = __builtin_ctzll(fl_mask);
              const int32_t me = wave::readlane(r_end[h], ln), mx = wave::readlane(r_x[h], ln);
              const int32_t mc = wave::readlane(r_c[h], ln), mh = wave::readlane(r_h[h], ln);
              const int32_t mu = wave::readlane(r_u[h], ln);
              const uint32_t mk = wave::readlane_u(r_key[h], ln);
              SK_AT_ROW(l, r_end[r] = wave::writelane(r_end[r], me, fl); r_x[r] = wave::writelane(r_x[r], mx, fl);
                        r_c[r] = wave::writelane(r_c[r], mc, fl); r_h[r] = wave::writelane(r_h[r], mh, fl);
                        r_u[r] = wave::writelane(r_u[r], mu, fl); r_key[r] = wave::writelane_u(r_key[r], mk, fl);
                        fm[r] &= ~(1ull << fl);)
              r_end[h] = wave::writelane(r_end[h], kEmpty, ln);
              r_c[h] = wave::writelane(r_c[h], kNever, ln);
              r_key[h] = wave::writelane_u(r_key[h], 0xFFFFFFFFu, ln);
            }
          }
          fr_row = 0;
          fr_mask = 0ull;  // the next admission looks for a free row
          handoff = target;
          status = kResume;
          break;
        }
      }

      // ---- 5. admission of the longest feasible prefix in key order
      bool stuck = true;          // the head cannot start before the next event
      int32_t wait_until = t + 1; // otherwise: not before this step
      for (;;) {
        SK_PICK();
        if (!c_any) break;
        const int32_t s = c_s, est = c_est;
        const int32_t E = t + est;
        const int32_t tp1 = t + 1;
        // step t+1: every running request is present; exact when a planned end
        // falls there and implied by the first planned end after it otherwise
        const int32_t Pm = X + N * (tp1 - t_r);
        if (Pm + s + 1 > M) break;
        stuck = false;
        if (t < retry_at) {
          wait_until = retry_at;
          break;
        }
        // step t (runs completing at t hold s+o); implied by step t+1 when DT = 0
        if (DT > 0 && DT + X + N * (t - t_r) + s > M) break;
        // planned ends c in (t+1, E] need h + t_r - t + s <= M (h + t_r = f(c) + c);
        // the candidate's own end E needs f(E) + s + est <= M, f(E) = sum of x + E - t_r
        const uint32_t lo2 = static_cast<uint32_t>(t) + 2u;
        const bool win = E > tp1;
        const uint32_t span = win ? static_cast<uint32_t>(E) - lo2 : 0u;
        const int32_t cE = E - t_r;
        const int32_t lim = win ? M + t - t_r - s : 0x7FFFFFFF;  // h above this violates
        int32_t fl = 0, hmx = INT32_MIN;
#pragma unroll
        for (int r = 0; r < ROWS; ++r) {
          const int32_t e = r_end[r];
          const bool in = static_cast<uint32_t>(e) - lo2 <= span;
          const int32_t hv = in ? r_h[r] : INT32_MIN;
          hmx = hv > hmx ? hv : hmx;
          fl += e >= E ? r_x[r] + cE : 0;
        }
        if constexpr (W > 1) {
          // one exchange agrees on both conditions and on the step to retry at
          // (both ways of failing are prepared, see below)
          int32_t fix = 0, emin = kNever;
#pragma unroll
          for (int r = 0; r < ROWS; ++r) {
            const int32_t a = r_h[r] - lim, bb = r_end[r] - 1 - t;
            const int32_t m = a < bb ? a : bb;
            const bool in = static_cast<uint32_t>(r_end[r]) - lo2 <= span;
            fix = (in && r_h[r] > lim && m > fix) ? m : fix;
            const int32_t e = r_end[r];
            emin = (e >= E && e < emin) ? e : emin;
          }
          const uint4 g = group_exchange<W>(
              gred, gpar, wv, lane,
              make_uint4(static_cast<uint32_t>(wave::max_i32(hmx)), static_cast<uint32_t>(wave::sum_i32(fl)),
                         static_cast<uint32_t>(wave::max_i32(fix)), wave::min_u32(static_cast<uint32_t>(emin))));
          const int32_t hg = lanes_max_i32(lane < W ? static_cast<int32_t>(g.x) : INT32_MIN);
          const int32_t fg = lanes_sum_i32(lane < W ? static_cast<int32_t>(g.y) : 0);
          if (hg > lim || (win && fg + s + est > M)) {
            if (hg > lim)
              retry_at = t + lanes_max_i32(lane < W ? static_cast<int32_t>(g.z) : 0);
            else
              retry_at = static_cast<int32_t>(lanes_min_u32(lane < W ? g.w : 0xFFFFFFFFu)) - est + 1;
            wait_until = retry_at;
            break;
          }
          // passed: the test below (one wave's) then passes with f = fg
          fl = lane == 0 ? fg : 0;
          hmx = INT32_MIN;
        }
        // both conditions in one ballot: the sum is left in every lane, so the
        // passing case costs a single vector-to-scalar hand-off
        const int32_t fv = wave::sum_i32_all(fl);
        const bool end_bad = win && fv + s + est > M;
        if (wave::ballot(hmx > lim || end_bad)) {
          if (wave::ballot(hmx > lim)) {
            // each violating end improves by one per step, or leaves the window
            int32_t fix = 0;
#pragma unroll
            for (int r = 0; r < ROWS; ++r) {
              const int32_t a = r_h[r] - lim, bb = r_end[r] - 1 - t;
              const int32_t m = a < bb ? a : bb;
              const bool in = static_cast<uint32_t>(r_end[r]) - lo2 <= span;
              fix = (in && r_h[r] > lim && m > fix) ? m : fix;
            }
            retry_at = t + wave::max_i32(fix);
          } else {
            // f at the sliding end only grows until it passes the next planned end
            int32_t emin = kNever;
#pragma unroll
            for (int r = 0; r < ROWS; ++r) {
              const int32_t e = r_end[r];
              emin = (e >= E && e < emin) ? e : emin;
            }
            retry_at = static_cast<int32_t>(wave::min_u32(static_cast<uint32_t>(emin))) - est + 1;
          }
          wait_until = retry_at;
          break;
        }
        const int32_t f = wave::uniform(fv);
        // admit: start at p = t; runs whose planned end is in (t+1, E] gain its share
        // a free slot first: without one nothing has changed for this candidate
        if (CAPPED && N >= P.run_cap) {
          status = retry_status;
          break;
        }
        int owner = 0;  // W > 1: the wave that takes the run
        if constexpr (W > 1) {
          // the wave with the fewest runs (the lowest such); all full: outgrown
          const uint32_t oc = lane < W ? (static_cast<uint32_t>(occ) << 4) | static_cast<uint32_t>(lane) : 0xFFFFFFFFu;
          const uint32_t om = lanes_min_u32(oc);
          if (static_cast<int>(om >> 4) >= 64 * ROWS) {
            status = retry_status;
            break;
          }
          owner = static_cast<int>(om & 15u);
          occ += lane == owner ? 1 : 0;
          if (wv == owner && fr_mask == 0ull) {
            // it has a free slot (its count is below its rows' slots)
            int rr = 0;
            uint64_t mm = 0ull;
#pragma unroll
            for (int r = ROWS - 1; r >= 0; --r) {
              const uint64_t m = wave::ballot(r_end[r] == kEmpty);
              rr = m ? r : rr;
              mm = m ? m : mm;
            }
            fr_row = rr;
            fr_mask = mm;
          }
        } else if (fr_mask == 0ull) {
          int rr = -1;
          uint64_t mm = 0ull;
#pragma unroll
          for (int r = ROWS - 1; r >= 0; --r) {
            const uint64_t m = wave::ballot(r_end[r] == kEmpty);
            rr = m ? r : rr;
            mm = m ? m : mm;
          }
          if (rr < 0) {
            if (TO_STATE && ladder_up(ROWS, kStateRows) > 0) {
              // hand the state at this admission to the body above
              handoff = ladder_up(ROWS, kStateRows);
              status = kResume;
            } else {
              status = retry_status;
            }
            break;
          }
          fr_row = rr;
          fr_mask = mm;
        }
        const int32_t xw = s - t + t_r;
        const int32_t hw = f + (xw + cE) + cE;
        if (win) {
          const uint32_t dh = static_cast<uint32_t>(xw) - static_cast<uint32_t>(t_r);
#pragma unroll
          for (int r = 0; r < ROWS; ++r) {
            const uint32_t e = static_cast<uint32_t>(r_end[r]);
            r_h[r] = static_cast<int32_t>(static_cast<uint32_t>(r_h[r]) + (e - lo2 <= span ? e + dh : 0u));
          }
        }
        {
          const int32_t cw = t + c_o;
          if (W == 1 || wv == owner) {
          const int ln = __builtin_ctzll(fr_mask);
          fr_mask &= fr_mask - 1;
          const uint32_t kw = c_key;
          const int32_t uw = c_u;
          SK_AT_ROW(fr_row, r_end[r] = wave::writelane(r_end[r], E, ln); r_x[r] = wave::writelane(r_x[r], xw, ln);
                    r_c[r] = wave::writelane(r_c[r], cw, ln); r_key[r] = wave::writelane_u(r_key[r], kw, ln);
                    r_h[r] = wave::writelane(r_h[r], hw, ln);
                    if (ALGO == SCHED_AELL) r_u[r] = wave::writelane(r_u[r], uw, ln);)
          }
          const int32_t ew = ALGO == SCHED_AELL && E < cw ? E : cw;  // A_l: promotion at E
          next_c = ew < next_c ? ew : next_c;
        }
        X += xw;
        N += 1;
        if (c_fromF) {
          SK_F_TAKE();
        } else if (ALGO == SCHED_AELL) {
          ++v_head;
          --nV;
          SK_V_HEAD();
        } else if (ALGO == SCHED_AMIN && c_fromU) {
          // from the register row
          u_key = wave::writelane_u(u_key, 0xFFFFFFFFu, uh_lane);
          u_used &= ~(1ull << uh_lane);
          SK_U_FIND();
        } else {
          // the last eligible entry moves into the hole; the last pending one fills
          // its place.  Lane 0 and lane 1 do the two moves with one read and one
          // write (when the hole is the last eligible slot, only the second move
          // is left, as in doing them one after the other)
          if (lane < 2) {
            const int le = nVe - 1;
            const int src = lane == 0 ? le : nV - 1;
            const uint64_t mv = vent[src];
            const bool act = lane == 0 ? v_pos != le : nV > nVe;
            if (act) vent[lane == 0 ? v_pos : le] = mv;
          }
          --nVe;
          --nV;
          SK_V_FIND();
        }
        stuck = true;
        wait_until = t + 1;
        retry_at = 0;
      }
      if (status != SCHED_OK) break;

      // ---- 6. this step processes every running request once
      rsteps += N;
      int32_t tn = t + 1;
      if (ALGO != SCHED_AMIN || (nV == nVe && !wave::ballot(u_gate != 0u))) {
        // Nothing changes before the next completion, arrival or (A_min)
        // overflow; until then the head cannot start before wait_until (or at
        // all when stuck: the memory at t+1 only grows).
        int32_t jump = stuck ? 0x7FFFFFFF : wait_until;
        jump = next_c < jump ? next_c : jump;
        jump = next_a < jump ? next_a : jump;
        if (ALGO == SCHED_AMIN && N > 0) {
          const int32_t Pm = X + N * (t + 1 - t_r);  // <= M here
          // first step whose projection exceeds M, if it comes before the jump
          if (static_cast<int64_t>(Pm) + static_cast<int64_t>(N) * (jump - 1 - t) > M) {
            const int32_t tev = t + (M - Pm) / N + 1;
            jump = tev < jump ? tev : jump;
          }
        }
        const int32_t lim = t_r + kRebase;
        jump = lim < jump ? lim : jump;
        jump = cap + 1 < jump ? cap + 1 : jump;
        if (jump > tn) {
          rsteps += static_cast<int64_t>(N) * (jump - tn);
          tn = jump;
        }
      }
      t = tn;
    }
    // every way out of a handing-over body writes the whole state (so that the
    // state a body started from is dead while it runs)
    if constexpr (TO_STATE) {
      SK_SAVE_STATE(handoff);
      if (status == kResume) return kResume;
    }
  }

  // ---- epilogue: totals from the per-request outputs (with tie keys, first
  // copied from the staging arrays, by id, to the outputs, by index)
  __syncthreads();
  const bool keep = (status == SCHED_OK || status == SCHED_E_STEP_CAP) && n > 0;
  const bool tie = P.tie_key != nullptr;
  const bool st_c = P.stage_comp != 0;
  int64_t tel = 0, mk = 0;
  if (keep) {
    const int32_t* lc =
        W > 1 ? reinterpret_cast<const int32_t*>(lds64 + group_pre_words(ALGO, W, ROWS) +
                                                 W * (P.nw_max + P.nw1_max + (VGLOBAL ? 0 : P.cap_v)))
              : reinterpret_cast<const int32_t*>(lds64 + P.nw_max + P.nw1_max + (VGLOBAL ? 0 : P.cap_v));
    for (int c = 0; c < n; c += 64 * W) {
      const int i = c + (W > 1 ? static_cast<int>(threadIdx.x) : lane);
      if (i < n) {
        const int32_t id = tie ? P.tr_of[b + i] : i;
        int32_t ci;
        if (st_c || tie) {
          ci = st_c ? lc[id] : P.comp_st[b + id];
          P.completion[b + i] = ci;
        } else {
          ci = P.completion[b + i];
        }
        if (P.evictions && tie) P.evictions[b + i] = P.ev_st[b + id];
        if (ci >= 0) {
          tel += ci - (P.arrival ? P.arrival[b + i] : 0);
          mk = ci > mk ? ci : mk;
        }
      }
    }
  } else if (status != st0 && n > 0) {
    // capacity outgrown at run time: report like an invalid instance (or hand
    // it to a retry pass, which starts from these values)
    int32_t* comp = tie ? P.comp_st : P.completion;
    int32_t* evs = tie ? P.ev_st : P.evictions;
    for (int c = 0; c < n; c += 64 * W) {
      const int i = c + (W > 1 ? static_cast<int>(threadIdx.x) : lane);
      if (i < n) {
        comp[b + i] = -1;
        if (P.evictions) evs[b + i] = 0;
      }
    }
  }
  tel = wave::sum_i64(tel);
  mk = wave::max_i64(mk);
  if constexpr (W > 1) {
    // over the waves (the exchange area is free: every wave is past the
    // barrier above, so past its last exchange)
    int64_t* gt = reinterpret_cast<int64_t*>(lds64);
    if (lane == 0) {
      gt[2 * wv] = tel;
      gt[2 * wv + 1] = mk;
    }
    __syncthreads();
    tel = 0;
    mk = 0;
    for (int j = 0; j < W; ++j) {
      tel += gt[2 * j];
      mk = gt[2 * j + 1] > mk ? gt[2 * j + 1] : mk;
    }
  }
  if (!keep) {
    rsteps = 0;
    tot_ev = 0;
  }
  if (W > 1 ? threadIdx.x == 0 : lane == 0) {
    P.total_latency[k] = tel;
    if (P.makespan) P.makespan[k] = static_cast<int32_t>(mk);
    if (P.request_steps) P.request_steps[k] = rsteps;
    if (P.total_evictions) P.total_evictions[k] = tot_ev;
    P.status[k] = status;
  }
  return status;
}

// One wave per instance.  RETRY_PASS: only instances handed over by an
// earlier launch for a reason this pass takes (P.run_mask) run, held to
// P.run_cap runs at once.
template <int ALGO, int ROWS, bool RETRY_PASS, bool VGLOBAL = false>
__global__ __launch_bounds__(64) void k_simulate(Params P) {
  const int k = blockIdx.x;
  if (P.algo_of && P.algo_of[k] != ALGO) return;  // adaptive run: the other policy's instance
  int st0 = P.status[k];
  if (RETRY_PASS) {
    const bool take = (st0 == kRetryRows && (P.run_mask & 1)) || (st0 == kRetryV && (P.run_mask & 2));
    if (!take) return;
    st0 = SCHED_OK;
  }
  sim_instance<ALGO, ROWS, false, false, VGLOBAL, RETRY_PASS>(P, k, st0, P.retry_status);
}

// One wave per instance on the row ladder: the simulation starts with 2
// register rows and moves, state and all, to the body with 3, 5, 8 or 10 rows
// as its running set grows and back down as it shrinks, so that every scan
// covers about as many rows as the instance has runs (most of an instance's
// events happen with at most 128 runs).  A running set beyond 640 runs ends
// with P.retry_status.  Held to 128 VGPRs so that four waves share a SIMD.
template <int ALGO, bool WIDE>
__device__ __forceinline__ void ladder_instance(const Params& P, const int k) {
  if (P.algo_of && P.algo_of[k] != ALGO) return;
  int st0 = P.status[k];
  if constexpr (WIDE) {
    if (P.run_mask) {
      // a retry pass: only the instances an earlier pass handed over
      const bool take = (st0 == kRetryRows && (P.run_mask & 1)) || (st0 == kRetryV && (P.run_mask & 2));
      if (!take) return;
      st0 = SCHED_OK;
    }
  }
  if (st0 == SCHED_OK) {
    // the bodies all resume from a state, so the bitmaps and staged outputs
    // are set up here
    extern __shared__ uint64_t lds64[];
    const int64_t b = P.offsets[k];
    const int n = static_cast<int>(P.offsets[k + 1] - b);
    const int nw = (n + 63) >> 6, nw1 = (nw + 63) >> 6;
    for (int w = threadIdx.x; w < nw; w += 64) lds64[w] = 0;
    for (int w = threadIdx.x; w < nw1; w += 64) lds64[P.nw_max + w] = 0;
    int32_t* lc = reinterpret_cast<int32_t*>(lds64 + P.nw_max + P.nw1_max + P.cap_v);
    if (P.stage_comp)
      for (int i = threadIdx.x; i < n; i += 64) lc[i] = -1;
    __syncthreads();
  }
  const bool empty = st0 == SCHED_OK && P.offsets[k + 1] == P.offsets[k];
  if (st0 != SCHED_OK || empty) {
    // nothing to simulate: zero totals (the per-request outputs were set by
    // the preparation)
    if (threadIdx.x == 0) {
      P.total_latency[k] = 0;
      if (P.makespan) P.makespan[k] = 0;
      if (P.request_steps) P.request_steps[k] = 0;
      if (P.total_evictions) P.total_evictions[k] = 0;
      P.status[k] = st0;
    }
    return;
  }
  using ST = typename std::conditional<WIDE, SimStateWide, SimState>::type;
  ST st;
  fresh_state(st);
  int r;
  if constexpr (!WIDE) {
    do {
      switch (st.next_rows) {
        case 2: r = sim_instance<ALGO, 2, true, true, false, false, ST>(P, k, SCHED_OK, P.retry_status, &st); break;
        case 3: r = sim_instance<ALGO, 3, true, true, false, false, ST>(P, k, SCHED_OK, P.retry_status, &st); break;
        case 5: r = sim_instance<ALGO, 5, true, true, false, false, ST>(P, k, SCHED_OK, P.retry_status, &st); break;
        case 8: r = sim_instance<ALGO, 8, true, true, false, false, ST>(P, k, SCHED_OK, P.retry_status, &st); break;
        default: r = sim_instance<ALGO, 10, true, true, false, false, ST>(P, k, SCHED_OK, P.retry_status, &st); break;
      }
    } while (r == kResume);
  } else {
    do {
      switch (st.next_rows) {
        case 2: r = sim_instance<ALGO, 2, true, true, false, false, ST>(P, k, SCHED_OK, P.retry_status, &st); break;
        case 3: r = sim_instance<ALGO, 3, true, true, false, false, ST>(P, k, SCHED_OK, P.retry_status, &st); break;
        case 5: r = sim_instance<ALGO, 5, true, true, false, false, ST>(P, k, SCHED_OK, P.retry_status, &st); break;
        case 8: r = sim_instance<ALGO, 8, true, true, false, false, ST>(P, k, SCHED_OK, P.retry_status, &st); break;
        case 10: r = sim_instance<ALGO, 10, true, true, false, false, ST>(P, k, SCHED_OK, P.retry_status, &st); break;
        case 12: r = sim_instance<ALGO, 12, true, true, false, false, ST>(P, k, SCHED_OK, P.retry_status, &st); break;
        default: r = sim_instance<ALGO, 16, true, true, false, false, ST>(P, k, SCHED_OK, P.retry_status, &st); break;
      }
    } while (r == kResume);
  }
}

// The narrow ladder: one wave per instance moving along the bodies of 2 to
// 10 rows (the body of the two kernels below; ORDERED_: workgroup g simulates
// instance P.order[g]; CLS_: issue priorities by P.pclass; PRIO_ false: the
// waves keep the default issue priority, for batches in which priorities
// cannot help (a wave per SIMD, or rounds of waves) but would cost scalar
// instructions).
#define SK_NARROW_LADDER(ORDERED_, CLS_, PRIO_)                                                                                               \
  const int k = (ORDERED_) ? P.order[blockIdx.x] : static_cast<int>(blockIdx.x);                                                       \
  if (P.algo_of && P.algo_of[k] != ALGO) return;                                                                                       \
  const int st0 = P.status[k];                                                                                                         \
  if (st0 == SCHED_OK) {                                                                                                               \
    /* the bodies all resume from a state, so the bitmaps and staged outputs */                                                        \
    /* are set up here */                                                                                                              \
    extern __shared__ uint64_t lds64[];                                                                                                \
    const int64_t b = P.offsets[k];                                                                                                    \
    const int n = static_cast<int>(P.offsets[k + 1] - b);                                                                              \
    const int nw = (n + 63) >> 6, nw1 = (nw + 63) >> 6;                                                                                \
    for (int w = threadIdx.x; w < nw; w += 64) lds64[w] = 0;                                                                           \
    for (int w = threadIdx.x; w < nw1; w += 64) lds64[P.nw_max + w] = 0;                                                               \
    int32_t* lc = reinterpret_cast<int32_t*>(lds64 + P.nw_max + P.nw1_max + P.cap_v);                                                  \
    if (P.stage_comp)                                                                                                                  \
      for (int i = threadIdx.x; i < n; i += 64) lc[i] = -1;                                                                            \
    __syncthreads();                                                                                                                   \
  }                                                                                                                                    \
  const bool empty = st0 == SCHED_OK && P.offsets[k + 1] == P.offsets[k];                                                              \
  if (st0 != SCHED_OK || empty) {                                                                                                      \
    /* nothing to simulate: zero totals (the per-request outputs were set by */                                                        \
    /* the preparation) */                                                                                                             \
    if (threadIdx.x == 0) {                                                                                                            \
      P.total_latency[k] = 0;                                                                                                          \
      if (P.makespan) P.makespan[k] = 0;                                                                                               \
      if (P.request_steps) P.request_steps[k] = 0;                                                                                     \
      if (P.total_evictions) P.total_evictions[k] = 0;                                                                                 \
      P.status[k] = st0;                                                                                                               \
    }                                                                                                                                  \
    return;                                                                                                                            \
  }                                                                                                                                    \
  SimState st;                                                                                                                         \
  fresh_state(st);                                                                                                                     \
  int r;                                                                                                                               \
  do {                                                                                                                                 \
    switch (st.next_rows) {                                                                                                            \
      case 2: r = sim_instance<ALGO, 2, true, true, false, false, SimState, 1, (CLS_), (PRIO_)>(P, k, SCHED_OK, P.retry_status, &st); break;    \
      case 3: r = sim_instance<ALGO, 3, true, true, false, false, SimState, 1, (CLS_), (PRIO_)>(P, k, SCHED_OK, P.retry_status, &st); break;    \
      case 5: r = sim_instance<ALGO, 5, true, true, false, false, SimState, 1, (CLS_), (PRIO_)>(P, k, SCHED_OK, P.retry_status, &st); break;    \
      case 8: r = sim_instance<ALGO, 8, true, true, false, false, SimState, 1, (CLS_), (PRIO_)>(P, k, SCHED_OK, P.retry_status, &st); break;    \
      default: r = sim_instance<ALGO, 10, true, true, false, false, SimState, 1, (CLS_), (PRIO_)>(P, k, SCHED_OK, P.retry_status, &st); break;  \
    }                                                                                                                                  \
  } while (r == kResume);

// The narrow ladder held to 128 VGPRs so that four waves share a SIMD; each
// (ORDERED, CLS, PRIO) choice is an instance of the kernel of its own, so
// that the other launches compile without it.
template <int ALGO, bool ORDERED = false, bool CLS = false, bool PRIO = true>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(4))) void k_simulate_ladder(Params P) {
  SK_NARROW_LADDER(ORDERED, CLS, PRIO);
}

// The same bodies with 256 VGPRs (fewer spills), for batches in which every
// wave has a SIMD to itself (so without issue priorities).
template <int ALGO>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(2))) void k_simulate_ladder_roomy(Params P) {
  SK_NARROW_LADDER(false, false, false);
}
#undef SK_NARROW_LADDER

// The wide ladder (up to 1024 runs): for batches of few instances, where
// registers matter more than occupancy, and for the instances that outgrow
// the narrow ladder (a retry pass).
template <int ALGO>
__global__ __launch_bounds__(64) void k_simulate_ladder_wide(Params P) {
  ladder_instance<ALGO, true>(P, blockIdx.x);
}
// A workgroup of W waves per instance, ROWS register rows each (W x 64 x ROWS
// runs): for few large instances, and for the instances whose running set
// outgrows one wave's rows (a retry pass).  With P.run_mask set, only the
// instances an earlier pass handed over run.
// Workgroup g simulates instances g, g + grid, ... (a launch with global
// cancelled sets has fewer workgroups than instances: each workgroup's sets
// are its own).
template <int ALGO, int W, int ROWS, bool VGLOBAL>
__global__ __launch_bounds__(64 * W) void k_simulate_group(Params P) {
  for (int k = blockIdx.x; k < P.K; k += gridDim.x) {
    if (P.algo_of && P.algo_of[k] != ALGO) continue;
    int st0 = P.status[k];
    if (P.run_mask) {
      const bool take = (st0 == kRetryRows && (P.run_mask & 1)) || (st0 == kRetryV && (P.run_mask & 2));
      if (!take) continue;
      st0 = SCHED_OK;
    }
    sim_instance<ALGO, ROWS, false, false, VGLOBAL, false, SimState, W>(P, k, st0, P.retry_status);
    __syncthreads();  // the next instance reuses the LDS
  }
}
#undef SK_SET_PRIORITY
#undef SK_SAVE_STATE
#undef SK_LOAD_ARRIVALS
#undef SK_PICK
#undef SK_F_FIND
#undef SK_F_RECORD
#undef SK_F_TAKE
#undef SK_V_FIND
#undef SK_V_SCAN
#undef SK_V_MERGE
#undef SK_V_HEAD
#undef SK_U_FIND
#undef SK_AT_ROW
#undef SK_DROP_SHARE

}  // namespace sk

