// opt_kernels.hip -- gfx950 kernels of the hindsight optimum on tiny instances.
//
// The hindsight optimum (the OPT of the competitive analysis, Section 2) is
// the minimum total latency (equation (3)) over every non-preemptive schedule
// that knows the true output lengths: request i starts at some p_i >= a_i,
// holds s_i + (tau - p_i) tokens for tau in [p_i, p_i + o_i], and the total
// may never exceed M (equation (1)).  A wave searches one instance (n <= 8)
// by depth-first branch and bound over start steps in request order:
//   * at every node the 64 lanes test 64 consecutive starts of the next
//     request at once; a ballot gives the feasible ones and the wave descends
//     into them in order, so the wave follows one path of the tree (no lane
//     divergence) and visits the nodes one lane would, in the same order;
//   * a start is feasible iff the total stays <= M at the completion step of
//     every placed run that overlaps the new one and at the new run's own
//     completion (between two completions the set of present runs only grows
//     and each run's memory grows, so the maximum is at a completion).  The
//     memory at each placed run's completion is kept up to date as runs are
//     placed and removed, so a test costs O(depth);
//   * each depth is its own template instance, so every index into the search
//     state is a compile-time constant and the state stays in registers;
//   * the cost of a partial assignment plus the remaining requests' output
//     lengths bounds any completion from below, and the cost grows with the
//     start, so the first start that reaches the best total ends the level;
//   * the first bound is the caller's (a known schedule's total, e.g. a
//     policy's) or else the schedule that runs the requests one at a time;
//   * requests are searched by arrival, then by decreasing s + o and o, and a
//     request identical to the previous one never starts before it (swapping
//     them gives the same schedule);
//   * starts range over [a_i, max a + sum(o + 1) + 1], a horizon within which
//     the sequential schedule already finishes every request (an instance
//     whose horizon reaches 2^27 is not searched: SCHED_E_UNSUPPORTED).
// A first launch gives every instance one wave and a short node budget.  The
// instances it leaves unfinished are listed, and a second launch of as many
// 16-wave workgroups as the device holds at once searches them together: the
// pieces of an instance (the subtrees below the starts of its first two
// requests) are claimed one at a time from a counter in global memory, so
// every workgroup that has finished its own instance joins the ones still
// open and the hardest instance ends up spread over the whole device.  The
// best total of an instance is kept in global memory (exchanged at every
// claim) and in LDS for the waves of a workgroup (read at every chunk of
// starts).  Node budgets guarantee every wave reaches the exit.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "schedsim.h"

namespace opt {

constexpr int kMaxN = 8;
// starts, ends and memory sums are int32: the horizon (max a + sum(o + 1) + 1)
// must stay below this
constexpr int64_t kHorizonLimit = int64_t(1) << 27;

struct OptParams {
  int32_t K;
  int64_t N;
  const int64_t* offsets;
  const int32_t* arrival;
  const int32_t* prompt;
  const int32_t* output;
  int32_t M;
  int64_t node_cap;
  const int64_t* upper_bound;
  int64_t* total_latency;
  int32_t* status;
  int64_t* nodes;
  int32_t unfinished;       // first launch: status of an instance not finished within node_cap
  // second launch: [0] the number U of unfinished instances, then four arrays
  // of K entries: the instances, their piece counters, best totals and flags
  // (bit 0: every piece claimed; bit 1: a wave ran out of nodes)
  int32_t* pool;
};

// status of an instance left to the second launch
constexpr int kSplit = -100;
// nodes of the first launch (one wave per instance)
constexpr int64_t kFirstPassNodes = int64_t(1) << 17;
// waves of a second-launch workgroup, and the depth below which they split
constexpr int kGroupWaves = 16;
constexpr int kSplitDepth = 2;
constexpr int kFlagClaimed = 1, kFlagStop = 2;

// One instance, sorted into search order.
struct Inst {
  int32_t a[kMaxN], s[kMaxN], o[kMaxN];
  int32_t rem[kMaxN + 1];   // rem[i] = o[i] + ... + o[n-1]
  uint32_t same;            // bit i: request i equals request i-1
  int n;
  int32_t M;
  int32_t horizon;          // < kHorizonLimit
};

// The search state.  mem[q] is the memory at the completion step of placed
// run q from every run placed so far (kept exact as runs are placed and
// removed), so testing a start costs O(depth).  Runs are kept by completion
// step (a start is c - o).
struct Search {
  int32_t c[kMaxN];         // completion step p + o of each placed run
  int32_t mem[kMaxN];
  int32_t best;             // below 8 * kHorizonLimit = 2^30
  int32_t nodes, cap;       // the budget is clamped to 2^31 - 1
  bool stop;
};

// The search below a node at depth D (runs 0..D-1 placed at total cost
// `cost`), the lanes of the wave testing 64 starts at a time.  SHARED: the
// best total is also shared with the other waves of the workgroup through *sb
// (read at every chunk of starts, lowered whenever this wave improves it).
// Nodes are counted per start tested.
template <int D, bool SHARED>
__device__ __forceinline__ void wplace(const Inst& I, Search& S, int32_t cost, int lane, int32_t* sb) {
  if constexpr (D < kMaxN) {
    const int32_t lo = (D > 0 && ((I.same >> D) & 1u)) ? S.c[D > 0 ? D - 1 : 0] - I.o[D > 0 ? D - 1 : 0] : I.a[D];
    for (int32_t base = lo; base <= I.horizon; base += 64) {
      if constexpr (SHARED) {
        const int32_t g = __hip_atomic_load(sb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        S.best = g < S.best ? g : S.best;
      }
      const int32_t pd = base + lane;
      const int32_t c = cost + (pd + I.o[D] - I.a[D]);
      const bool live = pd <= I.horizon && c + I.rem[D + 1] < S.best;
      const int32_t end = pd + I.o[D];
      bool ok = live;
      int32_t mend = I.s[D] + I.o[D];
#pragma unroll
      for (int q = 0; q < D; ++q) {
        const int32_t cq = S.c[q], pq = cq - I.o[q];
        if (cq >= pd && cq <= end) ok = ok && S.mem[q] + I.s[D] + (cq - pd) <= I.M;
        if (pq <= end && end <= cq) mend += I.s[q] + (end - pq);
      }
      ok = ok && mend <= I.M;
      uint64_t m = __builtin_amdgcn_ballot_w64(ok);
      const uint64_t lv = __builtin_amdgcn_ballot_w64(live);
      S.nodes += __builtin_popcountll(lv) + (lv != ~0ull ? 1 : 0);
      if (S.nodes > S.cap) {
        S.stop = true;
        return;
      }
      while (m) {
        const int j = __builtin_ctzll(m);
        m &= m - 1;
        const int32_t pj = base + j;
        const int32_t cj = cost + (pj + I.o[D] - I.a[D]);
        if (cj + I.rem[D + 1] >= S.best) return;  // the bound improved below an earlier start
        if (D == I.n - 1) {
          S.best = cj;  // a complete schedule; later starts here cost more
          if constexpr (SHARED) {
            if (lane == 0) atomicMin(sb, cj);
          }
          return;
        }
        const int32_t ej = pj + I.o[D];
        const int32_t mj = __builtin_amdgcn_readlane(mend, j);
        S.c[D] = ej;
#pragma unroll
        for (int q = 0; q < D; ++q) {
          const int32_t cq = S.c[q];
          if (cq >= pj && cq <= ej) S.mem[q] += I.s[D] + (cq - pj);
        }
        S.mem[D] = mj;
        wplace<D + 1, SHARED>(I, S, cj, lane, sb);
#pragma unroll
        for (int q = 0; q < D; ++q) {
          const int32_t cq = S.c[q];
          if (cq >= pj && cq <= ej) S.mem[q] -= I.s[D] + (cq - pj);
        }
        if (S.stop) return;
      }
      if (lv != ~0ull) return;
    }
  }
}

// The first kSplitDepth levels for the waves that share an instance: every
// wave walks the same feasible starts of the first kSplitDepth requests
// (without the bound's pruning, so that the walk, and the numbering of its
// leaves, is the same in every wave) and searches below the leaves it claims:
// a wave claims the next unclaimed leaf from the instance's counter in global
// memory (*cnt) whenever it has searched below its last one, and at every
// claim trades best totals with the instance's global best (*gb) and its
// workgroup's (*sb).
template <int D>
__device__ __forceinline__ void wtop(const Inst& I, Search& S, int32_t cost, int lane, int32_t* sb, int32_t* cnt,
                                     int32_t* gb, int32_t& leaf, int32_t& claim) {
  const int32_t lo = (D > 0 && ((I.same >> D) & 1u)) ? S.c[D > 0 ? D - 1 : 0] - I.o[D > 0 ? D - 1 : 0] : I.a[D];
  for (int32_t pd = lo; pd <= I.horizon; ++pd) {
    ++S.nodes;
    const int32_t c = cost + (pd + I.o[D] - I.a[D]);
    const int32_t end = pd + I.o[D];
    bool ok = true;
    int32_t mend = I.s[D] + I.o[D];
#pragma unroll
    for (int r = 0; r < D; ++r) {
      const int32_t cr = S.c[r], pr = cr - I.o[r];
      if (cr >= pd && cr <= end) ok = ok && S.mem[r] + I.s[D] + (cr - pd) <= I.M;
      if (pr <= end && end <= cr) mend += I.s[r] + (end - pr);
    }
    if (!ok || mend > I.M) continue;
    if (D == I.n - 1) {
      // a complete schedule above the split (n <= kSplitDepth): the same in every wave
      S.best = c < S.best ? c : S.best;
      return;
    }
    S.c[D] = end;
#pragma unroll
    for (int r = 0; r < D; ++r) {
      const int32_t cr = S.c[r];
      if (cr >= pd && cr <= end) S.mem[r] += I.s[D] + (cr - pd);
    }
    S.mem[D] = mend;
    if constexpr (D == kSplitDepth - 1) {
      if (leaf == claim) {
        const int32_t g = __hip_atomic_load(sb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        S.best = g < S.best ? g : S.best;
        if (c + I.rem[D + 1] < S.best) wplace<D + 1, true>(I, S, c, lane, sb);
        int32_t nx = 0, gbv = 0;
        if (lane == 0) {
          nx = atomicAdd(cnt, 1);
          gbv = atomicMin(gb, S.best);
        }
        claim = __builtin_amdgcn_readfirstlane(nx);
        gbv = __builtin_amdgcn_readfirstlane(gbv);
        if (gbv < S.best) S.best = gbv;
        if (lane == 0) atomicMin(sb, S.best);
      }
      ++leaf;
    } else {
      wtop<D + 1>(I, S, c, lane, sb, cnt, gb, leaf, claim);
    }
#pragma unroll
    for (int r = 0; r < D; ++r) {
      const int32_t cr = S.c[r];
      if (cr >= pd && cr <= end) S.mem[r] -= I.s[D] + (cr - pd);
    }
    if (S.stop) return;
  }
}

// Validates instance k and brings it into search order (I), with the first
// bound in S.best; returns its status.
__device__ __forceinline__ int setup(const OptParams& P, const int k, Inst& I, Search& S) {
  const int64_t b = P.offsets[k];
  const int64_t e = P.offsets[k + 1];
  int status = SCHED_OK;
  S.best = 0;
  if (b < 0 || e < b || e > P.N) status = SCHED_E_INVAL;
  const int n = status == SCHED_OK ? static_cast<int>(e - b) : 0;
  if (n > kMaxN) status = SCHED_E_UNSUPPORTED;
  I.n = n;
  I.M = P.M;
  if (status == SCHED_OK && n > 0) {
    bool arr_bad = false, int_bad = false, big_bad = false;
    int64_t amax = 0, span = 0;
#pragma unroll
    for (int i = 0; i < kMaxN; ++i) {
      I.a[i] = 0; I.s[i] = 0; I.o[i] = 1;
      if (i < n) {
        I.a[i] = P.arrival ? P.arrival[b + i] : 0;
        I.s[i] = P.prompt[b + i];
        I.o[i] = P.output[b + i];
        if (I.a[i] < 0 || (i > 0 && I.a[i] < I.a[i > 0 ? i - 1 : 0])) arr_bad = true;
        if (I.o[i] < 1 || I.s[i] < 0) int_bad = true;
        if (static_cast<int64_t>(I.s[i]) + I.o[i] > P.M) big_bad = true;
        amax = I.a[i] > amax ? I.a[i] : amax;
        span += static_cast<int64_t>(I.o[i]) + 1;
      }
    }
    status = arr_bad ? SCHED_E_ARRIVAL : int_bad ? SCHED_E_INTERVAL : big_bad ? SCHED_E_TOO_BIG : SCHED_OK;
    if (status == SCHED_OK && amax + span + 1 >= kHorizonLimit) status = SCHED_E_UNSUPPORTED;
    if (status == SCHED_OK) {
      I.horizon = static_cast<int32_t>(amax + span + 1);
      // first bound: one request at a time, each after the previous completes
      int32_t t = 0;
#pragma unroll
      for (int i = 0; i < kMaxN; ++i)
        if (i < n) {
          const int32_t start = t > I.a[i] ? t : I.a[i];
          S.best += start + I.o[i] - I.a[i];
          t = start + I.o[i] + 1;
        }
      if (P.upper_bound && P.upper_bound[k] > 0 && P.upper_bound[k] < S.best)
        S.best = static_cast<int32_t>(P.upper_bound[k]);
      // search order: arrival, then the largest s + o, then the longest o
      // first (big runs placed early prune the most); the optimum does not
      // depend on it, and equal keys mean identical requests.  A fixed
      // compare-exchange network over the first n slots (odd-even
      // transposition, n passes) keeps every index static.
#pragma unroll
      for (int pass = 0; pass < kMaxN; ++pass)
#pragma unroll
        for (int j = pass & 1; j + 1 < kMaxN; j += 2)
          if (j + 1 < n) {
            const int32_t wj = I.s[j + 1] + I.o[j + 1], wp = I.s[j] + I.o[j];
            const bool gt = I.a[j] > I.a[j + 1] ||
                            (I.a[j] == I.a[j + 1] && (wp < wj || (wp == wj && I.o[j] < I.o[j + 1])));
            if (gt) {
              const int32_t ta = I.a[j + 1], ts = I.s[j + 1], to = I.o[j + 1];
              I.a[j + 1] = I.a[j]; I.s[j + 1] = I.s[j]; I.o[j + 1] = I.o[j];
              I.a[j] = ta; I.s[j] = ts; I.o[j] = to;
            }
          }
      I.rem[kMaxN] = 0;
#pragma unroll
      for (int i = kMaxN - 1; i >= 0; --i) I.rem[i] = I.rem[i + 1] + (i < n ? I.o[i] : 0);
      I.same = 0u;
#pragma unroll
      for (int i = 1; i < kMaxN; ++i)
        if (i < n && I.a[i] == I.a[i - 1] && I.s[i] == I.s[i - 1] && I.o[i] == I.o[i - 1]) I.same |= 1u << i;
#pragma unroll
      for (int i = 0; i < kMaxN; ++i) {
        S.c[i] = 0;
        S.mem[i] = 0;
      }
    }
  }
  return status;
}

// First launch: one wave per instance, at most P.node_cap nodes; an instance
// not finished within them gets P.unfinished (the second launch's mark, with
// the best total found as its bound, or SCHED_E_STEP_CAP).
__global__ __launch_bounds__(64) void k_optimum(OptParams P) {
  const int k = blockIdx.x;
  const int lane = static_cast<int>(threadIdx.x);
  Search S;
  S.nodes = 0;
  S.cap = static_cast<int32_t>(P.node_cap < 0x7FFFFFFF ? P.node_cap : 0x7FFFFFFF);
  S.stop = false;
  Inst I;
  int status = setup(P, k, I, S);
  if (status == SCHED_OK && I.n > 0) {
    wplace<0, false>(I, S, 0, lane, nullptr);
    if (S.stop) status = P.unfinished;
  }
  if (status != SCHED_OK && status != SCHED_E_STEP_CAP && status != kSplit) S.best = 0;
  if (lane == 0) {
    P.total_latency[k] = S.best;
    P.status[k] = status;
    if (P.nodes) P.nodes[k] = S.nodes;
  }
}

// Between the launches: the list of unfinished instances (in no particular
// order) and their search state.  k_pool_reset clears the count first.
__global__ __launch_bounds__(64) void k_pool_reset(OptParams P) {
  if (threadIdx.x == 0) P.pool[0] = 0;
}

__global__ __launch_bounds__(256) void k_pool_list(OptParams P) {
  const int k = blockIdx.x * 256 + static_cast<int>(threadIdx.x);
  if (k >= P.K || P.status[k] != kSplit) return;
  int32_t* list = P.pool + 1;
  const int j = atomicAdd(P.pool, 1);
  list[j] = k;
  list[P.K + j] = 0;                                           // piece counter
  list[2 * P.K + j] = static_cast<int32_t>(P.total_latency[k]);  // best so far
  list[3 * P.K + j] = 0;                                       // flags
}

// Second launch: workgroups of kGroupWaves waves, as many as the device holds
// at once.  A workgroup starts at its own place in the list and goes through
// it once: at every instance whose pieces are not all claimed yet, its waves
// claim and search pieces (wtop) until none is left, then meet at a barrier
// and move on.  Each wave has at most P.node_cap nodes per instance it works
// on; a wave that runs out marks the instance stopped (its result is then an
// upper bound), and workgroups that come to it later skip it.
__global__ __launch_bounds__(64 * kGroupWaves) void k_optimum_pool(OptParams P) {
  __shared__ int32_t sbest, sflag;
  const int U = P.pool[0];
  if (U <= 0) return;
  const int32_t* list = P.pool + 1;
  int32_t* cnt = P.pool + 1 + P.K;
  int32_t* gbest = P.pool + 1 + 2 * P.K;
  int32_t* flags = P.pool + 1 + 3 * P.K;
  const int lane = static_cast<int>(threadIdx.x & 63u);
  const int j0 = static_cast<int>((static_cast<int64_t>(blockIdx.x) * U) / gridDim.x);
  for (int step = 0; step < U; ++step) {
    const int j = j0 + step < U ? j0 + step : j0 + step - U;
    if (threadIdx.x == 0) {
      sflag = __hip_atomic_load(&flags[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      sbest = __hip_atomic_load(&gbest[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    if (sflag == 0) {
      const int k = list[j];
      Search S;
      S.nodes = 0;
      S.cap = static_cast<int32_t>(P.node_cap < 0x7FFFFFFF ? P.node_cap : 0x7FFFFFFF);
      S.stop = false;
      Inst I;
      (void)setup(P, k, I, S);  // valid: the first launch searched it
      S.best = sbest;
      int32_t first = 0;
      if (lane == 0) first = atomicAdd(&cnt[j], 1);
      int32_t leaf = 0, claim = __builtin_amdgcn_readfirstlane(first);
      wtop<0>(I, S, 0, lane, &sbest, &cnt[j], &gbest[j], leaf, claim);
      if (lane == 0) {
        atomicMin(&gbest[j], S.best);
        if (P.nodes) atomicAdd(reinterpret_cast<unsigned long long*>(&P.nodes[k]),
                               static_cast<unsigned long long>(S.nodes));
        // a walk that ends finds every piece claimed; a stopped one gives up
        atomicOr(&flags[j], S.stop ? (kFlagClaimed | kFlagStop) : kFlagClaimed);
      }
    }
    __syncthreads();  // sflag and sbest are rewritten for the next instance
  }
}

// After the second launch: the results of the instances it searched.
__global__ __launch_bounds__(256) void k_pool_finish(OptParams P) {
  const int j = blockIdx.x * 256 + static_cast<int>(threadIdx.x);
  if (j >= P.pool[0]) return;
  const int32_t* list = P.pool + 1;
  const int k = list[j];
  P.total_latency[k] = list[2 * P.K + j];
  P.status[k] = (list[3 * P.K + j] & kFlagStop) ? SCHED_E_STEP_CAP : SCHED_OK;
}

}  // namespace opt

extern "C" int sched_optimum(const sched_instances_t* in, int64_t M, const int64_t* upper_bound,
                             int64_t* total_latency, int32_t* status, int64_t* nodes, int64_t node_cap,
                             void* stream) {
  if (!in || !total_latency || !status) return SCHED_E_INVAL;
  if (M <= 0 || M >= (int64_t(1) << 30)) return SCHED_E_INVAL;
  if (in->num_instances < 0 || in->total_requests < 0) return SCHED_E_INVAL;
  if (in->num_instances == 0) return SCHED_OK;
  if (!in->offsets || (in->total_requests > 0 && (!in->prompt || !in->output))) return SCHED_E_INVAL;
  if (in->max_requests > opt::kMaxN) return SCHED_E_UNSUPPORTED;
  opt::OptParams P{};
  P.K = in->num_instances;
  P.N = in->total_requests;
  P.offsets = in->offsets;
  P.arrival = in->arrival;
  P.prompt = in->prompt;
  P.output = in->output;
  P.M = static_cast<int32_t>(M);
  const int64_t cap = node_cap > 0 ? node_cap : (int64_t(1) << 26);
  P.upper_bound = upper_bound;
  P.total_latency = total_latency;
  P.status = status;
  P.nodes = nodes;
  // a first launch with a short budget, then the unfinished instances on workgroups
  const bool split = cap > opt::kFirstPassNodes;
  P.node_cap = split ? opt::kFirstPassNodes : cap;
  P.unfinished = split ? opt::kSplit : SCHED_E_STEP_CAP;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  // the second launch's grid: as many workgroups as the device holds at once
  int dev = 0, n_cu = 0, per_cu = 0;
  if (split) {
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, opt::k_optimum_pool, 64 * opt::kGroupWaves, 0) !=
            hipSuccess)
      return SCHED_E_HIP;
    if (per_cu < 1) per_cu = 1;
    // workspace: the count, then four arrays of K entries
    if (hipMallocAsync(reinterpret_cast<void**>(&P.pool), sizeof(int32_t) * (1 + 4 * static_cast<size_t>(P.K)), st) !=
        hipSuccess)
      return SCHED_E_HIP;
  }
  hipLaunchKernelGGL(opt::k_optimum, dim3(P.K), dim3(64), 0, st, P);
  hipError_t err = hipGetLastError();
  if (split) {
    const dim3 g256((P.K + 255) / 256);
    if (err == hipSuccess) {
      hipLaunchKernelGGL(opt::k_pool_reset, dim3(1), dim3(64), 0, st, P);
      hipLaunchKernelGGL(opt::k_pool_list, g256, dim3(256), 0, st, P);
      P.node_cap = cap;
      hipLaunchKernelGGL(opt::k_optimum_pool, dim3(n_cu * per_cu), dim3(64 * opt::kGroupWaves), 0, st, P);
      hipLaunchKernelGGL(opt::k_pool_finish, g256, dim3(256), 0, st, P);
      err = hipGetLastError();
    }
    const hipError_t ferr = hipFreeAsync(P.pool, st);
    if (err == hipSuccess) err = ferr;
  }
  return err == hipSuccess ? SCHED_OK : SCHED_E_HIP;
}
