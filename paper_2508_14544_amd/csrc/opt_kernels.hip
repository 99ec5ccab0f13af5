// opt_kernels.hip -- gfx950 kernel of the hindsight optimum on tiny instances.
//
// The hindsight optimum (the OPT of the competitive analysis, Section 2) is
// the minimum total latency (equation (3)) over every non-preemptive schedule
// that knows the true output lengths: request i starts at some p_i >= a_i,
// holds s_i + (tau - p_i) tokens for tau in [p_i, p_i + o_i], and the total
// may never exceed M (equation (1)).  One lane searches one instance (n <= 8)
// by depth-first branch and bound over start steps in request order:
//   * a start is feasible iff the total stays <= M at the completion step of
//     every placed run that overlaps the new one and at the new run's own
//     completion (between two completions the set of present runs only grows
//     and each run's memory grows, so the maximum is at a completion);
//   * the cost of a partial assignment plus the remaining requests' output
//     lengths bounds any completion from below, and the cost grows with the
//     start, so the first start that reaches the best total ends the level;
//   * the first bound is the caller's (a known schedule's total, e.g. a
//     policy's) or else the schedule that runs the requests one at a time;
//   * requests are searched by arrival, then by decreasing s + o and o, and a
//     request identical to the previous one never starts before it (swapping
//     them gives the same schedule);
//   * starts range over [a_i, max a + sum(o + 1) + 1], a horizon within which
//     the sequential schedule already finishes every request.
// A node budget per instance guarantees every lane reaches the exit.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "schedsim.h"

namespace opt {

constexpr int kMaxN = 8;

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
};

__global__ __launch_bounds__(64) void k_optimum(OptParams P) {
  const int k = blockIdx.x * 64 + threadIdx.x;
  if (k >= P.K) return;
  const int64_t b = P.offsets[k];
  const int64_t e = P.offsets[k + 1];
  int status = SCHED_OK;
  int64_t best = 0, nodes = 0;
  if (b < 0 || e < b || e > P.N) status = SCHED_E_INVAL;
  const int n = status == SCHED_OK ? static_cast<int>(e - b) : 0;
  if (n > kMaxN) status = SCHED_E_UNSUPPORTED;
  int32_t a[kMaxN], s[kMaxN], o[kMaxN], p[kMaxN];
  int64_t cost[kMaxN + 1], rem[kMaxN + 1];
  if (status == SCHED_OK && n > 0) {
    bool arr_bad = false, int_bad = false, big_bad = false;
    int64_t amax = 0, span = 0;
#pragma unroll
    for (int i = 0; i < kMaxN; ++i) {
      a[i] = 0; s[i] = 0; o[i] = 1;
      if (i < n) {
        a[i] = P.arrival ? P.arrival[b + i] : 0;
        s[i] = P.prompt[b + i];
        o[i] = P.output[b + i];
        if (a[i] < 0 || (i > 0 && a[i] < a[i - 1])) arr_bad = true;
        if (o[i] < 1 || s[i] < 0) int_bad = true;
        if (static_cast<int64_t>(s[i]) + o[i] > P.M) big_bad = true;
        amax = a[i] > amax ? a[i] : amax;
        span += static_cast<int64_t>(o[i]) + 1;
      }
    }
    status = arr_bad ? SCHED_E_ARRIVAL : int_bad ? SCHED_E_INTERVAL : big_bad ? SCHED_E_TOO_BIG : SCHED_OK;
    if (status == SCHED_OK) {
      const int64_t horizon = amax + span + 1;
      // first bound: one request at a time, each after the previous completes
      int64_t t = 0;
      for (int i = 0; i < n; ++i) {
        const int64_t start = t > a[i] ? t : a[i];
        best += start + o[i] - a[i];
        t = start + o[i] + 1;
      }
      if (P.upper_bound && P.upper_bound[k] > 0 && P.upper_bound[k] < best) best = P.upper_bound[k];
      // search order: arrival, then the largest s + o, then the longest o
      // first (big runs placed early prune the most); the optimum does not
      // depend on it, and equal keys mean identical requests
      for (int i = 1; i < n; ++i)
        for (int j = i; j > 0; --j) {
          const int32_t wj = s[j] + o[j], wp = s[j - 1] + o[j - 1];
          const bool gt = a[j - 1] > a[j] || (a[j - 1] == a[j] && (wp < wj || (wp == wj && o[j - 1] < o[j])));
          if (!gt) break;
          const int32_t ta = a[j], ts = s[j], to = o[j];
          a[j] = a[j - 1]; s[j] = s[j - 1]; o[j] = o[j - 1];
          a[j - 1] = ta; s[j - 1] = ts; o[j - 1] = to;
        }
      rem[n] = 0;
      for (int i = n - 1; i >= 0; --i) rem[i] = rem[i + 1] + o[i];
      int d = 0;
      cost[0] = 0;
      p[0] = a[0] - 1;
      while (d >= 0) {
        if (++nodes > P.node_cap) {
          status = SCHED_E_STEP_CAP;
          break;
        }
        const int64_t pd = ++p[d];
        const int64_t c = cost[d] + pd + o[d] - a[d];
        if (pd > horizon || c + rem[d + 1] >= best) {
          --d;  // later starts at this level only cost more
          continue;
        }
        // feasibility of run d starting at pd against runs 0..d-1
        const int64_t end = pd + o[d];
        bool ok = true;
        for (int q = 0; q <= d && ok; ++q) {
          const int64_t cq = q < d ? static_cast<int64_t>(p[q]) + o[q] : end;
          if (cq < pd || cq > end) continue;
          int64_t mem = s[d] + cq - pd;
          for (int j = 0; j < d; ++j)
            if (p[j] <= cq && cq <= static_cast<int64_t>(p[j]) + o[j]) mem += s[j] + cq - p[j];
          ok = mem <= P.M;
        }
        if (!ok) continue;
        if (d == n - 1) {
          best = c;  // a complete schedule; larger starts here cost more
          --d;
          continue;
        }
        cost[d + 1] = c;
        ++d;
        const bool same = a[d] == a[d - 1] && s[d] == s[d - 1] && o[d] == o[d - 1];
        p[d] = (same ? p[d - 1] : a[d]) - 1;
      }
    }
  }
  if (status != SCHED_OK && status != SCHED_E_STEP_CAP) best = 0;
  P.total_latency[k] = best;
  P.status[k] = status;
  if (P.nodes) P.nodes[k] = nodes;
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
  P.node_cap = node_cap > 0 ? node_cap : (int64_t(1) << 22);
  P.upper_bound = upper_bound;
  P.total_latency = total_latency;
  P.status = status;
  P.nodes = nodes;
  hipLaunchKernelGGL(opt::k_optimum, dim3((P.K + 63) / 64), dim3(64), 0, static_cast<hipStream_t>(stream), P);
  return hipGetLastError() == hipSuccess ? SCHED_OK : SCHED_E_HIP;
}
