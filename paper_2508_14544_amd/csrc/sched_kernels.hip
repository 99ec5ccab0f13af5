// sched_kernels.hip -- the C ABI of the scheduler simulator (host side) and
// the kernels it launches, except the wide row ladder (sched_wide.hip) and
// the workgroup kernels (sched_group.hip), each its own translation unit so
// that their large bodies do not change how the other kernels are compiled.
// The device code is in sim_device.hpp.
#include "sim_device.hpp"

namespace sk {
// defined in sched_wide.hip
extern template __global__ void k_simulate_ladder_wide<SCHED_AMAX>(Params);
extern template __global__ void k_simulate_ladder_wide<SCHED_AMIN>(Params);
extern template __global__ void k_simulate_ladder_wide<SCHED_HSF>(Params);
extern template __global__ void k_simulate_ladder_wide<SCHED_AELL>(Params);
extern template __global__ void k_simulate_ladder_wide<SCHED_ARANDOM>(Params);
// defined in sched_group.hip
extern template __global__ void k_simulate_group<SCHED_AMAX, 2, 8, false>(Params);
extern template __global__ void k_simulate_group<SCHED_AMAX, 4, 4, false>(Params);
extern template __global__ void k_simulate_group<SCHED_AMAX, 4, 16, false>(Params);
extern template __global__ void k_simulate_group<SCHED_AMAX, 8, 16, false>(Params);
extern template __global__ void k_simulate_group<SCHED_HSF, 2, 8, false>(Params);
extern template __global__ void k_simulate_group<SCHED_HSF, 4, 4, false>(Params);
extern template __global__ void k_simulate_group<SCHED_HSF, 4, 16, false>(Params);
extern template __global__ void k_simulate_group<SCHED_HSF, 8, 16, false>(Params);
extern template __global__ void k_simulate_group<SCHED_ARANDOM, 4, 16, false>(Params);
extern template __global__ void k_simulate_group<SCHED_ARANDOM, 8, 16, false>(Params);
extern template __global__ void k_simulate_group<SCHED_AELL, 4, 16, false>(Params);
extern template __global__ void k_simulate_group<SCHED_AELL, 8, 16, false>(Params);
extern template __global__ void k_simulate_group<SCHED_AMIN, 2, 8, false>(Params);
extern template __global__ void k_simulate_group<SCHED_AMIN, 2, 8, true>(Params);
extern template __global__ void k_simulate_group<SCHED_AMIN, 4, 4, false>(Params);
extern template __global__ void k_simulate_group<SCHED_AMIN, 4, 4, true>(Params);
extern template __global__ void k_simulate_group<SCHED_AMIN, 4, 16, false>(Params);
extern template __global__ void k_simulate_group<SCHED_AMIN, 4, 16, true>(Params);
extern template __global__ void k_simulate_group<SCHED_AMIN, 8, 16, true>(Params);

// Issue-priority classes (A_min with upper bounds, from k_prepare): kept only
// where they differ between the instances of the batch; a batch whose
// instances share one class keeps the priority by unfinished work alone.
__global__ __launch_bounds__(256) void k_prio_classes(Params P) {
  __shared__ int lo_s, hi_s;
  if (threadIdx.x == 0) {
    lo_s = 3;
    hi_s = -1;
  }
  __syncthreads();
  int lo = 3, hi = -1;
  for (int k = threadIdx.x; k < P.K; k += 256) {
    const int c = P.pclass[k];
    if (c < 3) {
      lo = c < lo ? c : lo;
      hi = c > hi ? c : hi;
    }
  }
  atomicMin(&lo_s, lo);
  atomicMax(&hi_s, hi);
  __syncthreads();
  if (lo_s >= hi_s)
    for (int k = threadIdx.x; k < P.K; k += 256) P.pclass[k] = -1;
}

// Launch order (A_min batches served in several rounds of waves): the
// instances by decreasing key, so that the longest expected simulations are
// not the last ones to start.  The order within a bucket is whatever the
// atomics give; outputs do not depend on the order.
__global__ __launch_bounds__(64) void k_order_clear(Params P) {
  P.obucket[threadIdx.x] = 0;
}
__global__ __launch_bounds__(64) void k_order_scan(Params P) {
  // bucket b starts after every bucket above it
  if (threadIdx.x == 0) {
    int32_t run = 0;
    for (int b = kOrderBuckets - 1; b >= 0; --b) {
      const int32_t c = P.obucket[b];
      P.obucket[b] = run;
      run += c;
    }
  }
}
__global__ __launch_bounds__(256) void k_order_scatter(Params P) {
  // one atomic per distinct key of a wave (neighbouring instances mostly
  // share their key), the lanes of a key placed in lane order
  const int k = blockIdx.x * 256 + static_cast<int>(threadIdx.x);
  const int lane = static_cast<int>(threadIdx.x & 63u);
  const bool act = k < P.K;
  const int key = act ? P.okey[k] : -1;
  uint64_t left = __builtin_amdgcn_ballot_w64(act);
  while (left) {
    const int lead = __builtin_ctzll(left);
    const int lkey = __builtin_amdgcn_readlane(key, lead);
    const uint64_t same = __builtin_amdgcn_ballot_w64(act && key == lkey) & left;
    int base = 0;
    if (lane == lead) base = atomicAdd(&P.obucket[lkey], __builtin_popcountll(same));
    base = __builtin_amdgcn_readlane(base, lead);
    if ((same >> lane) & 1ull) {
      const int below = __builtin_popcountll(same & ((1ull << lane) - 1ull));
      P.order[base + below] = k;
    }
    left &= ~same;
  }
}
}  // namespace sk

// ---------------------------------------------------------------------------
// The workspace of sched_simulate_noalloc: a fixed array in device memory
// (each device that runs the library holds its own copy until the process
// ends).  Host code never passes `scratch` itself to a kernel or a copy (in
// host code the name is a host-side stand-in): it uses the device address
// that hipGetSymbolAddress returns, taken once per device.
// ---------------------------------------------------------------------------
constexpr size_t kScratchBytes = size_t(96) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// ---------------------------------------------------------------------------
// host side: the C ABI
// ---------------------------------------------------------------------------
namespace {

// Device address of `scratch` on device `dev` (the current device), looked up
// on the first call on that device and kept.
hipError_t scratch_address(int dev, void** out) {
  constexpr int kMaxDev = 64;
  static std::mutex mu;
  static void* addr[kMaxDev] = {};
  if (dev < 0 || dev >= kMaxDev) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *out = addr[dev];
  return hipSuccess;
}

// One launch of the simulation kernel over the batch.
struct Tier {
  int rows;         // register rows (fixed-row kernels; per wave in a workgroup)
  bool grow;        // a row ladder: k_simulate_ladder, or k_simulate_ladder_wide with wide
  bool wide;
  bool retry;       // a retry pass: runs the instances an earlier pass handed over (run_mask)
  bool vglobal;     // cancelled set in global memory (16 rows)
  int cap_v;        // LDS slots of the cancelled set (LDS passes)
  int run_mask;     // retry: bit 0 takes kRetryRows, bit 1 kRetryV
  int rows_status;  // status for an outgrown running set
  int v_status;     // status for an outgrown cancelled set
  int stage;        // completion steps staged in LDS (1) or not (0)
  int gw;           // > 1: a workgroup of gw waves per instance (k_simulate_group)
  int grid;         // workgroups of the launch (0: one per instance)
  int roomy;        // the narrow ladder with 256 VGPRs (k_simulate_ladder_roomy)
};

// The workgroup kernels that exist (sched_group.hip), else NULL.
template <int ALGO>
const void* group_kernel(int w, int rows, bool vglobal) {
  using P = sk::Params;
  void (*f)(P) = nullptr;
  if constexpr (ALGO == SCHED_AMAX || ALGO == SCHED_HSF) {
    if (!vglobal) {
      if (w == 2 && rows == 8) f = &sk::k_simulate_group<ALGO, 2, 8, false>;
      if (w == 4 && rows == 4) f = &sk::k_simulate_group<ALGO, 4, 4, false>;
    }
  }
  if constexpr (ALGO != SCHED_AMIN) {
    if (!vglobal && w == 4 && rows == 16) f = &sk::k_simulate_group<ALGO, 4, 16, false>;
    if (!vglobal && w == 8 && rows == 16) f = &sk::k_simulate_group<ALGO, 8, 16, false>;
  } else {
    if (w == 2 && rows == 8) f = vglobal ? &sk::k_simulate_group<ALGO, 2, 8, true> : &sk::k_simulate_group<ALGO, 2, 8, false>;
    if (w == 4 && rows == 4) f = vglobal ? &sk::k_simulate_group<ALGO, 4, 4, true> : &sk::k_simulate_group<ALGO, 4, 4, false>;
    if (w == 4 && rows == 16)
      f = vglobal ? &sk::k_simulate_group<ALGO, 4, 16, true> : &sk::k_simulate_group<ALGO, 4, 16, false>;
    if (w == 8 && rows == 16 && vglobal) f = &sk::k_simulate_group<ALGO, 8, 16, true>;
  }
  return reinterpret_cast<const void*>(f);
}

template <int ALGO>
const void* sim_kernel(const Tier& tr, bool ordered, bool classes, bool rounds) {
  if (tr.gw > 1) return group_kernel<ALGO>(tr.gw, tr.rows, tr.vglobal);
  if constexpr (ALGO == SCHED_AMIN) {
    if (tr.grow && !tr.wide && ordered)
      return reinterpret_cast<const void*>(&sk::k_simulate_ladder<ALGO, true, false, false>);
    if (tr.grow && !tr.wide && classes)
      return reinterpret_cast<const void*>(&sk::k_simulate_ladder<ALGO, false, true>);
  }
  if (tr.grow && !tr.wide && tr.roomy) return reinterpret_cast<const void*>(&sk::k_simulate_ladder_roomy<ALGO>);
  if (tr.grow && !tr.wide && rounds)
    return reinterpret_cast<const void*>(&sk::k_simulate_ladder<ALGO, false, false, false>);
  if (tr.grow)
    return tr.wide ? reinterpret_cast<const void*>(&sk::k_simulate_ladder_wide<ALGO>)
                   : reinterpret_cast<const void*>(&sk::k_simulate_ladder<ALGO>);
  if constexpr (ALGO == SCHED_AMIN || ALGO == SCHED_AELL)
    if (tr.vglobal) return reinterpret_cast<const void*>(&sk::k_simulate<ALGO, 16, true, true>);
  if (tr.retry)
    return tr.rows <= 8    ? reinterpret_cast<const void*>(&sk::k_simulate<ALGO, 8, true>)
                           : reinterpret_cast<const void*>(&sk::k_simulate<ALGO, 16, true>);
  switch (tr.rows) {
    case 1: return reinterpret_cast<const void*>(&sk::k_simulate<ALGO, 1, false>);
    case 2: return reinterpret_cast<const void*>(&sk::k_simulate<ALGO, 2, false>);
    case 4: return reinterpret_cast<const void*>(&sk::k_simulate<ALGO, 4, false>);
    case 5: return reinterpret_cast<const void*>(&sk::k_simulate<ALGO, 5, false>);
    case 6: return reinterpret_cast<const void*>(&sk::k_simulate<ALGO, 6, false>);
    case 8: return reinterpret_cast<const void*>(&sk::k_simulate<ALGO, 8, false>);
    default: return reinterpret_cast<const void*>(&sk::k_simulate<ALGO, 16, false>);
  }
}

// ordered: A_min's narrow ladder takes the instances in the order P.order;
// classes: it sets issue priorities by P.pclass; rounds: the batch is served
// in rounds of waves (the narrow ladder without issue priorities)
const void* sim_kernel_any(int algo, const Tier& tr, bool ordered = false, bool classes = false,
                           bool rounds = false) {
  switch (algo) {
    case SCHED_AMAX: return sim_kernel<SCHED_AMAX>(tr, false, false, rounds);
    case SCHED_AMIN: return sim_kernel<SCHED_AMIN>(tr, ordered, classes, rounds);
    case SCHED_HSF: return sim_kernel<SCHED_HSF>(tr, false, false, rounds);
    case SCHED_ARANDOM: return sim_kernel<SCHED_ARANDOM>(tr, false, false, rounds);
    default: return sim_kernel<SCHED_AELL>(tr, false, false, rounds);
  }
}

// register rows that hold `want` runs
int rows_for(int64_t want) {
  const int64_t r = (want + 63) / 64;
  return r <= 1 ? 1 : r <= 2 ? 2 : r <= 4 ? 4 : r <= 5 ? 5 : r <= 6 ? 6 : r <= 8 ? 8 : 16;
}

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// The LDS of a launch: the bitmaps' words and the most a workgroup holds.
struct Room {
  size_t lds_max;
  int nw, nw1;
};

// LDS bytes of a workgroup launch (W waves, `rows` rows each) whose waves
// each hold cap_v cancelled-set slots (0: a global set), staging aside.
size_t group_lds(int algo, int w, int rows, const Room& rm, int cap_v) {
  return 8 * (static_cast<size_t>(sk::group_pre_words(algo, w, rows)) +
              static_cast<size_t>(w) * (static_cast<size_t>(rm.nw) + rm.nw1 + cap_v));
}

// Cancelled-set slots per wave that the LDS of such a launch leaves room for
// (-1: not even the bitmaps fit).
int64_t group_cap_fit(int algo, int w, int rows, const Room& rm) {
  const size_t base = group_lds(algo, w, rows, rm, 0);
  return base > rm.lds_max ? -1 : static_cast<int64_t>((rm.lds_max - base) / (8 * static_cast<size_t>(w)));
}

// The launches that simulate a batch under one policy.  The first holds an
// instance's running set in register rows whose number follows it (the row
// ladder: 2, 3, 5, 8, 10 rows, four waves a SIMD); an instance that needs more
// than 640 runs is simulated again from step 0 by the wide ladder (12 and 16
// more rows, 1024 runs, fewer waves a SIMD), which is also the first launch of a
// batch of few instances that may need it; one that needs more than 1024 runs,
// by a workgroup of 4 waves with 16 rows each (4096 runs), then of 8 waves
// (8192).  With workgroup_waves = W (2 or 4), the first launch is a workgroup
// of W waves with 1024 / (64 W) rows each instead.  The cancelled set (A_min)
// first gets cap0 LDS slots (a size chosen for occupancy); an instance that
// outgrows them is simulated again with as many slots as a workgroup's LDS
// holds, and one that outgrows those again with a global-memory set of n
// slots (per wave), which always suffices (at most n requests wait
// cancelled).  So whether an instance completes never depends on the other
// instances of the batch or on these sizes: only running sets above 8192 runs
// (4096 where eight waves' bitmaps do not fit the LDS), or above a caller's
// forced running capacity, are refused.
int build_tiers(int algo, int64_t nmax, int64_t K, int forced_rows, int cap0, int cap_fit, int ww, const Room& rm,
                bool simd_each, Tier* out) {
  // (A_l's queue lives in global memory and never overflows)
  const bool has_v = algo == SCHED_AMIN;
  const int64_t need_v = has_v ? std::max<int64_t>(nmax, 1) : 0;
  const int cap1 = has_v ? static_cast<int>(std::min<int64_t>(need_v, cap_fit)) : 0;
  const bool v_retry = has_v && cap0 < need_v && cap1 > cap0;  // a larger LDS set may help
  const bool v_lds_short = has_v && cap1 < need_v;              // even the largest LDS set may not
  int m = 0;
  // a workgroup launch: with an LDS cancelled set when `want` slots per wave
  // fit (and a global-set retry if that may be short), else a global set
  auto group = [&](int w, int rows, int mask) {
    if (!has_v) {
      out[m++] = Tier{rows, false, false, mask != 0, false, 0, mask, 0, 0, 0, w, 0};
      return;
    }
    const int64_t want = std::min<int64_t>(need_v, 16384);
    const int64_t fit = std::min<int64_t>(group_cap_fit(algo, w, rows, rm), cap_fit);
    const bool lds = fit >= want && group_kernel<SCHED_AMIN>(w, rows, false) != nullptr;
    if (lds) out[m++] = Tier{rows, false, false, mask != 0, false, static_cast<int>(want), mask, 0, 0, 0, w, 0};
    if (!lds || want < need_v) out[m++] = Tier{rows, false, false, true, true, 0, lds ? 2 : (mask ? mask : 0), 0, 0, 0, w, 0};
  };
  if (ww > 1) {
    group(ww, 1024 / (64 * ww), 0);
  } else if (forced_rows > 0) {
    out[m++] = Tier{forced_rows, false, false, false, false, cap0, 0, 0, 0, 0, 0, 0};
    if (v_retry) out[m++] = Tier{16, false, false, true, false, cap1, 2, 0, 0, 0, 0, 0};
    if (v_lds_short) out[m++] = Tier{16, false, false, true, true, 0, 2, 0, 0, 0, 0, 0};
  } else if (nmax <= 128) {
    out[m++] = Tier{rows_for(std::max<int64_t>(nmax, 1)), false, false, false, false, cap0, 0, 0, 0, 0, 0, 0};
    if (v_retry) out[m++] = Tier{8, false, false, true, false, cap1, 2, 0, 0, 0, 0, 0};
    if (v_lds_short) out[m++] = Tier{16, false, false, true, true, 0, 2, 0, 0, 0, 0, 0};
  } else {
    // few instances of many requests start on the wide ladder (they would
    // likely outgrow the narrow one, and the retry would simulate them again);
    // where every wave has a SIMD to itself (simd_each) the narrow bodies get
    // 256 VGPRs, which costs no occupancy there and spills less
    const bool wide0 = nmax > 4096 && K <= 256;
    out[m++] = Tier{0, true, wide0, false, false, cap0, 0, 0, 0, 0, 0, 0, !wide0 && simd_each ? 1 : 0};
    const int mask = (!wide0 && nmax > 640 ? 1 : 0) | (v_retry ? 2 : 0);
    if (mask) out[m++] = Tier{0, true, true, true, false, cap1, mask, 0, 0, 0, 0, 0};
    if (v_lds_short) out[m++] = Tier{16, false, false, true, true, 0, 2, 0, 0, 0, 0, 0};
  }
  // beyond 1024 runs: workgroups (a forced capacity holds instead)
  if (forced_rows == 0 && nmax > 1024) {
    group(4, 16, 1);
    // eight waves when their bitmaps (and lists) fit the LDS
    if (group_cap_fit(algo, 8, 16, rm) >= 0) {
      if (has_v)
        out[m++] = Tier{16, false, false, true, true, 0, 1, 0, 0, 0, 8, 0};
      else
        out[m++] = Tier{16, false, false, true, false, 0, 1, 0, 0, 0, 8, 0};
    }
  }
  // what a pass writes for an instance it cannot hold: a later pass that takes
  // it, or the final refusal
  for (int p = 0; p < m; ++p) {
    bool later_rows = false, later_v = false;
    for (int q = p + 1; q < m; ++q) {
      later_rows = later_rows || (out[q].run_mask & 1);
      later_v = later_v || (out[q].run_mask & 2);
    }
    out[p].rows_status = later_rows ? sk::kRetryRows : SCHED_E_UNSUPPORTED;
    out[p].v_status = later_v ? sk::kRetryV : SCHED_E_UNSUPPORTED;
  }
  return m;
}

// A second stream per device (default priority, created on first use and kept
// for the life of the process): the adaptive policy runs its A_l launches on
// it while the A_min launches run on the caller's stream.  The two touch
// disjoint instances.
hipError_t side_stream(int dev, hipStream_t* out) {
  constexpr int kMaxDev = 64;
  static std::mutex mu;
  static hipStream_t streams[kMaxDev] = {};
  if (dev < 0 || dev >= kMaxDev) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!streams[dev]) {
    const hipError_t e = hipStreamCreateWithFlags(&streams[dev], hipStreamNonBlocking);
    if (e != hipSuccess) {
      streams[dev] = nullptr;
      return e;
    }
  }
  *out = streams[dev];
  return hipSuccess;
}

// Argument checks shared by the entry points (no HIP call).
int check_args(const sched_instances_t* in, int32_t algo, int64_t M) {
  if (!in) return SCHED_E_INVAL;
  if (algo < SCHED_AMAX || algo > SCHED_ARANDOM) return SCHED_E_INVAL;
  if (M <= 0 || M >= (int64_t(1) << 30)) return SCHED_E_INVAL;
  if (in->num_instances < 0 || in->max_requests < 0 || in->total_requests < 0) return SCHED_E_INVAL;
  if (in->num_instances == 0) return SCHED_OK;
  if (!in->offsets) return SCHED_E_INVAL;
  const bool need_l = algo == SCHED_AMIN || algo == SCHED_AELL || algo == SCHED_ADAPTIVE;
  const bool need_u = algo == SCHED_AMAX || algo == SCHED_AELL || algo == SCHED_ADAPTIVE;
  if (in->total_requests > 0 && (!in->prompt || !in->output)) return SCHED_E_INVAL;
  if (in->total_requests > 0 && need_l && !in->lower) return SCHED_E_INVAL;
  if (in->total_requests > 0 && need_u && !in->upper) return SCHED_E_INVAL;
  if (in->total_requests > 0 && algo == SCHED_ARANDOM && !in->priority) return SCHED_E_INVAL;
  if (in->max_requests >= (1 << sk::kIdxBits)) return SCHED_E_UNSUPPORTED;
  return SCHED_OK;
}

sk::Params base_params(const sched_instances_t* in, int64_t M) {
  sk::Params P{};
  P.K = in->num_instances;
  P.max_requests = in->max_requests;
  P.N = in->total_requests;
  P.offsets = in->offsets;
  P.arrival = in->arrival;
  P.prompt = in->prompt;
  P.output = in->output;
  P.lower = in->lower;
  P.upper = in->upper;
  P.priority = in->priority;
  P.tie_key = in->total_requests > 0 ? in->tie_key : nullptr;
  P.M = static_cast<int32_t>(M);
  return P;
}

}  // namespace

extern "C" {

int sched_version(void) { return 131; }

const char* sched_strerror(int code) {
  switch (code) {
    case SCHED_OK: return "ok";
    case SCHED_E_INVAL: return "invalid argument";
    case SCHED_E_INTERVAL: return "invalid request data (o < 1, s < 0, or interval does not contain o)";
    case SCHED_E_TOO_BIG: return "a request can never fit in M";
    case SCHED_E_STEP_CAP: return "step cap reached with unfinished requests";
    case SCHED_E_HIP: return "HIP runtime error";
    case SCHED_E_UNSUPPORTED: return "beyond kernel capacity";
    case SCHED_E_ARRIVAL: return "arrivals negative or not non-decreasing";
    case SCHED_E_SCRATCH: return "workspace beyond the 96 MiB no-allocation scratch";
    default: return "unknown code";
  }
}

int sched_validate(const sched_instances_t* in, int32_t algo, int64_t M, int32_t* status, void* stream) {
  const int c = check_args(in, algo, M);
  if (c != SCHED_OK || in->num_instances == 0) return c;
  if (!status) return SCHED_E_INVAL;
  sk::Params P = base_params(in, M);
  P.status = status;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const dim3 grid(P.K), block(64);
  switch (algo) {
    case SCHED_AMAX: hipLaunchKernelGGL((sk::k_validate<SCHED_AMAX>), grid, block, 0, st, P); break;
    case SCHED_AMIN: hipLaunchKernelGGL((sk::k_validate<SCHED_AMIN>), grid, block, 0, st, P); break;
    case SCHED_HSF: hipLaunchKernelGGL((sk::k_validate<SCHED_HSF>), grid, block, 0, st, P); break;
    case SCHED_AELL: hipLaunchKernelGGL((sk::k_validate<SCHED_AELL>), grid, block, 0, st, P); break;
    case SCHED_ARANDOM: hipLaunchKernelGGL((sk::k_validate<SCHED_ARANDOM>), grid, block, 0, st, P); break;
    default: hipLaunchKernelGGL((sk::k_validate<SCHED_ADAPTIVE>), grid, block, 0, st, P); break;
  }
  return hipGetLastError() == hipSuccess ? SCHED_OK : SCHED_E_HIP;
}

}  // extern "C"

namespace {

// sched_simulate_opts and sched_simulate_noalloc.  no_alloc: the workspace is
// the device's `scratch` array, and the adaptive policy runs both of its
// policies' launches on the caller's stream (no side stream, no events), so
// nothing is allocated.
int simulate_impl(const sched_instances_t* in, int32_t algo, int64_t M, const sched_results_t* out,
                  void* stream, const sched_options_t* opts, bool no_alloc) {
  if (!in || !out) return SCHED_E_INVAL;
  {
    const int c = check_args(in, algo, M);
    if (c != SCHED_OK || in->num_instances == 0) return c;
  }
  if (!out->total_latency || !out->status) return SCHED_E_INVAL;
  if (in->total_requests > 0 && !out->completion) return SCHED_E_INVAL;
  sched_options_t o{};
  if (opts) o = *opts;
  if (o.step_cap > sk::kCapLimit) return SCHED_E_INVAL;
  if (o.running_capacity < 0 || o.evicted_capacity < 0 || o.evicted_lds_limit < 0) return SCHED_E_INVAL;
  if (o.running_capacity > 1024) return SCHED_E_UNSUPPORTED;
  const int ww = o.workgroup_waves <= 1 ? 0 : o.workgroup_waves;
  if (o.workgroup_waves < 0 || (ww != 0 && ww != 2 && ww != 4)) return SCHED_E_INVAL;
  if (ww && (o.running_capacity > 0 || (algo != SCHED_AMAX && algo != SCHED_AMIN && algo != SCHED_HSF)))
    return SCHED_E_INVAL;

  const int64_t nmax = in->max_requests;
  const bool tie = in->total_requests > 0 && in->tie_key != nullptr;
  hipStream_t st = static_cast<hipStream_t>(stream);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return SCHED_E_HIP;
  int lds_max = 0, n_cu = 0;
  if (hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess ||
      hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return SCHED_E_HIP;

  const int nw = static_cast<int>((nmax + 63) / 64);
  const int nw1 = (nw + 63) / 64;
  // LDS: the two bitmap levels, then the cancelled set (8 bytes a slot)
  const size_t lds_bitmaps = 8 * static_cast<size_t>(nw + nw1);
  if (lds_bitmaps + 8 > static_cast<size_t>(lds_max)) return SCHED_E_UNSUPPORTED;
  int cap_fit = static_cast<int>((static_cast<size_t>(lds_max) - lds_bitmaps) / 8);
  if (o.evicted_lds_limit > 0) cap_fit = std::min(cap_fit, o.evicted_lds_limit);
  // the first pass's cancelled-set slots (A_min; A_l's promoted queue is an
  // array of n entries in global memory).  Where many instances share a CU,
  // at most 1024, and for n_max <= 1024 what the LDS share of a wave leaves
  // next to the bitmaps and the staged completion steps (at least 512): an
  // instance whose set outgrows its slots is simulated again by a later pass
  const int64_t waves_cu = std::min<int64_t>(16, std::max<int64_t>(1, (in->num_instances + 255) / 256));
  const int64_t share_room =
      (static_cast<int64_t>(163840 / waves_cu) - 512 - static_cast<int64_t>(lds_bitmaps) - 4 * int64_t(nw) * 64) / 8;
  auto cap0_for = [&](int a) -> int {
    int64_t c = 0;
    if (a == SCHED_AMIN)
      c = std::min<int64_t>(std::max<int64_t>(nmax, 1),
                            in->num_instances <= 64 ? 16384
                            : nmax <= 1024          ? std::min<int64_t>(1024, std::max<int64_t>(512, share_room))
                                                    : 1024);
    if (o.evicted_capacity > 0 && a == SCHED_AMIN) c = o.evicted_capacity;
    return static_cast<int>(std::min<int64_t>(c, cap_fit));
  };
  const int forced_rows = o.running_capacity > 0 ? rows_for(o.running_capacity) : 0;
  // the adaptive policy runs the A_min passes and then the A_l passes; each
  // kernel skips the instances that k_prepare assigned to the other policy
  const int sim_algos[2] = {algo == SCHED_ADAPTIVE ? SCHED_AMIN : static_cast<int>(algo), SCHED_AELL};
  const int n_sim = algo == SCHED_ADAPTIVE ? 2 : 1;
  const Room rm{static_cast<size_t>(lds_max), nw, nw1};
  Tier tiers[2][8];
  int n_tiers[2] = {0, 0};
  bool any_global = algo == SCHED_AELL || algo == SCHED_ADAPTIVE;  // A_l's promoted queue
  // workgroup launches with global cancelled sets: each workgroup simulates
  // its instances one after the other, with n_max entries per wave of its own
  // (at most 64 MiB of them, and at least one workgroup)
  int64_t group_words = 0;
  for (int a = 0; a < n_sim; ++a) {
    n_tiers[a] = build_tiers(sim_algos[a], nmax, in->num_instances, forced_rows, cap0_for(sim_algos[a]), cap_fit,
                             ww, rm, in->num_instances <= 4 * int64_t(n_cu), tiers[a]);
    for (int p = 0; p < n_tiers[a]; ++p) {
      Tier& t = tiers[a][p];
      if (t.gw > 1 && t.vglobal) {
        const int64_t per = static_cast<int64_t>(t.gw) * std::max<int64_t>(nmax, 1);
        t.grid = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(in->num_instances, (int64_t(8) << 20) / per)));
        group_words = std::max<int64_t>(group_words, per * t.grid);
      } else {
        any_global = any_global || t.vglobal;
      }
      if (t.gw > 1 && !sim_kernel_any(sim_algos[a], t)) return SCHED_E_UNSUPPORTED;
    }
  }
  // LDS of a launch before staging (every launch fits, by the choices above)
  auto lds_base = [&](int a, const Tier& t) -> size_t {
    if (t.gw > 1) return group_lds(sim_algos[a], t.gw, t.rows, rm, t.vglobal ? 0 : t.cap_v);
    return lds_bitmaps + (t.vglobal ? 0 : 8 * static_cast<size_t>(t.cap_v));
  };
  for (int a = 0; a < n_sim; ++a)
    for (int p = 0; p < n_tiers[a]; ++p)
      if (lds_base(a, tiers[a][p]) > static_cast<size_t>(lds_max)) return SCHED_E_UNSUPPORTED;

  const size_t N = static_cast<size_t>(in->total_requests);
  const size_t K = static_cast<size_t>(in->num_instances);
  size_t off = 0;
  const size_t o_sa = off; off = align_up(off + 4 * N, 256);
  const size_t o_sb = off; off = align_up(off + 4 * N, 256);
  const size_t o_rec = off; off = align_up(off + 8 * N, 256);
  const size_t o_rk = off; off = align_up(off + 4 * N, 256);
  const size_t o_cap = off; off = align_up(off + 4 * K, 256);
  const size_t o_alg = off; off = align_up(off + (algo == SCHED_ADAPTIVE ? 4 * K : 0), 256);
  const size_t o_tr = off; off = align_up(off + (tie ? 4 * N : 0), 256);
  const size_t o_ix = off; off = align_up(off + (tie ? 4 * N : 0), 256);
  const size_t o_cs = off; off = align_up(off + (tie ? 4 * N : 0), 256);
  const size_t o_es = off; off = align_up(off + (tie && out->evictions ? 4 * N : 0), 256);
  const size_t o_vg = off; off = align_up(off + (any_global ? 8 * N : 0), 256);
  const size_t o_gv = off; off = align_up(off + 8 * static_cast<size_t>(group_words), 256);
  // Priority classes only where every instance of the batch is resident at
  // once (16 waves a CU), so that the launch lasts as long as its slowest
  // instance, and where waves share a SIMD at all (more than one wave on
  // each of a CU's four SIMDs); a batch served in several rounds of waves
  // keeps the priority by unfinished work.
  const bool pcl = (algo == SCHED_AMIN || algo == SCHED_ADAPTIVE) && in->upper != nullptr && in->total_requests > 0 &&
                   static_cast<int64_t>(K) > 4 * static_cast<int64_t>(n_cu) &&
                   static_cast<int64_t>(K) <= 16 * static_cast<int64_t>(n_cu);
  const size_t o_pc = off; off = align_up(off + (pcl ? 4 * K : 0), 256);
  // the launch order of A_min batches that take more than one round of waves
  const bool rounds = static_cast<int64_t>(K) > 16 * static_cast<int64_t>(n_cu);
  const bool ord = algo == SCHED_AMIN && in->total_requests > 0 && rounds;
  const size_t o_or = off; off = align_up(off + (ord ? 8 * K + 4 * sk::kOrderBuckets : 0), 256);
  // every workspace array is written before it is read (nothing needs clearing)
  void* ws = nullptr;
  if (no_alloc) {
    if (off > kScratchBytes) return SCHED_E_SCRATCH;
    if (scratch_address(dev, &ws) != hipSuccess) return SCHED_E_HIP;
  } else if (hipMallocAsync(&ws, off, st) != hipSuccess) {
    return SCHED_E_HIP;
  }
  char* base = static_cast<char*>(ws);

  sk::Params P = base_params(in, M);
  P.completion = out->completion;
  P.evictions = out->evictions;
  P.total_latency = out->total_latency;
  P.makespan = out->makespan;
  P.request_steps = out->request_steps;
  P.total_evictions = out->total_evictions;
  P.status = out->status;
  P.algo_used = out->algo_used;
  P.step_cap = o.step_cap;
  P.sort_a = reinterpret_cast<uint32_t*>(base + o_sa);
  P.sort_b = reinterpret_cast<uint32_t*>(base + o_sb);
  P.rec = reinterpret_cast<uint2*>(base + o_rec);
  P.rank_of = reinterpret_cast<int32_t*>(base + o_rk);
  P.u_of_rank = reinterpret_cast<int32_t*>(P.sort_b);  // free once the keys are sorted (A_l sorts none)
  P.cap = reinterpret_cast<int32_t*>(base + o_cap);
  P.algo_of = algo == SCHED_ADAPTIVE ? reinterpret_cast<int32_t*>(base + o_alg) : nullptr;
  P.tr_of = tie ? reinterpret_cast<int32_t*>(base + o_tr) : nullptr;
  P.idx_of = tie ? reinterpret_cast<int32_t*>(base + o_ix) : nullptr;
  P.comp_st = tie ? reinterpret_cast<int32_t*>(base + o_cs) : nullptr;
  P.ev_st = tie && out->evictions ? reinterpret_cast<int32_t*>(base + o_es) : nullptr;
  P.vglob = any_global ? reinterpret_cast<uint64_t*>(base + o_vg) : nullptr;
  P.vgroup = group_words ? reinterpret_cast<uint64_t*>(base + o_gv) : nullptr;
  P.pclass = pcl ? reinterpret_cast<int32_t*>(base + o_pc) : nullptr;
  P.order = ord ? reinterpret_cast<int32_t*>(base + o_or) : nullptr;
  P.okey = ord ? P.order + K : nullptr;
  P.obucket = ord ? P.okey + K : nullptr;
  P.nw_max = nw;
  P.nw1_max = nw1;
  P.run_cap = forced_rows > 0 ? forced_rows * 64 : INT32_MAX;

  hipError_t err = hipSuccess;
  const dim3 grid(P.K), block(64);
  // the preparation's key sort in LDS (two buffers of n_max keys) when they
  // take at most 32 KiB; with tie keys its index sorts use the workspace
  P.pre_lds = (!tie && algo != SCHED_AELL && 8 * nmax <= 32768) ? 1 : 0;
  const size_t pre_bytes = P.pre_lds ? 8 * static_cast<size_t>(nmax) : 0;
  if (P.order) hipLaunchKernelGGL(sk::k_order_clear, dim3(1), dim3(sk::kOrderBuckets), 0, st, P);
  switch (algo) {
    case SCHED_AMAX: hipLaunchKernelGGL((sk::k_prepare<SCHED_AMAX>), grid, block, pre_bytes, st, P); break;
    case SCHED_AMIN: hipLaunchKernelGGL((sk::k_prepare<SCHED_AMIN>), grid, block, pre_bytes, st, P); break;
    case SCHED_HSF: hipLaunchKernelGGL((sk::k_prepare<SCHED_HSF>), grid, block, pre_bytes, st, P); break;
    case SCHED_AELL: hipLaunchKernelGGL((sk::k_prepare<SCHED_AELL>), grid, block, pre_bytes, st, P); break;
    case SCHED_ARANDOM: hipLaunchKernelGGL((sk::k_prepare<SCHED_ARANDOM>), grid, block, pre_bytes, st, P); break;
    default: hipLaunchKernelGGL((sk::k_prepare<SCHED_ADAPTIVE>), grid, block, pre_bytes, st, P); break;
  }
  err = hipGetLastError();
  if (err == hipSuccess && P.pclass) {
    hipLaunchKernelGGL(sk::k_prio_classes, dim3(1), dim3(256), 0, st, P);
    err = hipGetLastError();
  }
  if (err == hipSuccess && P.order) {
    hipLaunchKernelGGL(sk::k_order_scan, dim3(1), dim3(64), 0, st, P);
    hipLaunchKernelGGL(sk::k_order_scatter, dim3((P.K + 255) / 256), dim3(256), 0, st, P);
    err = hipGetLastError();
  }
  // Staging the completion steps in LDS (written out coalesced at the end of
  // an instance instead of one scattered store per completion) when it fits
  // without costing occupancy: at most the LDS share of the waves a CU holds
  // at once (four per SIMD) or that the batch gives it.
  const int64_t nst = static_cast<int64_t>(nw) * 64;
  const int64_t per_cu = std::min<int64_t>(16, std::max<int64_t>(1, (static_cast<int64_t>(K) + 255) / 256));
  const size_t stage_budget = std::min<size_t>(static_cast<size_t>(lds_max), static_cast<size_t>(163840 / per_cu));
  for (int a = 0; a < n_sim; ++a)
    for (int p = 0; p < n_tiers[a]; ++p) {
      Tier& t = tiers[a][p];
      t.stage = 0;
      // (a workgroup launch: when it fits at all; few instances run at once)
      if (lds_base(a, t) + 4 * nst <= (t.gw > 1 ? static_cast<size_t>(lds_max) : stage_budget)) t.stage = 1;
    }
  auto lds_of = [&](int a, const Tier& t) -> size_t { return lds_base(a, t) + (t.stage ? 4 * nst : 0); };
  for (int a = 0; a < n_sim && err == hipSuccess; ++a)
    for (int p = 0; p < n_tiers[a] && err == hipSuccess; ++p)
      if (lds_of(a, tiers[a][p]) > 65536)
        err = hipFuncSetAttribute(sim_kernel_any(sim_algos[a], tiers[a][p], P.order && tiers[a][p].grid <= 0,
                                                 P.pclass != nullptr, rounds),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds_of(a, tiers[a][p])));
  if (err == hipSuccess && o.event_before) err = hipEventRecord(static_cast<hipEvent_t>(o.event_before), st);
  // adaptive: the A_l launches go to the side stream after the preparation,
  // and the caller's stream waits for them before the end (fork and join)
  hipStream_t side = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  if (err == hipSuccess && n_sim == 2 && !no_alloc) {
    err = side_stream(dev, &side);
    if (err == hipSuccess) err = hipEventCreateWithFlags(&fork, hipEventDisableTiming);
    if (err == hipSuccess) err = hipEventCreateWithFlags(&join, hipEventDisableTiming);
    if (err == hipSuccess) err = hipEventRecord(fork, st);
    if (err == hipSuccess) err = hipStreamWaitEvent(side, fork, 0);
  }
  for (int a = 0; a < n_sim && err == hipSuccess; ++a) {
    const hipStream_t sa = a == 1 && side ? side : st;
    for (int p = 0; p < n_tiers[a] && err == hipSuccess; ++p) {
      const Tier& t = tiers[a][p];
      sk::Params q = P;
      q.cap_v = t.cap_v;
      q.retry_status = t.rows_status;
      q.retry_v_status = t.v_status;
      q.run_mask = t.run_mask;
      q.stage_comp = t.stage;
      void* args[] = {&q};
      const dim3 tgrid(t.grid > 0 ? t.grid : P.K), tblock(64 * (t.gw > 1 ? t.gw : 1));
      // (a launch over every instance may take them in the launch order)
      err = hipLaunchKernel(sim_kernel_any(sim_algos[a], t, P.order && t.grid <= 0, P.pclass != nullptr, rounds), tgrid,
                            tblock, args, lds_of(a, t), sa);
    }
  }
  if (side) {
    // join even after a failed launch, so that the workspace is not freed
    // while work queued on the side stream may still use it
    hipError_t je = join ? hipEventRecord(join, side) : hipErrorInvalidValue;
    if (je == hipSuccess) je = hipStreamWaitEvent(st, join, 0);
    if (je != hipSuccess) je = hipStreamSynchronize(side);
    if (err == hipSuccess) err = je;
  }
  if (fork) (void)hipEventDestroy(fork);
  if (join) (void)hipEventDestroy(join);
  if (err == hipSuccess && o.event_after) err = hipEventRecord(static_cast<hipEvent_t>(o.event_after), st);
  const hipError_t ferr = no_alloc ? hipSuccess : hipFreeAsync(ws, st);
  if (err != hipSuccess || ferr != hipSuccess) return SCHED_E_HIP;
  return SCHED_OK;
}

}  // namespace

extern "C" {

int sched_simulate_opts(const sched_instances_t* in, int32_t algo, int64_t M,
                        const sched_results_t* out, void* stream, const sched_options_t* opts) {
  return simulate_impl(in, algo, M, out, stream, opts, false);
}

int sched_simulate_noalloc(const sched_instances_t* in, int32_t algo, int64_t M,
                           const sched_results_t* out, void* stream, const sched_options_t* opts) {
  return simulate_impl(in, algo, M, out, stream, opts, true);
}

int sched_simulate(const sched_instances_t* in, int32_t algo, int64_t M,
                   const sched_results_t* out, void* stream) {
  return sched_simulate_opts(in, algo, M, out, stream, nullptr);
}

}  // extern "C"
