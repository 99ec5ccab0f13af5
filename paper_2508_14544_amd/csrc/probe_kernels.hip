// probe_kernels.hip -- throughput probes that confirm, on the running GPU, the
// peaks the simulation kernel's roofline is priced against: 32-bit integer
// VALU lane-operations per second and LDS read bytes per second.  Measurement
// infrastructure only (a library of its own); no part of the simulator uses it.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "schedprobe.h"

namespace {

constexpr int kChains = 8;   // independent add chains per lane
constexpr int kUnroll = 16;  // adds per chain per loop iteration

// Every lane runs kChains independent chains of v_add_u32 (one instruction
// each, written as inline asm so the compiler cannot fold repeated adds).
__global__ __launch_bounds__(256) void k_probe_valu(uint32_t* out, int iters) {
  uint32_t x[kChains];
#pragma unroll
  for (int j = 0; j < kChains; ++j) x[j] = threadIdx.x + j;
  const uint32_t c = blockIdx.x | 1u;
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
#pragma unroll
      for (int j = 0; j < kChains; ++j) asm volatile("v_add_u32 %0, %1, %0" : "+v"(x[j]) : "s"(c));
    }
  }
  uint32_t acc = 0;
#pragma unroll
  for (int j = 0; j < kChains; ++j) acc ^= x[j];
  out[blockIdx.x * blockDim.x + threadIdx.x] = acc;
}

// Every lane reads 16 B per load from its own LDS slot (a wave covers 1 KiB,
// no bank conflicts); the slot moves with the iteration so no load repeats.
__global__ __launch_bounds__(256) void k_probe_lds(uint32_t* out, int iters) {
  __shared__ uint4 buf[4096];  // 64 KiB
  for (int i = threadIdx.x; i < 4096; i += blockDim.x) buf[i] = make_uint4(i, i + 1, i + 2, i + 3);
  __syncthreads();
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  uint4 acc = make_uint4(0, 0, 0, 0);
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int slot = (((i * 8 + u) * 4 + w) & 63) * 64 + lane;  // < 4096
      const uint4 v = buf[slot];
      acc.x += v.x;
      acc.y ^= v.y;
      acc.z += v.z;
      acc.w ^= v.w;
    }
  }
  out[blockIdx.x * blockDim.x + threadIdx.x] = acc.x ^ acc.y ^ acc.z ^ acc.w;
}

// Launches `kernel` (blocks x 256 threads) twice and times the second launch.
template <typename K>
int time_kernel(K kernel, int blocks, int iters, float* ms) {
  uint32_t* out = nullptr;
  if (hipMalloc(&out, sizeof(uint32_t) * static_cast<size_t>(blocks) * 256) != hipSuccess) return -1;
  hipEvent_t e0, e1;
  int rc = -1;
  if (hipEventCreate(&e0) == hipSuccess) {
    if (hipEventCreate(&e1) == hipSuccess) {
      hipLaunchKernelGGL(kernel, dim3(blocks), dim3(256), 0, nullptr, out, iters);
      const bool ok = hipGetLastError() == hipSuccess && hipEventRecord(e0, nullptr) == hipSuccess;
      hipLaunchKernelGGL(kernel, dim3(blocks), dim3(256), 0, nullptr, out, iters);
      if (ok && hipGetLastError() == hipSuccess && hipEventRecord(e1, nullptr) == hipSuccess &&
          hipEventSynchronize(e1) == hipSuccess && hipEventElapsedTime(ms, e0, e1) == hipSuccess)
        rc = 0;
      (void)hipEventDestroy(e1);
    }
    (void)hipEventDestroy(e0);
  }
  if (hipFree(out) != hipSuccess) rc = -1;
  return rc;
}

int blocks_for_device(int per_cu) {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return cus * per_cu;
}

}  // namespace

extern "C" int sched_probe_valu(int iters, double* lane_ops_per_s) {
  if (iters <= 0 || !lane_ops_per_s) return -1;
  const int blocks = blocks_for_device(8);  // 32 waves per CU
  if (blocks <= 0) return -1;
  float ms = 0.f;
  if (time_kernel(k_probe_valu, blocks, iters, &ms) != 0 || ms <= 0.f) return -1;
  const double ops = static_cast<double>(blocks) * 256.0 * iters * kUnroll * kChains;
  *lane_ops_per_s = ops / (ms * 1e-3);
  return 0;
}

extern "C" int sched_probe_lds(int iters, double* bytes_per_s) {
  if (iters <= 0 || !bytes_per_s) return -1;
  const int blocks = blocks_for_device(2);  // 64 KiB of LDS and 4 waves per block
  if (blocks <= 0) return -1;
  float ms = 0.f;
  if (time_kernel(k_probe_lds, blocks, iters, &ms) != 0 || ms <= 0.f) return -1;
  const double bytes = static_cast<double>(blocks) * 256.0 * iters * 8 * 16;
  *bytes_per_s = bytes / (ms * 1e-3);
  return 0;
}
