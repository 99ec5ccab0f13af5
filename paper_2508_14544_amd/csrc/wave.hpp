// wave.hpp -- wave64 primitives for gfx950 (CDNA4).
//
// Reductions run a DPP butterfly inside each row of 16 lanes (quad_perm
// 1,0,3,2 / 2,3,0,1, then row_half_mirror and row_mirror), after which every
// lane of a row holds the row result; the four row results are combined in
// scalar registers via v_readlane.  The result is wave-uniform.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wave {

constexpr int kDppQuadXor1 = 0xB1;    // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;    // quad_perm [2,3,0,1]
constexpr int kDppRowHalfMirror = 0x141;
constexpr int kDppRowMirror = 0x140;

__device__ __forceinline__ int lane_id() { return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)); }

__device__ __forceinline__ uint64_t ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }

__device__ __forceinline__ int32_t readlane(int32_t v, int lane) { return __builtin_amdgcn_readlane(v, lane); }

__device__ __forceinline__ uint32_t readlane_u(uint32_t v, int lane) {
  return static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int32_t>(v), lane));
}

__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int lane) {
  uint32_t lo = readlane_u(static_cast<uint32_t>(v), lane);
  uint32_t hi = readlane_u(static_cast<uint32_t>(v >> 32), lane);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// v with lane `lane` replaced by the uniform value s (the other lanes keep v).
// `lane` must come from scalar arithmetic (not straight from a VALU-written
// SGPR such as v_readlane's result), which needs no wait states.
__device__ __forceinline__ int32_t writelane(int32_t v, int32_t s, int lane) {
  const int32_t su = __builtin_amdgcn_readfirstlane(s);
  const int32_t lu = __builtin_amdgcn_readfirstlane(lane);
  asm("v_writelane_b32 %0, %1, %2" : "+v"(v) : "s"(su), "{m0}"(lu));
  return v;
}

__device__ __forceinline__ uint32_t writelane_u(uint32_t v, uint32_t s, int lane) {
  return static_cast<uint32_t>(writelane(static_cast<int32_t>(v), static_cast<int32_t>(s), lane));
}

__device__ __forceinline__ int32_t uniform(int32_t v) { return __builtin_amdgcn_readfirstlane(v); }

template <int CTRL>
__device__ __forceinline__ int32_t dpp(int32_t v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}

__device__ __forceinline__ int32_t max_i32(int32_t v) {
  v = max(v, dpp<kDppQuadXor1>(v));
  v = max(v, dpp<kDppQuadXor2>(v));
  v = max(v, dpp<kDppRowHalfMirror>(v));
  v = max(v, dpp<kDppRowMirror>(v));
  int32_t a = readlane(v, 0), b = readlane(v, 16), c = readlane(v, 32), d = readlane(v, 48);
  return max(max(a, b), max(c, d));
}

__device__ __forceinline__ int32_t sum_i32(int32_t v) {
  v += dpp<kDppQuadXor1>(v);
  v += dpp<kDppQuadXor2>(v);
  v += dpp<kDppRowHalfMirror>(v);
  v += dpp<kDppRowMirror>(v);
  return readlane(v, 0) + readlane(v, 16) + readlane(v, 32) + readlane(v, 48);
}

__device__ __forceinline__ uint32_t min_u32(uint32_t v) {
  auto m = [](uint32_t x, uint32_t y) { return x < y ? x : y; };
  v = m(v, static_cast<uint32_t>(dpp<kDppQuadXor1>(static_cast<int32_t>(v))));
  v = m(v, static_cast<uint32_t>(dpp<kDppQuadXor2>(static_cast<int32_t>(v))));
  v = m(v, static_cast<uint32_t>(dpp<kDppRowHalfMirror>(static_cast<int32_t>(v))));
  v = m(v, static_cast<uint32_t>(dpp<kDppRowMirror>(static_cast<int32_t>(v))));
  uint32_t a = readlane_u(v, 0), b = readlane_u(v, 16), c = readlane_u(v, 32), d = readlane_u(v, 48);
  return m(m(a, b), m(c, d));
}

// 64-bit sums for the epilogue (not on the hot path).
__device__ __forceinline__ int64_t sum_i64(int64_t v) {
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ int64_t max_i64(int64_t v) {
  for (int off = 32; off >= 1; off >>= 1) {
    int64_t o = __shfl_xor(v, off, 64);
    v = o > v ? o : v;
  }
  return v;
}

// Inclusive prefix sum over the wave (setup only).
__device__ __forceinline__ int32_t inclusive_scan_i32(int32_t v) {
  const int lane = lane_id();
  for (int off = 1; off < 64; off <<= 1) {
    int32_t o = __shfl_up(v, off, 64);
    if (lane >= off) v += o;
  }
  return v;
}

}  // namespace wave
