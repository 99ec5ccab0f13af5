// wave.hpp -- wave64 primitives for gfx950 (CDNA4).
//
// 32-bit reductions first fold the four 16-lane rows onto each other with the
// gfx950 lane swaps (v_permlane32_swap, v_permlane16_swap), then run a DPP
// butterfly inside each row (quad_perm 1,0,3,2 / 2,3,0,1, row_half_mirror,
// row_mirror); every lane then holds the result, read once with
// v_readfirstlane.  The result is wave-uniform.
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

// v_writelane_b32 through its LLVM intrinsic (this compiler has no clang builtin
// for it): the compiler knows its semantics and inserts the wait states.
extern "C" __device__ int32_t sk_llvm_writelane(int32_t src, int32_t lane, int32_t old)
    __asm("llvm.amdgcn.writelane");

// v with lane `lane` replaced by the uniform value s (the other lanes keep v)
__device__ __forceinline__ int32_t writelane(int32_t v, int32_t s, int lane) {
  return sk_llvm_writelane(s, lane, v);
}

__device__ __forceinline__ uint32_t writelane_u(uint32_t v, uint32_t s, int lane) {
  return static_cast<uint32_t>(writelane(static_cast<int32_t>(v), static_cast<int32_t>(s), lane));
}

__device__ __forceinline__ int32_t uniform(int32_t v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ uint32_t uniform_u(uint32_t v) {
  return static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int32_t>(v)));
}

// The same value, held in vector registers: the compiler treats the result
// as varying per lane.  For wave-uniform state that is used rarely (array
// base addresses, counters), so that it does not take scalar registers
// through the hot loops; loads and stores take vector addresses anyway.
template <typename T>
__device__ __forceinline__ T in_vgpr(T v) {
  asm volatile("" : "+v"(v));
  return v;
}

template <int CTRL>
__device__ __forceinline__ int32_t dpp(int32_t v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}

// Cross-row folds (gfx950): after fold_rows every lane holds OP over the four
// lanes {l mod 16 + 16 k}; v_permlane32_swap exchanges the two 32-lane halves
// and v_permlane16_swap the odd and even 16-lane rows.
template <typename F>
__device__ __forceinline__ uint32_t fold_rows(uint32_t v, F op) {
  const auto h = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  v = op(static_cast<uint32_t>(h[0]), static_cast<uint32_t>(h[1]));
  const auto q = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return op(static_cast<uint32_t>(q[0]), static_cast<uint32_t>(q[1]));
}

template <typename F>
__device__ __forceinline__ uint32_t fold_in_row(uint32_t v, F op) {
  v = op(v, static_cast<uint32_t>(dpp<kDppQuadXor1>(static_cast<int32_t>(v))));
  v = op(v, static_cast<uint32_t>(dpp<kDppQuadXor2>(static_cast<int32_t>(v))));
  v = op(v, static_cast<uint32_t>(dpp<kDppRowHalfMirror>(static_cast<int32_t>(v))));
  v = op(v, static_cast<uint32_t>(dpp<kDppRowMirror>(static_cast<int32_t>(v))));
  return v;
}

struct OpMaxI32 {
  __device__ uint32_t operator()(uint32_t a, uint32_t b) const {
    return static_cast<int32_t>(a) > static_cast<int32_t>(b) ? a : b;
  }
};
struct OpAddU32 {
  __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return a + b; }
};
struct OpMinU32 {
  __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return a < b ? a : b; }
};

__device__ __forceinline__ int32_t max_i32(int32_t v) {
  const uint32_t r = fold_in_row(fold_rows(static_cast<uint32_t>(v), OpMaxI32{}), OpMaxI32{});
  return uniform(static_cast<int32_t>(r));
}

__device__ __forceinline__ int32_t sum_i32(int32_t v) {
  const uint32_t r = fold_in_row(fold_rows(static_cast<uint32_t>(v), OpAddU32{}), OpAddU32{});
  return uniform(static_cast<int32_t>(r));
}

// The sum left in every lane (a vector value): for tests that combine it with
// other per-lane conditions before a single ballot.
__device__ __forceinline__ int32_t sum_i32_all(int32_t v) {
  return static_cast<int32_t>(fold_in_row(fold_rows(static_cast<uint32_t>(v), OpAddU32{}), OpAddU32{}));
}

// The minimum left in every lane, for locating it with a ballot without a
// round trip through a scalar register.
__device__ __forceinline__ uint32_t min_u32_all(uint32_t v) { return fold_in_row(fold_rows(v, OpMinU32{}), OpMinU32{}); }

__device__ __forceinline__ uint32_t min_u32(uint32_t v) {
  const uint32_t r = fold_in_row(fold_rows(v, OpMinU32{}), OpMinU32{});
  return static_cast<uint32_t>(uniform(static_cast<int32_t>(r)));
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
