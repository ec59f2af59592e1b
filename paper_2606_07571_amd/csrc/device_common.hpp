// Device-side building blocks shared by the gfx950 kernels: vector types,
// the bf16 MFMA wrapper, bf16 conversion and the XCD-aware block remap.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bc {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;
constexpr int kXcds = 8;  // MI355X: 8 accelerator complex dies, one L2 each

// D(32x32, fp32) += A(32x16, bf16) * B(16x32, bf16), one wave.
// Lane l (half = l/32, c = l%32) supplies A[row c][k slot (half, e)] and
// B[k slot (half, e)][col c], e = 0..7; it receives D[row 8j + 4*half + i][col c]
// in element 4j + i (i, j = 0..3).  A and B share the same k-slot order, so any
// consistent assignment of k indices to slots gives the same product.
__device__ __forceinline__ f32x16 mfma_32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}

// Round-to-nearest-even float -> bf16 (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ bf16 to_bf16(float x) { return (bf16)x; }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  bf16x2 v = {(bf16)lo, (bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float bf16_to_f32(bf16 x) { return (float)x; }

// Workgroups are dispatched round-robin over the XCDs (block i -> XCD i % 8).
// Returns a logical index such that each XCD receives a contiguous range of
// logical indices, so neighbouring tiles (which share operands) meet in one L2.
// A bijection on [0, n) for any n.
__device__ __forceinline__ int xcd_remap(int bid, int n) {
  const int q = n / kXcds, r = n % kXcds;
  const int x = bid % kXcds, k = bid / kXcds;
  return x * q + (x < r ? x : r) + k;
}

// v_permlane32_swap(x, x) returns, in every lane l, the pair {x[l], x[l ^ 32]}
// (in some order), so the max / sum over lanes l and l ^ 32 needs no LDS.
__device__ __forceinline__ float half_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float half_sum(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

}  // namespace bc
