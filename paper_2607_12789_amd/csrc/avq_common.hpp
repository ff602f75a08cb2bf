// Shared device helpers for the gfx950 AVQ kernels: element types, MFMA
// wrappers with their lane layouts, wave-level shuffles.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace avq {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// MFMA tiles used by every kernel (layouts checked on gfx950):
//
// v_mfma_f32_16x16x32_bf16  D[16x16] += A[16x32] * B[32x16]
//   lane l, g = l / 16, c = l % 16
//   A operand: A[c][8g .. 8g+7]        (8 bf16)
//   B operand: B[8g .. 8g+7][c]        (8 bf16)
//   D:         D[4g + r][c], r = 0..3  (4 fp32)
//
// v_mfma_f32_16x16x4_f32    D[16x16] += A[16x4] * B[4x16]
//   A operand: A[c][g]; B operand: B[g][c]; D as above.
//
// Both kernels that use them compute transposed products (codewords as the
// D rows, queries or keys as the D columns) so that each lane owns one token
// column and four consecutive codewords.
// ---------------------------------------------------------------------------
__device__ __forceinline__ f32x4 mfma_bf16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x4 mfma_f32(float a, float b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float shfl_xor(float v, int mask) { return __shfl_xor(v, mask, kWave); }
__device__ __forceinline__ int shfl_xor(int v, int mask) { return __shfl_xor(v, mask, kWave); }

// fp32 exp(x) for x <= 0 (every weight here is exp of a logit minus a running
// max): the hardware base-2 exponential of x * log2(e).
__device__ __forceinline__ float exp_neg(float x) {
  return __builtin_amdgcn_exp2f(x * 1.4426950408889634f);
}

template <typename T>
__device__ __forceinline__ float to_f32(T v) { return (float)v; }

template <typename T>
struct Elem;
template <>
struct Elem<float> {
  static constexpr bool kBf16 = false;
};
template <>
struct Elem<bf16> {
  static constexpr bool kBf16 = true;
};

// Maps a linear workgroup index to a tile index so that consecutive tiles run
// on the same XCD: workgroups are dispatched round-robin over the 8 XCDs, so
// workgroup i lands on XCD i % 8. With the remap, XCD x processes the
// contiguous tile range [x * n/8, (x+1) * n/8), which keeps the tiles of one
// (batch, head) and their shared codebook/aggregate rows in one L2.
__device__ __forceinline__ int xcd_remap(int i, int n) {
  constexpr int kXcd = 8;
  if (n % kXcd != 0) return i;
  return (i % kXcd) * (n / kXcd) + i / kXcd;
}

}  // namespace avq
