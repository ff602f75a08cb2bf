// Shared device helpers for the gfx950 AVQ kernels: element types, MFMA
// wrappers with their lane layouts, wave-level shuffles.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace avq {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
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

// Row swaps of gfx950 (v_permlane16_swap / v_permlane32_swap of a register
// with itself: VALU, no LDS round trip): every lane receives the value of the
// even and of the odd row of its pair of 16-lane (ROW = 16) or 32-lane rows,
// i.e. its own value and that of lane l ^ ROW, in row order.
template <int ROW>
__device__ __forceinline__ void row_pair(unsigned x, unsigned& even, unsigned& odd) {
  static_assert(ROW == 16 || ROW == 32, "rows of 16 or 32 lanes");
  if constexpr (ROW == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    even = r[0];
    odd = r[1];
  } else {
    const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
    even = r[0];
    odd = r[1];
  }
}
// x + (x of lane l ^ ROW) in every lane: the same sum as with a shuffle, as
// the addition commutes
template <int ROW>
__device__ __forceinline__ float add_xor(float x) {
  unsigned e, o;
  row_pair<ROW>(__float_as_uint(x), e, o);
  return __uint_as_float(e) + __uint_as_float(o);
}
template <int ROW>
__device__ __forceinline__ float max_xor(float x) {
  unsigned e, o;
  row_pair<ROW>(__float_as_uint(x), e, o);
  return fmaxf(__uint_as_float(e), __uint_as_float(o));
}
// The value of lane l % 16 (row 0) in every lane: row 0 into row 1 and row 2
// into row 3 (the even rows of the 16-lane swap), then the lower half into
// the upper one (the even row of the 32-lane swap).
__device__ __forceinline__ float from_row0(float x) {
  unsigned e, o, e2, o2;
  row_pair<16>(__float_as_uint(x), e, o);
  row_pair<32>(e, e2, o2);
  return __uint_as_float(e2);
}
// (value, index) of lanes l and l ^ ROW merged in both: the larger value
// (kMax) or the smaller one, the lower index on ties
template <int ROW, bool kMax>
__device__ __forceinline__ void merge_xor(float& v, int& i) {
  unsigned ve, vo, ie, io;
  row_pair<ROW>(__float_as_uint(v), ve, vo);
  row_pair<ROW>((unsigned)i, ie, io);
  const float a = __uint_as_float(ve), b = __uint_as_float(vo);
  const int ia = (int)ie, ib = (int)io;
  const bool take_b = (kMax ? b > a : b < a) || (b == a && ib < ia);
  v = take_b ? b : a;
  i = take_b ? ib : ia;
}

// Inclusive prefix sum over the 64 lanes of a wave with data-parallel-primitive
// adds (no LDS): a Hillis-Steele scan inside each row of 16 lanes (row_shr
// 1, 2, 4, 8; lanes whose source lies before the row start add 0), then the
// last lane of row 0 into row 1 and of row 2 into row 3 (row_bcast:15), and
// the last lane of row 1 into rows 2 and 3 (row_bcast:31).
__device__ __forceinline__ int wave_incl_scan(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, false);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, false);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, false);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, false);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);  // row_bcast:15, rows 1 and 3
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);  // row_bcast:31, rows 2 and 3
  return x;
}
// The value of the wave's last lane, in a scalar register.
__device__ __forceinline__ int last_lane(int x) { return __builtin_amdgcn_readlane(x, kWave - 1); }

// Set bits of a wave-wide mask in the lanes below the calling one (v_mbcnt:
// no lane mask held in registers).
__device__ __forceinline__ int bits_below(unsigned long long m) {
  return (int)__builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32),
                                        __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u));
}

// Data-parallel-primitive lane moves inside each row of 16 lanes (VALU, no
// LDS). CTRL encodings: quad_perm [1,0,3,2] = 0xB1, [2,3,0,1] = 0x4E,
// [3,2,1,0] = 0x1B, row_half_mirror = 0x141, row_ror:8 = 0x128.
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
// Value of lane (i ^ MASK) for MASK in {1, 2, 4, 8}, within a row of 16 lanes.
template <int MASK>
__device__ __forceinline__ float xor16(float v) {
  if constexpr (MASK == 1) return dpp<0xB1>(v);
  if constexpr (MASK == 2) return dpp<0x4E>(v);
  if constexpr (MASK == 4) return dpp<0x1B>(dpp<0x141>(v));  // i^7 then i^3
  if constexpr (MASK == 8) return dpp<0x128>(v);               // rotate a row by 8
  return v;
}

constexpr float kLog2e = 1.4426950408889634f;

// fp32 exp(x) (every weight here is exp of a logit minus a running max): the
// hardware base-2 exponential of x * log2(e).
__device__ __forceinline__ float exp_neg(float x) {
  return __builtin_amdgcn_exp2f(x * kLog2e);
}
// Hardware base-2 exponential and logarithm (fp32).
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float log2_hw(float x) { return __builtin_amdgcn_logf(x); }

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

// Exclusive prefix sums of n <= 128 counts (run by one whole wave): off[i] =
// cnt[0] + ... + cnt[i-1]; returns the total to every lane.
__device__ __forceinline__ int prefix128(const int* cnt, int* off, int n, int lane) {
  // the lane index passes an empty asm statement: the addresses below are
  // computed here, not hoisted out of the caller's loop and held (or spilled)
  asm volatile("" : "+v"(lane));
  const int a = lane < n ? cnt[lane] : 0;
  const int b = lane + kWave < n ? cnt[lane + kWave] : 0;
  const int ia = wave_incl_scan(a), ib = wave_incl_scan(b);
  const int ta = last_lane(ia);
  if (lane < n) off[lane] = ia - a;
  if (lane + kWave < n) off[lane + kWave] = ta + ib - b;
  return ta + last_lane(ib);
}

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

// Per-device facts the launchers need, queried once per device.
struct DeviceInfo {
  int lds_max = 0;  // bytes of LDS one workgroup may use
  int cus = 0;      // compute units
};
hipError_t device_info(DeviceInfo* out);

// Raises a kernel's dynamic-LDS limit once per device (the attribute is a
// property of the kernel on the current device).
hipError_t ensure_dynamic_lds(const void* kernel, int bytes, int slot);

}  // namespace avq
