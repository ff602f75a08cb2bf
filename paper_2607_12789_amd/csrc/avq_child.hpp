// The child compare of tree quantisation (Alg. 1's inner loop, Sec. 4.2):
// for 16 keys of one parent p, the nearest of p's Ch children, and whether it
// is strictly nearer than p itself.
//
// One MFMA tile holds the candidates as rows: row 0 the parent, rows 1..Ch
// its children (Ch = 16: a second tile for the last child; rows past Ch
// repeat the last child and are ignored). The keys are the tile's 16
// columns. Every candidate, the parent included, goes through the same
// routine: ||c||^2 summed in one fixed order, the row scaled by -2 (exact),
// and the product accumulated onto ||c||^2, so the accumulator holds
// ||c||^2 - 2 k.c, which has the argmin of ||k - c||^2; a child equal to its
// parent has exactly the parent's distance. The nearest child is the
// lexicographic (distance, child) minimum; it replaces the parent only when
// strictly nearer.
//
// Used by the assignment's child kernel and by the fused assign + aggregate
// kernel, so both give the same codes.
#pragma once

#include "avq_common.hpp"

#include <type_traits>

namespace avq {

// Sum of squares of the 8 (bf16) or 1 (fp32) values of a fragment, in order.
template <typename T>
__device__ __forceinline__ float frag_sq(
    const typename std::conditional<Elem<T>::kBf16, bf16x8, float>::type& v, float acc) {
  if constexpr (Elem<T>::kBf16) {
#pragma unroll
    for (int i = 0; i < 8; i += 2) {
      const bf16x2 p = {v[i], v[i + 1]};
      acc = __builtin_amdgcn_fdot2_f32_bf16(p, p, acc, false);
    }
    return acc;
  } else {
    return fmaf(v, v, acc);
  }
}

// -2 x, exactly (a power-of-two scale)
__device__ __forceinline__ bf16x8 times_minus2(const bf16x8& v) {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = (bf16)(-2.f * (float)v[i]);
  return r;
}
__device__ __forceinline__ float times_minus2(float v) { return -2.f * v; }

template <typename T, int D, int NT>
struct ChildTile {
  static constexpr bool kB = Elem<T>::kBf16;
  static constexpr int KQ = kB ? D / 32 : D / 4;  // MFMA k-steps over d
  using Frag = typename std::conditional<kB, bf16x8, float>::type;
};

// The candidate rows of parent p of head h (A operand): lane (g, c) holds row
// c of each tile, k-step kq at d = 32 kq + 8 g (bf16) or 4 kq + g (fp32).
// Then each row's ||c||^2 (each lane sums its quarter of row c in order, the
// quarters are combined in a fixed order, then moved to the lanes that hold
// the row's products), and the rows scaled by -2.
template <typename T, int D, int NT>
__device__ __forceinline__ void child_rows(
    const T* __restrict__ Cp, const T* __restrict__ Cc, int h, int M0, int Ch, int p, int g,
    int c, typename ChildTile<T, D, NT>::Frag (&cf)[NT][ChildTile<T, D, NT>::KQ],
    f32x4 (&cn)[NT]) {
  constexpr int KQ = ChildTile<T, D, NT>::KQ;
#pragma unroll
  for (int t2 = 0; t2 < NT; ++t2) {
    const int cand = 16 * t2 + c;
    const T* row = cand == 0 ? Cp + ((size_t)h * M0 + p) * D
                             : Cc + (((size_t)h * M0 + p) * Ch + min(cand - 1, Ch - 1)) * D;
#pragma unroll
    for (int kq = 0; kq < KQ; ++kq) {
      if constexpr (Elem<T>::kBf16)
        cf[t2][kq] = *reinterpret_cast<const bf16x8*>(row + 32 * kq + 8 * g);
      else
        cf[t2][kq] = row[4 * kq + g];
    }
  }
#pragma unroll
  for (int t2 = 0; t2 < NT; ++t2) {
    float part = 0.f;
#pragma unroll
    for (int kq = 0; kq < KQ; ++kq) part = frag_sq<T>(cf[t2][kq], part);
    // (lane groups 0 + 1, then + (2 + 3), the same order in every lane)
    const float nrm = add_xor<32>(add_xor<16>(part));
#pragma unroll
    for (int r = 0; r < 4; ++r) cn[t2][r] = __shfl(nrm, 4 * g + r, kWave);
#pragma unroll
    for (int kq = 0; kq < KQ; ++kq) cf[t2][kq] = times_minus2(cf[t2][kq]);
  }
}

// Key fragments of one key row (B operand, column c of the tile).
template <typename T, int D, int NT>
__device__ __forceinline__ void child_key(const T* __restrict__ krow, int g,
                                          typename ChildTile<T, D, NT>::Frag (&kf)[ChildTile<T, D, NT>::KQ]) {
  constexpr int KQ = ChildTile<T, D, NT>::KQ;
#pragma unroll
  for (int kq = 0; kq < KQ; ++kq) {
    if constexpr (Elem<T>::kBf16)
      kf[kq] = *reinterpret_cast<const bf16x8*>(krow + 32 * kq + 8 * g);
    else
      kf[kq] = krow[4 * kq + g];
  }
}

// The family-local row of the key in column c: 0 if the parent stays, else
// 1 + the nearest child. The same in all four lane groups.
template <typename T, int D, int NT>
__device__ __forceinline__ int child_pick(
    const typename ChildTile<T, D, NT>::Frag (&cf)[NT][ChildTile<T, D, NT>::KQ],
    const f32x4 (&cn)[NT], const typename ChildTile<T, D, NT>::Frag (&kf)[ChildTile<T, D, NT>::KQ],
    int Ch, int g, int c) {
  constexpr int KQ = ChildTile<T, D, NT>::KQ;
  float dpar = 0.f, dch = __builtin_inff();
  int cbest = 0;
#pragma unroll
  for (int t2 = 0; t2 < NT; ++t2) {
    f32x4 acc = cn[t2];
#pragma unroll
    for (int kq = 0; kq < KQ; ++kq) {
      if constexpr (Elem<T>::kBf16)
        acc = mfma_bf16(cf[t2][kq], kf[kq], acc);
      else
        acc = mfma_f32(cf[t2][kq], kf[kq], acc);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int cand = 16 * t2 + 4 * g + r;
      if (cand == 0) dpar = acc[r];
      if (cand >= 1 && cand <= Ch && acc[r] < dch) {
        dch = acc[r];
        cbest = cand - 1;
      }
    }
  }
  // parent distance from lane group 0; children by the lexicographic
  // (distance, child) minimum over the lane groups
  dpar = from_row0(dpar);
  merge_xor<16, false>(dch, cbest);
  merge_xor<32, false>(dch, cbest);
  return dch < dpar ? 1 + cbest : 0;
}

}  // namespace avq
