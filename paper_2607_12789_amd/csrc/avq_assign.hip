// Tree vector quantisation of the keys (Sec. 3.2 nearest-codeword assignment,
// Sec. 4.2 / Alg. 1 parent then child loop) for gfx950.
//
// One workgroup = 4 waves = 256 keys of one (batch, head). Each wave owns 64
// keys (4 subtiles of 16). The parent codebook of the head streams through LDS
// in chunks of 64 rows; every chunk is used by all four waves.
//
// Parent argmin: distances are evaluated as ||c||^2 - 2 k.c, the form whose
// argmin over c equals that of ||k - c||^2. k.c comes from MFMA computing the
// transposed product C . K^T (codewords as rows, keys as columns), so each lane
// owns one key column and four consecutive codewords; the lane keeps a running
// (distance, index) minimum over its rows in ascending codeword order (strict
// <, so the lowest index wins exact ties), and the four lane groups merge
// lexicographically. ||c||^2 is summed once per staged row in fixed order, so
// identical codewords give identical distances.
//
// Child compare: the key is compared with the Ch children of its parent and,
// with the same routine, with the parent itself, so that a child identical to
// its parent gives exactly the parent's distance. For bf16 the routine is
// ||c||^2 - 2 k.c with both dot products taken by packed bf16 dot2
// instructions (products exact, fp32 accumulation); for fp32 it is the direct
// sum of (k - c)^2. Each lane group sums its quarter of d and the quarters are
// combined by the same butterfly for every candidate. A key moves to its
// nearest child only if that value is strictly below the parent's (equal
// values keep the parent). Candidates are gathered four at a time so their
// loads overlap.
#include "avq_common.hpp"

namespace avq {

template <typename T, int D>
struct AssignCfg {
  static constexpr bool kB = Elem<T>::kBf16;
  static constexpr int kWaves = 4;
  static constexpr int KS = 4;                    // key subtiles (of 16) per wave
  static constexpr int kKeysPerBlock = kWaves * KS * 16;
  static constexpr int CW = 64;                   // codebook rows per LDS chunk
  static constexpr int KQ = kB ? D / 32 : D / 4;  // MFMA k-steps over d
  static constexpr int PAD = kB ? 8 : 4;          // 16 bytes of row padding
  static constexpr int ROW = D + PAD;
  static constexpr int SLOT = kB ? 8 : 1;         // d values per lane per k-step
};

template <typename T, int D>
__global__ __launch_bounds__(256) void assign_kernel(const T* __restrict__ K,
                                                     const T* __restrict__ Cp,
                                                     const T* __restrict__ Cc,
                                                     int32_t* __restrict__ parent_idx,
                                                     int32_t* __restrict__ code_idx, int H,
                                                     int N, int M0, int Ch,
                                                     int blocks_per_bh) {
  using Cfg = AssignCfg<T, D>;
  constexpr bool kB = Cfg::kB;
  constexpr int KS = Cfg::KS, CW = Cfg::CW, KQ = Cfg::KQ, ROW = Cfg::ROW;
  using Frag = typename std::conditional<kB, bf16x8, float>::type;

  __shared__ __attribute__((aligned(16))) T lc[CW * ROW];
  __shared__ float lnorm[CW];

  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = tid % kWave;
  const int g = lane / 16, c = lane % 16;
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = blk / blocks_per_bh;
  const int h = bh % H;
  const int key0 = (blk % blocks_per_bh) * Cfg::kKeysPerBlock + wave * KS * 16;

  // Key fragments: subtile s holds key key0 + 16 s + c; lane group g holds the
  // d values of k-step kq at 32 kq + 8 g (bf16) or 4 kq + g (fp32).
  Frag kf[KS][KQ];
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const int j = key0 + 16 * s + c;
    const T* row = K + ((size_t)bh * N + (j < N ? j : 0)) * D;
#pragma unroll
    for (int kq = 0; kq < KQ; ++kq) {
      if constexpr (kB) {
        bf16x8 v = *reinterpret_cast<const bf16x8*>(row + 32 * kq + 8 * g);
        kf[s][kq] = (j < N) ? v : bf16x8{};
      } else {
        float v = row[4 * kq + g];
        kf[s][kq] = (j < N) ? v : 0.f;
      }
    }
  }

  float best[KS];
  int bidx[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    best[s] = __builtin_inff();
    bidx[s] = 0;
  }

  const T* cp_head = Cp + (size_t)h * M0 * D;
  for (int base = 0; base < M0; base += CW) {
    // Stage rows [base, base + CW) of the parent codebook (zero rows past M0).
    constexpr int VEC = 16 / sizeof(T);
    constexpr int VPR = D / VEC;
    for (int v = tid; v < CW * VPR; v += blockDim.x) {
      const int r = v / VPR, col = (v % VPR) * VEC;
      uint4 val = {0u, 0u, 0u, 0u};
      if (base + r < M0)
        val = *reinterpret_cast<const uint4*>(cp_head + (size_t)(base + r) * D + col);
      *reinterpret_cast<uint4*>(&lc[r * ROW + col]) = val;
    }
    __syncthreads();
    {
      // ||c||^2 of every staged row: four threads per row, each summing a
      // quarter of d in order, combined in a fixed order (identical codewords
      // give identical norms).
      static_assert(CW * 4 == 256, "four threads per staged row");
      const int r = tid / 4, qd = tid % 4;
      float s2 = 0.f;
      for (int e = qd * (D / 4); e < (qd + 1) * (D / 4); ++e) {
        const float x = to_f32(lc[r * ROW + e]);
        s2 = fmaf(x, x, s2);
      }
      s2 += shfl_xor(s2, 1);
      s2 += shfl_xor(s2, 2);
      if (qd == 0) lnorm[r] = (base + r < M0) ? s2 : __builtin_inff();
    }
    __syncthreads();

#pragma unroll
    for (int tt = 0; tt < CW / 16; ++tt) {
      if (base + 16 * tt >= M0) break;
      f32x4 acc[KS];
#pragma unroll
      for (int s = 0; s < KS; ++s) acc[s] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kq = 0; kq < KQ; ++kq) {
        if constexpr (kB) {
          const bf16x8 a =
              *reinterpret_cast<const bf16x8*>(&lc[(16 * tt + c) * ROW + 32 * kq + 8 * g]);
#pragma unroll
          for (int s = 0; s < KS; ++s) acc[s] = mfma_bf16(a, kf[s][kq], acc[s]);
        } else {
          const float a = lc[(16 * tt + c) * ROW + 4 * kq + g];
#pragma unroll
          for (int s = 0; s < KS; ++s) acc[s] = mfma_f32(a, kf[s][kq], acc[s]);
        }
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 16 * tt + 4 * g + r;
        const float nrm = lnorm[row];
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const float dist = fmaf(-2.f, acc[s][r], nrm);
          if (dist < best[s]) {
            best[s] = dist;
            bidx[s] = base + row;
          }
        }
      }
    }
    __syncthreads();
  }

  // Merge the four lane groups: lexicographic (distance, index) minimum.
#pragma unroll
  for (int s = 0; s < KS; ++s) {
#pragma unroll
    for (int m = 16; m <= 32; m <<= 1) {
      const float ob = shfl_xor(best[s], m);
      const int oi = shfl_xor(bidx[s], m);
      if (ob < best[s] || (ob == best[s] && oi < bidx[s])) {
        best[s] = ob;
        bidx[s] = oi;
      }
    }
  }

  // Child compare (Alg. 1): the parent and its children through one routine.
  // Candidate 0 is the parent, candidate 1 + c is child c.
  constexpr int kBatch = 4;
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const int j = key0 + 16 * s + c;
    const int p = bidx[s];
    const T* kids = Cc + ((size_t)h * M0 + p) * Ch * D;
    float dpar = 0.f, dch = __builtin_inff();
    int cbest = 0;
    for (int b0 = 0; b0 <= Ch; b0 += kBatch) {
      Frag cv[kBatch][KQ];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int cand = min(b0 + u, Ch);  // clamped: slots past Ch are ignored
        const T* code = cand == 0 ? cp_head + (size_t)p * D : kids + (size_t)(cand - 1) * D;
#pragma unroll
        for (int kq = 0; kq < KQ; ++kq) {
          if constexpr (kB)
            cv[u][kq] = *reinterpret_cast<const bf16x8*>(code + 32 * kq + 8 * g);
          else
            cv[u][kq] = code[4 * kq + g];
        }
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        float part;
        if constexpr (kB) {
          float dotkc = 0.f, dotcc = 0.f;
#pragma unroll
          for (int kq = 0; kq < KQ; ++kq) {
#pragma unroll
            for (int i = 0; i < 8; i += 2) {
              const bf16x2 kk = {kf[s][kq][i], kf[s][kq][i + 1]};
              const bf16x2 cc = {cv[u][kq][i], cv[u][kq][i + 1]};
              dotkc = __builtin_amdgcn_fdot2_f32_bf16(kk, cc, dotkc, false);
              dotcc = __builtin_amdgcn_fdot2_f32_bf16(cc, cc, dotcc, false);
            }
          }
          dotkc += shfl_xor(dotkc, 16);
          dotkc += shfl_xor(dotkc, 32);
          dotcc += shfl_xor(dotcc, 16);
          dotcc += shfl_xor(dotcc, 32);
          part = fmaf(-2.f, dotkc, dotcc);
        } else {
          part = 0.f;
#pragma unroll
          for (int kq = 0; kq < KQ; ++kq) {
            const float diff = kf[s][kq] - cv[u][kq];
            part = fmaf(diff, diff, part);
          }
          part += shfl_xor(part, 16);
          part += shfl_xor(part, 32);
        }
        const int cand = b0 + u;
        if (cand == 0) {
          dpar = part;
        } else if (cand <= Ch && part < dch) {
          dch = part;
          cbest = cand - 1;
        }
      }
    }
    if (g == 0 && j < N) {
      const size_t o = (size_t)bh * N + j;
      parent_idx[o] = p;
      code_idx[o] = (dch < dpar) ? (M0 + p * Ch + cbest) : p;
    }
  }
}

template <typename T, int D>
hipError_t launch_assign(int BH, int H, int N, int M0, int Ch, const void* K, const void* Cp,
                         const void* Cc, int32_t* parent_idx, int32_t* code_idx,
                         hipStream_t stream) {
  using Cfg = AssignCfg<T, D>;
  const int per_bh = (N + Cfg::kKeysPerBlock - 1) / Cfg::kKeysPerBlock;
  const long long grid = (long long)BH * per_bh;
  if (grid > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((assign_kernel<T, D>), dim3((unsigned)grid), dim3(Cfg::kWaves * kWave), 0,
                     stream, static_cast<const T*>(K), static_cast<const T*>(Cp),
                     static_cast<const T*>(Cc), parent_idx, code_idx, H, N, M0, Ch, per_bh);
  return hipGetLastError();
}

template hipError_t launch_assign<bf16, 64>(int, int, int, int, int, const void*, const void*,
                                            const void*, int32_t*, int32_t*, hipStream_t);
template hipError_t launch_assign<bf16, 128>(int, int, int, int, int, const void*, const void*,
                                             const void*, int32_t*, int32_t*, hipStream_t);
template hipError_t launch_assign<float, 64>(int, int, int, int, int, const void*, const void*,
                                             const void*, int32_t*, int32_t*, hipStream_t);
template hipError_t launch_assign<float, 128>(int, int, int, int, int, const void*, const void*,
                                              const void*, int32_t*, int32_t*, hipStream_t);

}  // namespace avq
