// Tree vector quantisation of the keys (Sec. 3.2 nearest-codeword assignment,
// Sec. 4.2 / Alg. 1 parent then child loop) for gfx950, in two kernels.
//
// Distances are evaluated as ||c||^2 - 2 k.c, which has the argmin of
// ||k - c||^2. k.c comes from MFMA on the transposed product C . K^T
// (codewords as rows, keys as columns), so each lane owns one key column and
// four consecutive codewords; ||c||^2 is summed per codeword with one fixed
// routine, so identical codewords give identical distances.
//
// In both kernels one side of the product is scaled by -2 (exact in bf16 and
// fp32: the keys in the parent kernel, the candidate rows in the child
// kernel) and the MFMA accumulator starts at ||c||^2, so the accumulator holds
// the distance itself.
//
// parent_stream_kernel (below) when the head's parent codebook fits the LDS
// (always for bf16); otherwise (fp32 codebooks of more rows)
// parent_assign_kernel: one workgroup = 256 keys of one (batch, head), 4
// waves of 64 keys. The norms of the head's parents are summed once per
// workgroup (one row per thread, in order); the parent codebook streams
// through LDS in chunks of 64 rows by direct global->LDS copies, double
// buffered. Every lane keeps a running (distance, index) minimum over its
// rows in ascending codeword order with a strict <, and the four lane groups
// merge lexicographically, so exact ties go to the lowest index.
//
// child_assign_kernel: one workgroup owns one (batch, head) and a range of F
// parents. It scans the head's parent indices in rounds, buckets the keys of
// its parents by parent (integer LDS atomics: histogram, prefix sum,
// scatter), and turns each parent's bucket into groups of 16 keys. For a
// group, one MFMA tile holds the candidates of Alg. 1's child loop as rows:
// row 0 the parent, rows 1..Ch its children (Ch = 16: a second tile for the
// last child). All candidates, the parent included, go through the same
// routine, so a child equal to its parent has exactly the parent's distance.
// The nearest child (strict <, lowest index) replaces the parent only if its
// distance is strictly smaller.
#include "avq_child.hpp"
#include "avq_common.hpp"

#include <algorithm>
#include <type_traits>

namespace avq {

// XOR swizzle of the 16-byte units of a staged codebook row: the 16 rows a
// tile reads (16 tt + c) get distinct units for the same logical unit.
template <int U>
__device__ __forceinline__ int assign_swizzle(int r) {
  if constexpr (U >= 16) return r & 15;
  return (r >> 1) & 7;  // U = 8: two rows per 256 bytes
}

__device__ __forceinline__ void copy16_lds(const void* src, void* lds) {
  __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)src,
                                   (void __attribute__((address_space(3)))*)lds, 16, 0, 0);
}

// fp32 only (a bf16 codebook of up to 512 rows always fits the stream kernel)
template <int D>
struct AssignCfg {
  static constexpr int kWaves = 4;
  static constexpr int KS = 4;                    // key subtiles (of 16) per wave
  static constexpr int kKeysPerBlock = kWaves * KS * 16;
  static constexpr int CW = 64;                   // codebook rows per chunk
  static constexpr int KQ = D / 4;                // MFMA k-steps over d
  static constexpr int EPU = 4;                   // values per 16-byte unit
  static constexpr int U = D / 4;                 // 16-byte units per row
  static constexpr int COPIES = CW * U / 64;      // wave copies per chunk
  static constexpr int CPW = COPIES / kWaves;
  static constexpr int CHUNK_BYTES = CW * D * 4;
  static constexpr int BUF_BYTES = CHUNK_BYTES;
  static constexpr int M0MAX = 512;
  static constexpr int LDS_BYTES = 2 * BUF_BYTES + M0MAX * 4;  // two chunks + all norms
  static_assert(COPIES % kWaves == 0, "copies split evenly over the waves");
};

template <int D>
__global__ __launch_bounds__((AssignCfg<D>::kWaves * 64)) void parent_assign_kernel(
    const float* __restrict__ K, const float* __restrict__ Cp, int32_t* __restrict__ parent_idx,
    int32_t* __restrict__ code_idx, int H, int N, int M0, int blocks_per_bh) {
  using Cfg = AssignCfg<D>;
  using T = float;
  constexpr int KS = Cfg::KS, CW = Cfg::CW, KQ = Cfg::KQ, U = Cfg::U, EPU = Cfg::EPU,
                CPW = Cfg::CPW;
  extern __shared__ __attribute__((aligned(16))) unsigned char lds_raw[];

  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = tid % kWave;
  const int g = lane / 16, c = lane % 16;
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = blk / blocks_per_bh;
  const int h = bh % H;
  const int key0 = (blk % blocks_per_bh) * Cfg::kKeysPerBlock + wave * KS * 16;
  const T* cp_head = Cp + (size_t)h * M0 * D;

  // chunk staging: copy i of this wave covers rows (64 j + lane) / U
  auto issue = [&](int k) {
    unsigned char* B = lds_raw + (k % 2) * Cfg::BUF_BYTES;
#pragma unroll
    for (int i = 0; i < CPW; ++i) {
      const int j = wave + Cfg::kWaves * i;
      const int q = 64 * j + lane;
      const int r = q / U, pu = q % U;
      const T* src = cp_head + (size_t)min(CW * k + r, M0 - 1) * D + (pu ^ assign_swizzle<U>(r)) * EPU;
      copy16_lds(src, B + 1024 * j);
    }
  };
  const int n_chunks = (M0 + CW - 1) / CW;
  issue(0);
  float* lnorm = reinterpret_cast<float*>(lds_raw + 2 * Cfg::BUF_BYTES);  // [M0MAX]
  // ||row||^2 in one fixed order (ascending d)
  for (int r = tid; r < n_chunks * CW; r += blockDim.x) {
    float acc = __builtin_inff();
    if (r < M0) {
      const T* row = cp_head + (size_t)r * D;
      acc = 0.f;
#pragma unroll 8
      for (int d0 = 0; d0 < D; ++d0) acc = fmaf(row[d0], row[d0], acc);
    }
    lnorm[r] = acc;
  }

  // key fragments: subtile s holds key key0 + 16 s + c; lane group g holds
  // the d values of k-step kq at 4 kq + g
  float kf[KS][KQ];
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const int j = key0 + 16 * s + c;
    const T* row = K + ((size_t)bh * N + (j < N ? j : 0)) * D;
#pragma unroll
    for (int kq = 0; kq < KQ; ++kq) kf[s][kq] = times_minus2((j < N) ? row[4 * kq + g] : 0.f);
  }

  float best[KS];
  int bidx[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    best[s] = __builtin_inff();
    bidx[s] = 0;
  }

  for (int k = 0; k < n_chunks; ++k) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (k + 1 < n_chunks) issue(k + 1);
    const unsigned char* B = lds_raw + (k % 2) * Cfg::BUF_BYTES;
    const T* lc = reinterpret_cast<const T*>(B);
#pragma unroll
    for (int tt = 0; tt < CW / 16; ++tt) {
      const int r = 16 * tt + c;
      const int sw = assign_swizzle<U>(r);
      // the accumulator starts at ||c||^2 of the lane's rows 4 g + q
      const f32x4 nr = *reinterpret_cast<const f32x4*>(&lnorm[CW * k + 16 * tt + 4 * g]);
      f32x4 acc[KS];
#pragma unroll
      for (int kq = 0; kq < KQ; ++kq) {
        const float a = lc[r * D + (kq ^ sw) * EPU + g];
#pragma unroll
        for (int s = 0; s < KS; ++s) acc[s] = mfma_f32(a, kf[s][kq], kq == 0 ? nr : acc[s]);
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int row = CW * k + 16 * tt + 4 * g + q;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const float dist = acc[s][q];
          if (dist < best[s]) {
            best[s] = dist;
            bidx[s] = row;
          }
        }
      }
    }
  }

  // merge the four lane groups: lexicographic (distance, index) minimum
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    merge_xor<16, false>(best[s], bidx[s]);
    merge_xor<32, false>(best[s], bidx[s]);
    const int j = key0 + 16 * s + c;
    if (g == 0 && j < N) {
      parent_idx[(size_t)bh * N + j] = bidx[s];
      if (code_idx) code_idx[(size_t)bh * N + j] = bidx[s];  // flat codebook
    }
  }
}

// ---------------------------------------------------------------------------
// parent_stream_kernel: the same argmin when the head's whole parent codebook
// fits the LDS (bf16: one 16-wave workgroup per CU, up to 150 KB, every
// supported codebook; fp32: two 4-wave workgroups per CU, half the LDS
// each). Each workgroup is persistent over a run of consecutive steps
// (normally of one (batch, head)): the codebook and its norms are staged once
// per head, and the key fragments of the next step load while the current
// step runs, so K streams from HBM without the gaps of a one-shot workgroup.
// It keeps the keys unscaled and maximises k.c - ||c||^2 / 2, which is the
// distance times -1/2 exactly.
template <typename T, int D>
struct StreamCfg {
  static constexpr bool kB = Elem<T>::kBf16;
  // bf16: 16 waves of 32 keys (under 128 VGPRs, four waves per SIMD); fp32:
  // 4 waves of 64 keys (its fragments need the registers of two waves per
  // SIMD) and two workgroups per CU
  static constexpr int kWaves = kB ? 16 : 4;
  static constexpr int kPerCU = kB ? 1 : 2;       // workgroups per CU
  static constexpr int KS = kB ? 2 : 4;           // key subtiles (of 16) per wave
  static constexpr int kKeysPerStep = kWaves * KS * 16;
  static constexpr int KQ = kB ? D / 32 : D / 4;
  static constexpr int ESZ = sizeof(T);
  static constexpr int EPU = 16 / ESZ;
  static constexpr int U = D * ESZ / 16;
  static constexpr int ROW_BYTES = D * ESZ;
  static constexpr int LDS_CAP = kB ? 150 * 1024 : 80 * 1024;
  // codebook rows padded to whole pairs of 16-row tiles, then the norms
  static int lds_bytes(int M0) { return ((M0 + 31) / 32 * 32) * (ROW_BYTES + 4); }
  static bool fits(int M0) { return lds_bytes(M0) <= LDS_CAP; }
};

template <typename T, int D>
__global__ __launch_bounds__((StreamCfg<T, D>::kWaves * 64)) void parent_stream_kernel(
    const T* __restrict__ K, const T* __restrict__ Cp, int32_t* __restrict__ parent_idx,
    int32_t* __restrict__ code_idx, int H, int N, int M0, int steps_per_bh, int n_steps) {
  using Cfg = StreamCfg<T, D>;
  constexpr bool kB = Cfg::kB;
  constexpr int KS = Cfg::KS, KQ = Cfg::KQ, U = Cfg::U, EPU = Cfg::EPU;
  using Frag = typename std::conditional<kB, bf16x8, float>::type;
  extern __shared__ __attribute__((aligned(16))) unsigned char lds_raw[];

  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = tid % kWave;
  const int g = lane / 16, c = lane % 16;
  const int M16 = (M0 + 31) / 32 * 32;  // whole pairs of 16-row tiles
  const T* lc = reinterpret_cast<const T*>(lds_raw);                           // [M16][D]
  float* lnorm = reinterpret_cast<float*>(lds_raw + (size_t)M16 * Cfg::ROW_BYTES);  // [M16]

  // a contiguous run of steps per workgroup
  const int wg = xcd_remap(blockIdx.x, gridDim.x);
  const int per = (n_steps + gridDim.x - 1) / gridDim.x;
  const int s_begin = wg * per, s_end = min(s_begin + per, n_steps);
  if (s_begin >= s_end) return;  // whole workgroup

  // raw key fragments of step st: subtile s holds key key0 + 16 s + c, lane
  // group g the d values of k-step kq at 32 kq + 8 g (bf16) or 4 kq + g (fp32);
  // keys past N read key N - 1
  auto load_keys = [&](int st, Frag (&dst)[KS][KQ]) {
    const int bh = st / steps_per_bh;
    const int key0 = (st % steps_per_bh) * Cfg::kKeysPerStep + wave * KS * 16;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int j = min(key0 + 16 * s + c, N - 1);
      const T* row = K + ((size_t)bh * N + j) * D;
#pragma unroll
      for (int kq = 0; kq < KQ; ++kq) {
        if constexpr (kB)
          dst[s][kq] = *reinterpret_cast<const bf16x8*>(row + 32 * kq + 8 * g);
        else
          dst[s][kq] = row[4 * kq + g];
      }
    }
  };

  Frag kn[KS][KQ];
  load_keys(s_begin, kn);
  int cur_h = -1;
  for (int st = s_begin; st < s_end; ++st) {
    const int bh = st / steps_per_bh, h = bh % H;
    if (h != cur_h) {
      // stage head h's codebook: row r's 16-byte unit u at unit u ^ swizzle(r)
      __syncthreads();  // every wave is done with the previous head
      const T* cp_head = Cp + (size_t)h * M0 * D;
      const int copies = M16 * U / 64;
      for (int j = wave; j < copies; j += Cfg::kWaves) {
        const int q = 64 * j + lane;
        const int r = q / U, pu = q % U;
        copy16_lds(cp_head + (size_t)min(r, M0 - 1) * D + (pu ^ assign_swizzle<U>(r)) * EPU,
                   lds_raw + 1024 * j);
      }
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      // norms in one fixed order (consecutive units), +inf past M0 - 1
      for (int r = tid; r < M16; r += blockDim.x) {
        const int sw = assign_swizzle<U>(r);
        float acc = 0.f;
#pragma unroll
        for (int u = 0; u < U; ++u) {
          if constexpr (kB) {
            acc = frag_sq<T>(*reinterpret_cast<const bf16x8*>(&lc[r * D + (u ^ sw) * EPU]), acc);
          } else {
            const float4 v = *reinterpret_cast<const float4*>(&lc[r * D + (u ^ sw) * EPU]);
            acc = fmaf(v.x, v.x, acc);
            acc = fmaf(v.y, v.y, acc);
            acc = fmaf(v.z, v.z, acc);
            acc = fmaf(v.w, v.w, acc);
          }
        }
        // the products below give k.c - ||c||^2 / 2 = -(||c||^2 - 2 k.c) / 2
        // exactly (power-of-two scales), so the nearest row is the largest
        lnorm[r] = r < M0 ? -0.5f * acc : -__builtin_inff();
      }
      __syncthreads();
      cur_h = h;
    }

    // this step's keys and the next step's loads
    Frag kf[KS][KQ];
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int kq = 0; kq < KQ; ++kq) kf[s][kq] = kn[s][kq];
    if (st + 1 < s_end) load_keys(st + 1, kn);

    // per key subtile: the largest value so far, its 16-row tile, and that
    // tile's 4 values of the lane (the row within the tile is found once at
    // the end): 8 VALU per tile and subtile instead of 12 for a running
    // (value, row) pair
    float best[KS];
    int btile[KS];
    f32x4 bv[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      best[s] = -__builtin_inff();
      btile[s] = 0;
      if constexpr (kB) bv[s] = f32x4{best[s], best[s], best[s], best[s]};
    }
    // two 16-row tiles per step: all their row fragments are read before
    // the products, and the second tile's products overlap the first
    // tile's comparisons
    for (int tt = 0; tt < M16 / 16; tt += 2) {
      f32x4 acc[2][KS];
      Frag a[2][KQ];
      f32x4 nr[2];
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        const int r = 16 * (tt + h2) + c;
        const int sw = assign_swizzle<U>(r);
        // the accumulator starts at -||c||^2 / 2 of the lane's rows
        nr[h2] = *reinterpret_cast<const f32x4*>(&lnorm[16 * (tt + h2) + 4 * g]);
#pragma unroll
        for (int kq = 0; kq < KQ; ++kq) {
          if constexpr (kB)
            a[h2][kq] = *reinterpret_cast<const bf16x8*>(&lc[r * D + ((4 * kq + g) ^ sw) * EPU]);
          else
            a[h2][kq] = lc[r * D + (kq ^ sw) * EPU + g];
        }
      }
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
        for (int kq = 0; kq < KQ; ++kq)
#pragma unroll
          for (int s = 0; s < KS; ++s) {
            if constexpr (kB)
              acc[h2][s] = mfma_bf16(a[h2][kq], kf[s][kq], kq == 0 ? nr[h2] : acc[h2][s]);
            else
              acc[h2][s] = mfma_f32(a[h2][kq], kf[s][kq], kq == 0 ? nr[h2] : acc[h2][s]);
          }
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const f32x4 v = acc[h2][s];
          if constexpr (kB) {
            // the new best is a max of the tile's values and the old best
            // (two three-way maxima); it exceeds the old one only if the tile
            // holds a larger value (strict: the earlier tile keeps a tie)
            const float nb = fmaxf(fmaxf(fmaxf(fmaxf(v[0], v[1]), v[2]), v[3]), best[s]);
            const bool gt = nb > best[s];
            best[s] = nb;
            btile[s] = gt ? tt + h2 : btile[s];
#pragma unroll
            for (int q = 0; q < 4; ++q) bv[s][q] = gt ? v[q] : bv[s][q];
          } else {
            // fp32: no registers to spare for the tile's values; a running
            // (value, row) pair, the first (lowest) row keeping a tie
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const bool gt = v[q] > best[s];
              best[s] = gt ? v[q] : best[s];
              btile[s] = gt ? 4 * (tt + h2) + q : btile[s];
            }
          }
        }
    }
    // the row: bf16, the first of the best tile's 4 rows that holds the best
    // value; fp32, recorded as 4 tile + q
    int bidx[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      if constexpr (kB) {
        const int q = bv[s][0] == best[s] ? 0 : bv[s][1] == best[s] ? 1 : bv[s][2] == best[s] ? 2 : 3;
        bidx[s] = 16 * btile[s] + 4 * g + q;
      } else {
        bidx[s] = 16 * (btile[s] / 4) + 4 * g + btile[s] % 4;
      }
    }
    // merge the four lane groups: largest value, lowest index on ties
    const int key0 = (st % steps_per_bh) * Cfg::kKeysPerStep + wave * KS * 16;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      merge_xor<16, true>(best[s], bidx[s]);
      merge_xor<32, true>(best[s], bidx[s]);
      const int j = key0 + 16 * s + c;
      if (g == 0 && j < N) {
        parent_idx[(size_t)bh * N + j] = bidx[s];
        if (code_idx) code_idx[(size_t)bh * N + j] = bidx[s];  // flat codebook
      }
    }
  }
}

// ---------------------------------------------------------------------------
constexpr int kChildThreads = 1024;
constexpr int kChildWaves = kChildThreads / kWave;
constexpr int kScanPerThread = 8;
constexpr int kChildRound = kChildThreads * kScanPerThread;  // parent indices per round
constexpr int kMinChildChunk = 256;  // fewest keys a split of the child compare takes
constexpr int kMaxFam = 32;

struct ChildLds {
  int qkey[kChildRound];           // keys of this range, scan order
  unsigned char qfam[kChildRound]; // their family (parent - p0)
  int skey[kChildRound];           // keys bucketed by family
  int hist[kMaxFam];
  int start[kMaxFam + 1];
  int cursor[kMaxFam];
  int item_start[kMaxFam + 1];     // first group index of each family
  int wave_count[kScanPerThread][kChildWaves];  // queued keys per (round slot, wave)
  int wave_off[kScanPerThread][kChildWaves];    // their queue offsets
  int qlen;
};
static_assert(kScanPerThread * kChildWaves <= 128, "one wave scans the slot offsets");

// NT: 16-row candidate tiles (the parent and its Ch children): 1 for Ch < 16,
// 2 for Ch = 16.
template <typename T, int D, int NT>
__global__ __launch_bounds__(kChildThreads) void child_assign_kernel(
    const T* __restrict__ K, const T* __restrict__ Cp, const T* __restrict__ Cc,
    const int32_t* __restrict__ parent_idx, int32_t* __restrict__ code_idx, int H, int N, int M0,
    int Ch, int F, int ranges, int splits, int chunk) {
  using Frag = typename std::conditional<Elem<T>::kBf16, bf16x8, float>::type;
  constexpr bool kB = Elem<T>::kBf16;
  constexpr int KQ = kB ? D / 32 : D / 4;
  extern __shared__ __attribute__((aligned(16))) unsigned char lds_raw[];
  ChildLds& L = *reinterpret_cast<ChildLds*>(lds_raw);

  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int g = lane / 16, c = lane % 16;
  // workgroup (bh, family range, key split), the split fastest: the splits
  // of one family range share its candidate rows in one L2
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int split = blk % splits;
  const int bh = blk / splits / ranges;
  const int h = bh % H;
  const int p0 = (blk / splits % ranges) * F;
  const int kbegin = split * chunk, kend = min(N, kbegin + chunk);
  const int nfam = min(F, M0 - p0);
  const int32_t* pidx = parent_idx + (size_t)bh * N;
  const T* kh = K + (size_t)bh * N * D;
  constexpr bool kPrefetch = kB && D == 64;
  int cur_fam = -1;  // the family whose rows the wave holds
  Frag cf[NT][KQ];
  f32x4 cn[NT];

  // the 16 keys of group it (B operand); key index of lane c
  auto load_keys = [&](int f, int it, Frag (&kf)[KQ], int& key, bool& valid) {
    const int kb = L.start[f] + 16 * (it - L.item_start[f]);
    valid = kb + c < L.start[f + 1];
    key = L.skey[valid ? kb + c : kb];
    child_key<T, D, NT>(kh + (size_t)key * D, g, kf);
  };

  for (int base = kbegin; base < kend; base += kChildRound) {
    // 1. queue the keys of this range in scan order
    int cur[kScanPerThread];
#pragma unroll
    for (int k = 0; k < kScanPerThread; ++k) {
      const int j = base + k * kChildThreads + tid;
      const int p = j < kend ? pidx[j] : -1;
      cur[k] = (p >= p0 && p < p0 + nfam) ? p - p0 : -1;
    }
    unsigned long long mask[kScanPerThread];
#pragma unroll
    for (int k = 0; k < kScanPerThread; ++k) {
      mask[k] = __ballot(cur[k] >= 0);
      if (lane == 0) L.wave_count[k][wave] = __popcll(mask[k]);
    }
    if (tid < kMaxFam) L.hist[tid] = 0;
    __syncthreads();
    if (wave == 0) {
      const int tot = prefix128(&L.wave_count[0][0], &L.wave_off[0][0],
                                kScanPerThread * kChildWaves, lane);
      if (lane == 0) L.qlen = tot;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kScanPerThread; ++k) {
      if (cur[k] >= 0) {
        const int slot = L.wave_off[k][wave] + bits_below(mask[k]);
        L.qkey[slot] = base + k * kChildThreads + tid;
        L.qfam[slot] = (unsigned char)cur[k];
        atomicAdd(&L.hist[cur[k]], 1);
      }
    }
    const int qlen = L.qlen;
    __syncthreads();
    if (qlen == 0) continue;  // uniform
    // 2. bucket by family; groups of 16 keys per family
    if (wave == 0) {
      const int v = lane < nfam ? L.hist[lane] : 0;
      const int gv = (v + 15) / 16;
      const int incl = wave_incl_scan(v), gincl = wave_incl_scan(gv);
      if (lane < nfam) {
        L.start[lane] = incl - v;
        L.cursor[lane] = incl - v;
        L.item_start[lane] = gincl - gv;
      }
      if (lane == nfam - 1) {
        L.start[nfam] = incl;
        L.item_start[nfam] = gincl;
      }
    }
    __syncthreads();
    for (int e = tid; e < qlen; e += kChildThreads)
      L.skey[atomicAdd(&L.cursor[L.qfam[e]], 1)] = L.qkey[e];
    __syncthreads();
    // 3. each wave takes a contiguous run of groups (a group is 16 keys of
    //    one family), so that consecutive groups of a wave mostly share the
    //    family, whose rows stay in registers
    //    The next group's keys load while the current group is compared.
    const int n_items = L.item_start[nfam];
    const int per_wave = (n_items + kChildWaves - 1) / kChildWaves;
    const int it_begin = wave * per_wave, it_end = min(n_items, it_begin + per_wave);
    int f = 0;
    Frag kf[KQ];
    int key = 0;
    bool valid = false;
    if (it_begin < it_end) {
      while (L.item_start[f + 1] <= it_begin) ++f;  // wave-uniform
      load_keys(f, it_begin, kf, key, valid);
    }
    for (int it = it_begin; it < it_end; ++it) {
      const int p = p0 + f;
      Frag kn[KQ];
      int key_n = 0, fn = f;
      bool valid_n = false;
      if (it + 1 < it_end) {
        while (L.item_start[fn + 1] <= it + 1) ++fn;  // wave-uniform
        // a second set of key registers fits the 128 of a 1024-thread
        // workgroup for bf16 at d = 64 only; otherwise the keys load just in
        // time
        if constexpr (kPrefetch) load_keys(fn, it + 1, kn, key_n, valid_n);
      }
      if constexpr (!kPrefetch) {
        if (it > it_begin) load_keys(f, it, kf, key, valid);
      }
      if (p != cur_fam) {
        child_rows<T, D, NT>(Cp, Cc, h, M0, Ch, p, g, c, cf, cn);
        cur_fam = p;
      }
      const int row = child_pick<T, D, NT>(cf, cn, kf, Ch, g, c);
      if (g == 0 && valid) code_idx[(size_t)bh * N + key] = row > 0 ? M0 + p * Ch + row - 1 : p;
#pragma unroll
      for (int kq = 0; kq < KQ; ++kq) kf[kq] = kn[kq];
      key = key_n;
      valid = valid_n;
      f = fn;
    }
    __syncthreads();  // the queue is reused by the next round
  }
}

template <typename T, int D>
hipError_t launch_assign(int BH, int H, int N, int M0, int Ch, const void* K, const void* Cp,
                         const void* Cc, int32_t* parent_idx, int32_t* code_idx,
                         bool with_children, hipStream_t stream) {
  using SCfg = StreamCfg<T, D>;
  long long grid;
  DeviceInfo dev;
  hipError_t e = device_info(&dev);
  if (e != hipSuccess) return e;
  if (SCfg::fits(M0)) {
    // persistent: kPerCU workgroups per CU, each a run of whole steps
    const int per_bh = (N + SCfg::kKeysPerStep - 1) / SCfg::kKeysPerStep;
    const long long n_steps = (long long)BH * per_bh;
    if (n_steps > 0x7fffffff) return hipErrorInvalidConfiguration;
    const long long slots = (long long)SCfg::kPerCU * (dev.cus > 0 ? dev.cus : 1);
    const long long per = (n_steps + slots - 1) / slots;
    grid = (n_steps + per - 1) / per;
    const int lds = SCfg::lds_bytes(M0);
    constexpr int slot_s = 32 + (Elem<T>::kBf16 ? 0 : 2) + (D == 128 ? 1 : 0);
    e = ensure_dynamic_lds((const void*)parent_stream_kernel<T, D>, SCfg::LDS_CAP, slot_s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((parent_stream_kernel<T, D>), dim3((unsigned)grid),
                       dim3(SCfg::kWaves * kWave), lds, stream,
                       static_cast<const T*>(K), static_cast<const T*>(Cp), parent_idx,
                       Ch == 0 ? code_idx : nullptr, H, N, M0, per_bh, (int)n_steps);
  } else if constexpr (!Elem<T>::kBf16) {
    using Cfg = AssignCfg<D>;
    const int per_bh = (N + Cfg::kKeysPerBlock - 1) / Cfg::kKeysPerBlock;
    grid = (long long)BH * per_bh;
    if (grid > 0x7fffffff) return hipErrorInvalidConfiguration;
    constexpr int slot_a = 24 + (D == 128 ? 1 : 0);
    e = ensure_dynamic_lds((const void*)parent_assign_kernel<D>, Cfg::LDS_BYTES, slot_a);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((parent_assign_kernel<D>), dim3((unsigned)grid),
                       dim3(Cfg::kWaves * kWave), Cfg::LDS_BYTES, stream,
                       static_cast<const float*>(K), static_cast<const float*>(Cp), parent_idx,
                       Ch == 0 ? code_idx : nullptr, H, N, M0, per_bh);
  } else {
    return hipErrorInvalidValue;  // not reached: bf16 codebooks of up to 512 rows fit
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (Ch == 0) return hipSuccess;  // flat codebook: the parent is the code
  if (!with_children) return hipSuccess;  // the caller runs the child compare

  // child compare: F parents per workgroup, and the keys split into chunks
  // of at most one scan round each (the keys are independent: a workgroup
  // scans only its chunk, so the splits add no scan work; they shorten each
  // wave's chain of groups and let the grid fill the device in whole rounds).
  // When the family ranges alone would leave CUs idle (few heads, few
  // parents), the chunks shrink, to no fewer than kMinChildChunk keys, so
  // that about one workgroup per CU runs.
  const int F = kMaxFam;
  const int ranges = (M0 + F - 1) / F;
  const long long base_grid = (long long)BH * ranges;
  int chunk = kChildRound;
  if (base_grid < (long long)dev.cus) {
    const long long per = ((long long)dev.cus + base_grid - 1) / base_grid;  // splits wanted
    const long long c = ((long long)N + per - 1) / per;
    chunk = (int)std::min<long long>(kChildRound, std::max<long long>(kMinChildChunk, (c + 63) / 64 * 64));
  }
  const int splits = (N + chunk - 1) / chunk;
  grid = base_grid * splits;
  if (grid > 0x7fffffff) return hipErrorInvalidConfiguration;
  auto launch_child = [&](auto kernel, int slot) {
    hipError_t err = ensure_dynamic_lds((const void*)kernel, (int)sizeof(ChildLds), slot);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(kernel, dim3((unsigned)grid), dim3(kChildThreads), sizeof(ChildLds),
                       stream, static_cast<const T*>(K), static_cast<const T*>(Cp),
                       static_cast<const T*>(Cc), parent_idx, code_idx, H, N, M0, Ch, F, ranges,
                       splits, chunk);
    return hipGetLastError();
  };
  constexpr int slot_b = 100 + ((Elem<T>::kBf16 ? 0 : 2) + (D == 128 ? 1 : 0)) * 2;
  if (Ch + 1 > 16) return launch_child(child_assign_kernel<T, D, 2>, slot_b + 1);
  return launch_child(child_assign_kernel<T, D, 1>, slot_b);
}

template hipError_t launch_assign<bf16, 64>(int, int, int, int, int, const void*, const void*,
                                            const void*, int32_t*, int32_t*, bool, hipStream_t);
template hipError_t launch_assign<bf16, 128>(int, int, int, int, int, const void*, const void*,
                                             const void*, int32_t*, int32_t*, bool, hipStream_t);
template hipError_t launch_assign<float, 64>(int, int, int, int, int, const void*, const void*,
                                             const void*, int32_t*, int32_t*, bool, hipStream_t);
template hipError_t launch_assign<float, 128>(int, int, int, int, int, const void*, const void*,
                                              const void*, int32_t*, int32_t*, bool, hipStream_t);

}  // namespace avq
