// Fused refined-codebook attention (Sec. 4.3, Alg. 2) for gfx950.
//
// One workgroup processes one query tile (block_q consecutive tokens of one
// (batch, head)); each wave owns 32 query rows. Everything is computed
// transposed, codewords x queries: S^T = C . Q^T and Xbar^T = Vmean^T . W^T.
// With the 16x16 MFMA layouts a lane owns one query column and four
// consecutive codeword rows, so
//   - the weights that come out of exp2() are already in the register layout
//     of the MFMA operand of the next product (no shuffles);
//   - the Ch children of one parent sit in one lane's consecutive rows (plus
//     the partner lane groups for Ch = 8, 16): the recovered parent logit of
//     Eq. (parent_recovery) is an in-register sum;
//   - per-query softmax state is per lane.
//
// Log-count bias (App. D): a codeword's logit enters as
// t = S log2(e) + log2(n), so its weight exp2(t - m) is n exp(S - m'); empty
// codewords get t = -inf and drop out of the running max and of every sum
// without masks. The values are the means Vbar/n written by the aggregation
// (groups of 4 codes, [d][4]), so sum_j n_j exp(S_j - m') Vbar_j / n_j is the
// numerator of Eq. (vqflashattention). The parent logit recovered from the
// children uses the unbiased child logits, and the correcting weight of child
// c is n_c (exp(T_c - m') - exp(Srec - m')), Eq. (correcting_attention) times
// n_c. The denominator (the sum of the weights) comes out of the value MFMA
// through one extra d-tile whose first row is all ones, so numerator and
// denominator use the same rounded weights.
//
// Codewords stream through LDS in chunks of CW rows, copied by direct
// global->LDS loads (no registers, no VALU): codeword rows XOR-swizzled by
// 16-byte unit so that the 16 lanes reading 16 rows hit different banks, and
// the packed mean values as they lie in memory. Phases per tile:
//   1. parent sweep: per chunk, logits, running max, weights, fp32 parent
//      denominator, Xbar += Vmean^T W (online softmax);
//   2. importance (Eq. (importance)) with the final max and denominator: a
//      second sweep recomputes the parent logits chunk by chunk (or reuses
//      them when all parents fit one chunk) and sums W_ip / Z_i over the
//      tile's queries (a reduce-scatter butterfly over lanes, then a fixed
//      order over waves);
//   3. top-P: histogram of the importance exponents finds the bin holding
//      the P-th largest value; exact ranks (w desc, index asc) inside that bin
//      decide the rest; the selected parents are listed in index order;
//   4. child sweep over the selected parents' children, chunk by chunk:
//      logits, running max raised (Xbar rescaled), recovered parent logit,
//      correcting weights, Xbar += Vmean^T dW;
//   5. Y = Xbar / Z.
#include "avq_common.hpp"

#include <type_traits>

namespace avq {

template <typename T, int D, int MAXW>
struct AttnCfg {
  static constexpr bool kB = Elem<T>::kBf16;
  static constexpr int RPW = 32;                  // query rows per wave
  static constexpr int QS = RPW / 16;             // query subtiles per wave
  static constexpr int CW = 64;                   // codeword rows per chunk
  static constexpr int TPC = CW / 16;             // 16-row tiles per chunk
  static constexpr int KQ = kB ? D / 32 : D / 4;  // MFMA k-steps over d
  static constexpr int DT = D / 16;               // d tiles of Xbar
  static constexpr int XT = DT + 1;               // plus the denominator tile
  static constexpr int ESZ = sizeof(T);
  static constexpr int EPU = 16 / ESZ;            // elements per 16-byte unit
  static constexpr int U = D * ESZ / 16;          // 16-byte units per codeword row
  static constexpr int RB = (256 / (D * ESZ)) > 1 ? 256 / (D * ESZ) : 1;  // rows per 256 B
  static constexpr int M0MAX = 512;
  static constexpr int kWavesPerEu = (kB && D == 64 && MAXW == 4) ? 3 : 2;
  static constexpr int CHUNK_BYTES = CW * D * ESZ;  // codeword rows (= packed means)
  // dynamic LDS layout (bytes)
  static constexpr size_t OFF_C = 0;
  static constexpr size_t OFF_V = OFF_C + CHUNK_BYTES;
  static constexpr size_t OFF_N = OFF_V + CHUNK_BYTES;                // [CW] f32 n
  static constexpr size_t OFF_L = OFF_N + CW * 4;                     // [CW] f32 log2 n
  static constexpr size_t OFF_W = OFF_L + CW * 4;                     // [MAXW][M0MAX] f32
  static constexpr size_t OFF_WF = OFF_W + (size_t)MAXW * M0MAX * 4;  // [M0MAX] f32
  static constexpr size_t OFF_SEL = OFF_WF + M0MAX * 4;               // [M0MAX] i32
  static constexpr size_t OFF_FLAG = OFF_SEL + M0MAX * 4;             // [M0MAX] i32
  static constexpr size_t OFF_HIST = OFF_FLAG + M0MAX * 4;            // [256] i32
  static constexpr size_t OFF_MISC = OFF_HIST + 256 * 4;              // [4] i32
  static constexpr size_t LDS_BYTES = OFF_MISC + 16;
  static_assert(CHUNK_BYTES % 1024 == 0, "a chunk is a whole number of wave copies");
  static_assert(TPC * 4 == 16, "importance butterfly takes 16 codewords per lane");
};

struct AttnArgs {
  const void* Q;
  const void* Cp;
  const void* Cc;
  const void* Vmean;
  const int32_t* counts;
  void* Y;
  int32_t* topp_idx;
  float* importance;
  int H, N, M0, Ch, P, block_q, n_tiles;
};

// One wave copies 64 x 16 bytes from global memory to LDS: lane L's 16 bytes
// land at lds + 16 L (lds must be the same for the whole wave).
__device__ __forceinline__ void copy16_to_lds(const void* src, void* lds) {
  __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)src,
                                   (void __attribute__((address_space(3)))*)lds, 16, 0, 0);
}

// Register budget: two or three waves per SIMD (at most 256 or 168 registers
// each), so that other tiles' MFMA work runs while one workgroup waits for
// its chunk to arrive.
template <typename T, int D, int MAXW>
__global__ __launch_bounds__(MAXW * 64)
__attribute__((amdgpu_waves_per_eu(AttnCfg<T, D, MAXW>::kWavesPerEu)))
void attention_kernel(AttnArgs args) {
  using Cfg = AttnCfg<T, D, MAXW>;
  constexpr bool kB = Cfg::kB;
  constexpr int QS = Cfg::QS, CW = Cfg::CW, TPC = Cfg::TPC, KQ = Cfg::KQ, DT = Cfg::DT,
                XT = Cfg::XT, U = Cfg::U, EPU = Cfg::EPU, RB = Cfg::RB, M0MAX = Cfg::M0MAX;
  using QFrag = typename std::conditional<kB, bf16x8, float>::type;
  constexpr float kNegInf = -__builtin_inff();

  extern __shared__ __attribute__((aligned(16))) unsigned char lds_raw[];
  T* lc = reinterpret_cast<T*>(lds_raw + Cfg::OFF_C);            // codeword rows (swizzled)
  T* lv = reinterpret_cast<T*>(lds_raw + Cfg::OFF_V);            // mean values [CW/4][D][4]
  float* ln = reinterpret_cast<float*>(lds_raw + Cfg::OFF_N);    // counts of the rows
  float* ll = reinterpret_cast<float*>(lds_raw + Cfg::OFF_L);    // log2 of the counts
  float* lw = reinterpret_cast<float*>(lds_raw + Cfg::OFF_W);    // per-wave importance
  float* lwf = reinterpret_cast<float*>(lds_raw + Cfg::OFF_WF);  // importance
  int* lsel = reinterpret_cast<int*>(lds_raw + Cfg::OFF_SEL);    // selected, index order
  int* lflag = reinterpret_cast<int*>(lds_raw + Cfg::OFF_FLAG);  // selected flags
  int* lhist = reinterpret_cast<int*>(lds_raw + Cfg::OFF_HIST);  // exponent histogram
  int* lmisc = reinterpret_cast<int*>(lds_raw + Cfg::OFF_MISC);

  const T* __restrict__ Q = static_cast<const T*>(args.Q);
  const T* __restrict__ Cp = static_cast<const T*>(args.Cp);
  const T* __restrict__ Cc = static_cast<const T*>(args.Cc);
  const int32_t* __restrict__ counts = args.counts;
  const int N = args.N, M0 = args.M0, Ch = args.Ch, P = args.P;
  const int Mtot = M0 * (1 + Ch);
  const int PG = (M0 + 3) / 4, CG = (Ch + 3) / 4, PS = 4 * CG;  // groups; rows per parent

  const int tid = threadIdx.x, nthr = blockDim.x, nwaves = nthr / kWave;
  const int wave = tid / kWave, lane = tid % kWave;
  const int g = lane / 16, c = lane % 16;
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = tile / args.n_tiles, t = tile % args.n_tiles;
  const int h = bh % args.H;
  const int q_begin = t * args.block_q;
  const int q_end = min(q_begin + args.block_q, N);
  const int row0 = q_begin + wave * Cfg::RPW;
  const T* vm_par =
      static_cast<const T*>(args.Vmean) + (size_t)bh * (PG + (size_t)M0 * CG) * 4 * D;
  const T* vm_child = vm_par + (size_t)PG * 4 * D;
  const int32_t* cb = counts + (size_t)bh * Mtot;
  const T* cp_head = Cp + (size_t)h * M0 * D;
  const T* cc_head = Cc + (size_t)h * M0 * Ch * D;

  // ---- query fragments (B operand of S^T = C . Q^T) -------------------------
  QFrag qf[QS][KQ];
  bool qvalid[QS];
#pragma unroll
  for (int s = 0; s < QS; ++s) {
    const int i = row0 + 16 * s + c;
    qvalid[s] = i < q_end;
    const T* qrow = Q + ((size_t)bh * N + (qvalid[s] ? i : q_begin)) * D;
#pragma unroll
    for (int kq = 0; kq < KQ; ++kq) {
      if constexpr (kB) {
        bf16x8 v = *reinterpret_cast<const bf16x8*>(qrow + 32 * kq + 8 * g);
        qf[s][kq] = qvalid[s] ? v : bf16x8{};
      } else {
        float v = qrow[4 * kq + g];
        qf[s][kq] = qvalid[s] ? v : 0.f;
      }
    }
  }

  // ---- chunk staging --------------------------------------------------------
  // Codeword row r of the chunk holds its 16-byte unit u at unit u ^ swz(r).
  auto swz = [](int r) { return (r / RB) % U; };
  // stage(crow, vgroup, count, with_values): crow(r) = codebook row of chunk
  // row r (any valid row for padding), vgroup(k) = first element of the packed
  // means of chunk group k (rows 4k .. 4k+3), count(r) = n of chunk row r
  // (0 for padding).
  auto stage = [&](auto crow, auto vgroup, auto count, bool with_values) {
    constexpr int COPIES = CW * U / 64;  // wave copies per array
    for (int j = wave; j < COPIES; j += nwaves) {
      const int q = 64 * j + lane;
      const int r = q / U, pu = q % U;
      copy16_to_lds(crow(r) + (pu ^ swz(r)) * EPU, lds_raw + Cfg::OFF_C + 1024 * j);
    }
    if (with_values) {
      constexpr int UPG = D * 4 * Cfg::ESZ / 16;  // 16-byte units per group
      for (int j = wave; j < COPIES; j += nwaves) {
        const int q = 64 * j + lane;
        copy16_to_lds(vgroup(q / UPG) + (q % UPG) * EPU, lds_raw + Cfg::OFF_V + 1024 * j);
      }
    }
    for (int r = tid; r < CW; r += nthr) {
      const float n = (float)count(r);
      ln[r] = n;
      ll[r] = n > 0.f ? log2_hw(n) : kNegInf;
    }
    __builtin_amdgcn_s_waitcnt(0);
  };
  auto parent_crow = [=](int cbase) {
    return [=](int r) { return cp_head + (size_t)min(cbase + r, M0 - 1) * D; };
  };
  auto parent_vgroup = [=](int cbase) {
    return [=](int k) { return vm_par + (size_t)min(cbase / 4 + k, PG - 1) * 4 * D; };
  };
  auto parent_count = [=](int cbase) {
    return [=](int r) { return cbase + r < M0 ? cb[cbase + r] : 0; };
  };

  // ---- S^T tile (16 codewords x 16 queries) for chunk tile tt ----------------
  auto logits = [&](int tt, f32x4 (&out)[QS]) {
    const int r = 16 * tt + c;
#pragma unroll
    for (int s = 0; s < QS; ++s) out[s] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kq = 0; kq < KQ; ++kq) {
      if constexpr (kB) {
        const int u = 4 * kq + g;
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(&lc[r * D + (u ^ swz(r)) * EPU]);
#pragma unroll
        for (int s = 0; s < QS; ++s) out[s] = mfma_bf16(a, qf[s][kq], out[s]);
      } else {
        const float a = lc[r * D + (kq ^ swz(r)) * EPU + g];
#pragma unroll
        for (int s = 0; s < QS; ++s) out[s] = mfma_f32(a, qf[s][kq], out[s]);
      }
    }
  };

  // ---- Xbar^T += Vmean^T . W^T; the extra tile DT has an all-ones first row
  f32x4 X[XT][QS];
#pragma unroll
  for (int dt = 0; dt < XT; ++dt)
#pragma unroll
    for (int s = 0; s < QS; ++s) X[dt][s] = f32x4{0.f, 0.f, 0.f, 0.f};

  // bf16: the weights of chunk tiles tt and tt+1 form one B operand; k-slots
  // 8g .. 8g+3 are rows 4g .. 4g+3 of tile tt, 8g+4 .. 8g+7 those of tile tt+1
  auto accumulate_b = [&](int tt, const f32x4 (&w0)[QS], const f32x4 (&w1)[QS]) {
    bf16x8 b[QS];
#pragma unroll
    for (int s = 0; s < QS; ++s) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        b[s][r] = (bf16)w0[s][r];
        b[s][4 + r] = (bf16)w1[s][r];
      }
    }
    const bf16* g0 = reinterpret_cast<const bf16*>(lv) + (4 * tt + g) * 4 * D;
    const bf16* g1 = reinterpret_cast<const bf16*>(lv) + (4 * (tt + 1) + g) * 4 * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const int d = 16 * dt + c;
      const bf16x4 lo = *reinterpret_cast<const bf16x4*>(g0 + 4 * d);
      const bf16x4 hi = *reinterpret_cast<const bf16x4*>(g1 + 4 * d);
      const bf16x8 a = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
#pragma unroll
      for (int s = 0; s < QS; ++s) X[dt][s] = mfma_bf16(a, b[s], X[dt][s]);
    }
    const bf16 one = (bf16)(c == 0 ? 1.f : 0.f);
    const bf16x8 ones = {one, one, one, one, one, one, one, one};
#pragma unroll
    for (int s = 0; s < QS; ++s) X[DT][s] = mfma_bf16(ones, b[s], X[DT][s]);
  };
  // fp32: the r-th product of tile tt takes row 4g + r as k-slot g
  auto accumulate_f = [&](int tt, const f32x4 (&w0)[QS]) {
    const float* g0 = reinterpret_cast<const float*>(lv) + (4 * tt + g) * 4 * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const float4 a = *reinterpret_cast<const float4*>(g0 + 4 * (16 * dt + c));
#pragma unroll
      for (int s = 0; s < QS; ++s) {
        X[dt][s] = mfma_f32(a.x, w0[s][0], X[dt][s]);
        X[dt][s] = mfma_f32(a.y, w0[s][1], X[dt][s]);
        X[dt][s] = mfma_f32(a.z, w0[s][2], X[dt][s]);
        X[dt][s] = mfma_f32(a.w, w0[s][3], X[dt][s]);
      }
    }
    const float one = c == 0 ? 1.f : 0.f;
#pragma unroll
    for (int s = 0; s < QS; ++s)
#pragma unroll
      for (int r = 0; r < 4; ++r) X[DT][s] = mfma_f32(one, w0[s][r], X[DT][s]);
  };
  auto accumulate_chunk = [&](const f32x4 (&W)[TPC][QS]) {
    if constexpr (kB) {
#pragma unroll
      for (int tt = 0; tt < TPC; tt += 2) accumulate_b(tt, W[tt], W[tt + 1]);
    } else {
#pragma unroll
      for (int tt = 0; tt < TPC; ++tt) accumulate_f(tt, W[tt]);
    }
  };

  // Per-lane softmax state for query columns c + 16 s, in log2 units: m is
  // the running max of t, started at a finite floor so that t - m stays -inf
  // (weight 0) for empty codewords even before any non-empty one was seen.
  // zp is this lane group's partial fp32 sum of the parent weights (for
  // importance); the four groups are summed when needed.
  constexpr float kMaxFloor = -1e30f;
  float m[QS], zp[QS];
#pragma unroll
  for (int s = 0; s < QS; ++s) {
    m[s] = kMaxFloor;
    zp[s] = 0.f;
  }
  auto raise_max = [&](float (&mnew)[QS]) {
    bool moved = false;
#pragma unroll
    for (int s = 0; s < QS; ++s) {
      mnew[s] = fmaxf(mnew[s], shfl_xor(mnew[s], 16));
      mnew[s] = fmaxf(mnew[s], shfl_xor(mnew[s], 32));
      moved |= mnew[s] != m[s];
    }
    if (__ballot(moved) == 0) return;  // wave-uniform: nothing to rescale
#pragma unroll
    for (int s = 0; s < QS; ++s) {
      const float sc = exp2_hw(m[s] - mnew[s]);
      zp[s] *= sc;
#pragma unroll
      for (int dt = 0; dt < XT; ++dt) X[dt][s] *= sc;
      m[s] = mnew[s];
    }
  };
  // t = S log2(e) + log2 n over the chunk
  auto bias = [&](f32x4 (&S)[TPC][QS]) {
#pragma unroll
    for (int tt = 0; tt < TPC; ++tt) {
      const float4 l4 = *reinterpret_cast<const float4*>(&ll[16 * tt + 4 * g]);
#pragma unroll
      for (int s = 0; s < QS; ++s) {
        S[tt][s][0] = fmaf(S[tt][s][0], kLog2e, l4.x);
        S[tt][s][1] = fmaf(S[tt][s][1], kLog2e, l4.y);
        S[tt][s][2] = fmaf(S[tt][s][2], kLog2e, l4.z);
        S[tt][s][3] = fmaf(S[tt][s][3], kLog2e, l4.w);
      }
    }
  };
  auto chunk_max = [&](const f32x4 (&S)[TPC][QS], float (&mnew)[QS]) {
#pragma unroll
    for (int s = 0; s < QS; ++s) mnew[s] = m[s];
#pragma unroll
    for (int tt = 0; tt < TPC; ++tt)
#pragma unroll
      for (int s = 0; s < QS; ++s)
#pragma unroll
        for (int r = 0; r < 4; ++r) mnew[s] = fmaxf(mnew[s], S[tt][s][r]);
  };

  const bool need_importance =
      (P > 0 && P < M0) || args.importance != nullptr || (P > 0 && args.topp_idx != nullptr);
  const int n_pchunks = (M0 + CW - 1) / CW;
  float rz[QS];
  auto set_rz = [&]() {
#pragma unroll
    for (int s = 0; s < QS; ++s) {
      float z = zp[s];
      z += shfl_xor(z, 16);
      z += shfl_xor(z, 32);
      rz[s] = qvalid[s] ? 1.f / z : 0.f;
    }
  };
  // u_a = sum over this wave's queries of W_ia / Z_i for the chunk in W:
  // first over the query subtiles in registers, then over the 16 query
  // columns by a reduce-scatter butterfly over lane bits 3, 0, 1, 2 that
  // leaves lane c with value k = 8 b3 + 4 b0 + 2 b1 + b2 of its lane group
  // (value k = codeword row 16 (k / 4) + 4 g + k % 4 of the chunk).
  auto importance_partials = [&](const f32x4 (&W)[TPC][QS], int cbase) {
    float u[16];
#pragma unroll
    for (int tt = 0; tt < TPC; ++tt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float acc = 0.f;
#pragma unroll
        for (int s = 0; s < QS; ++s) acc = fmaf(W[tt][s][r], rz[s], acc);
        u[4 * tt + r] = acc;
      }
    auto step = [&](auto mask_tag, auto half_tag) {
      constexpr int MASK = decltype(mask_tag)::value, HALF = decltype(half_tag)::value;
      const bool upper = (c & MASK) != 0;
#pragma unroll
      for (int i = 0; i < HALF; ++i) {
        const float lo = u[i] + xor16<MASK>(u[i]);
        const float hi = u[i + HALF] + xor16<MASK>(u[i + HALF]);
        u[i] = upper ? hi : lo;
      }
    };
    step(std::integral_constant<int, 8>{}, std::integral_constant<int, 8>{});
    step(std::integral_constant<int, 1>{}, std::integral_constant<int, 4>{});
    step(std::integral_constant<int, 2>{}, std::integral_constant<int, 2>{});
    step(std::integral_constant<int, 4>{}, std::integral_constant<int, 1>{});
    const int k = 8 * ((c >> 3) & 1) + 4 * (c & 1) + 2 * ((c >> 1) & 1) + ((c >> 2) & 1);
    lw[wave * M0MAX + cbase + 16 * (k / 4) + 4 * g + (k % 4)] = u[0];
  };

  // ---- phase 1: parent sweep (online softmax over chunks) ---------------------
  for (int pc = 0; pc < n_pchunks; ++pc) {
    const int cbase = pc * CW;
    __syncthreads();
    stage(parent_crow(cbase), parent_vgroup(cbase), parent_count(cbase), true);
    __syncthreads();
    f32x4 S[TPC][QS];
#pragma unroll
    for (int tt = 0; tt < TPC; ++tt) logits(tt, S[tt]);
    bias(S);
    float mnew[QS];
    chunk_max(S, mnew);
    raise_max(mnew);
#pragma unroll
    for (int tt = 0; tt < TPC; ++tt)
#pragma unroll
      for (int s = 0; s < QS; ++s)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float w = exp2_hw(S[tt][s][r] - m[s]);
          S[tt][s][r] = w;
          zp[s] += w;
        }
    // a single chunk has its final max and denominators already: importance
    // comes straight from these weights
    if (n_pchunks == 1 && need_importance) {
      set_rz();
      importance_partials(S, cbase);
    }
    accumulate_chunk(S);
  }

  // ---- phase 2: importance with the final max and denominators ----------------
  if (need_importance) {
    if (n_pchunks > 1) {
      set_rz();
      for (int pc = 0; pc < n_pchunks; ++pc) {
        const int cbase = pc * CW;
        __syncthreads();
        stage(parent_crow(cbase), parent_vgroup(cbase), parent_count(cbase), false);
        __syncthreads();
        f32x4 S[TPC][QS];
#pragma unroll
        for (int tt = 0; tt < TPC; ++tt) logits(tt, S[tt]);
        bias(S);
#pragma unroll
        for (int tt = 0; tt < TPC; ++tt)
#pragma unroll
          for (int s = 0; s < QS; ++s)
#pragma unroll
            for (int r = 0; r < 4; ++r) S[tt][s][r] = exp2_hw(S[tt][s][r] - m[s]);
        importance_partials(S, cbase);
      }
    }
    __syncthreads();
    // sum the wave partials in a fixed order
    for (int a = tid; a < M0; a += nthr) {
      float acc = 0.f;
      for (int wv = 0; wv < nwaves; ++wv) acc += lw[wv * M0MAX + a];
      lwf[a] = acc;
      if (args.importance) args.importance[((size_t)bh * args.n_tiles + t) * M0 + a] = acc;
    }
    __syncthreads();
  }

  // ---- phase 3: top-P (w desc, index asc) -------------------------------------
  if (P > 0) {
    if (P < M0) {
      for (int i = tid; i < 256; i += nthr) lhist[i] = 0;
      if (tid == 0) lmisc[2] = 0;
      __syncthreads();
      for (int a = tid; a < M0; a += nthr)
        atomicAdd(&lhist[(__float_as_uint(lwf[a]) >> 23) & 255], 1);
      __syncthreads();
      if (wave == 0) {
        // lane l holds bins 255 - 4l - i (i = 0..3): lanes in descending bins
        int cnt[4], local = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          cnt[i] = lhist[255 - 4 * lane - i];
          local += cnt[i];
        }
        int incl = local;
#pragma unroll
        for (int off = 1; off < kWave; off <<= 1) {
          const int y = __shfl_up(incl, off, kWave);
          if (lane >= off) incl += y;
        }
        int above = incl - local;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (above < P && P <= above + cnt[i]) {
            lmisc[0] = 255 - 4 * lane - i;
            lmisc[1] = above;
          }
          above += cnt[i];
        }
      }
      __syncthreads();
      const int bstar = lmisc[0], need = P - lmisc[1];
      int* bmem = reinterpret_cast<int*>(lw);  // boundary-bin members (lw is free now)
      for (int a = tid; a < M0; a += nthr) {
        const int bin = (int)((__float_as_uint(lwf[a]) >> 23) & 255);
        lflag[a] = bin > bstar ? 1 : 0;
        if (bin == bstar) bmem[atomicAdd(&lmisc[2], 1)] = a;
      }
      __syncthreads();
      const int nbm = lmisc[2];
      for (int q = tid; q < nbm; q += nthr) {
        const int a = bmem[q];
        const float wa = lwf[a];
        int rank = 0;
        for (int k = 0; k < nbm; ++k) {
          const int b = bmem[k];
          const float wb = lwf[b];
          rank += (wb > wa) || (wb == wa && b < a);
        }
        if (rank < need) lflag[a] = 1;
      }
    } else {
      for (int a = tid; a < M0; a += nthr) lflag[a] = 1;
    }
    __syncthreads();
    if (wave == 0) {  // selected parents in ascending index order
      int filled = 0;
      for (int a0 = 0; a0 < M0; a0 += kWave) {
        const int a = a0 + lane;
        const bool f = a < M0 && lflag[a] != 0;
        const unsigned long long mask = __ballot(f);
        if (f) lsel[filled + __popcll(mask & ((1ull << lane) - 1ull))] = a;
        filled += __popcll(mask);
      }
    }
    __syncthreads();
    if (args.topp_idx) {  // canonical order (w desc, index asc) for the caller
      for (int q = tid; q < P; q += nthr) {
        const int a = lsel[q];
        const float wa = lwf[a];
        int rank = 0;
        for (int k = 0; k < P; ++k) {
          const int b = lsel[k];
          const float wb = lwf[b];
          rank += (wb > wa) || (wb == wa && b < a);
        }
        args.topp_idx[((size_t)bh * args.n_tiles + t) * P + rank] = a;
      }
    }

    // ---- phase 4: child sweep ----------------------------------------------
    // Each selected parent owns PS = 4 ceil(Ch/4) consecutive chunk rows: its
    // Ch children, padded to whole groups of 4 with rows of count 0. With one
    // child the recovered parent logit is that child's own logit, so every
    // correcting weight is exactly zero: nothing to do.
    const int rows = Ch > 1 ? P * PS : 0;
    for (int cbase = 0; cbase < rows; cbase += CW) {
      auto child_crow = [=](int r) {
        const int q = cbase + r;
        const int k = min(q / PS, P - 1), cc = min(q % PS, Ch - 1);
        return cc_head + ((size_t)lsel[k] * Ch + cc) * D;
      };
      auto child_vgroup = [=](int gl) {
        const int gg = cbase / 4 + gl;
        const int k = min(gg / CG, P - 1);
        return vm_child + ((size_t)lsel[k] * CG + gg % CG) * 4 * D;
      };
      auto child_count = [=](int r) {
        const int q = cbase + r;
        const int k = q / PS, cc = q % PS;
        return (q < rows && cc < Ch) ? cb[M0 + lsel[k] * Ch + cc] : 0;
      };
      __syncthreads();
      stage(child_crow, child_vgroup, child_count, true);
      __syncthreads();
      f32x4 Sc[TPC][QS];
      float sp[TPC][QS];  // recovered parent logit of the lane's rows
#pragma unroll
      for (int tt = 0; tt < TPC; ++tt) {
        logits(tt, Sc[tt]);
#pragma unroll
        for (int s = 0; s < QS; ++s) {
          const f32x4 v = Sc[tt][s];
          if (Ch == 2) {
            sp[tt][s] = (v[0] + v[1]) * 0.5f;  // rows 2, 3 are padding
          } else {
            float sum = (v[0] + v[1]) + (v[2] + v[3]);
            if (Ch >= 8) sum += shfl_xor(sum, 16);
            if (Ch >= 16) sum += shfl_xor(sum, 32);
            sp[tt][s] = sum * (1.f / (float)Ch);
          }
        }
      }
      bias(Sc);
      float mnew[QS];
      chunk_max(Sc, mnew);
      raise_max(mnew);
      // dW = n_c (exp(T_c - m) - exp(Srec - m)); padding and empty rows have
      // n = 0 and t = -inf, so dW = 0 (the recovered term is clamped finite)
#pragma unroll
      for (int tt = 0; tt < TPC; ++tt) {
        const float4 n4 = *reinterpret_cast<const float4*>(&ln[16 * tt + 4 * g]);
#pragma unroll
        for (int s = 0; s < QS; ++s) {
          const float e = exp2_hw(fminf(fmaf(sp[tt][s], kLog2e, -m[s]), 64.f));
          Sc[tt][s][0] = fmaf(-n4.x, e, exp2_hw(Sc[tt][s][0] - m[s]));
          Sc[tt][s][1] = fmaf(-n4.y, e, exp2_hw(Sc[tt][s][1] - m[s]));
          Sc[tt][s][2] = fmaf(-n4.z, e, exp2_hw(Sc[tt][s][2] - m[s]));
          Sc[tt][s][3] = fmaf(-n4.w, e, exp2_hw(Sc[tt][s][3] - m[s]));
        }
      }
      accumulate_chunk(Sc);
    }
  }

  // ---- phase 5: Y = Xbar / Z (Z from the denominator tile, lane group 0) ------
#pragma unroll
  for (int s = 0; s < QS; ++s) {
    const float z = __shfl(X[DT][s][0], c, kWave);
    if (!qvalid[s]) continue;
    const float rinv = 1.f / z;
    const int i = row0 + 16 * s + c;
    T* yrow = static_cast<T*>(args.Y) + ((size_t)bh * N + i) * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const f32x4 y = X[dt][s] * rinv;
      if constexpr (kB) {
        bf16x4 o = {(bf16)y[0], (bf16)y[1], (bf16)y[2], (bf16)y[3]};
        *reinterpret_cast<bf16x4*>(yrow + 16 * dt + 4 * g) = o;
      } else {
        *reinterpret_cast<f32x4*>(yrow + 16 * dt + 4 * g) = y;
      }
    }
  }
}

template <typename T, int D, int MAXW>
hipError_t launch_attention_cfg(const AttnArgs& a, int BH, hipStream_t stream) {
  const long long grid = (long long)BH * a.n_tiles;
  if (grid > 0x7fffffff) return hipErrorInvalidConfiguration;
  const int waves = (a.block_q + 31) / 32;
  using Cfg = AttnCfg<T, D, MAXW>;
  constexpr int slot = 8 + (Elem<T>::kBf16 ? 0 : 4) + (D == 128 ? 2 : 0) + (MAXW == 8 ? 1 : 0);
  hipError_t e = ensure_dynamic_lds((const void*)attention_kernel<T, D, MAXW>,
                                    (int)Cfg::LDS_BYTES, slot);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attention_kernel<T, D, MAXW>), dim3((unsigned)grid), dim3(waves * 64),
                     Cfg::LDS_BYTES, stream, a);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_attention(int BH, int H, int N, int M0, int Ch, int P, int block_q,
                            const void* Q, const void* Cp, const void* Cc, const void* Vmean,
                            const int32_t* counts, void* Y, int32_t* topp_idx,
                            float* importance, hipStream_t stream) {
  AttnArgs a;
  a.Q = Q;
  a.Cp = Cp;
  a.Cc = Cc;
  a.Vmean = Vmean;
  a.counts = counts;
  a.Y = Y;
  a.topp_idx = topp_idx;
  a.importance = importance;
  a.H = H;
  a.N = N;
  a.M0 = M0;
  a.Ch = Ch;
  a.P = P;
  a.block_q = block_q;
  a.n_tiles = (N + block_q - 1) / block_q;
  if (block_q <= 128) return launch_attention_cfg<T, D, 4>(a, BH, stream);
  return launch_attention_cfg<T, D, 8>(a, BH, stream);
}

#define AVQ_INSTANTIATE(T, D)                                                                \
  template hipError_t launch_attention<T, D>(int, int, int, int, int, int, int, const void*, \
                                             const void*, const void*, const void*,          \
                                             const int32_t*, void*, int32_t*, float*,        \
                                             hipStream_t);
AVQ_INSTANTIATE(bf16, 64)
AVQ_INSTANTIATE(bf16, 128)
AVQ_INSTANTIATE(float, 64)
AVQ_INSTANTIATE(float, 128)
#undef AVQ_INSTANTIATE

}  // namespace avq
