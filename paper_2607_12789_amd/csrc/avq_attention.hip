// Fused refined-codebook attention (Sec. 4.3, Alg. 2) for gfx950.
//
// One workgroup processes one query tile (block_q consecutive tokens of one
// (batch, head)); each wave owns 32 query rows. Everything is computed
// transposed, codewords x queries: S^T = C . Q^T and Xbar^T = Vmean^T . A^T.
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
// t = S log2(e) + log2(n), so the weight exp2(t - m) is n exp(S - m'); empty
// codewords get t = -inf and drop out of the running max and of every sum
// without masks. The values are staged as means Vbar/n, which gives
// sum_j n_j exp(S_j - m') Vbar_j / n_j = sum_j exp(S_j - m') Vbar_j, the
// numerator of Eq. (vqflashattention). The parent logit recovered from the
// children uses the unbiased child logits, and the correcting weight of
// child c is n_c (exp(T_c - m') - exp(Srec - m')), Eq. (correcting_attention)
// times n_c. The denominator (sum of the weights, n folded in) is produced by
// the value MFMA itself through one extra d-tile whose first row is all ones,
// so numerator and denominator use the same rounded weights; the parent-only
// denominator needed by Eq. (importance) is also summed in fp32.
//
// Phases per tile:
//   1. parent pass over the M0 parents in groups of 16*NT codewords held in
//      registers: logits, running max, weights, Xbar += Vmean^T W;
//   2. importance w_p = sum_i W_ip / Z_i with the final parent denominators
//      (Eq. (importance), n_p already inside W): straight from the registers
//      when all parents fit in one group, else from a second sweep that
//      recomputes the logits;
//   3. top-P: histogram of the importance exponents finds the bin holding the
//      P-th largest value; exact ranks (w desc, index asc) inside that bin
//      decide the rest; the selected parents are listed in index order;
//   4. child pass over the selected parents' children in chunks: logits,
//      running max raised (Xbar rescaled), recovered parent logit, correcting
//      weights, Xbar += Vmean^T dW;
//   5. Y = Xbar / Z.
#include "avq_common.hpp"

namespace avq {

template <typename T, int D, int NT, int MAXW>
struct AttnCfg {
  static constexpr bool kB = Elem<T>::kBf16;
  static constexpr int RPW = 32;                  // query rows per wave
  static constexpr int QS = RPW / 16;             // query subtiles per wave
  static constexpr int GROUP = 16 * NT;           // parents held in registers
  static constexpr int CW = kB ? GROUP : 32;      // codeword rows per LDS chunk
  static constexpr int KQ = kB ? D / 32 : D / 4;  // MFMA k-steps over d
  static constexpr int DT = D / 16;               // d tiles of Xbar
  static constexpr int XT = DT + 1;               // plus the denominator tile
  static constexpr int CPAD = kB ? 8 : 4;         // 16 bytes of row padding
  static constexpr int CROW = D + CPAD;
  static constexpr int VPAD = kB ? 8 : 4;
  static constexpr int VROW = CW + VPAD;
  static constexpr int M0MAX = 512;
  static_assert(GROUP % CW == 0, "a register group is a whole number of LDS chunks");
  using VT = typename std::conditional<kB, bf16, float>::type;
  // dynamic LDS layout (bytes)
  static constexpr size_t OFF_C = 0;                                      // [CW][CROW] T
  static constexpr size_t OFF_V = OFF_C + (size_t)CW * CROW * sizeof(T);   // [D][VROW] VT
  static constexpr size_t OFF_N = OFF_V + (size_t)D * VROW * sizeof(VT);   // [CW] f32 n
  static constexpr size_t OFF_L = OFF_N + (size_t)CW * 4;                  // [CW] f32 log2 n
  static constexpr size_t OFF_LP = OFF_L + (size_t)CW * 4;                 // [M0MAX] parents' log2 n
  static constexpr size_t OFF_W = OFF_LP + (size_t)M0MAX * 4;              // [MAXW][M0MAX] f32
  static constexpr size_t OFF_WF = OFF_W + (size_t)MAXW * M0MAX * 4;       // [M0MAX] f32
  static constexpr size_t OFF_SEL = OFF_WF + (size_t)M0MAX * 4;            // [M0MAX] i32
  static constexpr size_t OFF_FLAG = OFF_SEL + (size_t)M0MAX * 4;          // [M0MAX] i32
  static constexpr size_t OFF_HIST = OFF_FLAG + (size_t)M0MAX * 4;         // [256] i32
  static constexpr size_t OFF_MISC = OFF_HIST + 256 * 4;                   // [4] i32
  static constexpr size_t LDS_BYTES = OFF_MISC + 16;
  static_assert(OFF_V % 16 == 0 && OFF_N % 16 == 0 && OFF_W % 16 == 0, "aligned LDS regions");
};

struct AttnArgs {
  const void* Q;
  const void* Cp;
  const void* Cc;
  const float* Vbar;
  const int32_t* counts;
  void* Y;
  int32_t* topp_idx;
  float* importance;
  int H, N, M0, Ch, P, block_q, n_tiles;
};

template <typename T, int D, int NT, int MAXW>
__global__ __launch_bounds__(MAXW * 64) void attention_kernel(AttnArgs args) {
  using Cfg = AttnCfg<T, D, NT, MAXW>;
  constexpr bool kB = Cfg::kB;
  constexpr int QS = Cfg::QS, CW = Cfg::CW, KQ = Cfg::KQ, DT = Cfg::DT, XT = Cfg::XT;
  constexpr int CROW = Cfg::CROW, VROW = Cfg::VROW, M0MAX = Cfg::M0MAX;
  using QFrag = typename std::conditional<kB, bf16x8, float>::type;
  using VT = typename Cfg::VT;
  constexpr float kNegInf = -__builtin_inff();

  extern __shared__ __attribute__((aligned(16))) unsigned char lds_raw[];
  T* lc = reinterpret_cast<T*>(lds_raw + Cfg::OFF_C);          // staged codeword rows
  VT* lv = reinterpret_cast<VT*>(lds_raw + Cfg::OFF_V);        // their mean values, transposed
  float* ln = reinterpret_cast<float*>(lds_raw + Cfg::OFF_N);  // their counts
  float* ll = reinterpret_cast<float*>(lds_raw + Cfg::OFF_L);  // log2 of their counts
  float* lp = reinterpret_cast<float*>(lds_raw + Cfg::OFF_LP);   // log2 n of all parents
  float* lw = reinterpret_cast<float*>(lds_raw + Cfg::OFF_W);    // per-wave importance
  float* lwf = reinterpret_cast<float*>(lds_raw + Cfg::OFF_WF);  // importance
  int* lsel = reinterpret_cast<int*>(lds_raw + Cfg::OFF_SEL);    // selected, index order
  int* lflag = reinterpret_cast<int*>(lds_raw + Cfg::OFF_FLAG);  // selected flags
  int* lhist = reinterpret_cast<int*>(lds_raw + Cfg::OFF_HIST);  // exponent histogram
  int* lmisc = reinterpret_cast<int*>(lds_raw + Cfg::OFF_MISC);

  const T* __restrict__ Q = static_cast<const T*>(args.Q);
  const T* __restrict__ Cp = static_cast<const T*>(args.Cp);
  const T* __restrict__ Cc = static_cast<const T*>(args.Cc);
  const float* __restrict__ Vbar = args.Vbar;
  const int32_t* __restrict__ counts = args.counts;
  const int N = args.N, M0 = args.M0, Ch = args.Ch, P = args.P;
  const int Mtot = M0 * (1 + Ch);

  const int tid = threadIdx.x, nthr = blockDim.x, nwaves = nthr / kWave;
  const int wave = tid / kWave, lane = tid % kWave;
  const int g = lane / 16, c = lane % 16;
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = tile / args.n_tiles, t = tile % args.n_tiles;
  const int h = bh % args.H;
  const int q_begin = t * args.block_q;
  const int q_end = min(q_begin + args.block_q, N);
  const int row0 = q_begin + wave * Cfg::RPW;

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

  // ---- LDS staging of a chunk of CW codeword rows ---------------------------
  // Every thread first issues a batch of global loads, then writes them to
  // LDS, so a batch costs one memory latency instead of one per element.
  // stage_codes: row r of the chunk <- codebook row crow(r) (nullptr: zeros).
  auto stage_codes = [&](auto crow) {
    constexpr int VEC = 16 / sizeof(T);
    constexpr int VPR = D / VEC;
    constexpr int BATCH = 8;
    for (int v0 = tid; v0 < CW * VPR; v0 += BATCH * nthr) {
      uint4 val[BATCH];
#pragma unroll
      for (int b = 0; b < BATCH; ++b) {
        const int v = v0 + b * nthr;
        val[b] = uint4{0u, 0u, 0u, 0u};
        if (v < CW * VPR) {
          const T* src = crow(v / VPR);
          if (src) val[b] = *reinterpret_cast<const uint4*>(src + (v % VPR) * VEC);
        }
      }
#pragma unroll
      for (int b = 0; b < BATCH; ++b) {
        const int v = v0 + b * nthr;
        if (v < CW * VPR)
          *reinterpret_cast<uint4*>(&lc[(v / VPR) * CROW + (v % VPR) * VEC]) = val[b];
      }
    }
  };
  // stage_values: mean values Vbar/n (transposed), n and log2 n of aggregate
  // rows vrow(r) (-1: an empty row). A row's values and its count are loaded
  // together; an empty row has n = 0 and a zero sum, and is scaled by 0.
  const float* vb = Vbar + (size_t)bh * Mtot * D;
  const int32_t* cb = counts + (size_t)bh * Mtot;
  auto load_row = [&](int a, int col, float4& x, float& inv) {
    x = float4{0.f, 0.f, 0.f, 0.f};
    inv = 0.f;
    if (a >= 0) {
      x = *reinterpret_cast<const float4*>(vb + (size_t)a * D + col);
      const int n = cb[a];
      inv = n > 0 ? __builtin_amdgcn_rcpf((float)n) : 0.f;
    }
  };
  auto stage_values = [&](auto vrow) {
    if constexpr (kB) {
      // bf16, codewords of each 32-block permuted so that lane group g reads
      // its 8 MFMA k-slots {4g..4g+3, 16+4g..16+4g+3} as one 16-byte word:
      // position 8g' + i holds codeword perm(g', i).
      constexpr int ITEMS = (CW / 32) * 4 * (D / 4);
      constexpr int IB = 2;  // items in flight per thread
      for (int v0 = tid; v0 < ITEMS; v0 += IB * nthr) {
        float4 x[IB][8];
        float inv[IB][8];
#pragma unroll
        for (int b = 0; b < IB; ++b) {
          const int v = v0 + b * nthr;
          const int dq = v % (D / 4), gg = (v / (D / 4)) % 4, blk = v / (D / 4) / 4;
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const int r = 32 * blk + (i < 4 ? 4 * gg + i : 16 + 4 * gg + (i - 4));
            load_row(v < ITEMS ? vrow(r) : -1, 4 * dq, x[b][i], inv[b][i]);
          }
        }
#pragma unroll
        for (int b = 0; b < IB; ++b) {
          const int v = v0 + b * nthr;
          if (v >= ITEMS) continue;
          const int dq = v % (D / 4), gg = (v / (D / 4)) % 4, blk = v / (D / 4) / 4;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            bf16x8 o;
#pragma unroll
            for (int i = 0; i < 8; ++i) o[i] = (bf16)((&x[b][i].x)[e] * inv[b][i]);
            *reinterpret_cast<bf16x8*>(&lv[(4 * dq + e) * VROW + 32 * blk + 8 * gg]) = o;
          }
        }
      }
    } else {
      // fp32, natural codeword order, written as 4x4 transposes.
      constexpr int ITEMS = (CW / 4) * (D / 4);
      constexpr int IB = 2;
      for (int v0 = tid; v0 < ITEMS; v0 += IB * nthr) {
        float4 x[IB][4];
        float inv[IB][4];
#pragma unroll
        for (int b = 0; b < IB; ++b) {
          const int v = v0 + b * nthr;
          const int dq = v % (D / 4), rq = v / (D / 4);
#pragma unroll
          for (int i = 0; i < 4; ++i) load_row(v < ITEMS ? vrow(4 * rq + i) : -1, 4 * dq, x[b][i], inv[b][i]);
        }
#pragma unroll
        for (int b = 0; b < IB; ++b) {
          const int v = v0 + b * nthr;
          if (v >= ITEMS) continue;
          const int dq = v % (D / 4), rq = v / (D / 4);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            float4 o = {(&x[b][0].x)[e] * inv[b][0], (&x[b][1].x)[e] * inv[b][1],
                        (&x[b][2].x)[e] * inv[b][2], (&x[b][3].x)[e] * inv[b][3]};
            *reinterpret_cast<float4*>(&lv[(4 * dq + e) * VROW + 4 * rq]) = o;
          }
        }
      }
    }
    for (int r = tid; r < CW; r += nthr) {
      const int a = vrow(r);
      const float n = a >= 0 ? (float)cb[a] : 0.f;
      ln[r] = n;
      ll[r] = n > 0.f ? log2_hw(n) : kNegInf;
    }
  };

  // ---- S^T tile (16 codewords x 16 queries) for chunk tile tt ----------------
  auto logits = [&](int tt, f32x4 (&out)[QS]) {
#pragma unroll
    for (int s = 0; s < QS; ++s) out[s] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kq = 0; kq < KQ; ++kq) {
      if constexpr (kB) {
        const bf16x8 a =
            *reinterpret_cast<const bf16x8*>(&lc[(16 * tt + c) * CROW + 32 * kq + 8 * g]);
#pragma unroll
        for (int s = 0; s < QS; ++s) out[s] = mfma_bf16(a, qf[s][kq], out[s]);
      } else {
        const float a = lc[(16 * tt + c) * CROW + 4 * kq + g];
#pragma unroll
        for (int s = 0; s < QS; ++s) out[s] = mfma_f32(a, qf[s][kq], out[s]);
      }
    }
  };

  // ---- Xbar^T += Vmean^T . W^T for chunk tiles (tt, tt+1) (bf16) or tt (fp32);
  // the extra tile DT has an all-ones first row and accumulates sum W.
  f32x4 X[XT][QS];
#pragma unroll
  for (int dt = 0; dt < XT; ++dt)
#pragma unroll
    for (int s = 0; s < QS; ++s) X[dt][s] = f32x4{0.f, 0.f, 0.f, 0.f};

  // bf16: pack the weights of tiles (tt, tt+1) into the MFMA B operand.
  auto pack = [&](const f32x4 (&w0)[QS], const f32x4 (&w1)[QS], bf16x8 (&b)[QS]) {
#pragma unroll
    for (int s = 0; s < QS; ++s) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        b[s][r] = (bf16)w0[s][r];
        b[s][4 + r] = (bf16)w1[s][r];
      }
    }
  };
  auto accumulate_b = [&](int tt, const bf16x8 (&b)[QS]) {
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const bf16x8 a =
          *reinterpret_cast<const bf16x8*>(&lv[(16 * dt + c) * VROW + 16 * tt + 8 * g]);
#pragma unroll
      for (int s = 0; s < QS; ++s) X[dt][s] = mfma_bf16(a, b[s], X[dt][s]);
    }
    const bf16 one = (bf16)(c == 0 ? 1.f : 0.f);
    const bf16x8 ones = {one, one, one, one, one, one, one, one};
#pragma unroll
    for (int s = 0; s < QS; ++s) X[DT][s] = mfma_bf16(ones, b[s], X[DT][s]);
  };
  // fp32: weights of tile tt as scalar MFMA operands.
  auto accumulate_f = [&](int tt, const f32x4 (&w0)[QS]) {
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const float4 a =
          *reinterpret_cast<const float4*>(&lv[(16 * dt + c) * VROW + 16 * tt + 4 * g]);
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

  // Per-lane softmax state for query columns c + 16 s, in log2 units: m is
  // the running max of t, started at a finite floor so that t - m stays
  // -inf (weight 0) for empty codewords even before any non-empty one was
  // seen. zp holds this lane group's partial fp32 sum of the parent weights
  // (for importance); the four groups are summed when needed.
  constexpr float kMaxFloor = -1e30f;
  float m[QS], zp[QS];
#pragma unroll
  for (int s = 0; s < QS; ++s) {
    m[s] = kMaxFloor;
    zp[s] = 0.f;
  }
  auto full_zp = [&](int s) {
    float z = zp[s];
    z += shfl_xor(z, 16);
    z += shfl_xor(z, 32);
    return z;
  };
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

  const T* cp_head = Cp + (size_t)h * M0 * D;
  const int n_groups = (M0 + Cfg::GROUP - 1) / Cfg::GROUP;
  f32x4 S[NT][QS];

  // ---- phase 1: parent pass (online softmax over register groups) -----------
  for (int a = tid; a < M0MAX; a += nthr) {
    const int n = a < M0 ? cb[a] : 0;
    lp[a] = n > 0 ? log2_hw((float)n) : kNegInf;
  }
  __syncthreads();

  // t = S log2(e) + log2 n for the group's logits held in S
  auto bias_group = [&](int gbase) {
#pragma unroll
    for (int ti = 0; ti < NT; ++ti) {
      const float4 l4 = *reinterpret_cast<const float4*>(&lp[gbase + 16 * ti + 4 * g]);
#pragma unroll
      for (int s = 0; s < QS; ++s) {
        S[ti][s][0] = fmaf(S[ti][s][0], kLog2e, l4.x);
        S[ti][s][1] = fmaf(S[ti][s][1], kLog2e, l4.y);
        S[ti][s][2] = fmaf(S[ti][s][2], kLog2e, l4.z);
        S[ti][s][3] = fmaf(S[ti][s][3], kLog2e, l4.w);
      }
    }
  };
  auto group_logits = [&](int gbase, bool with_values) {
#pragma unroll
    for (int k = 0; k < NT * 16 / CW; ++k) {
      const int cbase = gbase + k * CW;
      if (cbase < M0) {
        __syncthreads();
        stage_codes([&](int r) -> const T* {
          return cbase + r < M0 ? cp_head + (size_t)(cbase + r) * D : nullptr;
        });
        if (with_values)
          stage_values([&](int r) -> int { return cbase + r < M0 ? cbase + r : -1; });
        __syncthreads();
      }
#pragma unroll
      for (int tt = 0; tt < CW / 16; ++tt) {
        const int ti = k * (CW / 16) + tt;
        if (cbase + 16 * tt < M0) {
          logits(tt, S[ti]);
        } else {
#pragma unroll
          for (int s = 0; s < QS; ++s) S[ti][s] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
      }
    }
    bias_group(gbase);
  };

  constexpr bool kOneChunk = (CW == Cfg::GROUP);
  const bool need_importance =
      (P > 0 && P < M0) || args.importance != nullptr || (P > 0 && args.topp_idx != nullptr);
  float rz[QS];

  // u_a = sum over this wave's queries of W_ia / Z_i for the group in S: first
  // over the query subtiles in registers, then over the 16 query columns by a
  // reduce-scatter butterfly over lane bits 3, 0, 1, 2, which leaves lane c
  // with the L values of block perm(c) = 8 b3 + 4 b0 + 2 b1 + b2.
  auto importance_partials = [&](int gbase) {
    constexpr int NV = NT * 4, L = NT / 4;
    float u[NV];
#pragma unroll
    for (int ti = 0; ti < NT; ++ti)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float acc = 0.f;
#pragma unroll
        for (int s = 0; s < QS; ++s) acc = fmaf(S[ti][s][r], rz[s], acc);
        u[4 * ti + r] = acc;
      }
    auto step = [&](auto mask_tag, int half) {
      constexpr int MASK = decltype(mask_tag)::value;
      const bool upper = (c & MASK) != 0;
#pragma unroll
      for (int i = 0; i < NV / 2; ++i) {
        if (i < half) {
          const float lo = u[i] + xor16<MASK>(u[i]);
          const float hi = u[i + half] + xor16<MASK>(u[i + half]);
          u[i] = upper ? hi : lo;
        }
      }
    };
    step(std::integral_constant<int, 8>{}, NV / 2);
    step(std::integral_constant<int, 1>{}, NV / 4);
    step(std::integral_constant<int, 2>{}, NV / 8);
    step(std::integral_constant<int, 4>{}, NV / 16);
    const int blk = 8 * ((c >> 3) & 1) + 4 * (c & 1) + 2 * ((c >> 1) & 1) + ((c >> 2) & 1);
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const int k = L * blk + i;
      const int a = gbase + 16 * (k / 4) + 4 * g + (k % 4);
      if (a < M0MAX) lw[wave * M0MAX + a] = u[i];
    }
  };
  auto set_rz = [&]() {
#pragma unroll
    for (int s = 0; s < QS; ++s) {
      const float z = full_zp(s);
      rz[s] = qvalid[s] ? 1.f / z : 0.f;
    }
  };

  for (int grp = 0; grp < n_groups; ++grp) {
    const int gbase = grp * Cfg::GROUP;
    group_logits(gbase, kOneChunk);
    float mnew[QS];
#pragma unroll
    for (int s = 0; s < QS; ++s) mnew[s] = m[s];
#pragma unroll
    for (int ti = 0; ti < NT; ++ti)
#pragma unroll
      for (int s = 0; s < QS; ++s)
#pragma unroll
        for (int r = 0; r < 4; ++r) mnew[s] = fmaxf(mnew[s], S[ti][s][r]);
    raise_max(mnew);
#pragma unroll
    for (int ti = 0; ti < NT; ++ti)
#pragma unroll
      for (int s = 0; s < QS; ++s)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float w = exp2_hw(S[ti][s][r] - m[s]);
          S[ti][s][r] = w;
          zp[s] += w;
        }
    // one group: its max and denominators are final, so importance comes
    // straight from these weights before they are consumed
    if (n_groups == 1 && need_importance) {
      set_rz();
      importance_partials(gbase);
    }
    if constexpr (kB) {
      bf16x8 Sb[NT / 2][QS];
#pragma unroll
      for (int ti = 0; ti < NT; ti += 2) pack(S[ti], S[ti + 1], Sb[ti / 2]);
#pragma unroll
      for (int k = 0; k < NT * 16 / CW; ++k) {
        const int cbase = gbase + k * CW;
        if (cbase >= M0) break;
        if constexpr (!kOneChunk) {
          __syncthreads();
          stage_values([&](int r) -> int { return cbase + r < M0 ? cbase + r : -1; });
          __syncthreads();
        }
#pragma unroll
        for (int tt = 0; tt < CW / 16; tt += 2) {
          const int ti = k * (CW / 16) + tt;
          if (cbase + 16 * tt < M0) accumulate_b(tt, Sb[ti / 2]);
        }
      }
    } else {
#pragma unroll
      for (int k = 0; k < NT * 16 / CW; ++k) {
        const int cbase = gbase + k * CW;
        if (cbase >= M0) break;
        if constexpr (!kOneChunk) {
          __syncthreads();
          stage_values([&](int r) -> int { return cbase + r < M0 ? cbase + r : -1; });
          __syncthreads();
        }
#pragma unroll
        for (int tt = 0; tt < CW / 16; ++tt) {
          const int ti = k * (CW / 16) + tt;
          if (cbase + 16 * tt < M0) accumulate_f(tt, S[ti]);
        }
      }
    }
  }

  // ---- phase 2: importance with the final denominators -----------------------
  if (need_importance) {
    if (n_groups > 1) {
      set_rz();
      for (int grp = 0; grp < n_groups; ++grp) {
        // recompute this group's logits and weights with the final max
        const int gbase = grp * Cfg::GROUP;
        group_logits(gbase, false);
#pragma unroll
        for (int ti = 0; ti < NT; ++ti)
#pragma unroll
          for (int s = 0; s < QS; ++s)
#pragma unroll
            for (int r = 0; r < 4; ++r) S[ti][s][r] = exp2_hw(S[ti][s][r] - m[s]);
        importance_partials(gbase);
      }
    }
    __syncthreads();
    // sum the wave partials in fixed order
    for (int a = tid; a < M0; a += nthr) {
      float acc = 0.f;
      for (int wv = 0; wv < nwaves; ++wv) acc += lw[wv * M0MAX + a];
      lwf[a] = acc;
      if (args.importance)
        args.importance[((size_t)bh * args.n_tiles + t) * M0 + a] = acc;
    }
    __syncthreads();
  }

  // ---- phase 3: top-P (w desc, index asc) -------------------------------------
  if (P > 0) {
    if (P < M0) {
      for (int i = tid; i < 256; i += nthr) lhist[i] = 0;
      if (tid == 0) lmisc[2] = 0;
      __syncthreads();
      for (int a = tid; a < M0; a += nthr) atomicAdd(&lhist[(__float_as_uint(lwf[a]) >> 23) & 255], 1);
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
      const bool have_w = need_importance;
      for (int q = tid; q < P; q += nthr) {
        const int a = lsel[q];
        const float wa = have_w ? lwf[a] : 0.f;
        int rank = 0;
        for (int k = 0; k < P; ++k) {
          const int b = lsel[k];
          const float wb = have_w ? lwf[b] : 0.f;
          rank += (wb > wa) || (wb == wa && b < a);
        }
        args.topp_idx[((size_t)bh * args.n_tiles + t) * P + rank] = a;
      }
    }

    // ---- phase 4: child refinement ------------------------------------------
    // With one child the recovered parent logit is that child's own logit, so
    // every correcting weight is exactly zero: nothing to do.
    const T* cc_head = Cc + (size_t)h * M0 * Ch * D;
    const int rows = Ch > 1 ? P * Ch : 0;
    for (int cbase = 0; cbase < rows; cbase += CW) {
      __syncthreads();
      stage_codes([&](int r) -> const T* {
        const int q = cbase + r;
        if (q >= rows) return nullptr;
        return cc_head + ((size_t)lsel[q / Ch] * Ch + (q % Ch)) * D;
      });
      stage_values([&](int r) -> int {
        const int q = cbase + r;
        return q < rows ? M0 + lsel[q / Ch] * Ch + (q % Ch) : -1;
      });
      __syncthreads();
      // tiles in halves of HT so that logits and weights of a half stay in
      // registers next to the accumulators
      constexpr int HT = (CW / 16) < (NT / 2) ? (CW / 16) : (NT / 2);
#pragma unroll
      for (int h0 = 0; h0 < CW / 16; h0 += HT) {
        if (cbase + 16 * h0 >= rows) break;
        f32x4 Sc[HT][QS];
        float sp[HT][QS][2];  // recovered parent logits (rows 0-1 / 2-3 for Ch = 2)
#pragma unroll
        for (int tt = 0; tt < HT; ++tt) {
          logits(h0 + tt, Sc[tt]);
#pragma unroll
          for (int s = 0; s < QS; ++s) {
            const f32x4 v = Sc[tt][s];
            if (Ch == 2) {
              sp[tt][s][0] = (v[0] + v[1]) * 0.5f;
              sp[tt][s][1] = (v[2] + v[3]) * 0.5f;
            } else {
              float sum = (v[0] + v[1]) + (v[2] + v[3]);
              if (Ch >= 8) sum += shfl_xor(sum, 16);
              if (Ch >= 16) sum += shfl_xor(sum, 32);
              sp[tt][s][0] = sum * (1.f / (float)Ch);
              sp[tt][s][1] = sp[tt][s][0];
            }
          }
          const float4 l4 = *reinterpret_cast<const float4*>(&ll[16 * (h0 + tt) + 4 * g]);
#pragma unroll
          for (int s = 0; s < QS; ++s) {
            Sc[tt][s][0] = fmaf(Sc[tt][s][0], kLog2e, l4.x);
            Sc[tt][s][1] = fmaf(Sc[tt][s][1], kLog2e, l4.y);
            Sc[tt][s][2] = fmaf(Sc[tt][s][2], kLog2e, l4.z);
            Sc[tt][s][3] = fmaf(Sc[tt][s][3], kLog2e, l4.w);
          }
        }
        float mnew[QS];
#pragma unroll
        for (int s = 0; s < QS; ++s) mnew[s] = m[s];
#pragma unroll
        for (int tt = 0; tt < HT; ++tt)
#pragma unroll
          for (int s = 0; s < QS; ++s)
#pragma unroll
            for (int r = 0; r < 4; ++r) mnew[s] = fmaxf(mnew[s], Sc[tt][s][r]);
        raise_max(mnew);
        // dW = n_c (exp(T_c - m) - exp(Srec - m)); empty rows have n = 0 and
        // t = -inf, so dW = 0 (the recovered term is clamped to stay finite)
#pragma unroll
        for (int tt = 0; tt < HT; ++tt) {
          const float4 n4 = *reinterpret_cast<const float4*>(&ln[16 * (h0 + tt) + 4 * g]);
#pragma unroll
          for (int s = 0; s < QS; ++s) {
            const float e0 = exp2_hw(fminf(fmaf(sp[tt][s][0], kLog2e, -m[s]), 64.f));
            const float e1 = Ch == 2 ? exp2_hw(fminf(fmaf(sp[tt][s][1], kLog2e, -m[s]), 64.f)) : e0;
            Sc[tt][s][0] = fmaf(-n4.x, e0, exp2_hw(Sc[tt][s][0] - m[s]));
            Sc[tt][s][1] = fmaf(-n4.y, e0, exp2_hw(Sc[tt][s][1] - m[s]));
            Sc[tt][s][2] = fmaf(-n4.z, e1, exp2_hw(Sc[tt][s][2] - m[s]));
            Sc[tt][s][3] = fmaf(-n4.w, e1, exp2_hw(Sc[tt][s][3] - m[s]));
          }
        }
        if constexpr (kB) {
#pragma unroll
          for (int tt = 0; tt < HT; tt += 2) {
            bf16x8 b[QS];
            pack(Sc[tt], Sc[tt + 1], b);
            accumulate_b(h0 + tt, b);
          }
        } else {
#pragma unroll
          for (int tt = 0; tt < HT; ++tt) accumulate_f(h0 + tt, Sc[tt]);
        }
      }
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

template <typename T, int D, int NT, int MAXW>
hipError_t launch_attention_cfg(const AttnArgs& a, int BH, hipStream_t stream) {
  const long long grid = (long long)BH * a.n_tiles;
  if (grid > 0x7fffffff) return hipErrorInvalidConfiguration;
  const int waves = (a.block_q + 31) / 32;
  using Cfg = AttnCfg<T, D, NT, MAXW>;
  constexpr int slot = 8 + (Elem<T>::kBf16 ? 0 : 4) + (D == 128 ? 2 : 0) + (MAXW == 8 ? 1 : 0);
  hipError_t e = ensure_dynamic_lds((const void*)attention_kernel<T, D, NT, MAXW>,
                                    (int)Cfg::LDS_BYTES, slot);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attention_kernel<T, D, NT, MAXW>), dim3((unsigned)grid), dim3(waves * 64),
                     Cfg::LDS_BYTES, stream, a);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_attention(int BH, int H, int N, int M0, int Ch, int P, int block_q,
                            const void* Q, const void* Cp, const void* Cc, const float* Vbar,
                            const int32_t* counts, void* Y, int32_t* topp_idx,
                            float* importance, hipStream_t stream) {
  AttnArgs a;
  a.Q = Q;
  a.Cp = Cp;
  a.Cc = Cc;
  a.Vbar = Vbar;
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
  if (block_q <= 128) return launch_attention_cfg<T, D, 16, 4>(a, BH, stream);
  return launch_attention_cfg<T, D, 8, 8>(a, BH, stream);
}

#define AVQ_INSTANTIATE(T, D)                                                                  \
  template hipError_t launch_attention<T, D>(int, int, int, int, int, int, int, const void*,   \
                                             const void*, const void*, const float*,           \
                                             const int32_t*, void*, int32_t*, float*,          \
                                             hipStream_t);
AVQ_INSTANTIATE(bf16, 64)
AVQ_INSTANTIATE(bf16, 128)
AVQ_INSTANTIATE(float, 64)
AVQ_INSTANTIATE(float, 128)
#undef AVQ_INSTANTIATE

}  // namespace avq
