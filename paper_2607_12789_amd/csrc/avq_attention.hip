// Fused refined-codebook attention (Sec. 4.3, Alg. 2) for gfx950.
//
// One workgroup processes one query tile (block_q consecutive tokens of one
// (batch, head)); each wave owns 32 query rows. Everything is computed
// transposed, codewords x queries: S^T = C . Q^T and Xbar^T = Vbar^T . A^T.
// With the 16x16 MFMA layouts, a lane then owns one query column and four
// consecutive codeword rows, which gives:
//   - the A^T tile that comes out of the exp() is already in the register
//     layout of the MFMA operand of the next product (no shuffles);
//   - the Ch children of one parent sit in one lane's consecutive rows (plus
//     the partner lane group for Ch = 8, 16), so the recovered parent logit of
//     Eq. (parent_recovery) is an in-register sum;
//   - per-query softmax state (running max, denominator) is per lane.
//
// Phases per tile:
//   1. parent pass over the M0 parents in groups of 16*NT codewords held in
//      registers: logits, masked running max (App. D), A = exp(S - m) zeroed
//      for empty parents, Zbar += A n, Xbar += Vbar^T A (Eq. (vqflashattention));
//   2. importance w_p = n_p sum_i A_ip / Zbar_i (Eq. (importance)) from the
//      final denominators: straight from the registers when all parents fit in
//      one group, otherwise from a second sweep that recomputes the logits;
//   3. top-P: every parent's rank under (w desc, index asc) by counting, in
//      LDS; parents of rank < P are selected;
//   4. child pass over the P*Ch gathered children in chunks of 64 rows:
//      logits, running max raised over non-empty children with Xbar/Zbar
//      rescaled, recovered parent logit, correcting weights
//      dA = exp(T - m) - exp(Srec - m) zeroed for empty children
//      (Eq. (correcting_attention)), Zbar += dA n, Xbar += Vbar^T dA;
//   5. Y = Xbar / Zbar.
// Codeword rows and (transposed) aggregated values are staged through LDS in
// chunks shared by all waves of the workgroup.
#include "avq_common.hpp"

namespace avq {

template <typename T, int D, int NT, int MAXW>
struct AttnCfg {
  static constexpr bool kB = Elem<T>::kBf16;
  static constexpr int RPW = 32;                  // query rows per wave
  static constexpr int QS = RPW / 16;             // query subtiles per wave
  static constexpr int CW = kB ? 64 : 32;         // codeword rows per LDS chunk
  static constexpr int KQ = kB ? D / 32 : D / 4;  // MFMA k-steps over d
  static constexpr int DT = D / 16;               // d tiles of Xbar
  static constexpr int CPAD = kB ? 8 : 4;         // 16 bytes of row padding
  static constexpr int CROW = D + CPAD;
  static constexpr int VPAD = kB ? 8 : 4;
  static constexpr int VROW = CW + VPAD;
  static constexpr int M0MAX = 512;
  static constexpr int GROUP = 16 * NT;           // parents held in registers
  static_assert(GROUP % CW == 0, "a register group is a whole number of LDS chunks");
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
  constexpr int QS = Cfg::QS, CW = Cfg::CW, KQ = Cfg::KQ, DT = Cfg::DT;
  constexpr int CROW = Cfg::CROW, VROW = Cfg::VROW, M0MAX = Cfg::M0MAX;
  using QFrag = typename std::conditional<kB, bf16x8, float>::type;
  using VT = typename std::conditional<kB, bf16, float>::type;

  __shared__ __attribute__((aligned(16))) T lc[CW * CROW];   // codeword rows
  __shared__ __attribute__((aligned(16))) VT lv[D * VROW];   // Vbar^T of those rows
  __shared__ float ln[CW];                                   // their counts
  __shared__ float lnp[M0MAX];                                     // parent counts
  __shared__ __attribute__((aligned(16))) float lw[MAXW * M0MAX];  // per-wave importance
  __shared__ __attribute__((aligned(16))) float lwf[M0MAX];        // importance
  __shared__ int lsel[M0MAX];                                      // selected parents

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

  // ---- LDS staging of a chunk of CW codeword rows -----------------------------
  // stage_codes: row r of the chunk <- codebook row crow(r) (nullptr: zeros).
  auto stage_codes = [&](auto crow) {
    constexpr int VEC = 16 / sizeof(T);
    constexpr int VPR = D / VEC;
    for (int v = tid; v < CW * VPR; v += nthr) {
      const int r = v / VPR, col = (v % VPR) * VEC;
      const T* src = crow(r);
      uint4 val = {0u, 0u, 0u, 0u};
      if (src) val = *reinterpret_cast<const uint4*>(src + col);
      *reinterpret_cast<uint4*>(&lc[r * CROW + col]) = val;
    }
  };
  // stage_values: Vbar^T and counts of aggregate rows vrow(r) (-1: zeros).
  auto stage_values = [&](auto vrow) {
    const float* vb = Vbar + (size_t)bh * Mtot * D;
    if constexpr (kB) {
      // Vbar^T in bf16, codewords of each 32-block permuted so that lane
      // group g reads its 8 MFMA k-slots {4g..4g+3, 16+4g..16+4g+3} as one
      // 16-byte word: position 8g' + i holds codeword perm(g', i).
      for (int v = tid; v < (CW / 32) * 4 * (D / 4); v += nthr) {
        const int dq = v % (D / 4), gg = (v / (D / 4)) % 4, blk = v / (D / 4) / 4;
        float4 x[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int r = 32 * blk + (i < 4 ? 4 * gg + i : 16 + 4 * gg + (i - 4));
          const int a = vrow(r);
          x[i] = (a >= 0) ? *reinterpret_cast<const float4*>(vb + (size_t)a * D + 4 * dq)
                          : float4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          bf16x8 o;
#pragma unroll
          for (int i = 0; i < 8; ++i) o[i] = (bf16)(&x[i].x)[e];
          *reinterpret_cast<bf16x8*>(&lv[(4 * dq + e) * VROW + 32 * blk + 8 * gg]) = o;
        }
      }
    } else {
      // Vbar^T in fp32, natural codeword order, written as 4x4 transposes.
      for (int v = tid; v < (CW / 4) * (D / 4); v += nthr) {
        const int dq = v % (D / 4), rq = v / (D / 4);
        float4 x[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int a = vrow(4 * rq + i);
          x[i] = (a >= 0) ? *reinterpret_cast<const float4*>(vb + (size_t)a * D + 4 * dq)
                          : float4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float4 o = {(&x[0].x)[e], (&x[1].x)[e], (&x[2].x)[e], (&x[3].x)[e]};
          *reinterpret_cast<float4*>(&lv[(4 * dq + e) * VROW + 4 * rq]) = o;
        }
      }
    }
    const int32_t* cb = counts + (size_t)bh * Mtot;
    for (int r = tid; r < CW; r += nthr) {
      const int a = vrow(r);
      ln[r] = (a >= 0) ? (float)cb[a] : 0.f;
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

  // ---- Xbar^T += Vbar^T . W^T for chunk tiles (tt, tt+1) (bf16) or tt (fp32) --
  f32x4 X[DT][QS];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int s = 0; s < QS; ++s) X[dt][s] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto accumulate = [&](int tt, const f32x4 (&w0)[QS], const f32x4 (&w1)[QS]) {
    if constexpr (kB) {
      bf16x8 b[QS];
#pragma unroll
      for (int s = 0; s < QS; ++s) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          b[s][r] = (bf16)w0[s][r];
          b[s][4 + r] = (bf16)w1[s][r];
        }
      }
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const bf16x8 a =
            *reinterpret_cast<const bf16x8*>(&lv[(16 * dt + c) * VROW + 16 * tt + 8 * g]);
#pragma unroll
        for (int s = 0; s < QS; ++s) X[dt][s] = mfma_bf16(a, b[s], X[dt][s]);
      }
    } else {
      (void)w1;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const float4 a = *reinterpret_cast<const float4*>(&lv[(16 * dt + c) * VROW + 16 * tt + 4 * g]);
#pragma unroll
        for (int s = 0; s < QS; ++s) {
          X[dt][s] = mfma_f32(a.x, w0[s][0], X[dt][s]);
          X[dt][s] = mfma_f32(a.y, w0[s][1], X[dt][s]);
          X[dt][s] = mfma_f32(a.z, w0[s][2], X[dt][s]);
          X[dt][s] = mfma_f32(a.w, w0[s][3], X[dt][s]);
        }
      }
    }
  };

  // Per-lane softmax state for query columns c + 16 s. zp holds this lane
  // group's partial denominator; the four groups are summed when needed.
  float m[QS], zp[QS];
#pragma unroll
  for (int s = 0; s < QS; ++s) {
    m[s] = -__builtin_inff();
    zp[s] = 0.f;
  }
  auto full_z = [&](int s) {
    float z = zp[s];
    z += shfl_xor(z, 16);
    z += shfl_xor(z, 32);
    return z;
  };
  auto rescale = [&](const float (&mnew)[QS]) {
#pragma unroll
    for (int s = 0; s < QS; ++s) {
      const float sc = (mnew[s] == -__builtin_inff()) ? 1.f : exp_neg(m[s] - mnew[s]);
      zp[s] *= sc;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) X[dt][s] *= sc;
      m[s] = mnew[s];
    }
  };

  const T* cp_head = Cp + (size_t)h * M0 * D;
  const int n_groups = (M0 + Cfg::GROUP - 1) / Cfg::GROUP;
  f32x4 S[NT][QS];

  // ---- phase 1: parent pass (online softmax over register groups) -----------
  const int32_t* nb = counts + (size_t)bh * Mtot;
  for (int a = tid; a < M0MAX; a += nthr) lnp[a] = a < M0 ? (float)nb[a] : 0.f;
  __syncthreads();
  auto parent_count = [&](int a) -> float { return lnp[a]; };

  for (int grp = 0; grp < n_groups; ++grp) {
    const int gbase = grp * Cfg::GROUP;
    // logits for the whole group (chunks staged one after another)
#pragma unroll
    for (int k = 0; k < NT * 16 / CW; ++k) {
      const int cbase = gbase + k * CW;
      if (cbase < M0) {
        __syncthreads();
        stage_codes([&](int r) -> const T* {
          return cbase + r < M0 ? cp_head + (size_t)(cbase + r) * D : nullptr;
        });
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
    // masked group max and rescale
    float mnew[QS];
#pragma unroll
    for (int s = 0; s < QS; ++s) mnew[s] = m[s];
#pragma unroll
    for (int ti = 0; ti < NT; ++ti)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float n = parent_count(gbase + 16 * ti + 4 * g + r);
#pragma unroll
        for (int s = 0; s < QS; ++s)
          if (n > 0.f) mnew[s] = fmaxf(mnew[s], S[ti][s][r]);
      }
#pragma unroll
    for (int s = 0; s < QS; ++s) {
      mnew[s] = fmaxf(mnew[s], shfl_xor(mnew[s], 16));
      mnew[s] = fmaxf(mnew[s], shfl_xor(mnew[s], 32));
    }
    rescale(mnew);
    // A = exp(S - m), zero for empty parents; Zbar += A n
#pragma unroll
    for (int ti = 0; ti < NT; ++ti)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float n = parent_count(gbase + 16 * ti + 4 * g + r);
#pragma unroll
        for (int s = 0; s < QS; ++s) {
          const float a = (n > 0.f) ? exp_neg(S[ti][s][r] - m[s]) : 0.f;
          S[ti][s][r] = a;
          zp[s] = fmaf(a, n, zp[s]);
        }
      }
    // Xbar += Vbar^T A, staging the Vbar rows of the group chunk by chunk
#pragma unroll
    for (int k = 0; k < NT * 16 / CW; ++k) {
      const int cbase = gbase + k * CW;
      if (cbase >= M0) break;
      __syncthreads();
      stage_values([&](int r) -> int { return cbase + r < M0 ? cbase + r : -1; });
      __syncthreads();
      if constexpr (kB) {
#pragma unroll
        for (int tt = 0; tt < CW / 16; tt += 2) {
          const int ti = k * (CW / 16) + tt;
          accumulate(tt, S[ti], S[ti + 1]);
        }
      } else {
#pragma unroll
        for (int tt = 0; tt < CW / 16; ++tt) {
          const int ti = k * (CW / 16) + tt;
          accumulate(tt, S[ti], S[ti]);
        }
      }
    }
  }

  // ---- phase 2: importance with the final denominators -----------------------
  const bool need_importance = (P > 0) || (args.importance != nullptr);
  if (need_importance) {
    float rz[QS];
#pragma unroll
    for (int s = 0; s < QS; ++s) {
      const float z = full_z(s);
      rz[s] = qvalid[s] ? 1.f / z : 0.f;
    }
    for (int grp = 0; grp < n_groups; ++grp) {
      const int gbase = grp * Cfg::GROUP;
      if (n_groups > 1) {
        // recompute this group's logits and weights with the final max
#pragma unroll
        for (int k = 0; k < NT * 16 / CW; ++k) {
          const int cbase = gbase + k * CW;
          if (cbase < M0) {
            __syncthreads();
            stage_codes([&](int r) -> const T* {
              return cbase + r < M0 ? cp_head + (size_t)(cbase + r) * D : nullptr;
            });
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
#pragma unroll
        for (int ti = 0; ti < NT; ++ti)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float n = parent_count(gbase + 16 * ti + 4 * g + r);
#pragma unroll
            for (int s = 0; s < QS; ++s)
              S[ti][s][r] = (n > 0.f) ? exp_neg(S[ti][s][r] - m[s]) : 0.f;
          }
      }
      // u_a = sum over this wave's queries of A_ia / Zbar_i: first over the
      // query subtiles in registers, then over the 16 query columns by a
      // reduce-scatter butterfly that leaves lane c with values [L c, L c + L).
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
#pragma unroll
      for (int step = 0; step < 4; ++step) {
        const int mask = 8 >> step;
        const int half = NV >> (step + 1);
        const bool upper = (c & mask) != 0;
#pragma unroll
        for (int i = 0; i < half; ++i) {
          const float lo = u[i], hi = u[i + half];
          const float send = upper ? lo : hi;
          const float keep = upper ? hi : lo;
          u[i] = keep + shfl_xor(send, mask);
        }
      }
#pragma unroll
      for (int i = 0; i < L; ++i) {
        const int k = L * c + i;
        const int a = gbase + 16 * (k / 4) + 4 * g + (k % 4);
        if (a < M0MAX) lw[wave * M0MAX + a] = u[i];
      }
    }
    __syncthreads();
    // sum the wave partials in fixed order, weight by the counts
    for (int a = tid; a < M0; a += nthr) {
      float acc = 0.f;
      for (int wv = 0; wv < nwaves; ++wv) acc += lw[wv * M0MAX + a];
      const float w = acc * (float)nb[a];
      lwf[a] = w;
      if (args.importance)
        args.importance[((size_t)bh * args.n_tiles + t) * M0 + a] = w;
    }
    __syncthreads();
  }

  // ---- phase 3: top-P by rank counting (w desc, index asc) --------------------
  if (P > 0) {
    for (int a = tid; a < M0; a += nthr) {
      const float wa = lwf[a];
      int rank = 0;
      for (int k = 0; k < M0; ++k) {
        const float wk = lwf[k];
        rank += (wk > wa) || (wk == wa && k < a);
      }
      if (rank < P) {
        lsel[rank] = a;
        if (args.topp_idx) args.topp_idx[((size_t)bh * args.n_tiles + t) * P + rank] = a;
      }
    }
    __syncthreads();

    // ---- phase 4: child refinement ------------------------------------------
    const T* cc_head = Cc + (size_t)h * M0 * Ch * D;
    const int rows = P * Ch;
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
      f32x4 Sc[CW / 16][QS];
#pragma unroll
      for (int tt = 0; tt < CW / 16; ++tt) logits(tt, Sc[tt]);
      // running max over the non-empty children of the chunk
      float mnew[QS];
#pragma unroll
      for (int s = 0; s < QS; ++s) mnew[s] = m[s];
#pragma unroll
      for (int tt = 0; tt < CW / 16; ++tt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float n = ln[16 * tt + 4 * g + r];
#pragma unroll
          for (int s = 0; s < QS; ++s)
            if (n > 0.f) mnew[s] = fmaxf(mnew[s], Sc[tt][s][r]);
        }
#pragma unroll
      for (int s = 0; s < QS; ++s) {
        mnew[s] = fmaxf(mnew[s], shfl_xor(mnew[s], 16));
        mnew[s] = fmaxf(mnew[s], shfl_xor(mnew[s], 32));
      }
      rescale(mnew);
      // recovered parent logit = mean of the Ch child logits of each parent
#pragma unroll
      for (int tt = 0; tt < CW / 16; ++tt) {
#pragma unroll
        for (int s = 0; s < QS; ++s) {
          f32x4 sp;
          if (Ch == 1) {
            sp = Sc[tt][s];
          } else if (Ch == 2) {
            const float a = Sc[tt][s][0] + Sc[tt][s][1], b = Sc[tt][s][2] + Sc[tt][s][3];
            sp = f32x4{a, a, b, b} * 0.5f;
          } else {
            float sum = (Sc[tt][s][0] + Sc[tt][s][1]) + (Sc[tt][s][2] + Sc[tt][s][3]);
            if (Ch >= 8) sum += shfl_xor(sum, 16);
            if (Ch >= 16) sum += shfl_xor(sum, 32);
            const float mean = sum * (1.f / (float)Ch);
            sp = f32x4{mean, mean, mean, mean};
          }
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float n = ln[16 * tt + 4 * g + r];
            const float da = exp_neg(Sc[tt][s][r] - m[s]) - exp_neg(sp[r] - m[s]);
            const float dA = (n > 0.f) ? da : 0.f;
            Sc[tt][s][r] = dA;
            zp[s] = fmaf(dA, n, zp[s]);
          }
        }
      }
      if constexpr (kB) {
#pragma unroll
        for (int tt = 0; tt < CW / 16; tt += 2) accumulate(tt, Sc[tt], Sc[tt + 1]);
      } else {
#pragma unroll
        for (int tt = 0; tt < CW / 16; ++tt) accumulate(tt, Sc[tt], Sc[tt]);
      }
    }
  }

  // ---- phase 5: Y = Xbar / Zbar ------------------------------------------------
#pragma unroll
  for (int s = 0; s < QS; ++s) {
    const float z = full_z(s);
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
  hipLaunchKernelGGL((attention_kernel<T, D, NT, MAXW>), dim3((unsigned)grid), dim3(waves * 64),
                     0, stream, a);
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

template hipError_t launch_attention<bf16, 64>(int, int, int, int, int, int, int, const void*,
                                               const void*, const void*, const float*,
                                               const int32_t*, void*, int32_t*, float*,
                                               hipStream_t);
template hipError_t launch_attention<bf16, 128>(int, int, int, int, int, int, int, const void*,
                                                const void*, const void*, const float*,
                                                const int32_t*, void*, int32_t*, float*,
                                                hipStream_t);
template hipError_t launch_attention<float, 64>(int, int, int, int, int, int, int, const void*,
                                                const void*, const void*, const float*,
                                                const int32_t*, void*, int32_t*, float*,
                                                hipStream_t);
template hipError_t launch_attention<float, 128>(int, int, int, int, int, int, int, const void*,
                                                 const void*, const void*, const float*,
                                                 const int32_t*, void*, int32_t*, float*,
                                                 hipStream_t);

}  // namespace avq
