// Fused refined-codebook attention (Sec. 4.3, Alg. 2) for gfx950.
//
// One workgroup processes one query tile (block_q consecutive tokens of one
// (batch, head)); each wave owns 32 query rows. Everything is computed
// transposed, codewords x queries: S^T = C . Q^T and Xbar^T = Vmean^T . W^T,
// with 16x16x32 bf16 (16x16x4 fp32) MFMA. A lane owns one query column and,
// in a pair of 16-row logit tiles, 8 consecutive codes (one octet of the
// packed aggregates): the 16 rows of tile tt are chunk rows
// 32 (tt/2) + 8 g + 4 (tt%2) + r for lane group g and r = 0..3. So
//   - the weights that come out of exp2() are already the B operand of the
//     value product, and its A operand, the 8 mean values of the octet at one
//     column, is one 16-byte LDS read;
//   - the 8 children of a parent (Ch = 8) are one lane's 8 values: the
//     recovered parent logit of Eq. (parent_recovery) is an in-register sum
//     (Ch = 16: plus one cross-lane-group exchange);
//   - per-query softmax state is per lane.
//
// Log-count bias (App. D): a parent's logit enters as t = S + ln n (the MFMA
// accumulator starts at ln n), so its weight exp(t - m) is n exp(S - m) and an
// empty parent (ln n = -inf) drops out of the max and of every sum without
// masks. It is applied to the parent's mean value Vbar/n, so
// sum_p n_p exp(S_p - m) Vbar_p / n_p is the numerator of
// Eq. (vqflashattention). The recovered parent logit is taken from the raw
// child logits T_c (all Ch children, empty ones included); then the children
// take the same bias, T_c + ln n_c, so that empty children and padding rows
// (-inf) take no part in the running max (App. D), and their correcting weight
// exp(T_c + ln n_c - m) - n_c exp(Srec - m), Eq. (correcting_attention) times
// n_c, is exactly zero for them however far their logits lie. The denominator
// Z is the fp32 sum of the same weights, per lane over its codes and then
// over the four lane groups (bf16: the value product takes the weights
// rounded to bf16, so numerator and denominator differ by that rounding, a
// relative 2^-9 per weight).
//
// Running max (in log2 units): it only moves when a chunk's logits exceed it
// by more than kLazy, so the rescaling of the accumulators and the reduction
// of the chunk max across lanes are rare; weights stay below 2^kLazy, far
// inside fp32 and bf16 range, and the result does not depend on the shift.
//
// Codewords stream through LDS in chunks of 64 rows (8 octets): codeword rows
// XOR-swizzled by 16-byte unit (the 16 rows of a logit tile hit different
// banks), packed mean octets and their count info as they lie in HBM, all by
// direct global->LDS loads (no registers, no VALU), double buffered: the next
// chunk is in flight while the current one is computed (fp32 at d = 128: one
// buffer, refilled after each chunk). Phases per tile:
//   1. parent sweep: logits, running max, weights, fp32 parent denominator,
//      Xbar += Vmean^T W;
//   2. importance (Eq. (importance)) with the final max and denominator: the
//      last parent chunk's weights are still in registers when both are
//      final, and are scaled by 1/Z there; a second sweep recomputes the
//      logits of the other chunks, with queries as the MFMA rows, and takes
//      exp(t - m - ln Z) directly; sums over the tile's queries in registers
//      and across lanes (a butterfly over the 16 query lanes of a row for the
//      last chunk, row swaps over the 4 lane groups in the sweep), then a
//      fixed order over waves. TILED instead takes the importance of App. B
//      inside phase 1, chunk by chunk, and skips the second sweep;
//   3. top-P in one wave: a threshold on the importance bits, built bit by
//      bit from the top, finds the P-th largest value; ties at it go to the
//      lowest indices; the selected parents are listed in index order;
//   4. child sweep over the child octets of the selected parents: logits,
//      recovered parent logit, log-count bias (running max over non-empty
//      children), correcting weights, Xbar += Vmean^T dW;
//   5. Y = Xbar / Z.
// With a query order, tile position i takes token order[i]: Q rows are read
// from, and Y rows written to, those tokens.
#include "avq_common.hpp"
#include "avq_packed.hpp"

#include <type_traits>

namespace avq {

template <typename T, int D, int MAXW>
struct AttnCfg {
  static constexpr bool kB = Elem<T>::kBf16;
  static constexpr int RPW = 32;                  // query rows per wave (16 QS)
  static constexpr int QS = RPW / 16;             // query subtiles per wave
  static constexpr int CW = 64;                   // codeword rows per chunk
  static constexpr int TPC = CW / 16;             // 16-row tiles per chunk
  static constexpr int KQ = kB ? D / 32 : D / 4;  // MFMA k-steps over d
  static constexpr int DT = D / 16;               // d tiles of Xbar
  static constexpr int ESZ = sizeof(T);
  static constexpr int EPU = 16 / ESZ;            // elements per 16-byte unit
  static constexpr int U = D * ESZ / 16;          // 16-byte units per codeword row
  static constexpr int COPIES = CW * U / 64;      // wave copies per array per chunk
  static constexpr int CPW = (COPIES + MAXW - 1) / MAXW;  // ... per wave, at most
  static constexpr int OCT_ELEMS = 8 * D;         // elements of one mean octet
  static constexpr int OCPY = OCT_ELEMS * ESZ / 1024;  // wave copies per mean octet
  static constexpr int M0MAX = 512;
  static constexpr int CHUNK_BYTES = CW * D * ESZ;
  // one chunk buffer: codeword rows, mean octets, count info
  static constexpr int OFF_C = 0;
  static constexpr int OFF_V = CHUNK_BYTES;
  static constexpr int OFF_I = 2 * CHUNK_BYTES;
  static constexpr int BUF_BYTES = 2 * CHUNK_BYTES + 8 * 64;
  static constexpr int NBUF = 2 * BUF_BYTES <= 72 * 1024 ? 2 : 1;
  // after the buffers
  static constexpr size_t OFF_LW = (size_t)NBUF * BUF_BYTES;    // [2][MAXW][CW] f32
  static constexpr size_t OFF_WF = OFF_LW + 2 * MAXW * CW * 4;  // [M0MAX] f32
  static constexpr size_t OFF_SEL = OFF_WF + M0MAX * 4;         // [M0MAX] i32
  static constexpr size_t LDS_BYTES = OFF_SEL + M0MAX * 4;
  static constexpr int kWavesPerEu = (kB && D == 64) ? 3 : 2;
  static_assert(COPIES % MAXW == 0 || COPIES < MAXW, "copies split evenly over the waves");
  static_assert(OCPY >= 1 && (OCPY & (OCPY - 1)) == 0, "whole wave copies per octet");
};

struct AttnArgs {
  const void* Q;
  const void* Cp;
  const void* Cc;
  const unsigned char* packed;
  void* Y;
  int32_t* topp_idx;
  float* importance;
  const int32_t* order;  // nullable: token row of each query position
  int H, N, M0, Ch, P, block_q, n_tiles;
};

// A raw buffer resource over bytes [p, p + bytes): stride 0, no format
// conversion (the gfx9 word-3 setting); loads past the end read 0.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// XOR swizzle of the 16-byte units of a staged codeword row: the 16 rows a
// logit tile reads (8 (c/4) + 4 h + c % 4 for lanes c) get distinct units for
// the same logical unit, so 16 lanes reading one unit each hit distinct banks.
template <int U>
__device__ __forceinline__ int row_swizzle(int r) {
  if constexpr (U >= 16) return ((r >> 3) & 3) * 4 + (r & 3);
  return ((r >> 3) & 3) * 2 + ((r >> 1) & 1);  // U = 8: two rows per 256 bytes
}

// Register budget: two or three waves per SIMD (at most 256 or 168 registers
// each), so that other tiles' MFMA work runs while one workgroup waits.
// TILED: importance with the count-extrapolated denominator of App. B, one
// codeword tile per chunk, computed in the parent sweep (no second sweep).
template <typename T, int D, int MAXW, bool TILED>
__global__ __launch_bounds__(MAXW * 64)
__attribute__((amdgpu_waves_per_eu(AttnCfg<T, D, MAXW>::kWavesPerEu)))
void attention_kernel(AttnArgs args) {
  using Cfg = AttnCfg<T, D, MAXW>;
  constexpr bool kB = Cfg::kB;
  constexpr int QS = Cfg::QS, CW = Cfg::CW, TPC = Cfg::TPC, KQ = Cfg::KQ, DT = Cfg::DT,
                U = Cfg::U, EPU = Cfg::EPU, CPW = Cfg::CPW,
                OCPY = Cfg::OCPY, OCT_ELEMS = Cfg::OCT_ELEMS;
  using QFrag = typename std::conditional<kB, bf16x8, float>::type;
  constexpr float kLn2 = 0.6931471805599453f;
  constexpr float kLazy = 8.f;         // log2 units the max may lag behind
  constexpr float kMaxFloor = -1e30f;  // finite start of the running max

  extern __shared__ __attribute__((aligned(16))) unsigned char lds_raw[];
  float* lw = reinterpret_cast<float*>(lds_raw + Cfg::OFF_LW);   // per-wave importance
  float* lwf = reinterpret_cast<float*>(lds_raw + Cfg::OFF_WF);  // importance
  int* lsel = reinterpret_cast<int*>(lds_raw + Cfg::OFF_SEL);    // selected, index order

  const T* __restrict__ Q = static_cast<const T*>(args.Q);
  const T* __restrict__ Cp = static_cast<const T*>(args.Cp);
  const T* __restrict__ Cc = static_cast<const T*>(args.Cc);
  const int N = args.N, M0 = args.M0, Ch = args.Ch, P = args.P;
  const PackedLayout PL = packed_layout(M0, Ch, D, Cfg::ESZ);
  const int PO = PL.PO, CO = PL.CO, ZO = PL.zero_oct;

  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = tid % kWave;
  const int g = lane / 16, c = lane % 16;
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = tile / args.n_tiles, t = tile % args.n_tiles;
  const int h = bh % args.H;
  const int q_begin = t * args.block_q;
  const int q_end = min(q_begin + args.block_q, N);
  const int row0 = q_begin + wave * Cfg::RPW;
  const bool has_rows = row0 < q_end;                                 // wave-uniform
  const int n_active = (q_end - q_begin + Cfg::RPW - 1) / Cfg::RPW;  // waves with rows
  const unsigned char* pk = args.packed + (size_t)bh * PL.bytes;
  const T* cp_head = Cp + (size_t)h * M0 * D;
  const T* cc_head = Cc + (size_t)h * M0 * Ch * D;

  // token row of query position i (the query order, if any; -1 for an entry
  // outside [0, N), which then takes no part)
  auto token_row = [&](int i) -> int {
    if (args.order == nullptr) return i;
    const int r = args.order[i];
    return (unsigned)r < (unsigned)N ? r : -1;
  };

  // ---- query fragments (B operand of S^T = C . Q^T) -------------------------
  QFrag qf[QS][KQ];
  bool qvalid[QS];
#pragma unroll
  for (int s = 0; s < QS; ++s) {
    const int i = row0 + 16 * s + c;
    const int src = i < q_end ? token_row(i) : -1;
    qvalid[s] = src >= 0;
    const T* qrow = Q + ((size_t)bh * N + (qvalid[s] ? src : 0)) * D;
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
  // Copies are buffer loads straight into LDS: one buffer resource per array
  // (base and size in scalar registers, made once per tile), the offset of
  // the chunk and copy in a scalar register, and a per-lane offset that is the
  // same for every chunk, computed here once; the LDS destination is uniform.
  // Copy i of this wave is wave copy j = wave + MAXW i of each array (every j
  // is below COPIES, a multiple of MAXW). A codeword copy covers RPC = 64 / U
  // consecutive chunk rows, RPC j + lane / U, inside one octet.
  static_assert(Cfg::COPIES % MAXW == 0, "copies split evenly over the waves");
  constexpr uint32_t RowB = D * Cfg::ESZ;
  constexpr uint32_t OctB = OCT_ELEMS * Cfg::ESZ;
  constexpr int RPC = 64 / U;
  const int lrow = lane / U;               // the lane's row inside its codeword copy
  const uint32_t loff = lrow * RowB;       // ... as a byte offset
  uint32_t uoff[CPW];                      // the lane's swizzled unit in codeword copy i
#pragma unroll
  for (int i = 0; i < CPW; ++i) {
    const int r = RPC * (wave + MAXW * i) + lrow;
    uoff[i] = (uint32_t)(((lane % U) ^ row_swizzle<U>(r)) * EPU * Cfg::ESZ);
  }
  const uint32_t moff = 16u * lane;  // lane offset of a mean or count-info copy
  // the wave index in a scalar register: the copy indices derived from it are
  // then computed on the scalar unit
  const int cwave = __builtin_amdgcn_readfirstlane(wave);
  auto buffer = [&](int b) { return lds_raw + b * Cfg::BUF_BYTES; };
  const __amdgpu_buffer_rsrc_t r_cp = make_rsrc(cp_head, (uint32_t)M0 * RowB);
  const __amdgpu_buffer_rsrc_t r_cc = make_rsrc(cc_head, (uint32_t)(M0 * Ch) * RowB);
  const __amdgpu_buffer_rsrc_t r_pk = make_rsrc(pk, (uint32_t)PL.bytes);
  // 16 bytes per lane from rsrc at soffset + voffset to LDS at lds_off + 16 lane
  auto copy = [&](__amdgpu_buffer_rsrc_t rs, uint32_t voffset, uint32_t soffset, uint32_t lds_off) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rs, (__attribute__((address_space(3))) void*)(lds_raw + __builtin_amdgcn_readfirstlane(lds_off)),
        16, voffset, __builtin_amdgcn_readfirstlane(soffset), 0, 0);
  };
  const uint32_t info_off = (uint32_t)PL.info_off;
  // parent chunk k into buffer b: rows past M0 - 1 read row M0 - 1 (only the
  // last chunk has such rows; its codeword offsets are clamped per lane)
  auto issue_parent = [&](int k, int b, bool with_values) {
    const uint32_t B = (uint32_t)(b * Cfg::BUF_BYTES);
    const uint32_t kb = (uint32_t)(64 * k) * RowB;
    if (64 * (k + 1) <= M0) {
#pragma unroll
      for (int i = 0; i < CPW; ++i) {
        const int j = cwave + MAXW * i;
        copy(r_cp, loff + uoff[i], kb + (uint32_t)(RPC * j) * RowB, B + Cfg::OFF_C + 1024 * j);
      }
    } else {
#pragma unroll
      for (int i = 0; i < CPW; ++i) {
        const int j = cwave + MAXW * i;
        const uint32_t r = (uint32_t)min(RPC * j + lrow, M0 - 1 - 64 * k);
        copy(r_cp, r * RowB + uoff[i], kb, B + Cfg::OFF_C + 1024 * j);
      }
    }
    if (with_values) {
#pragma unroll
      for (int i = 0; i < CPW; ++i) {
        const int j = cwave + MAXW * i;
        copy(r_pk, moff, (uint32_t)(8 * k + j / OCPY) * OctB + (uint32_t)(j % OCPY) * 1024u,
             B + Cfg::OFF_V + 1024 * j);
      }
    }
    if (cwave == MAXW - 1 && lane < 32)  // 8 octets x 64 bytes of count info
      copy(r_pk, moff, info_off + (uint32_t)(8 * k) * 64u, B + Cfg::OFF_I);
  };
  // child chunk k: octet o (o = 8k + os) belongs to selected parent o >> co_shift
  // (CO is 1 or 2); octets past the last read the empty octet (means and
  // counts) and the last octet's rows, rows past Ch - 1 the last child.
  // With Ch <= 4 the copies that hold only rows 4..7 of their octets
  // (padding, never read) are not made.
  const int n_child_oct = Ch > 1 ? P * CO : 0;
  const int co_shift = CO == 2 ? 1 : 0;
  const bool half_child = Ch <= 4;  // rows 4..7 of every child octet are padding
  auto issue_child = [&](int k, int b) {
    const uint32_t B = (uint32_t)(b * Cfg::BUF_BYTES);
    // lane l holds the selected parent of octet 8k + (l mod 8) (clamped to the
    // last octet); a copy takes the one of its octet with a lane read
    const int sel_l = lsel[min(8 * k + (lane & 7), n_child_oct - 1) >> co_shift];
    if (Ch >= 8) {  // every row of a copy is a child
#pragma unroll
      for (int i = 0; i < CPW; ++i) {
        const int j = cwave + MAXW * i;
        const int os = (RPC * j) / 8;
        const int o = min(8 * k + os, n_child_oct - 1);
        const int jj = o - ((o >> co_shift) << co_shift);  // child octet of the parent
        const int par = __builtin_amdgcn_readlane(sel_l, os);
        const int u = jj * 8 + (RPC * j) % 8;  // the copy's first row among the children
        copy(r_cc, loff + uoff[i], (uint32_t)(par * Ch + u) * RowB, B + Cfg::OFF_C + 1024 * j);
      }
    } else {
#pragma unroll
      for (int i = 0; i < CPW; ++i) {
        const int j = cwave + MAXW * i;
        if (RPC <= 4 && half_child && (RPC * j) % 8 >= 4) continue;
        const int os = (RPC * j) / 8;
        const int o = min(8 * k + os, n_child_oct - 1);
        const int jj = o - ((o >> co_shift) << co_shift);
        const int par = __builtin_amdgcn_readlane(sel_l, os);
        const int u = jj * 8 + (RPC * j) % 8;
        const uint32_t cc = (uint32_t)min(u + lrow, Ch - 1);
        copy(r_cc, cc * RowB + uoff[i], (uint32_t)(par * Ch) * RowB, B + Cfg::OFF_C + 1024 * j);
      }
    }
#pragma unroll
    for (int i = 0; i < CPW; ++i) {
      const int j = cwave + MAXW * i;
      const int os = j / OCPY;
      const int o = 8 * k + os;
      const int par = __builtin_amdgcn_readlane(sel_l, os);
      const int oct = o >= n_child_oct ? ZO : PO + (par << co_shift) + (o - ((o >> co_shift) << co_shift));
      copy(r_pk, moff, (uint32_t)oct * OctB + (uint32_t)(j % OCPY) * 1024u, B + Cfg::OFF_V + 1024 * j);
    }
    if (cwave == MAXW - 1 && lane < 32) {  // count info: lane's octet lane / 4
      const int o = 8 * k + lane / 4;
      const int sl = o >> co_shift;
      const int oct = o >= n_child_oct ? ZO : PO + (lsel[sl] << co_shift) + (o - (sl << co_shift));
      copy(r_pk, (uint32_t)oct * 64u + (uint32_t)(16 * (lane % 4)), info_off, B + Cfg::OFF_I);
    }
  };
  auto wait_chunk = [&]() {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  };

  // ---- S^T tile (16 codewords x 16 queries) for chunk tile tt ----------------
  // (qrows: the operands swapped, so the tile is S itself, queries as the D
  // rows: lane (g, c) holds queries 4 g + r of the codeword in chunk row
  // 32 (tt/2) + 8 (c/4) + 4 (tt%2) + c % 4; both MFMA operands have the same
  // lane layout)
  auto logits = [&](const unsigned char* B, int tt, f32x4 (&out)[QS], const f32x4& init,
                    bool qrows) {
    const T* lc = reinterpret_cast<const T*>(B + Cfg::OFF_C);
    const int r = 32 * (tt / 2) + 8 * (c / 4) + 4 * (tt % 2) + (c % 4);
    const int sw = row_swizzle<U>(r);
#pragma unroll
    for (int kq = 0; kq < KQ; ++kq) {
      if constexpr (kB) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(&lc[r * D + ((4 * kq + g) ^ sw) * EPU]);
#pragma unroll
        for (int s = 0; s < QS; ++s)
          out[s] = qrows ? mfma_bf16(qf[s][kq], a, kq == 0 ? init : out[s])
                         : mfma_bf16(a, qf[s][kq], kq == 0 ? init : out[s]);
      } else {
        const float a = lc[r * D + (kq ^ sw) * EPU + g];
#pragma unroll
        for (int s = 0; s < QS; ++s)
          out[s] = qrows ? mfma_f32(qf[s][kq], a, kq == 0 ? init : out[s])
                         : mfma_f32(a, qf[s][kq], kq == 0 ? init : out[s]);
      }
    }
  };
  // count info of the lane's 4 rows in tile tt: n (part 0) or ln n (part 1)
  auto info4 = [&](const unsigned char* B, int tt, int part) {
    const float* li = reinterpret_cast<const float*>(B + Cfg::OFF_I);
    return *reinterpret_cast<const f32x4*>(&li[(4 * (tt / 2) + g) * 16 + 8 * part + 4 * (tt % 2)]);
  };

  // ---- Xbar^T += Vmean^T . W^T ---------------------------------------------
  f32x4 X[DT][QS];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int s = 0; s < QS; ++s) X[dt][s] = f32x4{0.f, 0.f, 0.f, 0.f};

  // bf16: tiles 2b, 2b+1 form one B operand (k-slots 8 g .. 8 g + 7 = the 8
  // codes of octet 4 b + g); the A operand is that octet at column d
  auto accumulate_b = [&](const unsigned char* B, int b, const f32x4 (&w0)[QS],
                          const f32x4 (&w1)[QS]) {
    bf16x8 bw[QS];
#pragma unroll
    for (int s = 0; s < QS; ++s) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        bw[s][r] = (bf16)w0[s][r];
        bw[s][4 + r] = (bf16)w1[s][r];
      }
    }
    const bf16* oct = reinterpret_cast<const bf16*>(B + Cfg::OFF_V) + (4 * b + g) * OCT_ELEMS;
    // all of the pair's A operands are read before its products, so that the
    // products wait for the LDS once
    bf16x8 a[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) a[dt] = *reinterpret_cast<const bf16x8*>(oct + 8 * (16 * dt + c));
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int s = 0; s < QS; ++s) X[dt][s] = mfma_bf16(a[dt], bw[s], X[dt][s]);
  };
  // fp32: the r-th product of tile tt takes row r of the lane's half octet
  // as k-slot g
  auto accumulate_f = [&](const unsigned char* B, int tt, const f32x4 (&w0)[QS]) {
    const float* oct = reinterpret_cast<const float*>(B + Cfg::OFF_V) +
                       (4 * (tt / 2) + g) * OCT_ELEMS + 4 * (tt % 2);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const float4 a = *reinterpret_cast<const float4*>(oct + 8 * (16 * dt + c));
#pragma unroll
      for (int s = 0; s < QS; ++s) {
        X[dt][s] = mfma_f32(a.x, w0[s][0], X[dt][s]);
        X[dt][s] = mfma_f32(a.y, w0[s][1], X[dt][s]);
        X[dt][s] = mfma_f32(a.z, w0[s][2], X[dt][s]);
        X[dt][s] = mfma_f32(a.w, w0[s][3], X[dt][s]);
      }
    }
  };
  auto accumulate_pair = [&](const unsigned char* B, int b, const f32x4 (&W)[2][QS]) {
    if constexpr (kB) {
      accumulate_b(B, b, W[0], W[1]);
    } else {
      accumulate_f(B, 2 * b, W[0]);
      accumulate_f(B, 2 * b + 1, W[1]);
    }
  };
  // The value product of tile pair b in two steps, so that its A operands
  // (bf16: octet 4 b + g at the lane's columns) are read from LDS before the
  // weights they multiply are computed, and their latency is hidden by that
  // work. bf16 at d = 128 only: at d = 64 the three waves per SIMD leave no
  // registers for them (they are read where they are used), as for fp32.
  constexpr bool kValAhead = kB && D == 128;
  struct ValOps {
    bf16x8 a[kValAhead ? DT : 1];
  };
  auto load_vals = [&](const unsigned char* B, int b) {
    ValOps v;
    if constexpr (kValAhead) {
      const bf16* oct = reinterpret_cast<const bf16*>(B + Cfg::OFF_V) + (4 * b + g) * OCT_ELEMS;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) v.a[dt] = *reinterpret_cast<const bf16x8*>(oct + 8 * (16 * dt + c));
    }
    return v;
  };
  auto mfma_vals = [&](const unsigned char* B, int b, const ValOps& v, const f32x4 (&W)[2][QS]) {
    if constexpr (kValAhead) {
      bf16x8 bw[QS];
#pragma unroll
      for (int s = 0; s < QS; ++s)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          bw[s][r] = (bf16)W[0][s][r];
          bw[s][4 + r] = (bf16)W[1][s][r];
        }
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int s = 0; s < QS; ++s) X[dt][s] = mfma_bf16(v.a[dt], bw[s], X[dt][s]);
    } else {
      accumulate_pair(B, b, W);
    }
  };

  // Per-lane softmax state for query columns c + 16 s: m is the running max
  // in log2 units (lagging by at most kLazy), thr the raw logit (natural
  // units) that would pass m + kLazy, zp this lane group's partial fp32 sum of
  // the weights (the parents' alone for importance, then the denominator).
  float m[QS], thr[QS], zp[QS];
#pragma unroll
  for (int s = 0; s < QS; ++s) {
    m[s] = kMaxFloor;
    thr[s] = (kMaxFloor + kLazy) * kLn2;
    zp[s] = 0.f;
  }
  // Raises the running max if some lane's logit in the chunk (both tile pairs)
  // passed the threshold, rescaling the accumulators (rare: the max lags by
  // up to kLazy). One check per chunk keeps the weights and value products of
  // the chunk in one basic block, where the compiler interleaves the second
  // pair's exponentials with the first pair's MFMAs.
  auto check_chunk = [&](const f32x4 (&S0)[2][QS], const f32x4 (&S1)[2][QS]) {
    float mx[QS];
    bool over = false;
#pragma unroll
    for (int s = 0; s < QS; ++s) {
      // a running three-way max: two new values per instruction
      mx[s] = S0[0][s][0];
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
        for (int r = 0; r < 4; ++r) mx[s] = fmaxf(fmaxf(mx[s], S0[h2][s][r]), S1[h2][s][r]);
      over |= mx[s] > thr[s];
    }
    if (__ballot(over) == 0) return;
#pragma unroll
    for (int s = 0; s < QS; ++s) {
      mx[s] = max_xor<32>(max_xor<16>(mx[s]));
      const float mnew = mx[s] > thr[s] ? mx[s] * kLog2e : m[s];
      const float scs = exp2_hw(m[s] - mnew);
      zp[s] *= scs;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) X[dt][s] *= scs;
      m[s] = mnew;
      thr[s] = (mnew + kLazy) * kLn2;
    }
  };
  // parent weights n exp(S - m) = exp2((S + ln n) log2 e - m), in place
  auto parent_weights = [&](f32x4 (&S)[2][QS]) {
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
      for (int s = 0; s < QS; ++s)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float w = exp2_hw(fmaf(S[h2][s][r], kLog2e, -m[s]));
          S[h2][s][r] = w;
          zp[s] += w;
        }
  };
  // Recovered parent logit (Eq. (parent_recovery)) from the raw child logits
  // of tile pair b: the sum over all Ch children of the parent, empty ones
  // included (divided by Ch where it is used). Over the octet rows: Ch = 2:
  // rows 0-1 of the even tile (the rest is padding); Ch = 4: the 4 rows of
  // each tile (one parent per tile); Ch = 8: the whole octet; Ch = 16: and the
  // partner lane group's octet.
  // 0/1 weights of the recovered-logit cases (exact products and sums)
  const float w2 = Ch == 2 ? 1.f : 0.f, w4 = Ch == 4 ? 1.f : 0.f, w8 = Ch == 8 ? 1.f : 0.f,
              w16 = Ch == 16 ? 1.f : 0.f;
  auto child_recover = [&](const f32x4 (&S)[2][QS], float (&rs)[2][QS]) {
#pragma unroll
    for (int s = 0; s < QS; ++s) {
      // every case computed and one kept by 0/1 weights: no branch splits
      // the chunk's weights from its value products
      const f32x4 v0 = S[0][s], v1 = S[1][s];
      const float a01 = v0[0] + v0[1];
      const float a = a01 + (v0[2] + v0[3]);
      const float bs = (v1[0] + v1[1]) + (v1[2] + v1[3]);
      const float ab = a + bs;
      const float ab16 = add_xor<16>(ab);
      rs[0][s] = fmaf(w2, a01, fmaf(w4, a, fmaf(w8, ab, w16 * ab16)));
      rs[1][s] = fmaf(w2, a01, fmaf(w4, bs, fmaf(w8, ab, w16 * ab16)));
    }
  };
  // Ch = 8: the lane's octet is the whole family, so the recovered sum is the
  // sum of the lane's 8 values (the case child_recover keeps for Ch = 8,
  // without the other cases' arithmetic)
  auto child_recover8 = [&](const f32x4 (&S)[2][QS], float (&rs)[2][QS]) {
#pragma unroll
    for (int s = 0; s < QS; ++s) {
      const f32x4 v0 = S[0][s], v1 = S[1][s];
      const float ab = ((v0[0] + v0[1]) + (v0[2] + v0[3])) + ((v1[0] + v1[1]) + (v1[2] + v1[3]));
      rs[0][s] = ab;
      rs[1][s] = ab;
    }
  };
  // log-count bias of the child logits of tile pair b, in place: T + ln n,
  // -inf for empty children and padding rows (App. D: the running max is
  // taken over non-empty codes only)
  auto child_bias = [&](const unsigned char* B, int b, f32x4 (&S)[2][QS]) {
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
      const f32x4 l4 = info4(B, 2 * b + h2, 1);
#pragma unroll
      for (int s = 0; s < QS; ++s)
#pragma unroll
        for (int r = 0; r < 4; ++r) S[h2][s][r] += l4[r];
    }
  };
  // correcting weights exp(T + ln n - m) - n exp(Srec - m) of tile pair b
  // (biased logits in S, recovered sums in rs), in place. Empty children and
  // padding: exp2(-inf) = 0 and n = 0, so the weight is exactly 0; the
  // recovered term is clamped below 2^64, so 0 times it stays 0.
  // (full chunks only, Ch = 8 or 16: both tiles of the pair belong to one
  // parent, whose recovered sums rs[0] and rs[1] are equal, so its term is
  // computed once)
  auto child_weights = [&](const unsigned char* B, int b, f32x4 (&S)[2][QS],
                           const float (&rs)[2][QS]) {
    const float scale = kLog2e / (float)Ch;
    float er[QS];
#pragma unroll
    for (int s = 0; s < QS; ++s) er[s] = exp2_hw(fminf(fmaf(rs[0][s], scale, -m[s]), 64.f));
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
      const f32x4 n4 = info4(B, 2 * b + h2, 0);
#pragma unroll
      for (int s = 0; s < QS; ++s) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float w = fmaf(-n4[r], er[s], exp2_hw(fmaf(S[h2][s][r], kLog2e, -m[s])));
          S[h2][s][r] = w;
          zp[s] += w;
        }
      }
    }
  };
  // logits of the chunk's two tile pairs; parents start from ln n
  // (bf16: the A fragments of tile tt + 1 are read from LDS while the
  // products of tile tt run; scheduling barriers keep that order). qrows:
  // the tiles are S, queries as the D rows (see logits), each lane's column
  // starting from its codeword's ln n.
  auto chunk_logits = [&](const unsigned char* B, bool with_ln, f32x4 (&S0)[2][QS],
                          f32x4 (&S1)[2][QS], bool qrows = false) {
    const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
    f32x4 init[TPC];
#pragma unroll
    for (int tt = 0; tt < TPC; ++tt) {
      if (qrows) {
        const float* li = reinterpret_cast<const float*>(B + Cfg::OFF_I);
        const float l = li[(4 * (tt / 2) + c / 4) * 16 + 8 + 4 * (tt % 2) + c % 4];
        init[tt] = f32x4{l, l, l, l};
      } else {
        init[tt] = with_ln ? info4(B, tt, 1) : zero;
      }
    }
    if constexpr (kB) {
      const T* lc = reinterpret_cast<const T*>(B + Cfg::OFF_C);
      bf16x8 a[2][KQ];
      auto load_tile = [&](int tt, bf16x8 (&dst)[KQ]) {
        const int r = 32 * (tt / 2) + 8 * (c / 4) + 4 * (tt % 2) + (c % 4);
        const int sw = row_swizzle<U>(r);
#pragma unroll
        for (int kq = 0; kq < KQ; ++kq)
          dst[kq] = *reinterpret_cast<const bf16x8*>(&lc[r * D + ((4 * kq + g) ^ sw) * EPU]);
      };
      load_tile(0, a[0]);
#pragma unroll
      for (int tt = 0; tt < TPC; ++tt) {
        if (tt + 1 < TPC) load_tile(tt + 1, a[(tt + 1) % 2]);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int kq = 0; kq < KQ; ++kq)
#pragma unroll
          for (int s = 0; s < QS; ++s) {
            f32x4& o = tt < 2 ? S0[tt][s] : S1[tt - 2][s];
            o = qrows ? mfma_bf16(qf[s][kq], a[tt % 2][kq], kq == 0 ? init[tt] : o)
                      : mfma_bf16(a[tt % 2][kq], qf[s][kq], kq == 0 ? init[tt] : o);
          }
        __builtin_amdgcn_sched_barrier(0);
      }
    } else {
      logits(B, 0, S0[0], init[0], qrows);
      logits(B, 1, S0[1], init[1], qrows);
      logits(B, 2, S1[0], init[2], qrows);
      logits(B, 3, S1[1], init[3], qrows);
    }
  };

  // Child chunk with Ch <= 4: rows 4..7 of every octet are padding, so logit
  // tiles 1 and 3 (those rows) are never formed, and the valid halves of the
  // chunk's two pairs share one value product: k-slots 0..3 of lane group g
  // are codes 0..3 of octet g (pair 0), k-slots 4..7 codes 0..3 of octet
  // 4 + g (pair 1). Half the MFMAs and exponentials of a full chunk.
  auto child_chunk_half = [&](const unsigned char* B) {
    f32x4 S0[2][QS], S1[2][QS];
    const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
    const float ninf = -__builtin_inff();
    const f32x4 pad = {ninf, ninf, ninf, ninf};
    if constexpr (kB) {
      const T* lc = reinterpret_cast<const T*>(B + Cfg::OFF_C);
      bf16x8 a[2][KQ];
#pragma unroll
      for (int h = 0; h < 2; ++h) {  // tiles 0 and 2
        const int r = 32 * h + 8 * (c / 4) + (c % 4);
        const int sw = row_swizzle<U>(r);
#pragma unroll
        for (int kq = 0; kq < KQ; ++kq)
          a[h][kq] = *reinterpret_cast<const bf16x8*>(&lc[r * D + ((4 * kq + g) ^ sw) * EPU]);
      }
#pragma unroll
      for (int kq = 0; kq < KQ; ++kq)
#pragma unroll
        for (int s = 0; s < QS; ++s) {
          S0[0][s] = mfma_bf16(a[0][kq], qf[s][kq], kq == 0 ? zero : S0[0][s]);
          S1[0][s] = mfma_bf16(a[1][kq], qf[s][kq], kq == 0 ? zero : S1[0][s]);
        }
    } else {
      logits(B, 0, S0[0], zero, false);
      logits(B, 2, S1[0], zero, false);
    }
    // the recovered sums (Ch = 2, 4: only the even tile's rows enter; the odd
    // tile is zero here, as 0 * inf would poison the unused cases), then the
    // odd tiles as -inf: no part in the max
#pragma unroll
    for (int s = 0; s < QS; ++s) {
      S0[1][s] = zero;
      S1[1][s] = zero;
    }
    float rs0[2][QS], rs1[2][QS];
    child_recover(S0, rs0);
    child_recover(S1, rs1);
#pragma unroll
    for (int s = 0; s < QS; ++s) {
      S0[1][s] = pad;
      S1[1][s] = pad;
    }
#pragma unroll
    for (int s = 0; s < QS; ++s) {  // log-count bias of the valid rows
      const f32x4 l0 = info4(B, 0, 1), l2 = info4(B, 2, 1);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        S0[0][s][r] += l0[r];
        S1[0][s][r] += l2[r];
      }
    }
    check_chunk(S0, S1);
    // correcting weights of the valid rows, as child_weights
    const float scale = kLog2e / (float)Ch;
    const f32x4 n0 = info4(B, 0, 0), n2 = info4(B, 2, 0);
#pragma unroll
    for (int s = 0; s < QS; ++s) {
      const float e0 = exp2_hw(fminf(fmaf(rs0[0][s], scale, -m[s]), 64.f));
      const float e1 = exp2_hw(fminf(fmaf(rs1[0][s], scale, -m[s]), 64.f));
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float w0 = fmaf(-n0[r], e0, exp2_hw(fmaf(S0[0][s][r], kLog2e, -m[s])));
        const float w1 = fmaf(-n2[r], e1, exp2_hw(fmaf(S1[0][s][r], kLog2e, -m[s])));
        S0[0][s][r] = w0;
        S1[0][s][r] = w1;
        zp[s] += w0 + w1;
      }
    }
    if constexpr (kB) {
      bf16x8 bw[QS];
#pragma unroll
      for (int s = 0; s < QS; ++s)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          bw[s][r] = (bf16)S0[0][s][r];
          bw[s][4 + r] = (bf16)S1[0][s][r];
        }
      const bf16* o0 = reinterpret_cast<const bf16*>(B + Cfg::OFF_V) + g * OCT_ELEMS;
      const bf16* o1 = reinterpret_cast<const bf16*>(B + Cfg::OFF_V) + (4 + g) * OCT_ELEMS;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const bf16x4 lo = *reinterpret_cast<const bf16x4*>(o0 + 8 * (16 * dt + c));
        const bf16x4 hi = *reinterpret_cast<const bf16x4*>(o1 + 8 * (16 * dt + c));
        const bf16x8 a = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
#pragma unroll
        for (int s = 0; s < QS; ++s) X[dt][s] = mfma_bf16(a, bw[s], X[dt][s]);
      }
    } else {
      accumulate_f(B, 0, S0[0]);
      accumulate_f(B, 2, S1[0]);
    }
  };

  const bool need_importance =
      (P > 0 && P < M0) || args.importance != nullptr || (P > 0 && args.topp_idx != nullptr);
  const int n_pchunks = PO / 8;
  // importance: u_a = sum over this wave's queries of p_ia for the chunk in W
  // (already normalised): first over the query subtiles in registers, then
  // over the 16 query columns by a reduce-scatter butterfly over lane bits 3,
  // 0, 1, 2 that leaves lane c with value k = 8 b3 + 4 b0 + 2 b1 + b2 of its
  // lane group, value k being row r = k % 4 of tile tt = k / 4.
  auto importance_partials = [&](const f32x4 (&W0)[2][QS], const f32x4 (&W1)[2][QS],
                                 const float (&mul)[QS], int slot) {
    float u[16];
#pragma unroll
    for (int tt = 0; tt < TPC; ++tt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        // the first product starts the sum (a sum from 0.0 keeps an add of
        // zero per value: x + 0 is not x for x = -0)
        float acc = (tt < 2 ? W0[tt][0][r] : W1[tt - 2][0][r]) * mul[0];
#pragma unroll
        for (int s = 1; s < QS; ++s)
          acc = fmaf(tt < 2 ? W0[tt][s][r] : W1[tt - 2][s][r], mul[s], acc);
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
    const int tt = k / 4, r = k % 4;
    lw[(slot * MAXW + wave) * CW + 32 * (tt / 2) + 8 * g + 4 * (tt % 2) + r] = u[0];
  };
  // The same from the importance sweep's S tiles (chunk_logits with qrows):
  // normalised weights exp2(S log2 e - mz) with the shift of query
  // 16 s + 4 g + r in mzq[s][r]; each lane sums its 8 queries of a tile, then
  // the four lane groups are reduced by two 32-lane and one 16-lane row swap,
  // which leave lane group g with the sum of tile g.
  auto importance_qrows = [&](const f32x4 (&S0)[2][QS], const f32x4 (&S1)[2][QS],
                              const float (&mzq)[QS][4], int slot) {
    float u[TPC];
#pragma unroll
    for (int tt = 0; tt < TPC; ++tt) {
      float p[QS][4];
#pragma unroll
      for (int s = 0; s < QS; ++s)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          p[s][r] = exp2_hw(fmaf(tt < 2 ? S0[tt][s][r] : S1[tt - 2][s][r], kLog2e, -mzq[s][r]));
      float acc = (p[0][0] + p[0][1]) + (p[0][2] + p[0][3]);
#pragma unroll
      for (int s = 1; s < QS; ++s) acc += (p[s][0] + p[s][1]) + (p[s][2] + p[s][3]);
      u[tt] = acc;
    }
    // rows of 32 lanes: (u0, u2) -> lanes 0-31 hold u0 summed over groups
    // g and g + 2, lanes 32-63 u2; likewise (u1, u3); then rows of 16
    // (v_permlane32_swap / v_permlane16_swap: the odd rows of x trade places
    // with the even rows of y; the sum of the two results adds row pairs)
    auto swap_add = [](float x, float y, auto rows32_tag) {
      const unsigned ux = __float_as_uint(x), uy = __float_as_uint(y);
      if constexpr (decltype(rows32_tag)::value) {
        const auto xy = __builtin_amdgcn_permlane32_swap(ux, uy, false, false);
        return __uint_as_float(xy[0]) + __uint_as_float(xy[1]);
      } else {
        const auto xy = __builtin_amdgcn_permlane16_swap(ux, uy, false, false);
        return __uint_as_float(xy[0]) + __uint_as_float(xy[1]);
      }
    };
    const float a = swap_add(u[0], u[2], std::true_type{});
    const float b = swap_add(u[1], u[3], std::true_type{});
    const float tot = swap_add(a, b, std::false_type{});
    lw[(slot * MAXW + wave) * CW + 32 * (g / 2) + 8 * (c / 4) + 4 * (g % 2) + c % 4] = tot;
  };
  // sum the wave partials of chunk k (slot k % 2) in a fixed order
  auto importance_flush = [&](int k) {
    if (tid < CW) {
      const int a = CW * k + tid;
      float acc = 0.f;
      for (int wv = 0; wv < n_active; ++wv) acc += lw[((k % 2) * MAXW + wv) * CW + tid];
      if (a < M0) {
        lwf[a] = acc;
        if (args.importance) args.importance[((size_t)bh * args.n_tiles + t) * M0 + a] = acc;
      }
    }
  };
  // per-query log2 shift that turns exp2(t - m) into exp2(t - m) / Z
  float mz[QS];
  auto set_mz = [&]() {
#pragma unroll
    for (int s = 0; s < QS; ++s) {
      float z = zp[s];
      z = add_xor<32>(add_xor<16>(z));
      mz[s] = qvalid[s] ? m[s] + log2_hw(z) : __builtin_inff();
    }
  };

  // App. B: keys seen so far (the counts of the parents of the chunks up to
  // the current one), the same in every lane
  const bool tiled_importance = TILED && need_importance && n_pchunks > 1;
  float seen = 0.f;
  auto tiled_partials = [&](const unsigned char* B, const f32x4 (&W0)[2][QS],
                            const f32x4 (&W1)[2][QS], int k) {
    // this lane group's 16 rows of the chunk, then the other three groups'
    float cnt = 0.f;
#pragma unroll
    for (int tt = 0; tt < TPC; ++tt) {
      const f32x4 n4 = info4(B, tt, 0);
      cnt += (n4[0] + n4[1]) + (n4[2] + n4[3]);
    }
    cnt = add_xor<32>(add_xor<16>(cnt));
    seen += cnt;  // integers below 2^24: exact
    // weight / Ztilde = W * seen / (N * Z), W and Z relative to the same max
    float mul[QS];
#pragma unroll
    for (int s = 0; s < QS; ++s) {
      float z = zp[s];
      z = add_xor<32>(add_xor<16>(z));
      mul[s] = (qvalid[s] && seen > 0.f) ? seen / ((float)N * z) : 0.f;
    }
    importance_partials(W0, W1, mul, k % 2);
  };

  // ---- phase 1: parent sweep -------------------------------------------------
  // Per chunk: the logits of both tile pairs are issued first, then one max
  // check; the first pair's value MFMAs run while the second pair's weights
  // are computed.
  issue_parent(0, 0, true);
  for (int k = 0; k < n_pchunks; ++k) {
    wait_chunk();
    if (tiled_importance && k > 0) importance_flush(k - 1);
    if (Cfg::NBUF == 2 && k + 1 < n_pchunks) issue_parent(k + 1, (k + 1) % 2, true);
    const unsigned char* B = buffer(k % Cfg::NBUF);
    if (has_rows) {
      f32x4 S0[2][QS], S1[2][QS];
      chunk_logits(B, true, S0, S1);
      const ValOps v0 = load_vals(B, 0);  // in flight during the max check and weights
      __builtin_amdgcn_sched_barrier(0);
      check_chunk(S0, S1);
      parent_weights(S0);
      mfma_vals(B, 0, v0, S0);
      const ValOps v1 = load_vals(B, 1);
      parent_weights(S1);
      mfma_vals(B, 1, v1, S1);
      // the last chunk: max and denominators are final, so its normalised
      // weights are its weights times 1/Z (the other chunks' importance comes
      // from the second sweep)
      if (k == n_pchunks - 1 && need_importance && !tiled_importance) {
        set_mz();
        float rz[QS];
#pragma unroll
        for (int s = 0; s < QS; ++s) rz[s] = exp2_hw(m[s] - mz[s]);
        importance_partials(S0, S1, rz, k % 2);
      }
      if (tiled_importance) tiled_partials(B, S0, S1, k);
    }
    if (Cfg::NBUF == 1 && k + 1 < n_pchunks) {
      __syncthreads();
      issue_parent(k + 1, 0, true);
    }
  }

  // ---- phase 2: importance with the final max and denominators ---------------
  if (need_importance) {
    if (n_pchunks == 1 || TILED) {
      __syncthreads();
      importance_flush(n_pchunks - 1);
    } else {
      // chunks 0 .. n_pchunks - 2 again; the last one's partials (slot
      // (n_pchunks - 1) % 2) are summed before the sweep writes any slot
      const int n_sweep = n_pchunks - 1;
      // the shift of query 16 s + 4 g + r, from the lane that holds it
      float mzq[QS][4];
      if (has_rows) {
#pragma unroll
        for (int s = 0; s < QS; ++s)
#pragma unroll
          for (int r = 0; r < 4; ++r) mzq[s][r] = __shfl(mz[s], 4 * g + r, kWave);
      }
      __syncthreads();
      importance_flush(n_pchunks - 1);
      issue_parent(0, 0, false);
      for (int k = 0; k < n_sweep; ++k) {
        wait_chunk();
        if (k > 0) importance_flush(k - 1);
        if (Cfg::NBUF == 2 && k + 1 < n_sweep) issue_parent(k + 1, (k + 1) % 2, false);
        const unsigned char* B = buffer(k % Cfg::NBUF);
        if (has_rows) {
          f32x4 S0[2][QS], S1[2][QS];
          chunk_logits(B, true, S0, S1, true);
          importance_qrows(S0, S1, mzq, k % 2);
        }
        if (Cfg::NBUF == 1 && k + 1 < n_sweep) {
          __syncthreads();
          issue_parent(k + 1, 0, false);
        }
      }
      __syncthreads();
      importance_flush(n_sweep - 1);
    }
  }
  __syncthreads();

  // ---- phase 3: top-P (w desc, index asc) -------------------------------------
  // One wave. Lane l holds the keys of parents 64 i + l: the importance bits
  // plus one (importance is a non-negative float, so the integer order is the
  // value order; padding gets 0, below every parent). A threshold kp is built
  // bit by bit from the top, the largest with at least P keys >= kp (the P-th
  // largest key), or the first with exactly P; every key above kp is
  // selected, and of the keys equal to kp the lowest indices, as many as are
  // still missing. The selected parents are listed in index order. With
  // P >= M0 every parent is selected (all keys 1).
  if (P > 0) {
    // NV key registers per lane: the fewest that hold M0 parents
    auto select_top = [&](auto nv_tag) {
      constexpr int NV = decltype(nv_tag)::value;
      unsigned key[NV];
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const int a = kWave * i + lane;
        const unsigned kv = P < M0 ? __float_as_uint(lwf[a < M0 ? a : 0]) + 1u : 1u;
        key[i] = a < M0 ? kv : 0u;
      }
      auto count_ge = [&](unsigned v) {
        int n = 0;
#pragma unroll
        for (int i = 0; i < NV; ++i) n += __popcll(__ballot(key[i] >= v));
        return n;
      };
      unsigned kp = 0u;
      for (int bit = 30; bit >= 0; --bit) {  // keys stay below 2^31
        const unsigned cand = kp | (1u << bit);
        const int cnt = count_ge(cand);
        if (cnt >= P) {
          kp = cand;
          if (cnt == P) break;
        }
      }
      const int need = P - count_ge(kp + 1u);  // keys equal to kp still to take
      const unsigned long long below = (1ull << lane) - 1ull;
      int eq_before = 0, filled = 0;
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const bool eq = key[i] == kp;
        const unsigned long long me = __ballot(eq);
        const bool sel = key[i] > kp || (eq && eq_before + __popcll(me & below) < need);
        eq_before += __popcll(me);
        const unsigned long long ms = __ballot(sel);
        if (sel) lsel[filled + __popcll(ms & below)] = kWave * i + lane;
        filled += __popcll(ms);
      }
    };
    if (wave == 0) {
      if (M0 <= 2 * kWave) select_top(std::integral_constant<int, 2>{});
      else if (M0 <= 4 * kWave) select_top(std::integral_constant<int, 4>{});
      else select_top(std::integral_constant<int, Cfg::M0MAX / kWave>{});
    }
    __syncthreads();
    if (args.topp_idx) {  // canonical order (w desc, index asc) for the caller
      for (int q = tid; q < P; q += blockDim.x) {
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
    // The selected parents' child octets, 8 per chunk. With one child the
    // recovered parent logit is that child's own logit, so every correcting
    // weight is exactly zero: nothing to do.
    const int n_cchunks = (n_child_oct + 7) / 8;
    if (n_cchunks > 0) issue_child(0, 0);
    for (int k = 0; k < n_cchunks; ++k) {
      wait_chunk();
      if (Cfg::NBUF == 2 && k + 1 < n_cchunks) issue_child(k + 1, (k + 1) % 2);
      const unsigned char* B = buffer(k % Cfg::NBUF);
      if (has_rows && half_child) {
        child_chunk_half(B);
      } else if (has_rows) {
        f32x4 S0[2][QS], S1[2][QS];
        float rs0[2][QS], rs1[2][QS];
        chunk_logits(B, false, S0, S1);
        const ValOps v0 = load_vals(B, 0);  // in flight during the recovery, bias and weights
        __builtin_amdgcn_sched_barrier(0);
        if (Ch == 8) {
          child_recover8(S0, rs0);
          child_recover8(S1, rs1);
        } else {
          child_recover(S0, rs0);
          child_recover(S1, rs1);
        }
        child_bias(B, 0, S0);
        child_bias(B, 1, S1);
        check_chunk(S0, S1);
        child_weights(B, 0, S0, rs0);
        mfma_vals(B, 0, v0, S0);
        const ValOps v1 = load_vals(B, 1);
        child_weights(B, 1, S1, rs1);
        mfma_vals(B, 1, v1, S1);
      }
      if (Cfg::NBUF == 1 && k + 1 < n_cchunks) {  // one buffer: refill it when all are done
        __syncthreads();
        issue_child(k + 1, 0);
      }
    }
  }

  // ---- phase 5: Y = Xbar / Z (Z: the lane groups' partial sums) --------------
  // Each wave stages its 32 rows in LDS (the chunk buffers are free by now)
  // and stores them as whole rows: 16 bytes per lane, a row's 16-byte units
  // on consecutive lanes, instead of the fragments' 8-byte pieces of 16 rows
  // per store instruction. The units of a staged row are XOR-swizzled by
  // row, so the 16 rows a fragment write touches hit different banks.
  float rinv[QS];
#pragma unroll
  for (int s = 0; s < QS; ++s) {
    float z = zp[s];
    z = add_xor<32>(add_xor<16>(z));
    rinv[s] = 1.f / z;
  }
  constexpr int YROW = D * Cfg::ESZ;         // bytes of one Y row
  constexpr int YU = YROW / 16;              // 16-byte units per row
  constexpr int RPB = YROW >= 256 ? 1 : 256 / YROW;  // rows per 256 bytes of banks
  constexpr bool kStageY = (size_t)MAXW * Cfg::RPW * YROW <= (size_t)Cfg::NBUF * Cfg::BUF_BYTES;
  auto yswz = [](int r) { return (r / RPB) % YU; };
  if constexpr (kStageY) {
    __syncthreads();  // every wave is done with the chunk buffers
    unsigned char* ys = lds_raw + (size_t)wave * Cfg::RPW * YROW;  // this wave's rows
#pragma unroll
    for (int s = 0; s < QS; ++s) {
      const int r = 16 * s + c;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const f32x4 y = X[dt][s] * rinv[s];
        const int byte = (16 * dt + 4 * g) * Cfg::ESZ;  // of the lane's 4 values in the row
        unsigned char* dst = ys + r * YROW + (((byte / 16) ^ yswz(r)) * 16) + byte % 16;
        if constexpr (kB) {
          bf16x4 o = {(bf16)y[0], (bf16)y[1], (bf16)y[2], (bf16)y[3]};
          *reinterpret_cast<bf16x4*>(dst) = o;
        } else {
          *reinterpret_cast<f32x4*>(dst) = y;
        }
      }
    }
    // the wave reads back only what it wrote: LDS operations of one wave
    // complete in order
    constexpr int RPI = 64 / YU;  // rows per instruction
    const int u = lane % YU;
#pragma unroll
    for (int i = 0; i < Cfg::RPW / RPI; ++i) {
      const int r = RPI * i + lane / YU;
      const uint4 v = *reinterpret_cast<const uint4*>(ys + r * YROW + ((u ^ yswz(r)) * 16));
      const int q = row0 + r;
      const int tok = q < q_end ? token_row(q) : -1;
      if (tok >= 0)
        *reinterpret_cast<uint4*>(static_cast<unsigned char*>(args.Y) +
                                  ((size_t)bh * N + tok) * YROW + u * 16) = v;
    }
  } else {
#pragma unroll
    for (int s = 0; s < QS; ++s) {
      if (!qvalid[s]) continue;
      const int i = token_row(row0 + 16 * s + c);
      T* yrow = static_cast<T*>(args.Y) + ((size_t)bh * N + i) * D;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const f32x4 y = X[dt][s] * rinv[s];
        if constexpr (kB) {
          bf16x4 o = {(bf16)y[0], (bf16)y[1], (bf16)y[2], (bf16)y[3]};
          *reinterpret_cast<bf16x4*>(yrow + 16 * dt + 4 * g) = o;
        } else {
          *reinterpret_cast<f32x4*>(yrow + 16 * dt + 4 * g) = y;
        }
      }
    }
  }
}

template <typename T, int D, int MAXW, bool TILED>
hipError_t launch_attention_cfg(const AttnArgs& a, int BH, hipStream_t stream) {
  const long long grid = (long long)BH * a.n_tiles;
  if (grid > 0x7fffffff) return hipErrorInvalidConfiguration;
  using Cfg = AttnCfg<T, D, MAXW>;
  constexpr int slot = (TILED ? 48 : 8) + (Elem<T>::kBf16 ? 0 : 4) + (D == 128 ? 2 : 0) +
                       (MAXW == 8 ? 1 : 0);
  hipError_t e = ensure_dynamic_lds((const void*)attention_kernel<T, D, MAXW, TILED>,
                                    (int)Cfg::LDS_BYTES, slot);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attention_kernel<T, D, MAXW, TILED>), dim3((unsigned)grid),
                     dim3(MAXW * 64), Cfg::LDS_BYTES, stream, a);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_attention(int BH, int H, int N, int M0, int Ch, int P, int block_q,
                            const void* Q, const void* Cp, const void* Cc, const void* packed,
                            void* Y, int32_t* topp_idx, float* importance, bool tiled,
                            const int32_t* order, hipStream_t stream) {
  AttnArgs a;
  a.Q = Q;
  a.Cp = Cp;
  a.Cc = Cc;
  a.packed = static_cast<const unsigned char*>(packed);
  a.Y = Y;
  a.topp_idx = topp_idx;
  a.importance = importance;
  a.order = order;
  a.H = H;
  a.N = N;
  a.M0 = M0;
  a.Ch = Ch;
  a.P = P;
  a.block_q = block_q;
  a.n_tiles = (N + block_q - 1) / block_q;
  if (tiled) {
    if (block_q <= 128) return launch_attention_cfg<T, D, 4, true>(a, BH, stream);
    return launch_attention_cfg<T, D, 8, true>(a, BH, stream);
  }
  if (block_q <= 128) return launch_attention_cfg<T, D, 4, false>(a, BH, stream);
  return launch_attention_cfg<T, D, 8, false>(a, BH, stream);
}

#define AVQ_INSTANTIATE(T, D)                                                                \
  template hipError_t launch_attention<T, D>(int, int, int, int, int, int, int, const void*, \
                                             const void*, const void*, const void*, void*,   \
                                             int32_t*, float*, bool, const int32_t*,     \
                                             hipStream_t);
AVQ_INSTANTIATE(bf16, 64)
AVQ_INSTANTIATE(bf16, 128)
AVQ_INSTANTIATE(float, 64)
AVQ_INSTANTIATE(float, 128)
#undef AVQ_INSTANTIATE

}  // namespace avq
