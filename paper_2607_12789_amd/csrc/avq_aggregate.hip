// Per-codeword counts and value sums, Eq. (aggregates), with the Alg. 1
// convention that a parent row covers its whole cell and a child row the keys
// that moved to it.
//
// One workgroup owns one (batch, head) and a range of 32 parent families (a
// family = parent p and its Ch children); each half wave (32 lanes) owns one
// family and is the only writer of its rows, so no float atomics are needed
// (LDS float atomics serialise on gfx950; integer ones do not). The
// workgroup
//   1. scans the codes of every key of the head (the next round's codes are
//      prefetched while the current one is queued) and appends the keys whose
//      parent is in its range to an LDS queue, in key order (wave ballot +
//      prefix counts);
//   2. when the queue is full or the codes are exhausted, buckets the queued
//      keys by their row (stay row of the parent, or one of its children) with
//      integer LDS atomics: histogram, prefix sum, scatter;
//   3. lets each half wave walk its family's keys in bucket order through a
//      ring of 8 value rows (4 for Ch = 16) in flight, whatever rows they
//      belong to, each slot refilled as soon as its row is added (lane l
//      holds columns l*CPL .. l*CPL+CPL-1), summing in fp32 into a running
//      row sum that is added to the family's register table when the row
//      ends.
// At the end the parent row is the stay row plus the children (the whole
// cell), every row is written once, and counts come from the histograms.
// Optionally the packed aggregates are also written (avq_packed.hpp): the
// mean value (sum / count) of every code rounded to the input type, in octets
// of 8 codes laid out as the attention kernel's MFMA operands, [octet][d][8],
// with n and ln n per code.
#include "avq_child.hpp"
#include "avq_common.hpp"
#include "avq_launch.hpp"
#include "avq_packed.hpp"

namespace avq {

constexpr int kAggThreads = 1024;
constexpr int kAggWaves = kAggThreads / kWave;
constexpr int kFamLanes = 32;                          // lanes per family
constexpr int kFamilies = kAggThreads / kFamLanes;     // half waves = most families per workgroup
constexpr int kCodesPerThread = 8;                     // codes scanned per thread per round
constexpr int kRound = kAggThreads * kCodesPerThread;
constexpr int kQueueCap = 8192;                        // queued keys per flush
constexpr int kMaxRows = kFamilies * 17;               // families x (1 + Ch), Ch <= 16
// value rows in flight per family: as many as the registers beside the
// family table (1 + CHM rows of D / 32 sums per lane) allow
template <int CHM, typename T>
constexpr int kInFlight = CHM > 8 ? 4 : (CHM == 0 && sizeof(T) == 2) ? 16 : 8;

struct AggLds {
  int qkey[kQueueCap];       // queued keys, key order
  uint16_t qrow[kQueueCap];  // their family-local row
  int skey[kQueueCap];       // keys bucketed by row
  int hist[kMaxRows];        // keys per row in this flush
  int start[kMaxRows + 1];   // bucket starts
  int cursor[kMaxRows];      // scatter cursors
  int total[kMaxRows];       // keys per row over all flushes (the counts)
  int fstart[kFamilies + 1];      // fused: family buckets of the queue
  int fcursor[kFamilies];
  int item_start[kFamilies + 1];  // fused: first group of 16 keys of each family
  int wave_count[kCodesPerThread][kAggWaves];  // queued keys per (round slot, wave)
  int wave_off[kCodesPerThread][kAggWaves];    // their queue offsets in this round
  int round_total;
};
static_assert(kCodesPerThread * kAggWaves <= 128, "one wave scans the slot offsets");

// CPL values of type T as one load: 4, 8 or 16 bytes
template <int BYTES>
struct Chunk;
template <>
struct Chunk<4> {
  typedef uint32_t type;
};
template <>
struct Chunk<8> {
  typedef uint2 type;
};
template <>
struct Chunk<16> {
  typedef uint4 type;
};

// An empty asm statement on each 32-bit word of a loaded value: the value is
// first used here, as it was loaded, so the compiler can neither move work on
// it closer to the load nor wait for the load any earlier.
template <typename R>
__device__ __forceinline__ void pin_words(R& r) {
  constexpr int W = sizeof(R) / 4;
  uint32_t w[W];
  __builtin_memcpy(w, &r, sizeof(R));
#pragma unroll
  for (int j = 0; j < W; ++j) asm volatile("" : "+v"(w[j]));
  __builtin_memcpy(&r, w, sizeof(R));
}

// SPLIT half waves share one family (families per workgroup: kFamilies /
// SPLIT): each sums a contiguous share of the family's keys in every flush,
// and the shares are added in a fixed order at the end. More than one for
// heads with many keys per parent, where one half wave's chain of loads
// would set the time.
//
// FUSED (the child compare of Alg. 1 inside the same pass, Ch >= 1): the
// input is the parent index of every key instead of its code. Each flush
// first buckets the queued keys by family, then the waves take groups of 16
// keys of one family and run the child compare on them (the key rows are
// read here; the candidate rows stay in registers while a wave's groups share
// the family), write the code of every key and re-queue the keys with their
// rows; the flush then goes on as above. Keys, and so the K rows, are read
// once per head; no code round trip between two kernels.
struct FusedArgs {
  const void* K;   // [B][H][N][d]
  const void* Cp;  // [H][M0][d]
  const void* Cc;  // [H][M0][Ch][d]
  int32_t* code_idx;  // out: [B][H][N]
  int H;
};

template <typename T, int D, int CHM, int SPLIT, bool FUSED>
__global__ __launch_bounds__(kAggThreads) void aggregate_kernel(const T* __restrict__ V,
                                                                const int32_t* __restrict__ code_idx,
                                                                float* __restrict__ Vbar,
                                                                int32_t* __restrict__ counts,
                                                                unsigned char* __restrict__ packed,
                                                                int N, int M0, int Ch, int ranges,
                                                                FusedArgs fa) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds_raw[];
  AggLds& L = *reinterpret_cast<AggLds*>(lds_raw);
  constexpr int CPL = D / kFamLanes;  // columns per lane
  using Raw = typename Chunk<CPL * sizeof(T)>::type;
  static_assert(CPL % 2 == 0, "whole pairs of columns per lane");

  const int Mtot = M0 * (1 + Ch);
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = blk / ranges;
  constexpr int FAM = kFamilies / SPLIT;  // families of this workgroup
  const int p0 = (blk % ranges) * FAM;
  const int nfam = min(FAM, M0 - p0);
  const int rows = nfam * (1 + Ch);
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int sub = lane % kFamLanes, fam = tid / kFamLanes / SPLIT, part = tid / kFamLanes % SPLIT;
  const int ch_shift = Ch > 0 ? 31 - __builtin_clz(Ch) : 0;  // Ch = 0: a flat codebook

  for (int r = tid; r < kMaxRows; r += kAggThreads) L.total[r] = 0;

  const int32_t* codes = code_idx + (size_t)bh * N;  // FUSED: parent indices
  const T* vhead = V + (size_t)bh * N * D;
  static_assert(!FUSED || CHM == 8, "the fused child compare holds one 16-row candidate tile");

  // the family table of this half wave: row 0 = stay, row 1 + c = child c
  float acc[1 + CHM][CPL];
#pragma unroll
  for (int r = 0; r <= CHM; ++r)
#pragma unroll
    for (int i = 0; i < CPL; ++i) acc[r][i] = 0.f;

  // FUSED: the queue holds (key, family); bucket it by family, compare each
  // group of 16 keys with its family's candidates, and leave the queue as
  // (key, row) in family order, the code of every key written
  auto child_step = [&](int qlen) {
    constexpr int NT = 1;
    using CT = ChildTile<T, D, NT>;
    constexpr int KQ = CT::KQ;
    using Frag = typename CT::Frag;
    // at d = 64 the next group's key fragments stay in flight; at d = 128
    // they load when they are used (the family table, the candidate rows and
    // two sets of key fragments would pass the 128 registers of a lane)
    constexpr bool kPrefetch = D == 64;
    const int h = bh % fa.H;
    const T* kh = static_cast<const T*>(fa.K) + (size_t)bh * N * D;
    // thread and lane index through an empty asm statement: the LDS
    // addresses below are formed here, not held (or spilled) from the start
    int tq = tid, lq = lane;
    asm volatile("" : "+v"(tq), "+v"(lq));
    if (tq < kFamilies) L.hist[tq] = 0;
    __syncthreads();
    for (int e = tq; e < qlen; e += kAggThreads) atomicAdd(&L.hist[L.qrow[e]], 1);
    __syncthreads();
    if (wave == 0) {  // family starts and group starts (nfam <= 32 lanes)
      const int lane = lq;
      const int v = lane < nfam ? L.hist[lane] : 0;
      const int gv = (v + 15) / 16;
      const int incl = wave_incl_scan(v), gincl = wave_incl_scan(gv);
      if (lane < nfam) {
        L.fstart[lane] = incl - v;
        L.fcursor[lane] = incl - v;
        L.item_start[lane] = gincl - gv;
      }
      if (lane == nfam - 1) {
        L.fstart[nfam] = incl;
        L.item_start[nfam] = gincl;
      }
    }
    __syncthreads();
    for (int e = tid; e < qlen; e += kAggThreads)
      L.skey[atomicAdd(&L.fcursor[L.qrow[e]], 1)] = L.qkey[e];
    __syncthreads();
    // each wave a contiguous run of groups (consecutive groups mostly share
    // the family, whose candidate rows stay in registers)
    const int g = lane / 16, c = lane % 16;
    const int n_items = L.item_start[nfam];
    const int per_wave = (n_items + kAggWaves - 1) / kAggWaves;
    const int it_begin = wave * per_wave, it_end = min(n_items, it_begin + per_wave);
    auto group_keys = [&](int f, int it, Frag (&kf)[KQ], int& pos, bool& valid) {
      const int kb = L.fstart[f] + 16 * (it - L.item_start[f]);
      valid = kb + c < L.fstart[f + 1];
      pos = valid ? kb + c : kb;
      child_key<T, D, NT>(kh + (size_t)L.skey[pos] * D, g, kf);
    };
    Frag cf[NT][KQ];
    f32x4 cn[NT];
    Frag kf[KQ];
    int cur_f = -1, f = 0, pos = 0;
    bool valid = false;
    if (it_begin < it_end) {
      while (L.item_start[f + 1] <= it_begin) ++f;  // wave-uniform
      group_keys(f, it_begin, kf, pos, valid);
    }
    for (int it = it_begin; it < it_end; ++it) {
      Frag kn[KQ];
      int fn = f, pos_n = 0;
      bool valid_n = false;
      if (it + 1 < it_end) {
        while (L.item_start[fn + 1] <= it + 1) ++fn;  // wave-uniform
        if constexpr (kPrefetch) group_keys(fn, it + 1, kn, pos_n, valid_n);
      }
      if constexpr (!kPrefetch) {
        if (it > it_begin) group_keys(f, it, kf, pos, valid);
      }
      const int p = p0 + f;
      if (f != cur_f) {
        child_rows<T, D, NT>(static_cast<const T*>(fa.Cp), static_cast<const T*>(fa.Cc), h, M0,
                             Ch, p, g, c, cf, cn);
        cur_f = f;
      }
      const int r = child_pick<T, D, NT>(cf, cn, kf, Ch, g, c);
      if (g == 0 && valid) {
        const int key = L.skey[pos];
        fa.code_idx[(size_t)bh * N + key] = r > 0 ? M0 + p * Ch + r - 1 : p;
        L.qkey[pos] = key;
        L.qrow[pos] = (uint16_t)(f * (1 + Ch) + r);
      }
      if constexpr (kPrefetch) {
#pragma unroll
        for (int kq = 0; kq < KQ; ++kq) kf[kq] = kn[kq];
        pos = pos_n;
        valid = valid_n;
      }
      f = fn;
    }
    __syncthreads();
  };

  // 1. scan the head's codes and queue the keys of this range; bucket and
  //    sum the queue when it would overflow and once the codes are exhausted
  int qlen = 0;
  int next[kCodesPerThread];
  auto load_round = [&](int b, int (&dst)[kCodesPerThread]) {
#pragma unroll
    for (int k = 0; k < kCodesPerThread; ++k) {
      const int j = b + k * kAggThreads + tid;
      dst[k] = j < N ? codes[j] : -1;
    }
  };
  load_round(0, next);
  // family-local row of a code (or, FUSED, the family of a parent index);
  // -1 outside this range
  auto row_of = [&](int code) {
    int r = -1;
    if constexpr (FUSED) {  // the family; its row comes from the child compare
      if (code >= p0 && code < p0 + nfam) r = code - p0;
    } else if (code >= 0 && code < Mtot) {
      // Ch is a power of two: child code M0 + p Ch + c
      const int p = code < M0 ? code : (code - M0) >> ch_shift;
      if (p >= p0 && p < p0 + nfam)
        r = (p - p0) * (1 + Ch) + (code < M0 ? 0 : 1 + ((code - M0) & (Ch - 1)));
    }
    return r;
  };
  for (int base = 0;; base += kRound) {
    const bool done = base >= N;
    // this round's codes; their rows and ballots are taken again after a
    // flush rather than kept in registers through it
    int cur[kCodesPerThread];
    int round_total = 0;
    if (!done) {
#pragma unroll
      for (int k = 0; k < kCodesPerThread; ++k) cur[k] = next[k];
#pragma unroll
      for (int k = 0; k < kCodesPerThread; ++k) {
        const unsigned long long mk = __ballot(row_of(cur[k]) >= 0);
        if (lane == 0) L.wave_count[k][wave] = __popcll(mk);
      }
      __syncthreads();
      if (wave == 0) {
        const int tot = prefix128(&L.wave_count[0][0], &L.wave_off[0][0],
                                  kCodesPerThread * kAggWaves, lane);
        if (lane == 0) L.round_total = tot;
      }
      __syncthreads();
      round_total = L.round_total;
      load_round(base + kRound, next);  // prefetch the next round
    }
    // uniform across the workgroup
    const bool flush = done ? qlen > 0 : qlen + round_total > kQueueCap;
    if (flush) {
      if constexpr (FUSED) child_step(qlen);
      // as in child_step: indices through an empty asm statement
      int tq = tid, lq = lane;
      asm volatile("" : "+v"(tq), "+v"(lq));
      for (int r = tq; r < rows; r += kAggThreads) L.hist[r] = 0;
      __syncthreads();
      for (int e = tq; e < qlen; e += kAggThreads) atomicAdd(&L.hist[L.qrow[e]], 1);
      __syncthreads();
      if (wave == 0) {  // exclusive scan of the row histogram
        const int lane = lq;
        int carry = 0;
        for (int r0 = 0; r0 < rows; r0 += kWave) {
          const int r = r0 + lane;
          const int v = r < rows ? L.hist[r] : 0;
          const int incl = wave_incl_scan(v);
          if (r < rows) {
            L.start[r] = carry + incl - v;
            L.cursor[r] = carry + incl - v;
            L.total[r] += v;
          }
          carry += last_lane(incl);
        }
        if (lane == 0) L.start[rows] = carry;
      }
      __syncthreads();
      for (int e = tid; e < qlen; e += kAggThreads)
        L.skey[atomicAdd(&L.cursor[L.qrow[e]], 1)] = L.qkey[e];
      __syncthreads();
      if (fam < nfam) {
        // the family's keys, bucketed by row, in kInFlight<CHM, T> batches; the
        // running row sum goes into the table when its row ends. The family
        // index passes an empty asm statement: its row addresses are formed
        // here, not held (or spilled) from the kernel start.
        int fq = fam;
        asm volatile("" : "+v"(fq));
        const int r_begin = fq * (1 + Ch);
        const int fb = L.start[r_begin], fe = L.start[r_begin + 1 + Ch];
        // this half wave's share of the family's keys
        const int kb = fb + (fe - fb) * part / SPLIT, ke = fb + (fe - fb) * (part + 1) / SPLIT;
        int rr = 0;                          // current row of the family
        int row_end = L.start[r_begin + 1];  // end of its bucket
        float cur[CPL];
#pragma unroll
        for (int i = 0; i < CPL; ++i) cur[i] = 0.f;
        // every table row takes cur or zero: a plain add per row keeps the
        // table in registers (a conditional add on rr alone is turned into an
        // indexed access to scratch memory)
        auto close_row = [&]() {
#pragma unroll
          for (int r = 0; r <= CHM; ++r)
#pragma unroll
            for (int i = 0; i < CPL; ++i) acc[r][i] += r == rr ? cur[i] : 0.f;
#pragma unroll
          for (int i = 0; i < CPL; ++i) cur[i] = 0.f;
        };
        // a ring of kIF rows in flight: slot u holds key k0 + u; once it is
        // summed it is refilled with key k0 + kIF + u, so kIF - 1 loads stay
        // in flight while the rows are added. Keys past the share repeat its
        // last key: the refills are unconditional, so the compiler's count
        // of outstanding loads is exact and every wait leaves kIF - 1 of them
        // in flight (a conditional refill makes it wait for more).
        constexpr int kIF = kInFlight<CHM, T>;
        auto row_of = [&](int k) {
          return *reinterpret_cast<const Raw*>(vhead + (size_t)L.skey[min(k, ke - 1)] * D + sub * CPL);
        };
        Raw raw[kIF];
        if (kb < ke) {
#pragma unroll
          for (int u = 0; u < kIF; ++u) raw[u] = row_of(kb + u);
        }
        for (int k0 = kb; k0 < ke; k0 += kIF) {
#pragma unroll
          for (int u = 0; u < kIF; ++u) {
            if (k0 + u < ke) {
              while (k0 + u >= row_end) {  // uniform within the half wave
                close_row();
                ++rr;
                row_end = L.start[r_begin + rr + 1];
              }
              // the row is unpacked here, not where it was loaded: otherwise
              // the compiler moves the unpacking next to the loads and waits
              // for all of them there
              pin_words(raw[u]);
              const T* x = reinterpret_cast<const T*>(&raw[u]);
#pragma unroll
              for (int i = 0; i < CPL; ++i) cur[i] += to_f32(x[i]);
            }
            raw[u] = row_of(k0 + kIF + u);
          }
        }
        if (kb < ke) close_row();
      }
      __syncthreads();
      qlen = 0;
      // this round's codes and the next round's are loaded again rather than
      // held in registers through the flush
      if (!done) {
        load_round(base, cur);
        load_round(base + kRound, next);
      }
    }
    if (done) break;
#pragma unroll
    for (int k = 0; k < kCodesPerThread; ++k) {
      asm volatile("" : "+v"(cur[k]));  // rows from the codes, not held through the flush
      const int row = row_of(cur[k]);
      const unsigned long long mk = __ballot(row >= 0);
      if (row >= 0) {
        const int slot = qlen + L.wave_off[k][wave] + bits_below(mk);
        L.qkey[slot] = base + k * kAggThreads + tid;
        L.qrow[slot] = (uint16_t)row;
      }
    }
    qlen += round_total;
    __syncthreads();
  }

  // 2. parent row = stay + children; write every row once, and the counts.
  //    Packed aggregates (optional): the owner writes its children's octets
  //    directly; the parents' octets (8 parents from 8 owners each) are put
  //    together through LDS (the queue area is free now).
  const PackedLayout PL = packed_layout(M0, Ch, D, (int)sizeof(T));
  if constexpr (SPLIT > 1) {
    // add the shares of parts 1 .. SPLIT-1 into part 0's table, row by row,
    // in part order, through the free key queue
    float* share = reinterpret_cast<float*>(L.qkey);  // [SPLIT - 1][FAM][D]
    static_assert((SPLIT - 1) * FAM * D * 4 <= sizeof(L.qkey), "shares fit the key queue");
#pragma unroll
    for (int r = 0; r <= CHM; ++r) {
      if (r <= Ch) {  // uniform
        if (fam < nfam && part > 0) {
#pragma unroll
          for (int i = 0; i < CPL; ++i) share[((part - 1) * FAM + fam) * D + sub * CPL + i] = acc[r][i];
        }
        __syncthreads();
        if (fam < nfam && part == 0) {
#pragma unroll
          for (int q = 1; q < SPLIT; ++q)
#pragma unroll
            for (int i = 0; i < CPL; ++i) acc[r][i] += share[((q - 1) * FAM + fam) * D + sub * CPL + i];
        }
        __syncthreads();
      }
    }
  }
  float* pmean = reinterpret_cast<float*>(L.qkey);  // [FAM][D]
  int* pcell = reinterpret_cast<int*>(pmean + FAM * D);  // [FAM] cell sizes
  static_assert((kFamilies * D + kFamilies) * 4 <= sizeof(L.qkey), "parent means fit the key queue");
  // child octets leave through a 1 KB staging area per family (in the free
  // row and bucket queues), so that each store writes 16 consecutive bytes
  // per lane, contiguous over the half wave
  constexpr int kStageRows = 1024 / (8 * (int)sizeof(T));  // octet d-rows per pass
  static_assert(kFamilies * 1024 <= sizeof(L.qrow) + sizeof(L.skey), "staging fits the queues");
  static_assert(kStageRows % kFamLanes == 0 && D % kStageRows == 0, "whole passes");
  T* stage = reinterpret_cast<T*>(reinterpret_cast<unsigned char*>(L.qrow) + fam * 1024);
  float* vb = Vbar ? Vbar + (size_t)bh * Mtot * D : nullptr;
  unsigned char* pk = packed ? packed + (size_t)bh * PL.bytes : nullptr;
  T* means = reinterpret_cast<T*>(pk);
  float* info = reinterpret_cast<float*>(pk + PL.info_off);
  constexpr float kNegInf = -__builtin_inff();
  constexpr float kLn2 = 0.6931471805599453f;
  if (fam < nfam && part == 0) {
    const int p = p0 + fam;
    const int* tot = &L.total[fam * (1 + Ch)];
    float par[CPL];
#pragma unroll
    for (int i = 0; i < CPL; ++i) par[i] = acc[0][i];
    int ncell = tot[0];
#pragma unroll
    for (int r = 1; r <= CHM; ++r) {
      if (r <= Ch) {
        if (vb) {
          float* dst = vb + (size_t)(M0 + p * Ch + (r - 1)) * D + sub * CPL;
#pragma unroll
          for (int i = 0; i < CPL; i += 2)
            *reinterpret_cast<float2*>(dst + i) = float2{acc[r][i], acc[r][i + 1]};
        }
#pragma unroll
        for (int i = 0; i < CPL; ++i) par[i] += acc[r][i];
        ncell += tot[r];
      }
    }
    if (vb) {
      float* dst = vb + (size_t)p * D + sub * CPL;
#pragma unroll
      for (int i = 0; i < CPL; i += 2) *reinterpret_cast<float2*>(dst + i) = float2{par[i], par[i + 1]};
    }
    if (pk) {
      const float pinv = ncell > 0 ? 1.f / (float)ncell : 0.f;
#pragma unroll
      for (int i = 0; i < CPL; ++i) pmean[fam * D + sub * CPL + i] = par[i] * pinv;
      if (sub == 0) pcell[fam] = ncell;
      // this parent's child octets: [CO][D][8], and their info
#pragma unroll
      for (int j = 0; j < (CHM + 7) / 8; ++j) {
        if (j < PL.CO) {
          const int o = PL.PO + p * PL.CO + j;
          float inv[8];
#pragma unroll
          for (int sl = 0; sl < 8; ++sl) {
            const int c = 8 * j + sl;
            const int n = c < Ch ? tot[1 + c] : 0;
            inv[sl] = n > 0 ? 1.f / (float)n : 0.f;
          }
          // pass q: the lanes holding d-rows q R .. q R + R - 1 (R =
          // kStageRows) put them in the staging area, then lane sub stores
          // d-rows q R + sub + 32 t
#pragma unroll
          for (int q = 0; q < D / kStageRows; ++q) {
#pragma unroll
            for (int i = 0; i < CPL; ++i) {
              const int dr = sub * CPL + i - q * kStageRows;
              if (dr < 0 || dr >= kStageRows) continue;
              float v[8];
#pragma unroll
              for (int sl = 0; sl < 8; ++sl) {
                float a = 0.f;
#pragma unroll
                for (int r = 1; r <= CHM; ++r)
                  if (r == 1 + 8 * j + sl) a = acc[r][i];
                v[sl] = a * inv[sl];
              }
              T* sd = stage + dr * 8;
              if constexpr (Elem<T>::kBf16) {
                bf16x8 w = {(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3],
                            (bf16)v[4], (bf16)v[5], (bf16)v[6], (bf16)v[7]};
                *reinterpret_cast<bf16x8*>(sd) = w;
              } else {
                reinterpret_cast<float4*>(sd)[0] = float4{v[0], v[1], v[2], v[3]};
                reinterpret_cast<float4*>(sd)[1] = float4{v[4], v[5], v[6], v[7]};
              }
            }
            // the half wave's own LDS writes and reads stay in order
            __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int t = 0; t < kStageRows / kFamLanes; ++t) {
              const int dr = sub + kFamLanes * t;
              T* dst = means + ((size_t)o * D + q * kStageRows + dr) * 8;
              if constexpr (Elem<T>::kBf16) {
                *reinterpret_cast<bf16x8*>(dst) = *reinterpret_cast<const bf16x8*>(stage + dr * 8);
              } else {
                reinterpret_cast<float4*>(dst)[0] = reinterpret_cast<const float4*>(stage + dr * 8)[0];
                reinterpret_cast<float4*>(dst)[1] = reinterpret_cast<const float4*>(stage + dr * 8)[1];
              }
            }
            __builtin_amdgcn_s_waitcnt(0xc07f);
            __builtin_amdgcn_wave_barrier();
          }
          // lane sub < 16 writes info slot sub: n (slots 0..7), ln n (8..15)
          if (sub < 16) {
            const int c = 8 * j + (sub & 7);
            const int n = c < Ch ? tot[1 + c] : 0;
            info[(size_t)o * 16 + sub] =
                sub < 8 ? (float)n : (n > 0 ? log2_hw((float)n) * kLn2 : kNegInf);
          }
        }
      }
    }
  }
  __syncthreads();
  if (pk) {
    // the parent octets of this range (the last range also writes the padding
    // octets, the first one the empty octet)
    const int o_begin = p0 / 8;
    const int o_end = (p0 + nfam >= M0) ? PL.PO : (p0 + nfam) / 8;
    const int nrow = (o_end - o_begin) * D;
    for (int i = tid; i < nrow; i += kAggThreads) {
      const int o = o_begin + i / D, d = i % D;
      float v[8];
#pragma unroll
      for (int sl = 0; sl < 8; ++sl) {
        const int q = 8 * o + sl - p0;
        v[sl] = q < nfam ? pmean[q * D + d] : 0.f;
      }
      T* dst = means + ((size_t)o * D + d) * 8;
      if constexpr (Elem<T>::kBf16) {
        bf16x8 w = {(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3],
                    (bf16)v[4], (bf16)v[5], (bf16)v[6], (bf16)v[7]};
        *reinterpret_cast<bf16x8*>(dst) = w;
      } else {
        reinterpret_cast<float4*>(dst)[0] = float4{v[0], v[1], v[2], v[3]};
        reinterpret_cast<float4*>(dst)[1] = float4{v[4], v[5], v[6], v[7]};
      }
    }
    for (int i = tid; i < (o_end - o_begin) * 16; i += kAggThreads) {
      const int o = o_begin + i / 16, sl = i % 16;
      const int q = 8 * o + (sl & 7) - p0;
      const int n = q < nfam ? pcell[q] : 0;
      info[(size_t)o * 16 + sl] =
          sl < 8 ? (float)n : (n > 0 ? log2_hw((float)n) * kLn2 : kNegInf);
    }
    if (p0 == 0) {  // the empty octet
      for (int i = tid; i < D * 8; i += kAggThreads) means[(size_t)PL.zero_oct * D * 8 + i] = T(0.f);
      if (tid < 16) info[(size_t)PL.zero_oct * 16 + tid] = tid < 8 ? 0.f : kNegInf;
    }
  }
  int32_t* nb = counts + (size_t)bh * Mtot;
  for (int f = tid; f < nfam; f += kAggThreads) {
    const int* tot = &L.total[f * (1 + Ch)];
    int cell = 0;
    for (int c = 0; c <= Ch; ++c) cell += tot[c];
    nb[p0 + f] = cell;
    for (int c = 0; c < Ch; ++c) nb[M0 + (p0 + f) * Ch + c] = tot[1 + c];
  }
}

template <typename T, int D, int CHM, int SPLIT, bool FUSED>
hipError_t launch_aggregate_dcs(int BH, int N, int M0, int Ch, const void* V,
                                const int32_t* code_idx, float* Vbar, int32_t* counts,
                                void* packed, const FusedArgs& fa, hipStream_t stream) {
  // one range of kFamilies / SPLIT parents per workgroup: ranges start at
  // multiples of 8 parents, so each packed octet of parent means is written
  // by one workgroup
  constexpr int FAM = kFamilies / SPLIT;
  static_assert(FAM % 8 == 0, "parent octets are assembled by one workgroup");
  static_assert(kRound <= kQueueCap, "one round of codes fits the queue");
  const int ranges = (M0 + FAM - 1) / FAM;
  const int lds = (int)sizeof(AggLds);
  constexpr int chm_i = CHM == 0 ? 0 : CHM == 8 ? 1 : 2;
  constexpr int split_i = SPLIT == 1 ? 0 : SPLIT == 2 ? 1 : 2;
  constexpr int slot = (FUSED ? 128 : 64) +
                       (((Elem<T>::kBf16 ? 0 : 1) * 2 + (D == 128 ? 1 : 0)) * 3 + chm_i) * 3 +
                       split_i;
  hipError_t e =
      ensure_dynamic_lds((const void*)aggregate_kernel<T, D, CHM, SPLIT, FUSED>, lds, slot);
  if (e != hipSuccess) return e;
  const long long grid = (long long)BH * ranges;
  if (grid > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((aggregate_kernel<T, D, CHM, SPLIT, FUSED>), dim3((unsigned)grid),
                     dim3(kAggThreads), lds, stream, static_cast<const T*>(V), code_idx, Vbar,
                     counts, static_cast<unsigned char*>(packed), N, M0, Ch, ranges, fa);
  return hipGetLastError();
}

// Half waves per family. Each workgroup scans all codes of its head, so
// splitting a family over more half waves (more, smaller workgroups) costs
// scanning; it pays when some CUs would have no workgroup (few heads, few
// parents) and either one half wave per family would walk a long chain of
// value loads (at least 256 keys per parent) or the head's codes are one
// scan round (then the extra scanning is that one round). Then the fewest
// half waves (2 or 4) that give every CU a workgroup.
template <typename T, int D, int CHM, bool FUSED>
hipError_t launch_aggregate_dc(int BH, int N, int M0, int Ch, const void* V,
                               const int32_t* code_idx, float* Vbar, int32_t* counts,
                               void* packed, const FusedArgs& fa, hipStream_t stream) {
  DeviceInfo dev;
  hipError_t e = device_info(&dev);
  if (e != hipSuccess) return e;
  const long long cus = dev.cus > 1 ? dev.cus : 1;
  auto grid = [&](int split) {
    const int fam = kFamilies / split;
    return (long long)BH * ((M0 + fam - 1) / fam);
  };
  const bool long_chains = (long long)N >= 256LL * M0;
  if ((!long_chains && N > kRound) || grid(1) >= cus)
    return launch_aggregate_dcs<T, D, CHM, 1, FUSED>(BH, N, M0, Ch, V, code_idx, Vbar, counts,
                                                     packed, fa, stream);
  if (grid(2) >= cus)
    return launch_aggregate_dcs<T, D, CHM, 2, FUSED>(BH, N, M0, Ch, V, code_idx, Vbar, counts,
                                                     packed, fa, stream);
  return launch_aggregate_dcs<T, D, CHM, 4, FUSED>(BH, N, M0, Ch, V, code_idx, Vbar, counts,
                                                   packed, fa, stream);
}

template <typename T, int D>
hipError_t launch_aggregate_d(int BH, int N, int M0, int Ch, const void* V,
                              const int32_t* code_idx, float* Vbar, int32_t* counts,
                              void* packed, hipStream_t stream) {
  const FusedArgs none{};
  if (Ch == 0)  // flat codebook: a family is one parent
    return launch_aggregate_dc<T, D, 0, false>(BH, N, M0, Ch, V, code_idx, Vbar, counts, packed,
                                               none, stream);
  if (Ch <= 8)
    return launch_aggregate_dc<T, D, 8, false>(BH, N, M0, Ch, V, code_idx, Vbar, counts, packed,
                                               none, stream);
  if (Ch <= 16)
    return launch_aggregate_dc<T, D, 16, false>(BH, N, M0, Ch, V, code_idx, Vbar, counts,
                                                packed, none, stream);
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t launch_aggregate(int BH, int N, int d, int M0, int Ch, const void* V,
                            const int32_t* code_idx, float* Vbar, int32_t* counts, void* packed,
                            hipStream_t stream) {
  if (d == 64)
    return launch_aggregate_d<T, 64>(BH, N, M0, Ch, V, code_idx, Vbar, counts, packed, stream);
  if (d == 128)
    return launch_aggregate_d<T, 128>(BH, N, M0, Ch, V, code_idx, Vbar, counts, packed, stream);
  return hipErrorInvalidValue;
}

// Alg. 1 in two launches: the parent assignment (it reads K once and writes
// parent_idx), then the fused child compare + aggregation (bf16, 1 <= Ch <=
// 8). Ch = 0 (the parent is the code), Ch = 16 (two candidate tiles) and fp32
// (its fragments, the family table and the candidate rows pass the registers
// of a 1024-thread workgroup) take the parent and child kernels of the
// assignment and then the plain aggregation.
template <typename T>
hipError_t launch_assign_aggregate(int BH, int H, int N, int d, int M0, int Ch, const void* K,
                                   const void* V, const void* Cp, const void* Cc,
                                   int32_t* parent_idx, int32_t* code_idx, float* Vbar,
                                   int32_t* counts, void* packed, hipStream_t stream) {
  const bool fused = Elem<T>::kBf16 && Ch >= 1 && Ch <= 8;
  hipError_t e = d == 64 ? launch_assign<T, 64>(BH, H, N, M0, Ch, K, Cp, Cc, parent_idx, code_idx,
                                                !fused, stream)
                         : launch_assign<T, 128>(BH, H, N, M0, Ch, K, Cp, Cc, parent_idx,
                                                 code_idx, !fused, stream);
  if (e != hipSuccess) return e;
  if (!fused) return launch_aggregate<T>(BH, N, d, M0, Ch, V, code_idx, Vbar, counts, packed, stream);
  FusedArgs fa{K, Cp, Cc, code_idx, H};
  if constexpr (Elem<T>::kBf16) {
    if (d == 64)
      return launch_aggregate_dc<T, 64, 8, true>(BH, N, M0, Ch, V, parent_idx, Vbar, counts,
                                                 packed, fa, stream);
    return launch_aggregate_dc<T, 128, 8, true>(BH, N, M0, Ch, V, parent_idx, Vbar, counts,
                                                packed, fa, stream);
  }
  return hipErrorInvalidValue;  // not reached: fp32 takes the unfused path
}

template hipError_t launch_aggregate<bf16>(int, int, int, int, int, const void*, const int32_t*,
                                           float*, int32_t*, void*, hipStream_t);
template hipError_t launch_aggregate<float>(int, int, int, int, int, const void*, const int32_t*,
                                            float*, int32_t*, void*, hipStream_t);
template hipError_t launch_assign_aggregate<bf16>(int, int, int, int, int, int, const void*,
                                                  const void*, const void*, const void*,
                                                  int32_t*, int32_t*, float*, int32_t*, void*,
                                                  hipStream_t);
template hipError_t launch_assign_aggregate<float>(int, int, int, int, int, int, const void*,
                                                   const void*, const void*, const void*,
                                                   int32_t*, int32_t*, float*, int32_t*, void*,
                                                   hipStream_t);

}  // namespace avq
