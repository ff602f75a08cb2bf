// Packing of the paper's aggregates (Alg. 2 input: the value sums Vbar and
// the counts n of every code, Eq. (aggregates)) into the operand layout the
// attention kernel reads: per octet of 8 codes the mean values [d][8] in the
// storage type and the count info [16] fp32 (n, then ln n).
//
// The arithmetic is the aggregation kernel's own: mean = Vbar * fl(1/n) in
// fp32, rounded once to the storage type; ln n = log2(n) ln 2 by the hardware
// logarithm; -inf and a zero mean for an empty code and for padding slots. So
// the Vbar and counts that avq_aggregate writes pack into exactly the bytes of
// its packed output.
#include "avq_common.hpp"
#include "avq_packed.hpp"

namespace avq {

namespace {

constexpr int kPackThreads = 256;
constexpr float kLn2 = 0.6931471805599453f;

// code held by slot sl of octet o, or -1 for padding and the empty octet
__device__ __forceinline__ int octet_code(const PackedLayout& L, int M0, int Ch, int o, int sl) {
  if (o < L.PO) {
    const int p = 8 * o + sl;
    return p < M0 ? p : -1;
  }
  if (o >= L.zero_oct) return -1;
  const int p = (o - L.PO) / L.CO, c = 8 * ((o - L.PO) % L.CO) + sl;
  return c < Ch ? M0 + p * Ch + c : -1;
}

// One thread per (batch, head, octet, column): the 8 means of the column;
// threads of columns 0..15 also write info slot = column.
template <typename T>
__global__ __launch_bounds__(kPackThreads) void pack_kernel(const float* __restrict__ Vbar,
                                                            const int32_t* __restrict__ counts,
                                                            unsigned char* __restrict__ packed,
                                                            int M0, int Ch, int D,
                                                            long long total) {
  const long long i = (long long)blockIdx.x * kPackThreads + threadIdx.x;
  if (i >= total) return;
  const PackedLayout L = packed_layout(M0, Ch, D, (int)sizeof(T));
  const int Mtot = M0 * (1 + Ch);
  const long long per_bh = (long long)L.n_oct * D;
  const int bh = (int)(i / per_bh);
  const int rem = (int)(i % per_bh);
  const int o = rem / D, dr = rem % D;
  const float* vb = Vbar + (size_t)bh * Mtot * D;
  const int32_t* nb = counts + (size_t)bh * Mtot;
  unsigned char* pk = packed + (size_t)bh * L.bytes;
  float v[8];
#pragma unroll
  for (int sl = 0; sl < 8; ++sl) {
    const int x = octet_code(L, M0, Ch, o, sl);
    const int n = x >= 0 ? max(nb[x], 0) : 0;
    const float inv = n > 0 ? 1.f / (float)n : 0.f;
    v[sl] = x >= 0 ? vb[(size_t)x * D + dr] * inv : 0.f;
  }
  T* dst = reinterpret_cast<T*>(pk) + ((size_t)o * D + dr) * 8;
  if constexpr (Elem<T>::kBf16) {
    bf16x8 w = {(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3],
                (bf16)v[4], (bf16)v[5], (bf16)v[6], (bf16)v[7]};
    *reinterpret_cast<bf16x8*>(dst) = w;
  } else {
    reinterpret_cast<float4*>(dst)[0] = float4{v[0], v[1], v[2], v[3]};
    reinterpret_cast<float4*>(dst)[1] = float4{v[4], v[5], v[6], v[7]};
  }
  if (dr < 16) {
    const int x = octet_code(L, M0, Ch, o, dr & 7);
    const int n = x >= 0 ? max(nb[x], 0) : 0;
    float* info = reinterpret_cast<float*>(pk + L.info_off);
    info[(size_t)o * 16 + dr] =
        dr < 8 ? (float)n : (n > 0 ? log2_hw((float)n) * kLn2 : -__builtin_inff());
  }
}

}  // namespace

template <typename T>
hipError_t launch_pack(int BH, int M0, int Ch, int D, const float* Vbar, const int32_t* counts,
                       void* packed, hipStream_t stream) {
  const PackedLayout L = packed_layout(M0, Ch, D, (int)sizeof(T));
  const long long total = (long long)BH * L.n_oct * D;
  const long long blocks = (total + kPackThreads - 1) / kPackThreads;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(pack_kernel<T>, dim3((unsigned)blocks), dim3(kPackThreads), 0, stream, Vbar,
                     counts, static_cast<unsigned char*>(packed), M0, Ch, D, total);
  return hipGetLastError();
}

template hipError_t launch_pack<bf16>(int, int, int, int, const float*, const int32_t*, void*,
                                      hipStream_t);
template hipError_t launch_pack<float>(int, int, int, int, const float*, const int32_t*, void*,
                                       hipStream_t);

}  // namespace avq
