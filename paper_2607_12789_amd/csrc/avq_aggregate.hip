// Per-codeword counts and value sums, Eq. (aggregates), with the Alg. 1
// convention that a parent row covers its whole cell and a child row the keys
// that moved to it.
//
// One workgroup owns one (batch, head) and a slice of DS value columns. Its
// fp32 table for all Mtot codes x DS columns lives in LDS, so every atomic add
// stays on-chip; the table is written to HBM once, each row a contiguous
// DS-float segment. The workgroup holding slice 0 also counts keys per code
// in an LDS int table. DS is the widest power of two that divides d and lets
// both tables fit the 160 KB of LDS of a gfx950 CU.
#include "avq_common.hpp"

namespace avq {

constexpr int kAggThreads = 512;
constexpr int kLdsBytes = 160 * 1024;

template <typename T>
__global__ __launch_bounds__(kAggThreads) void aggregate_kernel(const T* __restrict__ V,
                                                                const int32_t* __restrict__ code_idx,
                                                                float* __restrict__ Vbar,
                                                                int32_t* __restrict__ counts,
                                                                int N, int d, int M0, int Ch,
                                                                int DS, int n_slices) {
  extern __shared__ __attribute__((aligned(16))) float lds[];
  const int Mtot = M0 * (1 + Ch);
  const int blk = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = blk / n_slices, slice = blk % n_slices;
  const bool do_counts = (slice == 0);
  float* table = lds;                                         // [Mtot][DS]
  int* cnt = reinterpret_cast<int*>(lds + (size_t)Mtot * DS);  // [Mtot]

  for (int i = threadIdx.x; i < Mtot * DS; i += blockDim.x) table[i] = 0.f;
  if (do_counts)
    for (int i = threadIdx.x; i < Mtot; i += blockDim.x) cnt[i] = 0;
  __syncthreads();

  const int e = threadIdx.x % DS;
  const int keys_per_iter = blockDim.x / DS;
  const T* vbase = V + (size_t)bh * N * d + (size_t)slice * DS + e;
  const int32_t* cbase = code_idx + (size_t)bh * N;
  for (int j = threadIdx.x / DS; j < N; j += keys_per_iter) {
    const int code = cbase[j];
    if (code < 0 || code >= Mtot) continue;  // not a code avq_assign writes
    const int p = code < M0 ? code : (code - M0) / Ch;
    const float v = to_f32(vbase[(size_t)j * d]);
    atomicAdd(&table[p * DS + e], v);
    if (code >= M0) atomicAdd(&table[code * DS + e], v);
    if (do_counts && e == 0) {
      atomicAdd(&cnt[p], 1);
      if (code >= M0) atomicAdd(&cnt[code], 1);
    }
  }
  __syncthreads();

  float* out = Vbar + (size_t)bh * Mtot * d + (size_t)slice * DS;
  for (int i = threadIdx.x; i < Mtot * DS; i += blockDim.x) {
    const int r = i / DS, col = i % DS;
    out[(size_t)r * d + col] = table[i];
  }
  if (do_counts)
    for (int i = threadIdx.x; i < Mtot; i += blockDim.x) counts[(size_t)bh * Mtot + i] = cnt[i];
}

// Widest d-slice (power of two dividing d, at most 16) whose tables fit in
// lds_bytes of LDS.
int aggregate_slice_width(int d, int M0, int Ch, long long lds_bytes) {
  const long long Mtot = (long long)M0 * (1 + Ch);
  for (int ds = 16; ds >= 1; ds >>= 1) {
    if (d % ds != 0) continue;
    if (Mtot * (ds + 1) * 4 <= lds_bytes) return ds;
  }
  return 0;
}

template <typename T>
hipError_t launch_aggregate(int BH, int N, int d, int M0, int Ch, const void* V,
                            const int32_t* code_idx, float* Vbar, int32_t* counts,
                            hipStream_t stream) {
  int dev = 0, lds_max = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
  if (e != hipSuccess) return e;
  if (lds_max > kLdsBytes) lds_max = kLdsBytes;
  const int DS = aggregate_slice_width(d, M0, Ch, lds_max);
  if (DS == 0) return hipErrorInvalidValue;
  const int n_slices = d / DS;
  const size_t lds = (size_t)M0 * (1 + Ch) * (DS + 1) * sizeof(float);
  if (lds > 65536) {
    e = hipFuncSetAttribute((const void*)aggregate_kernel<T>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  const long long grid = (long long)BH * n_slices;
  if (grid > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(aggregate_kernel<T>, dim3((unsigned)grid), dim3(kAggThreads), lds, stream,
                     static_cast<const T*>(V), code_idx, Vbar, counts, N, d, M0, Ch, DS,
                     n_slices);
  return hipGetLastError();
}

template hipError_t launch_aggregate<bf16>(int, int, int, int, int, const void*, const int32_t*,
                                           float*, int32_t*, hipStream_t);
template hipError_t launch_aggregate<float>(int, int, int, int, int, const void*, const int32_t*,
                                            float*, int32_t*, hipStream_t);

}  // namespace avq
