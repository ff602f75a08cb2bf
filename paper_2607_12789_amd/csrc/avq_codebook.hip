// Codebook update by exponential moving averages under the parent-child
// constraint (App. A, Eq. (child_constraint_solve)).
//
// Input: the key sums and counts of one batch per code (avq_aggregate run on
// the keys: parent rows cover the whole cell, child rows the keys that moved
// to the child), the EMA state (S, N) per code. One workgroup owns one parent
// family (the parent and its Ch children) of one head; thread e owns
// dimension e of every row of the family, so the projection needs no
// exchange between threads: for each row it sums the batch statistics in
// batch order, updates S and N, forms the unconstrained mean M = S / N, then
// the parent codeword C_p = M_p and the children
// C_pc = M_c - delta / (N_c sigma), delta = sum_c M_c - Ch C_p,
// sigma = sum_c 1 / N_c. All arithmetic is fp32; the codewords are stored in
// the codebook's type. Memory-bound: every byte is read or written once,
// rows are contiguous over the threads.
#include "avq_common.hpp"

namespace avq {

constexpr int kMaxCh = 16;

template <typename T>
__global__ __launch_bounds__(128) void codebook_update_kernel(
    const float* __restrict__ sums, const int32_t* __restrict__ counts, float* __restrict__ S,
    float* __restrict__ Nema, T* __restrict__ Cp_out, T* __restrict__ Cc_out, int B, int H, int d,
    int M0, int Ch, float lam) {
  const int fam = blockIdx.x;  // h * M0 + p
  const int h = fam / M0, p = fam % M0;
  const int e = threadIdx.x;
  const int Mtot = M0 * (1 + Ch);
  const float keep = lam, take = 1.f - lam;
  const size_t head = (size_t)h * Mtot;
  const size_t bstride = (size_t)H * Mtot;  // codes per batch entry

  // one code x: batch statistics in batch order, then the EMA; returns M_x[e]
  // (and N_x in n_out)
  auto update_row = [&](int x, float& n_out) {
    float n = 0.f;
    float s = 0.f;
    for (int b = 0; b < B; ++b) {
      const size_t r = (size_t)b * bstride + head + x;
      n += (float)counts[r];  // integers below 2^24: exact
      if (e < d) s += sums[r * d + e];
    }
    const size_t r = head + x;
    const float nn = fmaf(keep, Nema[r], take * n);
    n_out = nn;
    float m = 0.f;
    if (e < d) {
      const float ss = fmaf(keep, S[r * d + e], take * s);
      S[r * d + e] = ss;
      m = ss / nn;
    }
    return m;
  };

  float np_;
  const float cp = update_row(p, np_);
  float mc[kMaxCh], nc[kMaxCh];
#pragma unroll
  for (int c = 0; c < kMaxCh; ++c) {
    mc[c] = 0.f;
    nc[c] = 1.f;
    if (c < Ch) mc[c] = update_row(M0 + p * Ch + c, nc[c]);
  }
  // every thread has read the old N of the family's rows before one writes
  __syncthreads();
  if (e == 0) {
    Nema[head + p] = np_;
#pragma unroll
    for (int c = 0; c < kMaxCh; ++c)
      if (c < Ch) Nema[head + M0 + p * Ch + c] = nc[c];
  }
  if (e >= d) return;
  Cp_out[((size_t)h * M0 + p) * d + e] = (T)cp;
  if (Ch == 0) return;
  float sigma = 0.f, delta = 0.f;
#pragma unroll
  for (int c = 0; c < kMaxCh; ++c) {
    if (c < Ch) {
      sigma += 1.f / nc[c];
      delta += mc[c];
    }
  }
  delta = fmaf(-(float)Ch, cp, delta);
#pragma unroll
  for (int c = 0; c < kMaxCh; ++c) {
    if (c < Ch)
      Cc_out[(((size_t)h * M0 + p) * Ch + c) * d + e] = (T)(mc[c] - delta / (nc[c] * sigma));
  }
}

template <typename T>
hipError_t launch_codebook_update(int B, int H, int d, int M0, int Ch, float lam,
                                  const float* sums, const int32_t* counts, float* S,
                                  float* Nema, void* Cp_out, void* Cc_out, hipStream_t stream) {
  if (d > 128 || Ch > kMaxCh) return hipErrorInvalidValue;
  const long long grid = (long long)H * M0;
  if (grid > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((codebook_update_kernel<T>), dim3((unsigned)grid), dim3(128), 0, stream, sums,
                     counts, S, Nema, static_cast<T*>(Cp_out), static_cast<T*>(Cc_out), B, H, d,
                     M0, Ch, lam);
  return hipGetLastError();
}

template hipError_t launch_codebook_update<bf16>(int, int, int, int, int, float, const float*,
                                                 const int32_t*, float*, float*, void*, void*,
                                                 hipStream_t);
template hipError_t launch_codebook_update<float>(int, int, int, int, int, float, const float*,
                                                  const int32_t*, float*, float*, void*, void*,
                                                  hipStream_t);

}  // namespace avq
