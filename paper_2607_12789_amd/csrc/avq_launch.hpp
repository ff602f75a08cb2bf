// Host-side launchers of the gfx950 kernels (one per source file), called by
// the C ABI; each returns the HIP status of its launches.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace avq {
template <typename T, int D>
hipError_t launch_assign(int BH, int H, int N, int M0, int Ch, const void* K, const void* Cp,
                         const void* Cc, int32_t* parent_idx, int32_t* code_idx,
                         bool with_children, hipStream_t stream);
template <typename T>
hipError_t launch_aggregate(int BH, int N, int d, int M0, int Ch, const void* V,
                            const int32_t* code_idx, float* Vbar, int32_t* counts, void* packed,
                            hipStream_t stream);
template <typename T>
hipError_t launch_assign_aggregate(int BH, int H, int N, int d, int M0, int Ch, const void* K,
                                   const void* V, const void* Cp, const void* Cc,
                                   int32_t* parent_idx, int32_t* code_idx, float* Vbar,
                                   int32_t* counts, void* packed, hipStream_t stream);
template <typename T, int D>
hipError_t launch_attention(int BH, int H, int N, int M0, int Ch, int P, int block_q,
                            const void* Q, const void* Cp, const void* Cc, const void* packed,
                            void* Y, int32_t* topp_idx,
                            float* importance, bool tiled, const int32_t* order,
                            hipStream_t stream);
long long gilbert_order(int width, int height, int32_t* order);
template <typename T>
hipError_t launch_pack(int BH, int M0, int Ch, int D, const float* Vbar, const int32_t* counts,
                       void* packed, hipStream_t stream);
template <typename T>
hipError_t launch_codebook_update(int B, int H, int d, int M0, int Ch, float lam,
                                  const float* sums, const int32_t* counts, float* S,
                                  float* Nema, void* Cp_out, void* Cc_out, hipStream_t stream);
}  // namespace avq
