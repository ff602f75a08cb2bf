// C ABI of the AVQ-Attention forward pass: argument validation on the host,
// then dispatch to the gfx950 kernels. Nothing here allocates device memory or
// synchronises; no exception crosses the boundary.
#include <stdarg.h>
#include <stdio.h>

#include <atomic>

#include "../../include/avq.h"
#include "avq_common.hpp"
#include "avq_packed.hpp"

#include "avq_launch.hpp"

namespace avq {

constexpr int kMaxDevices = 64;
constexpr int kMaxSlots = 256;

hipError_t device_info(DeviceInfo* out) {
  static DeviceInfo cache[kMaxDevices];
  static std::atomic<int> ready[kMaxDevices];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  if (ready[dev].load(std::memory_order_acquire) == 0) {
    DeviceInfo info;
    e = hipDeviceGetAttribute(&info.lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&info.cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    cache[dev] = info;
    ready[dev].store(1, std::memory_order_release);
  }
  *out = cache[dev];
  return hipSuccess;
}

hipError_t ensure_dynamic_lds(const void* kernel, int bytes, int slot) {
  // largest limit already set for (device, slot)
  static std::atomic<int> done[kMaxDevices][kMaxSlots];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices || slot < 0 || slot >= kMaxSlots) return hipErrorInvalidValue;
  if (done[dev][slot].load(std::memory_order_acquire) >= bytes) return hipSuccess;
  e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e != hipSuccess) return e;
  int prev = done[dev][slot].load(std::memory_order_relaxed);
  while (prev < bytes && !done[dev][slot].compare_exchange_weak(prev, bytes)) {
  }
  return hipSuccess;
}

}  // namespace avq

namespace {

thread_local char g_err[512] = "";

avq_status_t fail(avq_status_t st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

avq_status_t ok() {
  g_err[0] = '\0';
  return AVQ_OK;
}

avq_status_t from_hip(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(AVQ_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

// Shared shape checks. Everything is validated before any HIP call.
avq_status_t check_common(avq_dtype_t dtype, int32_t B, int32_t H, int32_t N, int32_t d,
                          int32_t M0, int32_t Ch) {
  if (dtype != AVQ_F32 && dtype != AVQ_BF16)
    return fail(AVQ_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
  if (B < 1 || H < 1 || N < 1 || d < 1 || M0 < 1 || Ch < 0)
    return fail(AVQ_ERR_INVALID_ARG,
                "sizes must be positive, Ch not negative (B=%d H=%d N=%d d=%d M0=%d Ch=%d)", B, H,
                N, d, M0, Ch);
  if (d != 64 && d != 128) return fail(AVQ_ERR_UNSUPPORTED, "d=%d: only 64 and 128", d);
  if (Ch != 0 && Ch != 1 && Ch != 2 && Ch != 4 && Ch != 8 && Ch != 16)
    return fail(AVQ_ERR_UNSUPPORTED, "Ch=%d: only 0 (flat codebook), 1, 2, 4, 8, 16", Ch);
  if (M0 > 512) return fail(AVQ_ERR_UNSUPPORTED, "M0=%d: at most 512", M0);
  if (N > (1 << 24)) return fail(AVQ_ERR_UNSUPPORTED, "N=%d: at most 2^24 keys per head", N);
  const long long elems = (long long)B * H * N * d;
  if (elems >= (1LL << 31))
    return fail(AVQ_ERR_UNSUPPORTED, "B*H*N*d=%lld: must stay below 2^31", elems);
  return AVQ_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

extern "C" {

int avq_version(void) { return 202; }

const char* avq_last_error(void) { return g_err; }

int64_t avq_packed_bytes(avq_dtype_t dtype, int32_t M0, int32_t Ch, int32_t d) {
  if (dtype != AVQ_F32 && dtype != AVQ_BF16) return -1;
  if (M0 < 1 || Ch < 0 || d < 1 || M0 > 512 || Ch > 16 || d > 128) return -1;
  return (int64_t)avq::packed_layout(M0, Ch, d, dtype == AVQ_BF16 ? 2 : 4).bytes;
}

avq_status_t avq_assign(avq_dtype_t dtype, int32_t B, int32_t H, int32_t N, int32_t d,
                        int32_t M0, int32_t Ch, const void* K, const void* Cp, const void* Cc,
                        int32_t* parent_idx, int32_t* code_idx, void* stream) {
  avq_status_t st = check_common(dtype, B, H, N, d, M0, Ch);
  if (st != AVQ_OK) return st;
  if (!K || !Cp || (!Cc && Ch > 0) || !parent_idx || !code_idx)
    return fail(AVQ_ERR_INVALID_ARG, "avq_assign: null pointer argument");
  if (!aligned16(K) || !aligned16(Cp) || !aligned16(Cc) || !aligned16(parent_idx) ||
      !aligned16(code_idx))
    return fail(AVQ_ERR_INVALID_ARG, "avq_assign: arrays must be 16-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int BH = B * H;
  hipError_t e;
  if (dtype == AVQ_BF16)
    e = d == 64 ? avq::launch_assign<avq::bf16, 64>(BH, H, N, M0, Ch, K, Cp, Cc, parent_idx, code_idx, true, s)
                : avq::launch_assign<avq::bf16, 128>(BH, H, N, M0, Ch, K, Cp, Cc, parent_idx, code_idx, true, s);
  else
    e = d == 64 ? avq::launch_assign<float, 64>(BH, H, N, M0, Ch, K, Cp, Cc, parent_idx, code_idx, true, s)
                : avq::launch_assign<float, 128>(BH, H, N, M0, Ch, K, Cp, Cc, parent_idx, code_idx, true, s);
  return from_hip(e, "avq_assign launch");
}

avq_status_t avq_aggregate(avq_dtype_t dtype, int32_t B, int32_t H, int32_t N, int32_t d,
                           int32_t M0, int32_t Ch, const void* V, const int32_t* code_idx,
                           float* Vbar, int32_t* counts, void* packed, void* stream) {
  avq_status_t st = check_common(dtype, B, H, N, d, M0, Ch);
  if (st != AVQ_OK) return st;
  if (!V || !code_idx || !counts)
    return fail(AVQ_ERR_INVALID_ARG, "avq_aggregate: null pointer argument");
  if (!Vbar && !packed)
    return fail(AVQ_ERR_INVALID_ARG, "avq_aggregate: Vbar and packed are both null");
  if (!aligned16(V) || !aligned16(code_idx) || !aligned16(Vbar) || !aligned16(counts) ||
      !aligned16(packed))
    return fail(AVQ_ERR_INVALID_ARG, "avq_aggregate: arrays must be 16-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int BH = B * H;
  hipError_t e =
      dtype == AVQ_BF16
          ? avq::launch_aggregate<avq::bf16>(BH, N, d, M0, Ch, V, code_idx, Vbar, counts, packed, s)
          : avq::launch_aggregate<float>(BH, N, d, M0, Ch, V, code_idx, Vbar, counts, packed, s);
  return from_hip(e, "avq_aggregate launch");
}

avq_status_t avq_assign_aggregate(avq_dtype_t dtype, int32_t B, int32_t H, int32_t N,
                                  int32_t d, int32_t M0, int32_t Ch, const void* K,
                                  const void* V, const void* Cp, const void* Cc,
                                  int32_t* parent_idx, int32_t* code_idx, float* Vbar,
                                  int32_t* counts, void* packed, void* stream) {
  avq_status_t st = check_common(dtype, B, H, N, d, M0, Ch);
  if (st != AVQ_OK) return st;
  if (!K || !V || !Cp || (!Cc && Ch > 0) || !parent_idx || !code_idx || !counts)
    return fail(AVQ_ERR_INVALID_ARG, "avq_assign_aggregate: null pointer argument");
  if (!Vbar && !packed)
    return fail(AVQ_ERR_INVALID_ARG, "avq_assign_aggregate: Vbar and packed are both null");
  if (!aligned16(K) || !aligned16(V) || !aligned16(Cp) || !aligned16(Cc) ||
      !aligned16(parent_idx) || !aligned16(code_idx) || !aligned16(Vbar) || !aligned16(counts) ||
      !aligned16(packed))
    return fail(AVQ_ERR_INVALID_ARG, "avq_assign_aggregate: arrays must be 16-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int BH = B * H;
  hipError_t e =
      dtype == AVQ_BF16
          ? avq::launch_assign_aggregate<avq::bf16>(BH, H, N, d, M0, Ch, K, V, Cp, Cc, parent_idx,
                                                    code_idx, Vbar, counts, packed, s)
          : avq::launch_assign_aggregate<float>(BH, H, N, d, M0, Ch, K, V, Cp, Cc, parent_idx,
                                                code_idx, Vbar, counts, packed, s);
  return from_hip(e, "avq_assign_aggregate launch");
}

avq_status_t avq_pack_aggregates(avq_dtype_t dtype, int32_t B, int32_t H, int32_t d,
                                 int32_t M0, int32_t Ch, const float* Vbar,
                                 const int32_t* counts, void* packed, void* stream) {
  avq_status_t st = check_common(dtype, B, H, 1, d, M0, Ch);
  if (st != AVQ_OK) return st;
  if (!Vbar || !counts || !packed)
    return fail(AVQ_ERR_INVALID_ARG, "avq_pack_aggregates: null pointer argument");
  if (!aligned16(Vbar) || !aligned16(counts) || !aligned16(packed))
    return fail(AVQ_ERR_INVALID_ARG, "avq_pack_aggregates: arrays must be 16-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int BH = B * H;
  hipError_t e = dtype == AVQ_BF16
                     ? avq::launch_pack<avq::bf16>(BH, M0, Ch, d, Vbar, counts, packed, s)
                     : avq::launch_pack<float>(BH, M0, Ch, d, Vbar, counts, packed, s);
  return from_hip(e, "avq_pack_aggregates launch");
}

}  // extern "C"

namespace {

// avq_attention_fwd and avq_attention_fwd_tiled: the same checks and launch;
// tiled selects the App. B importance.
avq_status_t attention(const char* name, bool tiled, const int32_t* order, avq_dtype_t dtype,
                       int32_t B, int32_t H, int32_t N, int32_t d, int32_t M0, int32_t Ch,
                       int32_t P, int32_t block_q, const void* Q, const void* Cp, const void* Cc,
                       const void* packed, void* Y, int32_t* topp_idx, float* importance,
                       void* stream) {
  avq_status_t st = check_common(dtype, B, H, N, d, M0, Ch);
  if (st != AVQ_OK) return st;
  if (P < 0 || P > M0) return fail(AVQ_ERR_INVALID_ARG, "P=%d outside [0, M0=%d]", P, M0);
  if (Ch == 0 && P != 0)
    return fail(AVQ_ERR_INVALID_ARG, "P=%d with a flat codebook (Ch=0): must be 0", P);
  if (block_q < 1) return fail(AVQ_ERR_INVALID_ARG, "block_q=%d must be positive", block_q);
  if (block_q > 256) return fail(AVQ_ERR_UNSUPPORTED, "block_q=%d: at most 256", block_q);
  if (!Q || !Cp || (!Cc && Ch > 0) || !packed || !Y)
    return fail(AVQ_ERR_INVALID_ARG, "%s: null pointer argument", name);
  if (!aligned16(Q) || !aligned16(Cp) || !aligned16(Cc) || !aligned16(packed) ||
      !aligned16(Y) || !aligned16(topp_idx) || !aligned16(importance) || !aligned16(order))
    return fail(AVQ_ERR_INVALID_ARG, "%s: arrays must be 16-byte aligned", name);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int BH = B * H;
  hipError_t e;
  if (dtype == AVQ_BF16)
    e = d == 64 ? avq::launch_attention<avq::bf16, 64>(BH, H, N, M0, Ch, P, block_q, Q, Cp, Cc,
                                                       packed, Y, topp_idx, importance, tiled, order, s)
                : avq::launch_attention<avq::bf16, 128>(BH, H, N, M0, Ch, P, block_q, Q, Cp, Cc,
                                                        packed, Y, topp_idx, importance, tiled, order, s);
  else
    e = d == 64 ? avq::launch_attention<float, 64>(BH, H, N, M0, Ch, P, block_q, Q, Cp, Cc,
                                                   packed, Y, topp_idx, importance, tiled, order, s)
                : avq::launch_attention<float, 128>(BH, H, N, M0, Ch, P, block_q, Q, Cp, Cc,
                                                    packed, Y, topp_idx, importance, tiled, order, s);
  return from_hip(e, "attention launch");
}

}  // namespace

extern "C" {

avq_status_t avq_attention_fwd(avq_dtype_t dtype, int32_t B, int32_t H, int32_t N, int32_t d,
                               int32_t M0, int32_t Ch, int32_t P, int32_t block_q,
                               const void* Q, const void* Cp, const void* Cc,
                               const void* packed, void* Y,
                               int32_t* topp_idx, float* importance, void* stream) {
  return attention("avq_attention_fwd", false, nullptr, dtype, B, H, N, d, M0, Ch, P, block_q, Q, Cp, Cc,
                   packed, Y, topp_idx, importance, stream);
}

avq_status_t avq_attention_fwd_tiled(avq_dtype_t dtype, int32_t B, int32_t H, int32_t N,
                                     int32_t d, int32_t M0, int32_t Ch, int32_t P,
                                     int32_t block_q, const void* Q, const void* Cp,
                                     const void* Cc, const void* packed, void* Y,
                                     int32_t* topp_idx, float* importance, void* stream) {
  return attention("avq_attention_fwd_tiled", true, nullptr, dtype, B, H, N, d, M0, Ch, P, block_q, Q, Cp,
                   Cc, packed, Y, topp_idx, importance, stream);
}

avq_status_t avq_codebook_update(avq_dtype_t dtype, int32_t B, int32_t H, int32_t d,
                                 int32_t M0, int32_t Ch, float lambda, const float* sums,
                                 const int32_t* counts, float* S, float* Nema, void* Cp_out,
                                 void* Cc_out, void* stream) {
  avq_status_t st = check_common(dtype, B, H, 1, d, M0, Ch);
  if (st != AVQ_OK) return st;
  if (!(lambda > 0.f && lambda <= 1.f))
    return fail(AVQ_ERR_INVALID_ARG, "lambda=%g outside (0, 1]", (double)lambda);
  if (!sums || !counts || !S || !Nema || !Cp_out || (!Cc_out && Ch > 0))
    return fail(AVQ_ERR_INVALID_ARG, "avq_codebook_update: null pointer argument");
  if (!aligned16(sums) || !aligned16(counts) || !aligned16(S) || !aligned16(Nema) ||
      !aligned16(Cp_out) || !aligned16(Cc_out))
    return fail(AVQ_ERR_INVALID_ARG, "avq_codebook_update: arrays must be 16-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e =
      dtype == AVQ_BF16
          ? avq::launch_codebook_update<avq::bf16>(B, H, d, M0, Ch, lambda, sums, counts, S, Nema,
                                                   Cp_out, Cc_out, s)
          : avq::launch_codebook_update<float>(B, H, d, M0, Ch, lambda, sums, counts, S, Nema,
                                               Cp_out, Cc_out, s);
  return from_hip(e, "avq_codebook_update launch");
}

avq_status_t avq_attention_fwd_ordered(avq_dtype_t dtype, int32_t B, int32_t H, int32_t N,
                                       int32_t d, int32_t M0, int32_t Ch, int32_t P,
                                       int32_t block_q, const int32_t* query_order,
                                       int32_t tiled_importance, const void* Q, const void* Cp,
                                       const void* Cc, const void* packed, void* Y,
                                       int32_t* topp_idx, float* importance, void* stream) {
  if (!query_order)
    return fail(AVQ_ERR_INVALID_ARG, "avq_attention_fwd_ordered: null query_order");
  if (tiled_importance != 0 && tiled_importance != 1)
    return fail(AVQ_ERR_INVALID_ARG, "tiled_importance=%d: must be 0 or 1", tiled_importance);
  return attention("avq_attention_fwd_ordered", tiled_importance == 1, query_order, dtype, B, H,
                   N, d, M0, Ch, P, block_q, Q, Cp, Cc, packed, Y, topp_idx, importance, stream);
}

avq_status_t avq_gilbert_order(int32_t width, int32_t height, int32_t* order, int32_t* rank) {
  if (width < 1 || height < 1)
    return fail(AVQ_ERR_INVALID_ARG, "grid %d x %d: sizes must be positive", width, height);
  if ((long long)width * height > (1LL << 24))
    return fail(AVQ_ERR_UNSUPPORTED, "grid %d x %d: at most 2^24 cells", width, height);
  if (!order) return fail(AVQ_ERR_INVALID_ARG, "avq_gilbert_order: null order");
  const long long n = avq::gilbert_order(width, height, order);
  if (n != (long long)width * height)
    return fail(AVQ_ERR_INVALID_ARG, "avq_gilbert_order: internal count mismatch");
  if (rank)
    for (long long k = 0; k < n; ++k) rank[order[k]] = (int32_t)k;
  return ok();
}

}  // extern "C"
