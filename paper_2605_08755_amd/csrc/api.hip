// C ABI of the library (include/laq.h): argument validation on the host,
// then an asynchronous launch on the caller's stream.  Nothing is enqueued
// when validation fails.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>

#include "laq.h"
#include "laq_internal.h"

namespace {

thread_local std::string g_last_error;
thread_local laq::LaunchEvents g_next_events;  // measurement hook, consumed by the next launch

laq::LaunchEvents take_events() {
  laq::LaunchEvents ev = g_next_events;
  g_next_events = laq::LaunchEvents{};
  return ev;
}

laq_status fail(laq_status st, const char* fn, const char* what) {
  char buf[256];
  std::snprintf(buf, sizeof(buf), "%s: %s", fn, what);
  g_last_error = buf;
  return st;
}

laq_status ok() {
  g_last_error.clear();
  return LAQ_OK;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

laq_status check_shape(const char* fn, int64_t N, int64_t K) {
  if (N < 1) return fail(LAQ_ERR_BAD_SHAPE, fn, "N must be >= 1");
  if (K < 128 || K % 128 != 0) return fail(LAQ_ERR_BAD_SHAPE, fn, "K must be a positive multiple of 128");
  if (N > 0x7FFFFFFFLL) return fail(LAQ_ERR_BAD_SHAPE, fn, "N must be < 2^31");
  if (K > (1LL << 24)) return fail(LAQ_ERR_BAD_SHAPE, fn, "K must be <= 2^24");
  if (N * K >= (1LL << 40)) return fail(LAQ_ERR_BAD_SHAPE, fn, "N*K must be < 2^40");
  return LAQ_OK;
}

laq_status hip_status(const char* fn, hipError_t e) {
  if (e != hipSuccess) return fail(LAQ_ERR_HIP, fn, hipGetErrorString(e));
  return ok();
}

template <int BITS>
laq_status quantize(const char* fn, const void* w, int64_t N, int64_t K, uint32_t* qweight,
                    void* scales, uint8_t* zeros, void* stream) {
  const laq::LaunchEvents ev = take_events();  // consumed whether or not the call launches
  if (!w || !qweight || !scales || !zeros) return fail(LAQ_ERR_NULL_POINTER, fn, "null pointer argument");
  laq_status st = check_shape(fn, N, K);
  if (st != LAQ_OK) return st;
  if (!aligned(w, 16) || !aligned(qweight, 16)) return fail(LAQ_ERR_MISALIGNED, fn, "w and qweight must be 16-byte aligned");
  if (!aligned(scales, 2)) return fail(LAQ_ERR_MISALIGNED, fn, "scales must be 2-byte aligned");
  return hip_status(fn, laq::launch_quantize<BITS>(static_cast<const uint16_t*>(w), N, K, qweight,
                                                   static_cast<uint16_t*>(scales), zeros,
                                                   static_cast<hipStream_t>(stream), ev));
}

template <int BITS>
laq_status pack(const char* fn, const void* w, const void* scales, const uint8_t* zeros, int64_t N,
                int64_t K, uint32_t* qweight, void* stream) {
  const laq::LaunchEvents ev = take_events();  // consumed whether or not the call launches
  if (!w || !qweight || !scales || !zeros) return fail(LAQ_ERR_NULL_POINTER, fn, "null pointer argument");
  laq_status st = check_shape(fn, N, K);
  if (st != LAQ_OK) return st;
  if (!aligned(w, 16) || !aligned(qweight, 16)) return fail(LAQ_ERR_MISALIGNED, fn, "w and qweight must be 16-byte aligned");
  if (!aligned(scales, 2)) return fail(LAQ_ERR_MISALIGNED, fn, "scales must be 2-byte aligned");
  return hip_status(fn, laq::launch_pack<BITS>(static_cast<const uint16_t*>(w),
                                               static_cast<const uint16_t*>(scales), zeros, N, K, qweight,
                                               static_cast<hipStream_t>(stream), ev));
}

template <int BITS>
laq_status linear(const char* fn, const void* x, const uint32_t* qweight, const void* scales,
                  const uint8_t* zeros, void* y, int64_t M, int64_t N, int64_t K, void* stream) {
  const laq::LaunchEvents ev = take_events();  // consumed whether or not the call launches
  if (!x || !qweight || !scales || !zeros || !y) return fail(LAQ_ERR_NULL_POINTER, fn, "null pointer argument");
  laq_status st = check_shape(fn, N, K);
  if (st != LAQ_OK) return st;
  if (M < 1 || M > LAQ_MAX_M) return fail(LAQ_ERR_BAD_M, fn, "M must be in 1..16");
  if (!aligned(x, 16) || !aligned(qweight, 16)) return fail(LAQ_ERR_MISALIGNED, fn, "x and qweight must be 16-byte aligned");
  if (!aligned(scales, 2) || !aligned(y, 2)) return fail(LAQ_ERR_MISALIGNED, fn, "scales and y must be 2-byte aligned");
  return hip_status(fn, laq::launch_linear<BITS>(static_cast<const uint16_t*>(x), qweight,
                                                 static_cast<const uint16_t*>(scales), zeros,
                                                 static_cast<uint16_t*>(y), (int)M, N, K,
                                                 static_cast<hipStream_t>(stream), ev));
}

template <int BITS>
laq_status linear_ws(const char* fn, const void* x, const uint32_t* qweight, const void* scales,
                     const uint8_t* zeros, void* y, int64_t M, int64_t N, int64_t K, void* workspace,
                     int64_t workspace_bytes, void* stream) {
  const laq::LaunchEvents ev = take_events();  // consumed whether or not the call launches
  if (!x || !qweight || !scales || !zeros || !y) return fail(LAQ_ERR_NULL_POINTER, fn, "null pointer argument");
  if (workspace_bytes < 0) return fail(LAQ_ERR_BAD_SHAPE, fn, "workspace_bytes must be >= 0");
  if (workspace_bytes > 0 && !workspace) return fail(LAQ_ERR_NULL_POINTER, fn, "null workspace with workspace_bytes > 0");
  laq_status st = check_shape(fn, N, K);
  if (st != LAQ_OK) return st;
  if (M < 1 || M > LAQ_MAX_M) return fail(LAQ_ERR_BAD_M, fn, "M must be in 1..16");
  if (!aligned(x, 16) || !aligned(qweight, 16)) return fail(LAQ_ERR_MISALIGNED, fn, "x and qweight must be 16-byte aligned");
  if (!aligned(scales, 2) || !aligned(y, 2)) return fail(LAQ_ERR_MISALIGNED, fn, "scales and y must be 2-byte aligned");
  if (workspace && !aligned(workspace, 16)) return fail(LAQ_ERR_MISALIGNED, fn, "workspace must be 16-byte aligned");
  return hip_status(fn, laq::launch_linear<BITS>(static_cast<const uint16_t*>(x), qweight,
                                                 static_cast<const uint16_t*>(scales), zeros,
                                                 static_cast<uint16_t*>(y), (int)M, N, K,
                                                 static_cast<hipStream_t>(stream), ev,
                                                 workspace_bytes > 0 ? static_cast<float*>(workspace) : nullptr,
                                                 (size_t)workspace_bytes));
}

template <int BITS>
laq_status linear_group(const char* fn, const laq_linear_call* calls, int32_t count, int64_t M, void* stream) {
  const laq::LaunchEvents ev = take_events();  // consumed whether or not the call launches
  if (!calls) return fail(LAQ_ERR_NULL_POINTER, fn, "null calls array");
  if (count < 1 || count > LAQ_MAX_GROUP) return fail(LAQ_ERR_BAD_SHAPE, fn, "count must be in 1..8");
  if (M < 1 || M > LAQ_MAX_M) return fail(LAQ_ERR_BAD_M, fn, "M must be in 1..16");
  laq::LinearCall lc[laq::kMaxGroup];
  int64_t blocks = 0;
  for (int i = 0; i < count; ++i) {
    const laq_linear_call& c = calls[i];
    if (!c.x || !c.qweight || !c.scales || !c.zeros || !c.y) return fail(LAQ_ERR_NULL_POINTER, fn, "null pointer in a call");
    laq_status st = check_shape(fn, c.N, c.K);
    if (st != LAQ_OK) return st;
    if (!aligned(c.x, 16) || !aligned(c.qweight, 16)) return fail(LAQ_ERR_MISALIGNED, fn, "x and qweight must be 16-byte aligned");
    if (!aligned(c.scales, 2) || !aligned(c.y, 2)) return fail(LAQ_ERR_MISALIGNED, fn, "scales and y must be 2-byte aligned");
    blocks += c.N;  // an upper bound of the grid: at least one row per block
    lc[i] = laq::LinearCall{static_cast<const uint16_t*>(c.x), c.qweight, static_cast<const uint16_t*>(c.scales),
                            c.zeros, static_cast<uint16_t*>(c.y), (int)c.N, (int)(c.K / 128), 0, 0, 0.0f};
  }
  if (blocks >= (1LL << 31)) return fail(LAQ_ERR_BAD_SHAPE, fn, "the calls' rows must total < 2^31");
  return hip_status(fn, laq::launch_linear_group<BITS>(lc, count, (int)M, static_cast<hipStream_t>(stream), ev));
}

}  // namespace

extern "C" {

int32_t laq_abi_version(void) { return LAQ_ABI_VERSION; }

const char* laq_status_string(laq_status status) {
  switch (status) {
    case LAQ_OK: return "ok";
    case LAQ_ERR_NULL_POINTER: return "null pointer argument";
    case LAQ_ERR_BAD_SHAPE: return "bad shape (need N >= 1, K >= 128, K % 128 == 0)";
    case LAQ_ERR_BAD_M: return "M outside 1..16";
    case LAQ_ERR_MISALIGNED: return "misaligned pointer";
    case LAQ_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* laq_last_error(void) { return g_last_error.c_str(); }

laq_status laq_profile_next_launch(void* start_event, void* stop_event) {
  g_next_events.start = static_cast<hipEvent_t>(start_event);
  g_next_events.stop = static_cast<hipEvent_t>(stop_event);
  return LAQ_OK;
}

laq_status laq_quantize_w3g128(const void* w, int64_t N, int64_t K, uint32_t* qweight, void* scales,
                               uint8_t* zeros, void* stream) {
  return quantize<3>("laq_quantize_w3g128", w, N, K, qweight, scales, zeros, stream);
}

laq_status laq_quantize_w4g128(const void* w, int64_t N, int64_t K, uint32_t* qweight, void* scales,
                               uint8_t* zeros, void* stream) {
  return quantize<4>("laq_quantize_w4g128", w, N, K, qweight, scales, zeros, stream);
}

laq_status laq_pack_w3g128(const void* w, const void* scales, const uint8_t* zeros, int64_t N, int64_t K,
                           uint32_t* qweight, void* stream) {
  return pack<3>("laq_pack_w3g128", w, scales, zeros, N, K, qweight, stream);
}

laq_status laq_pack_w4g128(const void* w, const void* scales, const uint8_t* zeros, int64_t N, int64_t K,
                           uint32_t* qweight, void* stream) {
  return pack<4>("laq_pack_w4g128", w, scales, zeros, N, K, qweight, stream);
}

laq_status laq_linear_w3g128(const void* x, const uint32_t* qweight, const void* scales,
                             const uint8_t* zeros, void* y, int64_t M, int64_t N, int64_t K,
                             void* stream) {
  return linear<3>("laq_linear_w3g128", x, qweight, scales, zeros, y, M, N, K, stream);
}

int64_t laq_linear_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  if (M < 1 || M > LAQ_MAX_M || N < 1 || N > 0x7FFFFFFFLL || K < 128 || K % 128 != 0 || K > (1LL << 24) ||
      N * K >= (1LL << 40))
    return 0;
  const laq::SplitPlan p = laq::mfma_split_plan((int)M, N, (int)(K / 128));
  return (int64_t)laq::split_workspace_bytes(p, (int)M, N);
}

laq_status laq_linear_ws_w3g128(const void* x, const uint32_t* qweight, const void* scales,
                                const uint8_t* zeros, void* y, int64_t M, int64_t N, int64_t K,
                                void* workspace, int64_t workspace_bytes, void* stream) {
  return linear_ws<3>("laq_linear_ws_w3g128", x, qweight, scales, zeros, y, M, N, K, workspace, workspace_bytes,
                      stream);
}

laq_status laq_linear_ws_w4g128(const void* x, const uint32_t* qweight, const void* scales,
                                const uint8_t* zeros, void* y, int64_t M, int64_t N, int64_t K,
                                void* workspace, int64_t workspace_bytes, void* stream) {
  return linear_ws<4>("laq_linear_ws_w4g128", x, qweight, scales, zeros, y, M, N, K, workspace, workspace_bytes,
                      stream);
}

laq_status laq_linear_group_w3g128(const laq_linear_call* calls, int32_t count, int64_t M, void* stream) {
  return linear_group<3>("laq_linear_group_w3g128", calls, count, M, stream);
}

laq_status laq_linear_group_w4g128(const laq_linear_call* calls, int32_t count, int64_t M, void* stream) {
  return linear_group<4>("laq_linear_group_w4g128", calls, count, M, stream);
}

laq_status laq_linear_w4g128(const void* x, const uint32_t* qweight, const void* scales,
                             const uint8_t* zeros, void* y, int64_t M, int64_t N, int64_t K,
                             void* stream) {
  return linear<4>("laq_linear_w4g128", x, qweight, scales, zeros, y, M, N, K, stream);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Decode-step operations
// ---------------------------------------------------------------------------
namespace {
constexpr int64_t kHeadDimAbi = 128;

laq_status check_heads(const char* fn, int64_t Hq, int64_t Hkv, int64_t head_dim) {
  if (head_dim != kHeadDimAbi) return fail(LAQ_ERR_BAD_SHAPE, fn, "head_dim must be 128");
  if (Hq < 1 || Hkv < 1 || Hq % Hkv != 0) return fail(LAQ_ERR_BAD_SHAPE, fn, "Hq must be a positive multiple of Hkv");
  const int64_t r = Hq / Hkv;
  if (r != 1 && r != 2 && r != 4 && r != 8) return fail(LAQ_ERR_BAD_SHAPE, fn, "Hq / Hkv must be 1, 2, 4 or 8");
  if (Hq > 4096) return fail(LAQ_ERR_BAD_SHAPE, fn, "Hq must be <= 4096");
  return LAQ_OK;
}
}  // namespace

extern "C" {

laq_status laq_add_rmsnorm_f16(float* residual, const void* delta, const void* weight, void* y, int64_t M,
                               int64_t D, float eps, void* stream) {
  const char* fn = "laq_add_rmsnorm_f16";
  const laq::LaunchEvents ev = take_events();
  if (!residual || !weight || !y) return fail(LAQ_ERR_NULL_POINTER, fn, "null pointer argument");
  if (M < 1 || M > 0x7FFFFFFFLL || D < 1 || D > (1LL << 20)) return fail(LAQ_ERR_BAD_SHAPE, fn, "need 1 <= M < 2^31 and 1 <= D <= 2^20");
  if (!(eps >= 0.0f) || !(eps < INFINITY)) return fail(LAQ_ERR_BAD_SHAPE, fn, "eps must be finite and >= 0");
  if (!aligned(residual, 4) || !aligned(weight, 2) || !aligned(y, 2) || (delta && !aligned(delta, 2)))
    return fail(LAQ_ERR_MISALIGNED, fn, "residual must be 4-byte, fp16 arrays 2-byte aligned");
  return hip_status(fn, laq::launch_add_rmsnorm(residual, static_cast<const uint16_t*>(delta),
                                                static_cast<const uint16_t*>(weight), static_cast<uint16_t*>(y), M, D,
                                                eps, static_cast<hipStream_t>(stream), ev));
}

laq_status laq_qk_norm_rope_f16(const void* qkv, const void* q_norm_weight, const void* k_norm_weight,
                                const float* cos_sin, int64_t pos, int64_t Hq, int64_t Hkv, int64_t head_dim,
                                float eps, void* q_out, void* k_cache, void* v_cache, int64_t S_max, void* stream) {
  const char* fn = "laq_qk_norm_rope_f16";
  const laq::LaunchEvents ev = take_events();
  if (!qkv || !q_norm_weight || !k_norm_weight || !cos_sin || !q_out || !k_cache || !v_cache)
    return fail(LAQ_ERR_NULL_POINTER, fn, "null pointer argument");
  laq_status st = check_heads(fn, Hq, Hkv, head_dim);
  if (st != LAQ_OK) return st;
  if (S_max < 1 || S_max > (1LL << 21) || pos < 0 || pos >= S_max)
    return fail(LAQ_ERR_BAD_SHAPE, fn, "need 1 <= S_max <= 2^21 and 0 <= pos < S_max");
  if (!(eps >= 0.0f) || !(eps < INFINITY)) return fail(LAQ_ERR_BAD_SHAPE, fn, "eps must be finite and >= 0");
  if (!aligned(qkv, 2) || !aligned(q_norm_weight, 2) || !aligned(k_norm_weight, 2) || !aligned(cos_sin, 4) ||
      !aligned(q_out, 2) || !aligned(k_cache, 16) || !aligned(v_cache, 16))
    return fail(LAQ_ERR_MISALIGNED, fn, "caches must be 16-byte, cos_sin 4-byte, fp16 arrays 2-byte aligned");
  return hip_status(fn, laq::launch_qk_norm_rope(
                            static_cast<const uint16_t*>(qkv), static_cast<const uint16_t*>(q_norm_weight),
                            static_cast<const uint16_t*>(k_norm_weight), cos_sin, pos, Hq, Hkv, eps,
                            static_cast<uint16_t*>(q_out), static_cast<uint16_t*>(k_cache),
                            static_cast<uint16_t*>(v_cache), S_max, static_cast<hipStream_t>(stream), ev));
}

int64_t laq_decode_attention_workspace_bytes(int64_t Hq, int64_t L) {
  if (Hq < 1 || L < 1 || Hq > 4096 || L > (1LL << 21)) return 0;
  return Hq * laq::decode_attention_tiles(L) * (kHeadDimAbi + 2) * (int64_t)sizeof(float);
}

laq_status laq_decode_attention_f16(const void* q, const void* k_cache, const void* v_cache, int64_t Hq,
                                    int64_t Hkv, int64_t head_dim, int64_t L, int64_t S_max, void* out,
                                    void* workspace, int64_t workspace_bytes, void* stream) {
  const char* fn = "laq_decode_attention_f16";
  const laq::LaunchEvents ev = take_events();
  if (!q || !k_cache || !v_cache || !out || !workspace) return fail(LAQ_ERR_NULL_POINTER, fn, "null pointer argument");
  laq_status st = check_heads(fn, Hq, Hkv, head_dim);
  if (st != LAQ_OK) return st;
  if (S_max < 1 || S_max > (1LL << 21) || L < 1 || L > S_max)
    return fail(LAQ_ERR_BAD_SHAPE, fn, "need 1 <= L <= S_max <= 2^21");
  if (workspace_bytes < laq_decode_attention_workspace_bytes(Hq, L))
    return fail(LAQ_ERR_BAD_SHAPE, fn, "workspace_bytes below laq_decode_attention_workspace_bytes(Hq, L)");
  if (!aligned(q, 2) || !aligned(out, 2) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(workspace, 16))
    return fail(LAQ_ERR_MISALIGNED, fn, "caches and workspace must be 16-byte, q and out 2-byte aligned");
  return hip_status(fn, laq::launch_decode_attention(
                            static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k_cache),
                            static_cast<const uint16_t*>(v_cache), Hq, Hkv, L, S_max, static_cast<uint16_t*>(out),
                            static_cast<float*>(workspace), static_cast<hipStream_t>(stream), ev));
}

int64_t laq_decode_attention_qkv_workspace_bytes(int64_t Hq, int64_t Hkv, int64_t L) {
  if (Hq < 1 || Hkv < 1 || L < 1 || Hq > 4096 || Hkv > Hq || L > (1LL << 21)) return 0;
  // The tile length grows with the context, so the tile count is largest at
  // the end of a tile-length regime: the maximum over every L' <= L.
  int64_t tiles = 0;
  for (int64_t lp : {L, std::min(L, 32767 / Hkv), std::min(L, 4095 / Hkv)})
    if (lp >= 1) tiles = std::max(tiles, laq::decode_attention_qkv_tiles(Hkv, lp));
  return Hq * tiles * (kHeadDimAbi + 2) * (int64_t)sizeof(float);
}

laq_status laq_decode_attention_qkv_f16(const void* qkv, const void* q_norm_weight, const void* k_norm_weight,
                                        const float* cos_sin, int64_t pos, int64_t Hq, int64_t Hkv,
                                        int64_t head_dim, float eps, void* k_cache, void* v_cache, int64_t S_max,
                                        void* out, void* workspace, int64_t workspace_bytes, void* stream) {
  const char* fn = "laq_decode_attention_qkv_f16";
  const laq::LaunchEvents ev = take_events();
  if (!qkv || !q_norm_weight || !k_norm_weight || !cos_sin || !k_cache || !v_cache || !out || !workspace)
    return fail(LAQ_ERR_NULL_POINTER, fn, "null pointer argument");
  laq_status st = check_heads(fn, Hq, Hkv, head_dim);
  if (st != LAQ_OK) return st;
  if (S_max < 1 || S_max > (1LL << 21) || pos < 0 || pos >= S_max)
    return fail(LAQ_ERR_BAD_SHAPE, fn, "need 1 <= S_max <= 2^21 and 0 <= pos < S_max");
  if (!(eps >= 0.0f) || !(eps < INFINITY)) return fail(LAQ_ERR_BAD_SHAPE, fn, "eps must be finite and >= 0");
  if (workspace_bytes < laq_decode_attention_qkv_workspace_bytes(Hq, Hkv, pos + 1))
    return fail(LAQ_ERR_BAD_SHAPE, fn, "workspace_bytes below laq_decode_attention_qkv_workspace_bytes(Hq, Hkv, pos + 1)");
  if (!aligned(qkv, 2) || !aligned(q_norm_weight, 2) || !aligned(k_norm_weight, 2) || !aligned(cos_sin, 4) ||
      !aligned(out, 2) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(workspace, 16))
    return fail(LAQ_ERR_MISALIGNED, fn,
                "caches and workspace must be 16-byte, cos_sin 4-byte, fp16 arrays 2-byte aligned");
  return hip_status(fn, laq::launch_decode_attention_qkv(
                            static_cast<const uint16_t*>(qkv), static_cast<const uint16_t*>(q_norm_weight),
                            static_cast<const uint16_t*>(k_norm_weight), cos_sin, pos, Hq, Hkv, eps,
                            static_cast<uint16_t*>(k_cache), static_cast<uint16_t*>(v_cache), S_max,
                            static_cast<uint16_t*>(out), static_cast<float*>(workspace),
                            static_cast<hipStream_t>(stream), ev));
}

}  // extern "C"

namespace {

template <int BITS>
laq_status linear_swiglu(const char* fn, const void* x, const uint32_t* qweight, const void* scales,
                         const uint8_t* zeros, void* y, int64_t M, int64_t N, int64_t K, void* stream) {
  const laq::LaunchEvents ev = take_events();
  if (!x || !qweight || !scales || !zeros || !y) return fail(LAQ_ERR_NULL_POINTER, fn, "null pointer argument");
  laq_status st = check_shape(fn, N, K);
  if (st != LAQ_OK) return st;
  if (M < 1 || M > 4) return fail(LAQ_ERR_BAD_M, fn, "M must be in 1..4");
  if (N % 2 != 0) return fail(LAQ_ERR_BAD_SHAPE, fn, "N (gate and up rows interleaved) must be even");
  if (!laq::swiglu_fits((int)M, K))
    return fail(LAQ_ERR_BAD_SHAPE, fn, "need K <= 16384 / M' (M' = M rounded up to 1, 2 or 4)");
  if (!aligned(x, 16) || !aligned(qweight, 16)) return fail(LAQ_ERR_MISALIGNED, fn, "x and qweight must be 16-byte aligned");
  if (!aligned(scales, 2) || !aligned(y, 2)) return fail(LAQ_ERR_MISALIGNED, fn, "scales and y must be 2-byte aligned");
  return hip_status(fn, laq::launch_linear_swiglu<BITS>(static_cast<const uint16_t*>(x), qweight,
                                                        static_cast<const uint16_t*>(scales), zeros,
                                                        static_cast<uint16_t*>(y), (int)M, N, K,
                                                        static_cast<hipStream_t>(stream), ev));
}

template <int BITS>
laq_status norm_linear(const char* fn, const float* residual, const void* delta, const void* norm_weight, float eps,
                       float* residual_out, const uint32_t* qweight, const void* scales, const uint8_t* zeros,
                       void* y, int64_t N, int64_t K, bool swiglu, void* stream) {
  const laq::LaunchEvents ev = take_events();
  if (!residual || !norm_weight || !qweight || !scales || !zeros || !y)
    return fail(LAQ_ERR_NULL_POINTER, fn, "null pointer argument");
  laq_status st = check_shape(fn, N, K);
  if (st != LAQ_OK) return st;
  if (!laq::norm_linear_fits(K)) return fail(LAQ_ERR_BAD_SHAPE, fn, "need K <= 8192");
  if (swiglu && N % 2 != 0) return fail(LAQ_ERR_BAD_SHAPE, fn, "N (gate and up rows interleaved) must be even");
  if (!(eps >= 0.0f) || !(eps < INFINITY)) return fail(LAQ_ERR_BAD_SHAPE, fn, "eps must be finite and >= 0");
  if (residual_out != nullptr && residual_out < residual + K && residual < residual_out + K)
    return fail(LAQ_ERR_BAD_SHAPE, fn, "residual_out must not overlap residual");
  if (!aligned(residual, 16) || !aligned(delta, 16) || !aligned(norm_weight, 16) || !aligned(residual_out, 16) ||
      !aligned(qweight, 16))
    return fail(LAQ_ERR_MISALIGNED, fn, "residual, residual_out, delta, norm_weight and qweight must be 16-byte aligned");
  if (!aligned(scales, 2) || !aligned(y, 2)) return fail(LAQ_ERR_MISALIGNED, fn, "scales and y must be 2-byte aligned");
  laq::NormPrologue np;
  np.res_in = residual;
  np.delta = static_cast<const uint16_t*>(delta);
  np.weight = static_cast<const uint16_t*>(norm_weight);
  np.res_out = residual_out;
  np.eps = eps;
  return hip_status(fn, laq::launch_linear_norm<BITS>(np, qweight, static_cast<const uint16_t*>(scales), zeros,
                                                      static_cast<uint16_t*>(y), N, K, swiglu,
                                                      static_cast<hipStream_t>(stream), ev));
}

template <int BITS>
laq_status linear_residual(const char* fn, const void* x, const uint32_t* qweight, const void* scales,
                           const uint8_t* zeros, void* y, const float* residual_in, float* residual_out, int64_t N,
                           int64_t K, void* stream) {
  const laq::LaunchEvents ev = take_events();
  if (!x || !qweight || !scales || !zeros || !residual_in || !residual_out)  // y may be NULL
    return fail(LAQ_ERR_NULL_POINTER, fn, "null pointer argument");
  laq_status st = check_shape(fn, N, K);
  if (st != LAQ_OK) return st;
  if (!laq::residual_linear_fits(N, K))
    return fail(LAQ_ERR_BAD_SHAPE, fn, "need K >= 2048 and rows whose activation tile fits in LDS (K <= ~28000)");
  if (residual_out != residual_in && residual_out < residual_in + N && residual_in < residual_out + N)
    return fail(LAQ_ERR_BAD_SHAPE, fn, "residual_out must equal residual_in or not overlap it");
  if (!aligned(x, 16) || !aligned(qweight, 16)) return fail(LAQ_ERR_MISALIGNED, fn, "x and qweight must be 16-byte aligned");
  if (!aligned(scales, 2) || !aligned(y, 2)) return fail(LAQ_ERR_MISALIGNED, fn, "scales and y must be 2-byte aligned");
  if (!aligned(residual_in, 4) || !aligned(residual_out, 4))
    return fail(LAQ_ERR_MISALIGNED, fn, "residual_in and residual_out must be 4-byte aligned");
  return hip_status(fn, laq::launch_linear_residual<BITS>(
                            static_cast<const uint16_t*>(x), qweight, static_cast<const uint16_t*>(scales), zeros,
                            static_cast<uint16_t*>(y), residual_in, residual_out, N, K,
                            static_cast<hipStream_t>(stream), ev));
}

template <int BITS>
laq_status norm_mlp(const char* fn, const float* residual, const void* delta, const void* norm_weight, float eps,
                    float* residual_out, const uint32_t* gu_qweight, const void* gu_scales, const uint8_t* gu_zeros,
                    const uint32_t* down_qweight, const void* down_scales, const uint8_t* down_zeros, void* y,
                    int64_t D, int64_t I, void* workspace, int64_t workspace_bytes, void* stream) {
  const laq::LaunchEvents ev = take_events();
  if (!residual || !norm_weight || !gu_qweight || !gu_scales || !gu_zeros || !down_qweight || !down_scales ||
      !down_zeros || !y || !workspace)
    return fail(LAQ_ERR_NULL_POINTER, fn, "null pointer argument");
  const laq::MlpPlan p = laq::mlp_plan(D, I, BITS);
  if (p.S == 0)
    return fail(LAQ_ERR_BAD_SHAPE, fn,
                "need D and I positive multiples of 128, D <= 2560, I <= 2^20, and the down group's codes in LDS");
  if (!(eps >= 0.0f) || !(eps < INFINITY)) return fail(LAQ_ERR_BAD_SHAPE, fn, "eps must be finite and >= 0");
  if (residual_out != nullptr && residual_out < residual + D && residual < residual_out + D)
    return fail(LAQ_ERR_BAD_SHAPE, fn, "residual_out must not overlap residual");
  if (workspace_bytes < (int64_t)laq::mlp_workspace_bytes(p, D))
    return fail(LAQ_ERR_BAD_SHAPE, fn, "workspace smaller than laq_mlp_workspace_bytes(D, I)");
  if (!aligned(residual, 16) || !aligned(delta, 16) || !aligned(norm_weight, 16) || !aligned(residual_out, 16) ||
      !aligned(gu_qweight, 16) || !aligned(down_qweight, 16) || !aligned(workspace, 16))
    return fail(LAQ_ERR_MISALIGNED, fn,
                "residual, residual_out, delta, norm_weight, both qweights and workspace must be 16-byte aligned");
  if (!aligned(gu_scales, 2) || !aligned(down_scales, 2) || !aligned(y, 2))
    return fail(LAQ_ERR_MISALIGNED, fn, "scales and y must be 2-byte aligned");
  laq::NormPrologue np;
  np.res_in = residual;
  np.delta = static_cast<const uint16_t*>(delta);
  np.weight = static_cast<const uint16_t*>(norm_weight);
  np.res_out = residual_out;
  np.eps = eps;
  return hip_status(fn, laq::launch_mlp<BITS>(np, gu_qweight, static_cast<const uint16_t*>(gu_scales), gu_zeros,
                                               down_qweight, static_cast<const uint16_t*>(down_scales), down_zeros,
                                               static_cast<uint16_t*>(y), D, I, workspace,
                                               static_cast<hipStream_t>(stream), ev));
}

}  // namespace

extern "C" {

laq_status laq_linear_residual_w3g128(const void* x, const uint32_t* qweight, const void* scales,
                                      const uint8_t* zeros, void* y, const float* residual_in, float* residual_out,
                                      int64_t N, int64_t K, void* stream) {
  return linear_residual<3>("laq_linear_residual_w3g128", x, qweight, scales, zeros, y, residual_in, residual_out, N,
                            K, stream);
}

laq_status laq_linear_residual_w4g128(const void* x, const uint32_t* qweight, const void* scales,
                                      const uint8_t* zeros, void* y, const float* residual_in, float* residual_out,
                                      int64_t N, int64_t K, void* stream) {
  return linear_residual<4>("laq_linear_residual_w4g128", x, qweight, scales, zeros, y, residual_in, residual_out, N,
                            K, stream);
}

int64_t laq_mlp_workspace_bytes(int64_t D, int64_t I) {
  const laq::MlpPlan p = laq::mlp_plan(D, I, 3);
  return (int64_t)laq::mlp_workspace_bytes(p, D);
}

laq_status laq_add_rmsnorm_mlp_w3g128(const float* residual, const void* delta, const void* norm_weight, float eps,
                                      float* residual_out, const uint32_t* gu_qweight, const void* gu_scales,
                                      const uint8_t* gu_zeros, const uint32_t* down_qweight, const void* down_scales,
                                      const uint8_t* down_zeros, void* y, int64_t D, int64_t I, void* workspace,
                                      int64_t workspace_bytes, void* stream) {
  return norm_mlp<3>("laq_add_rmsnorm_mlp_w3g128", residual, delta, norm_weight, eps, residual_out, gu_qweight,
                     gu_scales, gu_zeros, down_qweight, down_scales, down_zeros, y, D, I, workspace, workspace_bytes,
                     stream);
}

laq_status laq_linear_swiglu_w3g128(const void* x, const uint32_t* qweight, const void* scales,
                                    const uint8_t* zeros, void* y, int64_t M, int64_t N, int64_t K, void* stream) {
  return linear_swiglu<3>("laq_linear_swiglu_w3g128", x, qweight, scales, zeros, y, M, N, K, stream);
}

laq_status laq_linear_swiglu_w4g128(const void* x, const uint32_t* qweight, const void* scales,
                                    const uint8_t* zeros, void* y, int64_t M, int64_t N, int64_t K, void* stream) {
  return linear_swiglu<4>("laq_linear_swiglu_w4g128", x, qweight, scales, zeros, y, M, N, K, stream);
}

laq_status laq_add_rmsnorm_linear_w3g128(const float* residual, const void* delta, const void* norm_weight, float eps,
                                         float* residual_out, const uint32_t* qweight, const void* scales,
                                         const uint8_t* zeros, void* y, int64_t N, int64_t K, void* stream) {
  return norm_linear<3>("laq_add_rmsnorm_linear_w3g128", residual, delta, norm_weight, eps, residual_out, qweight,
                        scales, zeros, y, N, K, false, stream);
}

laq_status laq_add_rmsnorm_linear_w4g128(const float* residual, const void* delta, const void* norm_weight, float eps,
                                         float* residual_out, const uint32_t* qweight, const void* scales,
                                         const uint8_t* zeros, void* y, int64_t N, int64_t K, void* stream) {
  return norm_linear<4>("laq_add_rmsnorm_linear_w4g128", residual, delta, norm_weight, eps, residual_out, qweight,
                        scales, zeros, y, N, K, false, stream);
}

laq_status laq_add_rmsnorm_linear_swiglu_w3g128(const float* residual, const void* delta, const void* norm_weight,
                                                float eps, float* residual_out, const uint32_t* qweight,
                                                const void* scales, const uint8_t* zeros, void* y, int64_t N,
                                                int64_t K, void* stream) {
  return norm_linear<3>("laq_add_rmsnorm_linear_swiglu_w3g128", residual, delta, norm_weight, eps, residual_out,
                        qweight, scales, zeros, y, N, K, true, stream);
}

laq_status laq_add_rmsnorm_linear_swiglu_w4g128(const float* residual, const void* delta, const void* norm_weight,
                                                float eps, float* residual_out, const uint32_t* qweight,
                                                const void* scales, const uint8_t* zeros, void* y, int64_t N,
                                                int64_t K, void* stream) {
  return norm_linear<4>("laq_add_rmsnorm_linear_swiglu_w4g128", residual, delta, norm_weight, eps, residual_out,
                        qweight, scales, zeros, y, N, K, true, stream);
}

laq_status laq_silu_mul_f16(const void* gate_up, void* y, int64_t M, int64_t I, void* stream) {
  const char* fn = "laq_silu_mul_f16";
  const laq::LaunchEvents ev = take_events();
  if (!gate_up || !y) return fail(LAQ_ERR_NULL_POINTER, fn, "null pointer argument");
  if (M < 1 || I < 1 || M > 65535 || I > (1LL << 30))
    return fail(LAQ_ERR_BAD_SHAPE, fn, "need 1 <= M <= 65535 and 1 <= I <= 2^30");
  if (!aligned(gate_up, 2) || !aligned(y, 2)) return fail(LAQ_ERR_MISALIGNED, fn, "fp16 arrays must be 2-byte aligned");
  return hip_status(fn, laq::launch_silu_mul(static_cast<const uint16_t*>(gate_up), static_cast<uint16_t*>(y), M, I,
                                             static_cast<hipStream_t>(stream), ev));
}

}  // extern "C"

// ---------------------------------------------------------------------------
// The linear without a caller workspace and without allocation: split-K
// partial sums in a scratch array the library holds on each GPU.
// ---------------------------------------------------------------------------
namespace {

// Each GPU the library runs on holds its own copy of this array until the
// process ends.  In host code the name is only a symbol handle, never an
// address: the device address comes from hipGetSymbolAddress, per device.
static __device__ __align__(256) float scratch[LAQ_NOALLOC_SCRATCH_BYTES / sizeof(float)];

constexpr int kScratchDevices = 64;
std::atomic<float*> g_scratch_ptr[kScratchDevices];
std::mutex g_scratch_mutex;

// Device address of `scratch` on the device that runs `stream` (looked up
// once per device, with that device current).
laq_status scratch_on_stream_device(const char* fn, hipStream_t stream, float** out) {
  int cur = 0;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return fail(LAQ_ERR_HIP, fn, hipGetErrorString(e));
  int dev = cur;
  if (stream) {
    hipDevice_t d = 0;
    e = hipStreamGetDevice(stream, &d);
    if (e != hipSuccess) return fail(LAQ_ERR_HIP, fn, hipGetErrorString(e));
    dev = (int)d;
  }
  if (dev < 0 || dev >= kScratchDevices) return fail(LAQ_ERR_HIP, fn, "device index beyond the scratch table");
  float* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
      if (dev != cur && (e = hipSetDevice(dev)) != hipSuccess) return fail(LAQ_ERR_HIP, fn, hipGetErrorString(e));
      void* addr = nullptr;
      e = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
      const hipError_t e2 = dev != cur ? hipSetDevice(cur) : hipSuccess;
      if (e != hipSuccess) return fail(LAQ_ERR_HIP, fn, hipGetErrorString(e));
      if (e2 != hipSuccess) return fail(LAQ_ERR_HIP, fn, hipGetErrorString(e2));
      if (!addr) return fail(LAQ_ERR_HIP, fn, "no device address for the scratch array");
      p = static_cast<float*>(addr);
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return LAQ_OK;
}

}  // namespace

extern "C" laq_status laq_linear_noalloc_w3g128(const void* x, const uint32_t* qweight, const void* scales,
                                                const uint8_t* zeros, void* y, int64_t M, int64_t N, int64_t K,
                                                void* stream) {
  const char* fn = "laq_linear_noalloc_w3g128";
  const laq::LaunchEvents ev = take_events();  // consumed whether or not the call launches
  if (!x || !qweight || !scales || !zeros || !y) return fail(LAQ_ERR_NULL_POINTER, fn, "null pointer argument");
  laq_status st = check_shape(fn, N, K);
  if (st != LAQ_OK) return st;
  if (M < 1 || M > LAQ_MAX_M) return fail(LAQ_ERR_BAD_M, fn, "M must be in 1..16");
  if (!aligned(x, 16) || !aligned(qweight, 16)) return fail(LAQ_ERR_MISALIGNED, fn, "x and qweight must be 16-byte aligned");
  if (!aligned(scales, 2) || !aligned(y, 2)) return fail(LAQ_ERR_MISALIGNED, fn, "scales and y must be 2-byte aligned");
  const size_t need = laq::split_workspace_bytes(laq::mfma_split_plan((int)M, N, (int)(K / 128)), (int)M, N);
  if (need > (size_t)LAQ_NOALLOC_SCRATCH_BYTES)
    return fail(LAQ_ERR_BAD_SHAPE, fn,
                "the split-K partial sums of this shape exceed the scratch array (LAQ_NOALLOC_SCRATCH_BYTES)");
  float* ws = nullptr;
  if (need > 0) {
    st = scratch_on_stream_device(fn, static_cast<hipStream_t>(stream), &ws);
    if (st != LAQ_OK) return st;
  }
  return hip_status(fn, laq::launch_linear<3>(static_cast<const uint16_t*>(x), qweight,
                                              static_cast<const uint16_t*>(scales), zeros,
                                              static_cast<uint16_t*>(y), (int)M, N, K,
                                              static_cast<hipStream_t>(stream), ev, ws, need));
}
