// Driver for a sanitizer build (AddressSanitizer + UndefinedBehaviorSanitizer
// on the host code) of the library's C ABI: every entry point with arguments
// that its host-side validation must reject -- null pointers, bad shapes and
// activation-row counts, misaligned pointers, sizes at and past every limit,
// extreme integers for the workspace-size queries -- checking the returned
// status and the last-error text.  Nothing here passes validation, so no
// HIP call is reached and no GPU is needed.  Any sanitizer report aborts the
// run; a wrong status returns 1.  Prints "ok N" (N checks) on success.
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <initializer_list>
#include <limits>

#include "laq.h"

namespace {

int g_checks = 0, g_bad = 0;

void expect(int line, laq_status got, laq_status want, const char* fn) {
  ++g_checks;
  const char* msg = laq_last_error();
  if (got != want || (fn && !std::strstr(msg, fn))) {
    std::printf("line %d: status %d (want %d), last error \"%s\"\n", line, got, want, msg);
    ++g_bad;
  }
}
#define EXPECT(call, want, fn) expect(__LINE__, (call), (want), (fn))

void* const P = reinterpret_cast<void*>(0x100000);  // aligned, never dereferenced
void* off(int b) { return static_cast<char*>(P) + b; }
uint32_t* const Q = static_cast<uint32_t*>(P);
uint8_t* const Z = static_cast<uint8_t*>(P);
float* const F = static_cast<float*>(P);
const int64_t kMax = std::numeric_limits<int64_t>::max();
const int64_t kMin = std::numeric_limits<int64_t>::min();

typedef laq_status (*quant_fn)(const void*, int64_t, int64_t, uint32_t*, void*, uint8_t*, void*);
typedef laq_status (*pack_fn)(const void*, const void*, const uint8_t*, int64_t, int64_t, uint32_t*, void*);
typedef laq_status (*lin_fn)(const void*, const uint32_t*, const void*, const uint8_t*, void*, int64_t, int64_t,
                             int64_t, void*);
typedef laq_status (*lin_ws_fn)(const void*, const uint32_t*, const void*, const uint8_t*, void*, int64_t, int64_t,
                                int64_t, void*, int64_t, void*);
typedef laq_status (*group_fn)(const laq_linear_call*, int32_t, int64_t, void*);

const int64_t kBadShapes[][2] = {{0, 128},        {-1, 128},       {kMin, 128},     {4, 0},
                                 {4, 64},         {4, 200},        {4, -128},       {4, kMin},
                                 {1LL << 31, 128}, {kMax, 128},    {4, (1LL << 24) + 128},
                                 {4, kMax & ~127LL}, {1LL << 30, 1 << 11}, {1LL << 16, 1LL << 24}};

void quantize_cases(quant_fn f, const char* fn) {
  EXPECT(f(nullptr, 4, 128, Q, P, Z, nullptr), LAQ_ERR_NULL_POINTER, fn);
  EXPECT(f(P, 4, 128, nullptr, P, Z, nullptr), LAQ_ERR_NULL_POINTER, fn);
  EXPECT(f(P, 4, 128, Q, nullptr, Z, nullptr), LAQ_ERR_NULL_POINTER, fn);
  EXPECT(f(P, 4, 128, Q, P, nullptr, nullptr), LAQ_ERR_NULL_POINTER, fn);
  for (const auto& s : kBadShapes) EXPECT(f(P, s[0], s[1], Q, P, Z, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  EXPECT(f(off(8), 4, 128, Q, P, Z, nullptr), LAQ_ERR_MISALIGNED, fn);
  EXPECT(f(P, 4, 128, static_cast<uint32_t*>(off(4)), P, Z, nullptr), LAQ_ERR_MISALIGNED, fn);
  EXPECT(f(P, 4, 128, Q, off(1), Z, nullptr), LAQ_ERR_MISALIGNED, fn);
}

void pack_cases(pack_fn f, const char* fn) {
  EXPECT(f(nullptr, P, Z, 4, 128, Q, nullptr), LAQ_ERR_NULL_POINTER, fn);
  EXPECT(f(P, nullptr, Z, 4, 128, Q, nullptr), LAQ_ERR_NULL_POINTER, fn);
  EXPECT(f(P, P, nullptr, 4, 128, Q, nullptr), LAQ_ERR_NULL_POINTER, fn);
  EXPECT(f(P, P, Z, 4, 128, nullptr, nullptr), LAQ_ERR_NULL_POINTER, fn);
  for (const auto& s : kBadShapes) EXPECT(f(P, P, Z, s[0], s[1], Q, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  EXPECT(f(off(2), P, Z, 4, 128, Q, nullptr), LAQ_ERR_MISALIGNED, fn);
  EXPECT(f(P, off(1), Z, 4, 128, Q, nullptr), LAQ_ERR_MISALIGNED, fn);
  EXPECT(f(P, P, Z, 4, 128, static_cast<uint32_t*>(off(8)), nullptr), LAQ_ERR_MISALIGNED, fn);
}

void linear_cases(lin_fn f, const char* fn, int64_t max_m) {
  EXPECT(f(nullptr, Q, P, Z, P, 1, 4, 128, nullptr), LAQ_ERR_NULL_POINTER, fn);
  EXPECT(f(P, nullptr, P, Z, P, 1, 4, 128, nullptr), LAQ_ERR_NULL_POINTER, fn);
  EXPECT(f(P, Q, nullptr, Z, P, 1, 4, 128, nullptr), LAQ_ERR_NULL_POINTER, fn);
  EXPECT(f(P, Q, P, nullptr, P, 1, 4, 128, nullptr), LAQ_ERR_NULL_POINTER, fn);
  EXPECT(f(P, Q, P, Z, nullptr, 1, 4, 128, nullptr), LAQ_ERR_NULL_POINTER, fn);
  for (const auto& s : kBadShapes) EXPECT(f(P, Q, P, Z, P, 1, s[0], s[1], nullptr), LAQ_ERR_BAD_SHAPE, fn);
  for (int64_t m : {(int64_t)0, (int64_t)-1, max_m + 1, kMax, kMin})
    EXPECT(f(P, Q, P, Z, P, m, 4, 128, nullptr), LAQ_ERR_BAD_M, fn);
  EXPECT(f(off(4), Q, P, Z, P, 1, 4, 128, nullptr), LAQ_ERR_MISALIGNED, fn);
  EXPECT(f(P, static_cast<uint32_t*>(off(4)), P, Z, P, 1, 4, 128, nullptr), LAQ_ERR_MISALIGNED, fn);
  EXPECT(f(P, Q, off(1), Z, P, 1, 4, 128, nullptr), LAQ_ERR_MISALIGNED, fn);
  EXPECT(f(P, Q, P, Z, off(1), 1, 4, 128, nullptr), LAQ_ERR_MISALIGNED, fn);
}

void linear_ws_cases(lin_ws_fn f, const char* fn) {
  EXPECT(f(nullptr, Q, P, Z, P, 2, 4, 128, P, 16, nullptr), LAQ_ERR_NULL_POINTER, fn);
  EXPECT(f(P, Q, P, Z, nullptr, 2, 4, 128, P, 16, nullptr), LAQ_ERR_NULL_POINTER, fn);
  EXPECT(f(P, Q, P, Z, P, 2, 4, 128, nullptr, 16, nullptr), LAQ_ERR_NULL_POINTER, fn);
  EXPECT(f(P, Q, P, Z, P, 2, 4, 128, P, -1, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  EXPECT(f(P, Q, P, Z, P, 2, 4, 128, P, kMin, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  for (const auto& s : kBadShapes) EXPECT(f(P, Q, P, Z, P, 2, s[0], s[1], P, 16, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  EXPECT(f(P, Q, P, Z, P, 17, 4, 128, P, 16, nullptr), LAQ_ERR_BAD_M, fn);
  EXPECT(f(P, Q, P, Z, P, 2, 4, 128, off(8), 16, nullptr), LAQ_ERR_MISALIGNED, fn);
  EXPECT(f(off(2), Q, P, Z, P, 2, 4, 128, P, 16, nullptr), LAQ_ERR_MISALIGNED, fn);
}

void group_cases(group_fn f, const char* fn) {
  laq_linear_call c[LAQ_MAX_GROUP + 1];
  for (auto& ci : c) ci = laq_linear_call{P, Q, P, Z, P, 4, 128};
  EXPECT(f(nullptr, 1, 1, nullptr), LAQ_ERR_NULL_POINTER, fn);
  for (int32_t n : {0, -1, LAQ_MAX_GROUP + 1, std::numeric_limits<int32_t>::min()})
    EXPECT(f(c, n, 1, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  EXPECT(f(c, 2, 0, nullptr), LAQ_ERR_BAD_M, fn);
  EXPECT(f(c, 2, 17, nullptr), LAQ_ERR_BAD_M, fn);
  for (int i = 0; i < LAQ_MAX_GROUP; ++i) {
    laq_linear_call d[LAQ_MAX_GROUP];
    for (auto& di : d) di = laq_linear_call{P, Q, P, Z, P, 4, 128};
    d[i].y = nullptr;
    EXPECT(f(d, LAQ_MAX_GROUP, 1, nullptr), LAQ_ERR_NULL_POINTER, fn);
    d[i].y = P;
    d[i].K = 200;
    EXPECT(f(d, LAQ_MAX_GROUP, 1, nullptr), LAQ_ERR_BAD_SHAPE, fn);
    d[i].K = 128;
    d[i].x = off(2);
    EXPECT(f(d, LAQ_MAX_GROUP, 1, nullptr), LAQ_ERR_MISALIGNED, fn);
  }
  // rows of all calls must total < 2^31
  laq_linear_call big[2] = {{P, Q, P, Z, P, 1LL << 30, 128}, {P, Q, P, Z, P, 1LL << 30, 128}};
  EXPECT(f(big, 2, 1, nullptr), LAQ_ERR_BAD_SHAPE, fn);
}

}  // namespace

int main() {
  // status strings and version
  for (int s = -3; s < 10; ++s) ++g_checks, g_bad += laq_status_string(s) == nullptr;
  ++g_checks, g_bad += laq_abi_version() != LAQ_ABI_VERSION;
  ++g_checks, g_bad += laq_profile_next_launch(nullptr, nullptr) != LAQ_OK;

  quantize_cases(laq_quantize_w3g128, "laq_quantize_w3g128");
  quantize_cases(laq_quantize_w4g128, "laq_quantize_w4g128");
  pack_cases(laq_pack_w3g128, "laq_pack_w3g128");
  pack_cases(laq_pack_w4g128, "laq_pack_w4g128");
  linear_cases(laq_linear_w3g128, "laq_linear_w3g128", 16);
  linear_cases(laq_linear_w4g128, "laq_linear_w4g128", 16);
  linear_cases(laq_linear_noalloc_w3g128, "laq_linear_noalloc_w3g128", 16);
  linear_cases(laq_linear_swiglu_w3g128, "laq_linear_swiglu_w3g128", 4);
  linear_cases(laq_linear_swiglu_w4g128, "laq_linear_swiglu_w4g128", 4);
  linear_ws_cases(laq_linear_ws_w3g128, "laq_linear_ws_w3g128");
  linear_ws_cases(laq_linear_ws_w4g128, "laq_linear_ws_w4g128");
  group_cases(laq_linear_group_w3g128, "laq_linear_group_w3g128");
  group_cases(laq_linear_group_w4g128, "laq_linear_group_w4g128");

  // the fused gate|up linear: even rows, activation tile within LDS
  EXPECT(laq_linear_swiglu_w3g128(P, Q, P, Z, P, 1, 5, 128, nullptr), LAQ_ERR_BAD_SHAPE, "swiglu");
  EXPECT(laq_linear_swiglu_w3g128(P, Q, P, Z, P, 1, 4, 16384 + 128, nullptr), LAQ_ERR_BAD_SHAPE, "swiglu");
  EXPECT(laq_linear_swiglu_w3g128(P, Q, P, Z, P, 3, 4, 4096 + 128, nullptr), LAQ_ERR_BAD_SHAPE, "swiglu");

  // residual add + RMSNorm inside the linear (M = 1)
  typedef laq_status (*norm_lin_fn)(const float*, const void*, const void*, float, float*, const uint32_t*,
                                    const void*, const uint8_t*, void*, int64_t, int64_t, void*);
  const norm_lin_fn nls[] = {laq_add_rmsnorm_linear_w3g128, laq_add_rmsnorm_linear_w4g128,
                             laq_add_rmsnorm_linear_swiglu_w3g128, laq_add_rmsnorm_linear_swiglu_w4g128};
  float* const RO = static_cast<float*>(off(1 << 16));
  for (int i = 0; i < 4; ++i) {
    const norm_lin_fn f = nls[i];
    EXPECT(f(nullptr, P, P, 1e-6f, RO, Q, P, Z, P, 4, 128, nullptr), LAQ_ERR_NULL_POINTER, "laq_add_rmsnorm_linear");
    EXPECT(f(F, P, nullptr, 1e-6f, RO, Q, P, Z, P, 4, 128, nullptr), LAQ_ERR_NULL_POINTER, "laq_add_rmsnorm_linear");
    EXPECT(f(F, P, P, 1e-6f, RO, nullptr, P, Z, P, 4, 128, nullptr), LAQ_ERR_NULL_POINTER, "laq_add_rmsnorm_linear");
    EXPECT(f(F, P, P, 1e-6f, RO, Q, P, Z, nullptr, 4, 128, nullptr), LAQ_ERR_NULL_POINTER, "laq_add_rmsnorm_linear");
    for (const auto& sh : kBadShapes)
      EXPECT(f(F, P, P, 1e-6f, RO, Q, P, Z, P, sh[0], sh[1], nullptr), LAQ_ERR_BAD_SHAPE, "laq_add_rmsnorm_linear");
    EXPECT(f(F, P, P, 1e-6f, RO, Q, P, Z, P, 4, 8192 + 128, nullptr), LAQ_ERR_BAD_SHAPE, "laq_add_rmsnorm_linear");
    EXPECT(f(F, P, P, -1.0f, RO, Q, P, Z, P, 4, 128, nullptr), LAQ_ERR_BAD_SHAPE, "laq_add_rmsnorm_linear");
    EXPECT(f(F, P, P, std::numeric_limits<float>::quiet_NaN(), RO, Q, P, Z, P, 4, 128, nullptr), LAQ_ERR_BAD_SHAPE,
           "laq_add_rmsnorm_linear");
    EXPECT(f(F, P, P, 1e-6f, F, Q, P, Z, P, 4, 128, nullptr), LAQ_ERR_BAD_SHAPE, "laq_add_rmsnorm_linear");
    EXPECT(f(F, P, P, 1e-6f, F + 100, Q, P, Z, P, 4, 128, nullptr), LAQ_ERR_BAD_SHAPE, "laq_add_rmsnorm_linear");
    EXPECT(f(F + 2, P, P, 1e-6f, RO, Q, P, Z, P, 4, 128, nullptr), LAQ_ERR_MISALIGNED, "laq_add_rmsnorm_linear");
    EXPECT(f(F, off(8), P, 1e-6f, RO, Q, P, Z, P, 4, 128, nullptr), LAQ_ERR_MISALIGNED, "laq_add_rmsnorm_linear");
    EXPECT(f(F, P, P, 1e-6f, RO, Q, off(1), Z, P, 4, 128, nullptr), LAQ_ERR_MISALIGNED, "laq_add_rmsnorm_linear");
    if (i >= 2)
      EXPECT(f(F, P, P, 1e-6f, RO, Q, P, Z, P, 5, 128, nullptr), LAQ_ERR_BAD_SHAPE, "laq_add_rmsnorm_linear_swiglu");
  }
  // the no-allocation linear: split-K partial sums beyond its scratch array
  EXPECT(laq_linear_noalloc_w3g128(P, Q, P, Z, P, 16, 16000, 1LL << 20, nullptr), LAQ_ERR_BAD_SHAPE, "scratch");
  EXPECT(laq_linear_noalloc_w3g128(P, Q, P, Z, P, 16, 16368, 1LL << 24, nullptr), LAQ_ERR_BAD_SHAPE, "scratch");

  // workspace-size queries over extreme arguments: defined results only
  const int64_t ms[] = {kMin, -1, 0, 1, 2, 3, 16, 17, kMax};
  const int64_t ns[] = {kMin, -1, 0, 1, 3, 1000, 5120, 16368, 16384, 0x7FFFFFFF, 1LL << 31, kMax};
  const int64_t ks[] = {kMin, -128, 0, 100, 128, 19968, 20480, 25600, 1LL << 20, 1LL << 24, (1LL << 24) + 128,
                        kMax & ~127LL};
  for (int64_t m : ms)
    for (int64_t n : ns)
      for (int64_t k : ks) {
        const int64_t b = laq_linear_workspace_bytes(m, n, k);
        ++g_checks;
        const bool valid = m >= 1 && m <= 16 && n >= 1 && n <= 0x7FFFFFFF && k >= 128 && k % 128 == 0 &&
                           k <= (1LL << 24) && n * k < (1LL << 40);
        if (b < 0 || (!valid && b != 0) || (b > 0 && b % (m * n * 4) != 0)) {
          std::printf("workspace_bytes(%lld, %lld, %lld) = %lld\n", (long long)m, (long long)n, (long long)k,
                      (long long)b);
          ++g_bad;
        }
      }
  const int64_t hs[] = {kMin, -1, 0, 1, 8, 32, 4096, 4097, kMax};
  const int64_t ls[] = {kMin, -1, 0, 1, 63, 64, 65, 1 << 20, 1 << 21, (1 << 21) + 1, kMax};
  for (int64_t h : hs)
    for (int64_t l : ls) {
      const int64_t b = laq_decode_attention_workspace_bytes(h, l);
      ++g_checks;
      const bool valid = h >= 1 && h <= 4096 && l >= 1 && l <= (1 << 21);
      if (b < 0 || (valid != (b > 0))) {
        std::printf("attention_workspace_bytes(%lld, %lld) = %lld\n", (long long)h, (long long)l, (long long)b);
        ++g_bad;
      }
    }

  // decode-step operations
  const char* fn = "laq_add_rmsnorm_f16";
  EXPECT(laq_add_rmsnorm_f16(nullptr, P, P, P, 1, 2560, 1e-6f, nullptr), LAQ_ERR_NULL_POINTER, fn);
  EXPECT(laq_add_rmsnorm_f16(F, P, nullptr, P, 1, 2560, 1e-6f, nullptr), LAQ_ERR_NULL_POINTER, fn);
  EXPECT(laq_add_rmsnorm_f16(F, P, P, nullptr, 1, 2560, 1e-6f, nullptr), LAQ_ERR_NULL_POINTER, fn);
  for (int64_t m : {(int64_t)0, (int64_t)-1, (int64_t)1 << 31, kMax, kMin})
    EXPECT(laq_add_rmsnorm_f16(F, P, P, P, m, 2560, 1e-6f, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  for (int64_t d : {(int64_t)0, (int64_t)-1, (int64_t)(1 << 20) + 1, kMax, kMin})
    EXPECT(laq_add_rmsnorm_f16(F, P, P, P, 1, d, 1e-6f, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  for (float e : {-1e-6f, std::numeric_limits<float>::quiet_NaN(), std::numeric_limits<float>::infinity()})
    EXPECT(laq_add_rmsnorm_f16(F, P, P, P, 1, 2560, e, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  EXPECT(laq_add_rmsnorm_f16(reinterpret_cast<float*>(off(2)), P, P, P, 1, 2560, 1e-6f, nullptr),
         LAQ_ERR_MISALIGNED, fn);
  EXPECT(laq_add_rmsnorm_f16(F, off(1), P, P, 1, 2560, 1e-6f, nullptr), LAQ_ERR_MISALIGNED, fn);

  fn = "laq_qk_norm_rope_f16";
  EXPECT(laq_qk_norm_rope_f16(nullptr, P, P, F, 0, 32, 8, 128, 1e-6f, P, P, P, 1024, nullptr), LAQ_ERR_NULL_POINTER, fn);
  EXPECT(laq_qk_norm_rope_f16(P, P, P, F, 0, 32, 8, 128, 1e-6f, P, nullptr, P, 1024, nullptr), LAQ_ERR_NULL_POINTER, fn);
  EXPECT(laq_qk_norm_rope_f16(P, P, P, F, 0, 32, 8, 64, 1e-6f, P, P, P, 1024, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  for (int64_t hq : {(int64_t)0, (int64_t)24, (int64_t)128, (int64_t)8192, kMax, kMin})
    EXPECT(laq_qk_norm_rope_f16(P, P, P, F, 0, hq, 8, 128, 1e-6f, P, P, P, 1024, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  EXPECT(laq_qk_norm_rope_f16(P, P, P, F, 0, 32, 0, 128, 1e-6f, P, P, P, 1024, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  for (int64_t pos : {(int64_t)-1, (int64_t)1024, kMax, kMin})
    EXPECT(laq_qk_norm_rope_f16(P, P, P, F, pos, 32, 8, 128, 1e-6f, P, P, P, 1024, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  EXPECT(laq_qk_norm_rope_f16(P, P, P, F, 0, 32, 8, 128, 1e-6f, P, P, P, (1 << 21) + 1, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  EXPECT(laq_qk_norm_rope_f16(P, P, P, F, 0, 32, 8, 128, 1e-6f, P, off(8), P, 1024, nullptr), LAQ_ERR_MISALIGNED, fn);
  EXPECT(laq_qk_norm_rope_f16(P, P, P, reinterpret_cast<float*>(off(2)), 0, 32, 8, 128, 1e-6f, P, P, P, 1024, nullptr),
         LAQ_ERR_MISALIGNED, fn);

  fn = "laq_decode_attention_f16";
  const int64_t ws = laq_decode_attention_workspace_bytes(32, 1024);
  EXPECT(laq_decode_attention_f16(nullptr, P, P, 32, 8, 128, 1024, 1024, P, P, ws, nullptr), LAQ_ERR_NULL_POINTER, fn);
  EXPECT(laq_decode_attention_f16(P, P, P, 32, 8, 128, 1024, 1024, P, nullptr, ws, nullptr), LAQ_ERR_NULL_POINTER, fn);
  for (int64_t l : {(int64_t)0, (int64_t)1025, kMax, kMin})
    EXPECT(laq_decode_attention_f16(P, P, P, 32, 8, 128, l, 1024, P, P, ws, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  EXPECT(laq_decode_attention_f16(P, P, P, 32, 8, 128, 1024, 1024, P, P, ws - 1, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  EXPECT(laq_decode_attention_f16(P, P, P, 32, 8, 128, 1024, 1024, P, P, kMin, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  EXPECT(laq_decode_attention_f16(P, P, P, 32, 3, 128, 1024, 1024, P, P, ws, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  EXPECT(laq_decode_attention_f16(P, P, P, 32, 8, 128, 1024, 1024, P, off(4), ws, nullptr), LAQ_ERR_MISALIGNED, fn);

  fn = "laq_decode_attention_qkv_f16";
  const int64_t wq = laq_decode_attention_qkv_workspace_bytes(32, 8, 1024);
  EXPECT(laq_decode_attention_qkv_f16(nullptr, P, P, F, 10, 32, 8, 128, 1e-6f, P, P, 1024, P, P, wq, nullptr),
         LAQ_ERR_NULL_POINTER, fn);
  EXPECT(laq_decode_attention_qkv_f16(P, P, P, F, 10, 32, 8, 128, 1e-6f, P, P, 1024, P, nullptr, wq, nullptr),
         LAQ_ERR_NULL_POINTER, fn);
  for (int64_t pos : {(int64_t)-1, (int64_t)1024, kMax, kMin})
    EXPECT(laq_decode_attention_qkv_f16(P, P, P, F, pos, 32, 8, 128, 1e-6f, P, P, 1024, P, P, wq, nullptr),
           LAQ_ERR_BAD_SHAPE, fn);
  EXPECT(laq_decode_attention_qkv_f16(P, P, P, F, 1023, 32, 8, 128, 1e-6f, P, P, 1024, P, P, wq - 1, nullptr),
         LAQ_ERR_BAD_SHAPE, fn);
  EXPECT(laq_decode_attention_qkv_f16(P, P, P, F, 10, 32, 8, 128, 1e-6f, P, P, 1024, P, P, kMin, nullptr),
         LAQ_ERR_BAD_SHAPE, fn);
  EXPECT(laq_decode_attention_qkv_f16(P, P, P, F, 10, 32, 8, 128, -1.0f, P, P, 1024, P, P, wq, nullptr),
         LAQ_ERR_BAD_SHAPE, fn);
  EXPECT(laq_decode_attention_qkv_f16(P, P, P, F, 10, 32, 8, 128, 1e-6f, P, off(8), 1024, P, P, wq, nullptr),
         LAQ_ERR_MISALIGNED, fn);
  for (int64_t h : hs)
    for (int64_t kv : {kMin, (int64_t)-1, (int64_t)0, (int64_t)1, (int64_t)8, (int64_t)4096, kMax})
      for (int64_t l : ls) {
        const int64_t b = laq_decode_attention_qkv_workspace_bytes(h, kv, l);
        ++g_checks;
        const bool valid = h >= 1 && h <= 4096 && kv >= 1 && kv <= h && l >= 1 && l <= (1 << 21);
        if (b < 0 || (valid != (b > 0))) {
          std::printf("attention_qkv_workspace_bytes(%lld, %lld, %lld) = %lld\n", (long long)h, (long long)kv,
                      (long long)l, (long long)b);
          ++g_bad;
        }
      }

  fn = "laq_silu_mul_f16";
  EXPECT(laq_silu_mul_f16(nullptr, P, 1, 9728, nullptr), LAQ_ERR_NULL_POINTER, fn);
  for (int64_t m : {(int64_t)0, (int64_t)65536, kMax, kMin})
    EXPECT(laq_silu_mul_f16(P, P, m, 9728, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  for (int64_t i : {(int64_t)0, (int64_t)(1LL << 30) + 1, kMax, kMin})
    EXPECT(laq_silu_mul_f16(P, P, 1, i, nullptr), LAQ_ERR_BAD_SHAPE, fn);
  EXPECT(laq_silu_mul_f16(P, off(1), 1, 9728, nullptr), LAQ_ERR_MISALIGNED, fn);

  if (g_bad) {
    std::printf("%d of %d checks failed\n", g_bad, g_checks);
    return 1;
  }
  std::printf("ok %d\n", g_checks);
  return 0;
}
