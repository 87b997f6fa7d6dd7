// Driver for a ThreadSanitizer build of the library's C ABI (host code): eight
// host threads call the entry points at the same time, each with its own
// argument that the host-side validation must reject, and check that the
// status and the calling thread's last-error text are those of its own call
// (the error detail is per thread); they also query the workspace sizes, which
// must not depend on what other threads do.  Nothing passes validation, so no
// HIP call is reached and no GPU is needed.  Prints "ok N" (N checks) on
// success; a wrong result returns 1, a sanitizer report aborts.
#include <atomic>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <thread>
#include <vector>

#include "laq.h"

namespace {

std::atomic<int> g_checks{0}, g_bad{0};
void* const P = reinterpret_cast<void*>(0x100000);  // aligned, never dereferenced
uint32_t* const Q = static_cast<uint32_t*>(P);
uint8_t* const Z = static_cast<uint8_t*>(P);

void check(bool cond, int thread, const char* what) {
  g_checks.fetch_add(1, std::memory_order_relaxed);
  if (!cond) {
    if (g_bad.fetch_add(1) < 10) std::printf("thread %d: %s (last error \"%s\")\n", thread, what, laq_last_error());
  }
}

// One failing call per thread kind; returns the status and checks the text.
void call(int kind, int thread) {
  laq_status st;
  const char* fn;
  switch (kind) {
    case 0: st = laq_linear_w3g128(P, Q, P, Z, P, 17, 4, 128, nullptr); fn = "laq_linear_w3g128"; break;
    case 1: st = laq_quantize_w4g128(nullptr, 4, 128, Q, P, Z, nullptr); fn = "laq_quantize_w4g128"; break;
    case 2: st = laq_pack_w3g128(P, P, Z, 4, 200, Q, nullptr); fn = "laq_pack_w3g128"; break;
    case 3: st = laq_linear_swiglu_w4g128(P, Q, P, Z, P, 1, 3, 128, nullptr); fn = "laq_linear_swiglu_w4g128"; break;
    case 4: st = laq_add_rmsnorm_linear_w3g128(static_cast<float*>(P), nullptr, P, 1e-6f, static_cast<float*>(P), Q, P,
                                               Z, P, 4, 128, nullptr);
      fn = "laq_add_rmsnorm_linear_w3g128"; break;
    case 5: st = laq_add_rmsnorm_f16(static_cast<float*>(P), P, P, P, 1, 2560, -1.0f, nullptr);
      fn = "laq_add_rmsnorm_f16"; break;
    case 6: st = laq_linear_ws_w3g128(static_cast<char*>(P) + 2, Q, P, Z, P, 1, 4, 128, P, 1 << 20, nullptr);
      fn = "laq_linear_ws_w3g128"; break;
    default: st = laq_decode_attention_qkv_f16(P, P, P, static_cast<float*>(P), 5, 32, 8, 128, 1e-6f, P, P, 4, P, P,
                                               1 << 20, nullptr);
      fn = "laq_decode_attention_qkv_f16"; break;
  }
  check(st != LAQ_OK, thread, "call passed validation");
  check(std::strstr(laq_last_error(), fn) != nullptr, thread, "last error names another call");
}

}  // namespace

int main() {
  const int64_t ws_lin = laq_linear_workspace_bytes(16, 1030, 25600);
  const int64_t ws_att = laq_decode_attention_qkv_workspace_bytes(32, 8, 4096);
  std::vector<std::thread> threads;
  for (int t = 0; t < 8; ++t) {
    threads.emplace_back([t, ws_lin, ws_att] {
      for (int i = 0; i < 3000; ++i) {
        call(t, t);
        if (i % 7 == 0) {
          check(laq_linear_workspace_bytes(16, 1030, 25600) == ws_lin, t, "workspace size changed");
          check(laq_decode_attention_qkv_workspace_bytes(32, 8, 4096) == ws_att, t, "attention workspace size changed");
        }
      }
    });
  }
  for (auto& th : threads) th.join();
  if (g_bad.load() != 0) {
    std::printf("%d of %d checks failed\n", g_bad.load(), g_checks.load());
    return 1;
  }
  std::printf("ok %d\n", g_checks.load());
  return 0;
}
