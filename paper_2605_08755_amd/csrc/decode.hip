// Decode-step operations between the quantized linears of a decoder layer
// (the model the paper quantizes and times, Sec. 5, Table 3): residual add
// with RMSNorm, per-head q/k RMSNorm with the rotary embedding and the
// key/value cache append, single-token attention over the cache, and
// SiLU-and-multiply.  fp16 in and out, fp32 arithmetic, fixed reduction
// orders (deterministic).  Head dimension 128.
#include <math.h>

#include "laq_internal.h"

namespace laq {

namespace {

constexpr int kHeadDim = 128;
constexpr int kNormThreads = 256;
constexpr int kAttnTile = 64;  // positions per attention block (one wave)

__device__ __forceinline__ float h2f(uint16_t h) { return (float)__builtin_bit_cast(_Float16, h); }
__device__ __forceinline__ uint16_t f2h(float f) { return __builtin_bit_cast(uint16_t, (_Float16)f); }

// Sum / maximum over the 64 lanes of a wave, every lane receiving the result
// (a fixed butterfly, so the order is the same on every call).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// One row per block: r = residual + delta (written back), y = r / rms(r) * w.
__global__ __launch_bounds__(kNormThreads) void add_rmsnorm_kernel(float* __restrict__ res,
                                                                   const uint16_t* __restrict__ delta,
                                                                   const uint16_t* __restrict__ w,
                                                                   uint16_t* __restrict__ y, int D, float eps) {
  __shared__ float part[kNormThreads / 64];
  const int64_t row = blockIdx.x;
  float* r = res + row * D;
  const uint16_t* dl = delta ? delta + row * D : nullptr;
  uint16_t* yr = y + row * D;
  float ss = 0.0f;
  for (int i = threadIdx.x; i < D; i += kNormThreads) {
    float v = r[i];
    if (dl) v += h2f(dl[i]);
    r[i] = v;
    ss = fmaf(v, v, ss);
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.0f;
#pragma unroll
  for (int i = 0; i < kNormThreads / 64; ++i) tot += part[i];
  const float inv = 1.0f / sqrtf(tot / (float)D + eps);
  for (int i = threadIdx.x; i < D; i += kNormThreads) yr[i] = f2h(r[i] * inv * h2f(w[i]));
}

// One head per block (64 lanes; lane i holds dimensions i and i + 64, the
// pair the rotary embedding turns): q heads are normalized, rotated and
// written to q_out, k heads normalized, rotated and written to the key cache
// at position pos, v heads copied to the value cache.  cs points at the
// table row of pos: cos of the 64 angles, then their sin.
__global__ __launch_bounds__(64) void qk_norm_rope_kernel(const uint16_t* __restrict__ qkv,
                                                          const uint16_t* __restrict__ qw,
                                                          const uint16_t* __restrict__ kw,
                                                          const float* __restrict__ cs, int Hq, int Hkv,
                                                          float eps, uint16_t* __restrict__ q_out,
                                                          uint16_t* __restrict__ kc, uint16_t* __restrict__ vc,
                                                          int64_t pos, int64_t S_max) {
  const int h = blockIdx.x;
  const int i = threadIdx.x;
  const uint16_t* src = qkv + (int64_t)h * kHeadDim;
  if (h >= Hq + Hkv) {
    uint16_t* dst = vc + ((int64_t)(h - Hq - Hkv) * S_max + pos) * kHeadDim;
    dst[i] = src[i];
    dst[i + 64] = src[i + 64];
    return;
  }
  const bool isq = h < Hq;
  const uint16_t* wn = isq ? qw : kw;
  float a = h2f(src[i]), b = h2f(src[i + 64]);
  const float ss = wave_sum(fmaf(a, a, b * b));
  const float inv = 1.0f / sqrtf(ss / (float)kHeadDim + eps);
  a = a * inv * h2f(wn[i]);
  b = b * inv * h2f(wn[i + 64]);
  const float c = cs[i], s = cs[64 + i];
  uint16_t* dst = isq ? q_out + (int64_t)h * kHeadDim : kc + ((int64_t)(h - Hq) * S_max + pos) * kHeadDim;
  dst[i] = f2h(a * c - b * s);
  dst[i + 64] = f2h(b * c + a * s);
}

// Partial attention of one key/value head over 64 positions (one wave):
// lane t scores position 64*tile + t against the R query heads of the group,
// then the softmax statistics (max m, sum l of exp(s - m)) and the weighted
// value sums o (lane i: dimensions i and i + 64) go to the workspace,
// ws[((h * T) + tile) * 130 + {0: m, 1: l, 2..129: o}].
template <int R>
__global__ __launch_bounds__(64) void attn_partial_kernel(const uint16_t* __restrict__ q,
                                                          const uint16_t* __restrict__ kc,
                                                          const uint16_t* __restrict__ vc, int64_t S_max,
                                                          int L, int T, float* __restrict__ ws) {
  __shared__ float qs[R][kHeadDim];
  const int g = blockIdx.x;
  const int tile = blockIdx.y;
  const int lane = threadIdx.x;
  const int p = tile * kAttnTile + lane;
  const bool valid = p < L;
  const float scale = 0.08838834764831845f;  // 1 / sqrt(128)
  for (int k = lane; k < R * kHeadDim; k += 64)
    qs[k / kHeadDim][k % kHeadDim] = h2f(q[((int64_t)g * R) * kHeadDim + k]) * scale;
  __syncthreads();

  float s[R];
#pragma unroll
  for (int r = 0; r < R; ++r) s[r] = 0.0f;
  const uint16_t* krow = kc + ((int64_t)g * S_max + (valid ? p : 0)) * kHeadDim;
#pragma unroll 4
  for (int c = 0; c < kHeadDim / 8; ++c) {
    const u32x4 kv = *reinterpret_cast<const u32x4*>(krow + c * 8);
    const uint32_t wv[4] = {kv.x, kv.y, kv.z, kv.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float kf = h2f((uint16_t)(wv[e >> 1] >> (16 * (e & 1))));
#pragma unroll
      for (int r = 0; r < R; ++r) s[r] = fmaf(kf, qs[r][c * 8 + e], s[r]);
    }
  }
  float m[R], l[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const float sv = valid ? s[r] : -INFINITY;
    m[r] = wave_max(sv);
    s[r] = valid ? expf(sv - m[r]) : 0.0f;
    l[r] = wave_sum(s[r]);
  }
  float o0[R], o1[R];
#pragma unroll
  for (int r = 0; r < R; ++r) o0[r] = o1[r] = 0.0f;
  const uint16_t* vrow = vc + ((int64_t)g * S_max + (int64_t)tile * kAttnTile) * kHeadDim;
  const int npos = min(kAttnTile, L - tile * kAttnTile);
  for (int t = 0; t < npos; ++t, vrow += kHeadDim) {
    const float v0 = h2f(vrow[lane]), v1 = h2f(vrow[lane + 64]);
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const float pt = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, s[r]), t));
      o0[r] = fmaf(pt, v0, o0[r]);
      o1[r] = fmaf(pt, v1, o1[r]);
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    float* wp = ws + ((int64_t)(g * R + r) * T + tile) * (kHeadDim + 2);
    if (lane == 0) {
      wp[0] = m[r];
      wp[1] = l[r];
    }
    wp[2 + lane] = o0[r];
    wp[2 + 64 + lane] = o1[r];
  }
}

// Combines the T partials of each query head in tile order.
__global__ __launch_bounds__(kHeadDim) void attn_combine_kernel(const float* __restrict__ ws, int T,
                                                                 uint16_t* __restrict__ out) {
  const int h = blockIdx.x;
  const int d = threadIdx.x;
  const float* base = ws + (int64_t)h * T * (kHeadDim + 2);
  float M = -INFINITY;
  for (int t = 0; t < T; ++t) M = fmaxf(M, base[(int64_t)t * (kHeadDim + 2)]);
  float num = 0.0f, den = 0.0f;
  for (int t = 0; t < T; ++t) {
    const float* pt = base + (int64_t)t * (kHeadDim + 2);
    const float e = expf(pt[0] - M);
    den = fmaf(e, pt[1], den);
    num = fmaf(e, pt[2 + d], num);
  }
  out[(int64_t)h * kHeadDim + d] = f2h(num / den);
}

// y[m][i] = silu(g) * u with g = gu[m][i], u = gu[m][I + i].
__global__ __launch_bounds__(256) void silu_mul_kernel(const uint16_t* __restrict__ gu, uint16_t* __restrict__ y,
                                                       int64_t M, int64_t I) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= M * I) return;
  const int64_t m = idx / I;
  const int64_t i = idx - m * I;
  const float g = h2f(gu[m * 2 * I + i]);
  const float u = h2f(gu[m * 2 * I + I + i]);
  y[idx] = f2h(g / (1.0f + expf(-g)) * u);
}

}  // namespace

int64_t decode_attention_tiles(int64_t L) { return (L + kAttnTile - 1) / kAttnTile; }

hipError_t launch_add_rmsnorm(float* res, const uint16_t* delta, const uint16_t* w, uint16_t* y, int64_t M,
                              int64_t D, float eps, hipStream_t stream, const LaunchEvents& ev) {
  launch(add_rmsnorm_kernel, dim3((unsigned)M), dim3(kNormThreads), 0, stream, ev, res, delta, w, y, (int)D, eps);
  return hipGetLastError();
}

hipError_t launch_qk_norm_rope(const uint16_t* qkv, const uint16_t* qw, const uint16_t* kw, const float* cos_sin,
                               int64_t pos, int64_t Hq, int64_t Hkv, float eps, uint16_t* q_out, uint16_t* kc,
                               uint16_t* vc, int64_t S_max, hipStream_t stream, const LaunchEvents& ev) {
  launch(qk_norm_rope_kernel, dim3((unsigned)(Hq + 2 * Hkv)), dim3(64), 0, stream, ev, qkv, qw, kw,
         cos_sin + pos * kHeadDim, (int)Hq, (int)Hkv, eps, q_out, kc, vc, pos, S_max);
  return hipGetLastError();
}

hipError_t launch_decode_attention(const uint16_t* q, const uint16_t* kc, const uint16_t* vc, int64_t Hq,
                                   int64_t Hkv, int64_t L, int64_t S_max, uint16_t* out, float* ws,
                                   hipStream_t stream, const LaunchEvents& ev) {
  const int T = (int)decode_attention_tiles(L);
  const int R = (int)(Hq / Hkv);
  LaunchEvents e1, e2;  // the measurement hook spans both kernels
  e1.start = ev.start;
  e2.stop = ev.stop;
  const dim3 grid((unsigned)Hkv, (unsigned)T);
  switch (R) {
    case 1: launch(attn_partial_kernel<1>, grid, dim3(64), 0, stream, e1, q, kc, vc, S_max, (int)L, T, ws); break;
    case 2: launch(attn_partial_kernel<2>, grid, dim3(64), 0, stream, e1, q, kc, vc, S_max, (int)L, T, ws); break;
    case 4: launch(attn_partial_kernel<4>, grid, dim3(64), 0, stream, e1, q, kc, vc, S_max, (int)L, T, ws); break;
    default: launch(attn_partial_kernel<8>, grid, dim3(64), 0, stream, e1, q, kc, vc, S_max, (int)L, T, ws); break;
  }
  launch(attn_combine_kernel, dim3((unsigned)Hq), dim3(kHeadDim), 0, stream, e2, (const float*)ws, T, out);
  return hipGetLastError();
}

hipError_t launch_silu_mul(const uint16_t* gu, uint16_t* y, int64_t M, int64_t I, hipStream_t stream,
                           const LaunchEvents& ev) {
  const int64_t n = M * I;
  launch(silu_mul_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, ev, gu, y, M, I);
  return hipGetLastError();
}

}  // namespace laq
