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

// Sum / maximum over the 64 lanes of a wave, every lane receiving the result:
// DPP within each 16-lane row (xor 1, xor 2, the half-row mirror, the row
// mirror; each step combines a lane with its partner commutatively, so the 16
// lanes end with the same bits), then the four row results read from lanes
// 0, 16, 32 and 48 and combined in that order.  No LDS round trips; the same
// order on every call.
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float lane_value(float v, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp<0x141>(v);  // row_half_mirror
  v += dpp<0x140>(v);  // row_mirror
  return ((lane_value(v, 0) + lane_value(v, 16)) + lane_value(v, 32)) + lane_value(v, 48);
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp<0xB1>(v));
  v = fmaxf(v, dpp<0x4E>(v));
  v = fmaxf(v, dpp<0x141>(v));
  v = fmaxf(v, dpp<0x140>(v));
  return fmaxf(fmaxf(lane_value(v, 0), lane_value(v, 16)), fmaxf(lane_value(v, 32), lane_value(v, 48)));
}

// One row per block: r = residual + delta (written back), y = r / rms(r) * w.
// Rows of up to 16 elements per thread take one pass: every load is issued
// (indices clamped into the row, so no branch stands between loads) before
// any arithmetic, and r stays in registers.  HAS_DELTA: delta is not null.
constexpr int kNormRegs = 16;
template <bool HAS_DELTA>
__global__ __launch_bounds__(kNormThreads) void add_rmsnorm_kernel(float* __restrict__ res,
                                                                   const uint16_t* __restrict__ delta,
                                                                   const uint16_t* __restrict__ w,
                                                                   uint16_t* __restrict__ y, int D, float eps) {
  __shared__ float part[kNormThreads / 64];
  const int64_t row = blockIdx.x;
  float* r = res + row * D;
  const uint16_t* dl = HAS_DELTA ? delta + row * D : nullptr;
  uint16_t* yr = y + row * D;
  const int t = threadIdx.x;
  float ss = 0.0f;
  if (D <= kNormRegs * kNormThreads) {
    float v[kNormRegs], wv[kNormRegs], dv[kNormRegs];
#pragma unroll
    for (int k = 0; k < kNormRegs; ++k) {
      const int i = min(t + k * kNormThreads, D - 1);
      v[k] = r[i];
      wv[k] = h2f(w[i]);
      dv[k] = HAS_DELTA ? h2f(dl[i]) : 0.0f;
    }
#pragma unroll
    for (int k = 0; k < kNormRegs; ++k) {
      const bool in = t + k * kNormThreads < D;
      v[k] = in ? v[k] + dv[k] : 0.0f;
      ss = fmaf(v[k], v[k], ss);
    }
#pragma unroll
    for (int k = 0; k < kNormRegs; ++k)
      if (t + k * kNormThreads < D) r[t + k * kNormThreads] = v[k];
    ss = wave_sum(ss);
    if ((t & 63) == 0) part[t >> 6] = ss;
    __syncthreads();
    float tot = 0.0f;
#pragma unroll
    for (int i = 0; i < kNormThreads / 64; ++i) tot += part[i];
    const float inv = 1.0f / sqrtf(tot / (float)D + eps);
#pragma unroll
    for (int k = 0; k < kNormRegs; ++k)
      if (t + k * kNormThreads < D) yr[t + k * kNormThreads] = f2h(v[k] * inv * wv[k]);
    return;
  }
  for (int i = t; i < D; i += kNormThreads) {
    float v = r[i];
    if (HAS_DELTA) v += h2f(dl[i]);
    r[i] = v;
    ss = fmaf(v, v, ss);
  }
  ss = wave_sum(ss);
  if ((t & 63) == 0) part[t >> 6] = ss;
  __syncthreads();
  float tot = 0.0f;
#pragma unroll
  for (int i = 0; i < kNormThreads / 64; ++i) tot += part[i];
  const float inv = 1.0f / sqrtf(tot / (float)D + eps);
  for (int i = t; i < D; i += kNormThreads) yr[i] = f2h(r[i] * inv * h2f(w[i]));
}

// RMSNorm of one 128-value head held by a wave (lane i: dimensions i and
// i + 64, a and b) with weights wn, then the rotary embedding of the pair
// (a, b) by the angle whose cosine and sine are cs[i] and cs[64 + i].
// The same with the lane's norm weights (wa, wb) and rotation (c, s) given.
__device__ __forceinline__ void norm_rope_vals(float& a, float& b, float wa, float wb, float c, float s, float eps) {
  const float ss = wave_sum(fmaf(a, a, b * b));
  const float inv = 1.0f / sqrtf(ss / (float)kHeadDim + eps);
  const float na = a * inv * wa;
  const float nb = b * inv * wb;
  a = na * c - nb * s;
  b = nb * c + na * s;
}

__device__ __forceinline__ void norm_rope_pair(float& a, float& b, const uint16_t* __restrict__ wn,
                                               const float* __restrict__ cs, float eps, int i) {
  norm_rope_vals(a, b, h2f(wn[i]), h2f(wn[i + 64]), cs[i], cs[64 + i], eps);
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
  float a = h2f(src[i]), b = h2f(src[i + 64]);
  norm_rope_pair(a, b, isq ? qw : kw, cs, eps, i);
  uint16_t* dst = isq ? q_out + (int64_t)h * kHeadDim : kc + ((int64_t)(h - Hq) * S_max + pos) * kHeadDim;
  dst[i] = f2h(a);
  dst[i + 64] = f2h(b);
}

// Weighted value sums of one wave over the P rows of a value tile in LDS
// (row-major, 128 fp16 per row): lane i accumulates dimensions 2i and 2i + 1
// (one 32-bit LDS read per row), with row t's weight taken from lane t of pr.
// Row t goes to accumulator t % 4 (rows in order within each), and the four
// are added as (a0 + a1) + (a2 + a3): four independent chains instead of one.
// Rows past the key length must hold finite values (zeros) and weight zero.
// Fully unrolled, so the LDS reads of a batch of 8 rows are in flight together.
template <int P>
__device__ __forceinline__ void value_sums(const u32x4* vt, float pr, int lane, float& o_even, float& o_odd) {
  const uint32_t* vw = reinterpret_cast<const uint32_t*>(vt);
  float e[4] = {0.0f, 0.0f, 0.0f, 0.0f}, o[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int t0 = 0; t0 < P; t0 += 8) {
    uint32_t v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = vw[(t0 + j) * (kHeadDim / 2) + lane];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float pt = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, pr), t0 + j));
      e[j & 3] = fmaf(pt, h2f((uint16_t)(v[j] & 0xFFFFu)), e[j & 3]);
      o[j & 3] = fmaf(pt, h2f((uint16_t)(v[j] >> 16)), o[j & 3]);
    }
  }
  o_even = (e[0] + e[1]) + (e[2] + e[3]);
  o_odd = (o[0] + o[1]) + (o[2] + o[3]);
}

// Partial attention of one key/value head over 64 positions: a block of R
// waves, wave w for query head g*R + w of the group.  The block loads the
// tile's key and value rows (16 KiB each, contiguous) into LDS with
// coalesced 16-byte loads, all issued before the first is used; rows past L
// read zero (buffer extent).  Lane t then scores position 64*tile + t, the
// wave forms its softmax statistics (max m, sum l of exp(s - m)) and the
// weighted value sums o (lane i: dimensions 2i and 2i + 1), written to
// ws[((h * T) + tile) * 130 + {0: m, 1: l, 2..129: o}].  Key rows sit in LDS
// with a 16-byte pad (a stride of 17 units), so that lanes reading their own
// rows spread over the banks.
constexpr int kKeyStrideU4 = kHeadDim / 8 + 1;
template <int R>
__global__ __launch_bounds__(64 * R) void attn_partial_kernel(const uint16_t* __restrict__ q,
                                                              const uint16_t* __restrict__ kc,
                                                              const uint16_t* __restrict__ vc, int64_t S_max,
                                                              int L, int T, float* __restrict__ ws) {
  __shared__ u32x4 qh[R][kHeadDim / 8];  // the group's query heads, fp16, 8 per unit
  __shared__ u32x4 kt[kAttnTile * kKeyStrideU4];
  __shared__ u32x4 vt[kAttnTile * kHeadDim / 8];
  constexpr int kUnits = kAttnTile * kHeadDim / 8;  // 16-byte units per tile
  constexpr int kPer = kUnits / (64 * R);           // per thread
  const int g = blockIdx.x;
  const int tile = blockIdx.y;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int npos = __builtin_amdgcn_readfirstlane(min(kAttnTile, L - tile * kAttnTile));
  const int64_t row0 = (int64_t)g * S_max + (int64_t)tile * kAttnTile;
  const __amdgpu_buffer_rsrc_t kr = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(kc + row0 * kHeadDim),
                                                                     (short)0, npos * kHeadDim * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(vc + row0 * kHeadDim),
                                                                     (short)0, npos * kHeadDim * 2, 0x00020000);
  u32x4 ka[kPer], va[kPer];
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const uint32_t u = (uint32_t)(i * 64 * R + tid);
    ka[i] = __builtin_amdgcn_raw_buffer_load_b128(kr, u * 16, 0, 0);
    va[i] = __builtin_amdgcn_raw_buffer_load_b128(vr, u * 16, 0, 0);
  }
  uint16_t qv[2];  // the group's R query heads: R * 128 values, two per thread, both loads in flight
#pragma unroll
  for (int i = 0; i < 2; ++i) qv[i] = q[((int64_t)g * R) * kHeadDim + tid + i * 64 * R];
  uint16_t* qh16 = reinterpret_cast<uint16_t*>(&qh[0][0]);
#pragma unroll
  for (int i = 0; i < 2; ++i) qh16[tid + i * 64 * R] = qv[i];
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int u = i * 64 * R + tid;
    kt[(u >> 4) * kKeyStrideU4 + (u & 15)] = ka[i];
    vt[u] = va[i];
  }
  __syncthreads();

  // score of position p: key and query pairs through v_dot2_f32_f16 into four
  // accumulators (pair j of a unit to accumulator j), (a0 + a1) + (a2 + a3),
  // scaled by 1/sqrt(128)
  const int p = tile * kAttnTile + lane;
  const bool valid = p < L;
  float sa[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int c = 0; c < kHeadDim / 8; ++c) {
    const u32x4 kv = kt[lane * kKeyStrideU4 + c];
    const u32x4 qu = qh[w][c];
    sa[0] = __builtin_amdgcn_fdot2(as_half2(kv.x), as_half2(qu.x), sa[0], false);
    sa[1] = __builtin_amdgcn_fdot2(as_half2(kv.y), as_half2(qu.y), sa[1], false);
    sa[2] = __builtin_amdgcn_fdot2(as_half2(kv.z), as_half2(qu.z), sa[2], false);
    sa[3] = __builtin_amdgcn_fdot2(as_half2(kv.w), as_half2(qu.w), sa[3], false);
  }
  const float sc = ((sa[0] + sa[1]) + (sa[2] + sa[3])) * 0.08838834764831845f;  // 1 / sqrt(128)
  const float sv = valid ? sc : -INFINITY;
  const float m = wave_max(sv);
  const float pr = valid ? expf(sv - m) : 0.0f;
  const float l = wave_sum(pr);
  // value rows past L were loaded as zeros (buffer extent) and weigh zero
  float oe, oo;
  value_sums<kAttnTile>(vt, pr, lane, oe, oo);
  float* wp = ws + ((int64_t)(g * R + w) * T + tile) * (kHeadDim + 2);
  if (lane == 0) {
    wp[0] = m;
    wp[1] = l;
  }
  *reinterpret_cast<float2*>(wp + 2 + 2 * lane) = float2{oe, oo};
}

// Combines the T partials of each query head in tile order: one wave per
// head; the per-tile weights exp(m_t - M) are computed by lane t (batches of
// 64 tiles), and each lane adds dimensions i and i + 64 over the tiles with
// eight partial rows loaded at a time.
__global__ __launch_bounds__(64) void attn_combine_kernel(const float* __restrict__ ws, int T,
                                                          uint16_t* __restrict__ out) {
  const int h = blockIdx.x;
  const int lane = threadIdx.x;
  const float* base = ws + (int64_t)h * T * (kHeadDim + 2);
  float M = -INFINITY;
  for (int t0 = 0; t0 < T; t0 += 64)
    M = fmaxf(M, wave_max(t0 + lane < T ? base[(int64_t)(t0 + lane) * (kHeadDim + 2)] : -INFINITY));
  float den = 0.0f, n0 = 0.0f, n1 = 0.0f;
  for (int t0 = 0; t0 < T; t0 += 64) {
    const int t = t0 + lane;
    const float e = t < T ? expf(base[(int64_t)t * (kHeadDim + 2)] - M) : 0.0f;
    den += wave_sum(t < T ? e * base[(int64_t)t * (kHeadDim + 2) + 1] : 0.0f);
    const int nt = min(64, T - t0);
    for (int j0 = 0; j0 < nt; j0 += 8) {
      float a0[8], a1[8], ej[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int jj = min(j0 + j, nt - 1);
        const float* pt = base + (int64_t)(t0 + jj) * (kHeadDim + 2) + 2;
        a0[j] = pt[lane];
        a1[j] = pt[lane + 64];
        ej[j] = (j0 + j < nt) ? __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, e), jj)) : 0.0f;
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        n0 = fmaf(ej[j], a0[j], n0);
        n1 = fmaf(ej[j], a1[j], n1);
      }
    }
  }
  out[(int64_t)h * kHeadDim + lane] = f2h(n0 / den);
  out[(int64_t)h * kHeadDim + lane + 64] = f2h(n1 / den);
}


// The attention of one decode token straight from the q|k|v projection
// output: per-head RMSNorm and rotary embedding of q and k, the key/value
// cache append at pos, and the partial attention over tiles of P positions
// (L = pos + 1), in one kernel.  Block (g, tile) of R waves, wave w for query
// head g*R + w:
//  - issues the tile's cache rows before pos (16-byte loads, all in flight
//    before the first use; rows at pos and beyond are not loaded),
//  - normalizes and rotates its query head (rounded to fp16, as the separate
//    qk-norm-rope call stores it, then scaled by 1/sqrt(128)),
//  - the block whose tile holds pos also forms that token's key (normalized,
//    rotated, rounded to fp16) and value, writes them to the caches and into
//    its tile in LDS,
//  - scores the tile's positions (64/P lanes per position, each a slice of
//    the 128 dimensions, added by a fixed butterfly), forms the softmax
//    statistics and the weighted value sums as attn_partial_kernel does.
// Partials go to ws[((h * T) + tile) * 130 + {0: m, 1: l, 2..129: o}].
// Argument order: what the tile's loads and the query's norm need first
// (the first fourteen dwords arrive preloaded in scalar registers).
template <int R, int P>
__global__ __launch_bounds__(64 * R) void attn_qkv_partial_kernel(
    uint16_t* __restrict__ kc, uint16_t* __restrict__ vc, int S_max, int pos, const uint16_t* __restrict__ qkv,
    const uint16_t* __restrict__ qw, const float* __restrict__ cs, float eps, int Hq,
    const uint16_t* __restrict__ kw, int Hkv, int T, float* __restrict__ ws) {
  static_assert(P == 16 || P == 32 || P == 64, "tile of 16, 32 or 64 positions");
  constexpr int DS = 64 / P;                   // lanes per position (dimension slices)
  constexpr int kUnits = P * kHeadDim / 8;     // 16-byte units of keys (and of values) per tile
  constexpr int kThreads = 64 * R;
  constexpr int kPer = (kUnits + kThreads - 1) / kThreads;
  __shared__ u32x4 qh[R][kHeadDim / 8];  // the wave's query head, fp16, 8 per unit
  __shared__ u32x4 kt[P * kKeyStrideU4];
  __shared__ u32x4 vt[P * kHeadDim / 8];
  const int g = blockIdx.x;
  const int tile = blockIdx.y;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int L = pos + 1;
  const int p0 = tile * P;
  const int nload = __builtin_amdgcn_readfirstlane(max(0, min(P, pos - p0)));  // cache rows read from memory
  const int64_t row0 = (int64_t)g * S_max + p0;
  const __amdgpu_buffer_rsrc_t kr = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(kc + row0 * kHeadDim),
                                                                     (short)0, nload * kHeadDim * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(vc + row0 * kHeadDim),
                                                                     (short)0, nload * kHeadDim * 2, 0x00020000);
  u32x4 ka[kPer], va[kPer];
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const uint32_t u = (uint32_t)(i * kThreads + tid);
    ka[i] = __builtin_amdgcn_raw_buffer_load_b128(kr, u * 16, 0, 0);
    va[i] = __builtin_amdgcn_raw_buffer_load_b128(vr, u * 16, 0, 0);
  }
  __builtin_amdgcn_sched_barrier(0);  // the tile's loads go out first
  // This wave's query head, its norm weights and the rotation of pos; then
  // the new token's key and value of head g with the key norm weights, which
  // only wave 0 of the block holding pos uses: every wave loads them (a few
  // bytes) because a load under a branch would be waited for inside it,
  // putting a second round trip on that block's path.
  const uint16_t* qsrc = qkv + (int64_t)(g * R + w) * kHeadDim;
  const uint16_t* ksrc = qkv + (int64_t)(Hq + g) * kHeadDim;
  const uint16_t qa = qsrc[lane], qb = qsrc[lane + 64];
  const uint16_t wqa = qw[lane], wqb = qw[lane + 64];
  const float rc = cs[lane], rs = cs[64 + lane];
  const uint16_t kra = ksrc[lane], krb = ksrc[lane + 64];
  __builtin_amdgcn_sched_barrier(0);  // then these, before the loads that wait for kw and Hkv
  const uint16_t wka = kw[lane], wkb = kw[lane + 64];
  const uint16_t* vsrc = ksrc + (int64_t)Hkv * kHeadDim;
  const uint16_t v0 = vsrc[lane], v1 = vsrc[lane + 64];
  // T and ws follow the preloaded arguments: read them now, not at the end.
  asm volatile("" : "+s"(T), "+s"(ws));
  const bool own = pos >= p0 && pos < p0 + P;  // uniform over the block
  float a = h2f(qa), b = h2f(qb);
  norm_rope_vals(a, b, h2f(wqa), h2f(wqb), rc, rs, eps);
  uint16_t* qh16 = reinterpret_cast<uint16_t*>(qh[w]);
  qh16[lane] = f2h(a);
  qh16[lane + 64] = f2h(b);
  // Rows past nload were read as zeros (buffer extent), so the tile holds
  // finite values only; in the block holding pos, wave 0 then overwrites the
  // new token's row (zeros here) after a barrier.  (Staging every row, with no
  // test of the row, keeps the compiler from sinking the tile's loads into a
  // conditional store, behind the query's round trip.)
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int u = i * kThreads + tid;
    if (kPer * kThreads == kUnits || u < kUnits) {
      kt[(u >> 4) * kKeyStrideU4 + (u & 15)] = ka[i];
      vt[u] = va[i];
    }
  }
  if (own) __syncthreads();  // uniform over the block
  if (own && w == 0) {
    float ka0 = h2f(kra), kb0 = h2f(krb);
    norm_rope_vals(ka0, kb0, h2f(wka), h2f(wkb), rc, rs, eps);
    const uint16_t k0 = f2h(ka0), k1 = f2h(kb0);
    const int64_t crow = ((int64_t)g * S_max + pos) * kHeadDim;
    kc[crow + lane] = k0;
    kc[crow + lane + 64] = k1;
    vc[crow + lane] = v0;
    vc[crow + lane + 64] = v1;
    uint16_t* kl = reinterpret_cast<uint16_t*>(kt + (pos - p0) * kKeyStrideU4);
    uint16_t* vl = reinterpret_cast<uint16_t*>(vt + (pos - p0) * (kHeadDim / 8));
    kl[lane] = k0;
    kl[lane + 64] = k1;
    vl[lane] = v0;
    vl[lane + 64] = v1;
  }
  __syncthreads();

  // scores: lane = (slice c, position t) with t = lane % P, c = lane / P; the
  // slice's key and query pairs through v_dot2_f32_f16 into four accumulators
  // (pair j of a unit to accumulator j), added as (a0 + a1) + (a2 + a3), then
  // the slices by a fixed butterfly and the product scaled by 1/sqrt(128).
  // (Vector elements pass through as_half2 by value: a bit cast applied to an
  // element expression was compiled as a cast of element 0.)
  const int t = lane % P;
  const int c = lane / P;
  const int p = p0 + t;
  const bool valid = p < L;
  float sa[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int cc = 0; cc < (kHeadDim / 8) / DS; ++cc) {
    const int unit = c * ((kHeadDim / 8) / DS) + cc;
    const u32x4 kv = kt[t * kKeyStrideU4 + unit];
    const u32x4 qv = qh[w][unit];
    sa[0] = __builtin_amdgcn_fdot2(as_half2(kv.x), as_half2(qv.x), sa[0], false);
    sa[1] = __builtin_amdgcn_fdot2(as_half2(kv.y), as_half2(qv.y), sa[1], false);
    sa[2] = __builtin_amdgcn_fdot2(as_half2(kv.z), as_half2(qv.z), sa[2], false);
    sa[3] = __builtin_amdgcn_fdot2(as_half2(kv.w), as_half2(qv.w), sa[3], false);
  }
  float sc = (sa[0] + sa[1]) + (sa[2] + sa[3]);
#pragma unroll
  for (int o = P; o < 64; o <<= 1) sc += __shfl_xor(sc, o, 64);
  sc *= 0.08838834764831845f;  // 1 / sqrt(128)
  const float sv = valid && c == 0 ? sc : -INFINITY;
  const float m = wave_max(sv);
  const float pr = (valid && c == 0) ? expf(sv - m) : 0.0f;
  const float l = wave_sum(pr);
  float oe, oo;
  value_sums<P>(vt, pr, lane, oe, oo);
  float* wp = ws + ((int64_t)(g * R + w) * T + tile) * (kHeadDim + 2);
  if (lane == 0) {
    wp[0] = m;
    wp[1] = l;
  }
  *reinterpret_cast<float2*>(wp + 2 + 2 * lane) = float2{oe, oo};
}

// Combines the T partials of one query head (block h of NW waves): every wave
// forms the maximum M of the tiles' maxima and the denominator sum_t l_t
// exp(m_t - M) itself (the same fixed order in every wave); wave w adds
// exp(m_t - M) o_t over its tiles t = w, w + NW, ... in order; the waves'
// sums are added in wave order.  A wave's loads of a batch of 8 tiles are
// issued before the statistics pass, so up to 8 * NW tiles cost one memory
// round trip.
template <int NW>
__global__ __launch_bounds__(64 * NW) void attn_combine2_kernel(const float* __restrict__ ws, int T,
                                                                uint16_t* __restrict__ out) {
  __shared__ float num[NW][kHeadDim];
  const int h = blockIdx.x;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const float* base = ws + (int64_t)h * T * (kHeadDim + 2);
  // this wave's first batch of value sums, issued before the statistics
  constexpr int kB = 8;
  float a0[kB], a1[kB], mt[kB];
#pragma unroll
  for (int j = 0; j < kB; ++j) {
    const int tt = min(w + NW * j, T - 1);
    const float* pt = base + (int64_t)tt * (kHeadDim + 2);
    mt[j] = pt[0];
    a0[j] = pt[2 + lane];
    a1[j] = pt[2 + 64 + lane];
  }
  // Statistics: lane t holds tile t's maximum and denominator.  Up to 64
  // tiles one pass loads both; beyond, a pass per 64 tiles for M, then one
  // for the denominator.
  float M = -INFINITY, den = 0.0f;
  if (T <= 64) {
    const float* pt = base + (int64_t)min(lane, T - 1) * (kHeadDim + 2);
    const float ml = pt[0], ll = pt[1];
    M = wave_max(lane < T ? ml : -INFINITY);
    den = wave_sum(lane < T ? expf(ml - M) * ll : 0.0f);
  } else {
    for (int t0 = 0; t0 < T; t0 += 64)
      M = fmaxf(M, wave_max(t0 + lane < T ? base[(int64_t)(t0 + lane) * (kHeadDim + 2)] : -INFINITY));
    for (int t0 = 0; t0 < T; t0 += 64) {
      const int tt = t0 + lane;
      const float* pt = base + (int64_t)min(tt, T - 1) * (kHeadDim + 2);
      den += wave_sum(tt < T ? expf(pt[0] - M) * pt[1] : 0.0f);
    }
  }
  float n0 = 0.0f, n1 = 0.0f;
  for (int j0 = 0; w + NW * j0 < T; j0 += kB) {
    if (j0 > 0) {
#pragma unroll
      for (int j = 0; j < kB; ++j) {
        const int tt = min(w + NW * (j0 + j), T - 1);
        const float* pt = base + (int64_t)tt * (kHeadDim + 2);
        mt[j] = pt[0];
        a0[j] = pt[2 + lane];
        a1[j] = pt[2 + 64 + lane];
      }
    }
#pragma unroll
    for (int j = 0; j < kB; ++j) {
      const float e = (w + NW * (j0 + j) < T) ? expf(mt[j] - M) : 0.0f;
      n0 = fmaf(e, a0[j], n0);
      n1 = fmaf(e, a1[j], n1);
    }
  }
  num[w][lane] = n0;
  num[w][lane + 64] = n1;
  __syncthreads();
  if (w == 0) {
    float s0 = 0.0f, s1 = 0.0f;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      s0 += num[i][lane];
      s1 += num[i][lane + 64];
    }
    out[(int64_t)h * kHeadDim + lane] = f2h(s0 / den);
    out[(int64_t)h * kHeadDim + lane + 64] = f2h(s1 / den);
  }
}

// y[m][i] = silu(g) * u with g = gu[m][i], u = gu[m][I + i]; row m = blockIdx.y.
__global__ __launch_bounds__(256) void silu_mul_kernel(const uint16_t* __restrict__ gu, uint16_t* __restrict__ y,
                                                       int64_t I) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= I) return;
  const int64_t m = blockIdx.y;
  const float g = h2f(gu[m * 2 * I + i]);
  const float u = h2f(gu[m * 2 * I + I + i]);
  y[m * I + i] = f2h(g / (1.0f + expf(-g)) * u);
}

}  // namespace

int64_t decode_attention_tiles(int64_t L) { return (L + kAttnTile - 1) / kAttnTile; }

hipError_t launch_add_rmsnorm(float* res, const uint16_t* delta, const uint16_t* w, uint16_t* y, int64_t M,
                              int64_t D, float eps, hipStream_t stream, const LaunchEvents& ev) {
  if (delta)
    launch(add_rmsnorm_kernel<true>, dim3((unsigned)M), dim3(kNormThreads), 0, stream, ev, res, delta, w, y, (int)D, eps);
  else
    launch(add_rmsnorm_kernel<false>, dim3((unsigned)M), dim3(kNormThreads), 0, stream, ev, res, delta, w, y, (int)D, eps);
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
    case 2: launch(attn_partial_kernel<2>, grid, dim3(128), 0, stream, e1, q, kc, vc, S_max, (int)L, T, ws); break;
    case 4: launch(attn_partial_kernel<4>, grid, dim3(256), 0, stream, e1, q, kc, vc, S_max, (int)L, T, ws); break;
    default: launch(attn_partial_kernel<8>, grid, dim3(512), 0, stream, e1, q, kc, vc, S_max, (int)L, T, ws); break;
  }
  launch(attn_combine_kernel, dim3((unsigned)Hq), dim3(64), 0, stream, e2, (const float*)ws, T, out);
  return hipGetLastError();
}

// Positions per tile of the fused attention: enough blocks (Hkv x tiles) to
// give every compute unit work at short contexts, longer tiles (fewer
// partials to combine) at long ones.
int attention_qkv_tile(int64_t Hkv, int64_t L) {
  const int64_t work = Hkv * L;
  return work >= 32768 ? 64 : work >= 4096 ? 32 : 16;
}

int64_t decode_attention_qkv_tiles(int64_t Hkv, int64_t L) {
  const int P = attention_qkv_tile(Hkv, L);
  return (L + P - 1) / P;
}

hipError_t launch_decode_attention_qkv(const uint16_t* qkv, const uint16_t* qw, const uint16_t* kw,
                                       const float* cos_sin, int64_t pos, int64_t Hq, int64_t Hkv, float eps,
                                       uint16_t* kc, uint16_t* vc, int64_t S_max, uint16_t* out, float* ws,
                                       hipStream_t stream, const LaunchEvents& ev) {
  const int64_t L = pos + 1;
  const int P = attention_qkv_tile(Hkv, L);
  const int T = (int)((L + P - 1) / P);
  const int R = (int)(Hq / Hkv);
  LaunchEvents e1, e2;  // the measurement hook spans both kernels
  e1.start = ev.start;
  e2.stop = ev.stop;
  const dim3 grid((unsigned)Hkv, (unsigned)T);
  const float* cs = cos_sin + pos * kHeadDim;
#define LAQ_ATTN_QKV(RV, PV)                                                                                 \
  launch(attn_qkv_partial_kernel<RV, PV>, grid, dim3(64 * RV), 0, stream, e1, kc, vc, (int)S_max, (int)pos, qkv, \
         qw, cs, eps, (int)Hq, kw, (int)Hkv, T, ws)
#define LAQ_ATTN_QKV_P(RV)                 \
  do {                                     \
    if (P == 64) LAQ_ATTN_QKV(RV, 64);     \
    else if (P == 32) LAQ_ATTN_QKV(RV, 32); \
    else LAQ_ATTN_QKV(RV, 16);             \
  } while (0)
  switch (R) {
    case 1: LAQ_ATTN_QKV_P(1); break;
    case 2: LAQ_ATTN_QKV_P(2); break;
    case 4: LAQ_ATTN_QKV_P(4); break;
    default: LAQ_ATTN_QKV_P(8); break;
  }
#undef LAQ_ATTN_QKV_P
#undef LAQ_ATTN_QKV
  launch(attn_combine2_kernel<4>, dim3((unsigned)Hq), dim3(256), 0, stream, e2, (const float*)ws, T, out);
  return hipGetLastError();
}

hipError_t launch_silu_mul(const uint16_t* gu, uint16_t* y, int64_t M, int64_t I, hipStream_t stream,
                           const LaunchEvents& ev) {
  launch(silu_mul_kernel, dim3((unsigned)((I + 255) / 256), (unsigned)M), dim3(256), 0, stream, ev, gu, y, I);
  return hipGetLastError();
}

}  // namespace laq
