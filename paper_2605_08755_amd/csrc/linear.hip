// Dequantize-fused GEMV / skinny GEMM:
//   y[m][n] = sum_g s[n][g] * sum_{k in g} x[m][k] * (q[n][k] - z[n][g])
// i.e. Eq. 1's w_hat = s (q - z) applied inside the dot product, with fp16
// activations, fp32 accumulation and one fp16 rounding per output.
//
// Work mapping: a 256-thread block owns 256/L consecutive output rows; the L
// lanes of a row (a power of two, <= 64, so a row never leaves its wave)
// take groups j, j+L, j+2L, ... of that row.  For a group a lane issues one
// 16-byte load per plane (planes are K-contiguous per row, so the L lanes of
// a row read L*16 contiguous bytes per plane), keeps the codes in registers
// and reads the group's activations from LDS.  The row's partial sums are
// combined with a fixed butterfly over its L lanes: results are
// deterministic and no cross-block reduction is needed.
//
// Unpack without offsets: a code field at bits [p, p+3) of a 16-bit half,
// masked out of its word with every other bit cleared, is an fp16 subnormal
// of value q * 2^(p-24), exactly.  One AND therefore yields two fp16
// operands (the low and high halves hold consecutive k), and v_dot2_f32_f16
// multiplies them with two activations and accumulates in fp32.  Fields at
// the same p share an accumulator; the accumulators are rescaled by their
// exact power of two once per group, and the zero point enters once per
// group as z * sum_k x[m][k] (the per-group activation sums are computed
// while staging x).
#include <algorithm>

#include "laq_internal.h"

namespace laq {

namespace {

constexpr int kThreads = 256;
constexpr int kMaxGroupsPerLane = 4;   // groups a lane holds in registers per K tile
constexpr int kGroupStrideU4 = 17;     // 16 u32x4 of activations + 1 pad (bank spread)
constexpr int kLdsBudget = 64 * 1024;  // bytes of activation tile per block

__device__ __forceinline__ float dot2(uint32_t codes, uint32_t xpair, float acc) {
  return __builtin_amdgcn_fdot2(as_half2(codes), as_half2(xpair), acc, false);
}

// Accumulate one 32-code chunk (plane words w[0..BITS-1]) against the
// chunk's 16 activation pairs xp[0..15] (pair t = x[2t], x[2t+1]).
template <int BITS>
__device__ __forceinline__ void chunk_dot(const uint32_t (&w)[BITS], const uint32_t (&xp)[16],
                                          float (&acc)[4]) {
  if constexpr (BITS == 3) {
    // acc[0]: fields at bits 0-2 (x 2^-24), acc[1]: bits 3-5 (x 2^-21),
    // acc[2]: bits 6-8 (x 2^-18), acc[3]: bits 7-9 (x 2^-17)
#pragma unroll
    for (int p = 0; p < 3; ++p) {
      const uint32_t t = w[p] >> 10;
      acc[0] = dot2(w[p] & 0x00070007u, xp[5 * p + 0], acc[0]);
      acc[1] = dot2(w[p] & 0x00380038u, xp[5 * p + 1], acc[1]);
      acc[2] = dot2(w[p] & 0x01C001C0u, xp[5 * p + 2], acc[2]);
      acc[0] = dot2(t & 0x00070007u, xp[5 * p + 3], acc[0]);
      acc[1] = dot2(t & 0x00380038u, xp[5 * p + 4], acc[1]);
    }
    // codes 30/31: bit j of the code is bit 9 (low) / 25 (high) of plane j;
    // move plane 0's bit to 7 and plane 1's to 8 to rebuild a 3-bit field.
    const uint32_t spare = ((w[0] >> 2) & 0x00800080u) | ((w[1] >> 1) & 0x01000100u) |
                           (w[2] & 0x02000200u);
    acc[3] = dot2(spare, xp[15], acc[3]);
  } else {
    // acc[0]: nibbles at bits 0-3 (x 2^-24), acc[1]: bits 4-7 (x 2^-20)
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const uint32_t t = w[p] >> 8;
      acc[0] = dot2(w[p] & 0x000F000Fu, xp[4 * p + 0], acc[0]);
      acc[1] = dot2(w[p] & 0x00F000F0u, xp[4 * p + 1], acc[1]);
      acc[0] = dot2(t & 0x000F000Fu, xp[4 * p + 2], acc[0]);
      acc[1] = dot2(t & 0x00F000F0u, xp[4 * p + 3], acc[1]);
    }
  }
}

template <int BITS>
__device__ __forceinline__ float classes_to_value(const float (&acc)[4]) {
  if constexpr (BITS == 3)
    return fmaf(acc[0], 16777216.0f, fmaf(acc[1], 2097152.0f, fmaf(acc[2], 262144.0f, acc[3] * 131072.0f)));
  else
    return fmaf(acc[0], 16777216.0f, acc[1] * 1048576.0f);
}

template <int BITS, int MT>
__global__ __launch_bounds__(kThreads) void linear_kernel(
    const u32x4* __restrict__ x4, const u32x4* __restrict__ qw4, const uint16_t* __restrict__ scales,
    const uint8_t* __restrict__ zeros, uint16_t* __restrict__ y, int M, int N, int G, int lpr_log2,
    int tile_groups) {
  extern __shared__ u32x4 lds[];
  float* xsum = reinterpret_cast<float*>(lds + (size_t)MT * tile_groups * kGroupStrideU4);

  const int L = 1 << lpr_log2;
  const int t = threadIdx.x;
  const int j = t & (L - 1);
  const int rows_per_block = kThreads >> lpr_log2;
  const int n = blockIdx.x * rows_per_block + (t >> lpr_log2);
  const bool row_ok = n < N;
  const int n_c = row_ok ? n : N - 1;  // clamped row for address arithmetic

  float yacc[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) yacc[m] = 0.0f;

  for (int tg0 = 0; tg0 < G; tg0 += tile_groups) {
    const int tgn = min(tile_groups, G - tg0);

    // 1. Issue this lane's weight loads for the tile (kept in registers).
    u32x4 wv[kMaxGroupsPerLane][BITS];
    float sv[kMaxGroupsPerLane];
    float zv[kMaxGroupsPerLane];
#pragma unroll
    for (int i = 0; i < kMaxGroupsPerLane; ++i) {
      const int gl = j + i * L;
      const bool ok = row_ok && gl < tgn;
      const int g = ok ? tg0 + gl : 0;  // in-bounds address even when predicated off
#pragma unroll
      for (int p = 0; p < BITS; ++p)
        wv[i][p] = ok ? __builtin_nontemporal_load(qw4 + ((int64_t)n_c * BITS + p) * G + g) : u32x4{0u, 0u, 0u, 0u};
      sv[i] = ok ? (float)__builtin_bit_cast(_Float16, scales[(int64_t)n_c * G + g]) : 0.0f;
      zv[i] = ok ? (float)zeros[(int64_t)n_c * G + g] : 0.0f;
    }

    // 2. Stage the activation tile into LDS with its per-group sums.
    const int units = MT * tgn * 16;  // u32x4 units of the tile
    for (int u = t; u < units; u += kThreads) {
      const int m = u / (tgn * 16);
      const int rem = u - m * tgn * 16;
      const int gg = rem >> 4;
      const int bb = rem & 15;
      u32x4 v = u32x4{0u, 0u, 0u, 0u};
      if (m < M) v = x4[((int64_t)m * G + tg0 + gg) * 16 + bb];
      const uint32_t vw[4] = {v.x, v.y, v.z, v.w};
      float s = 0.0f;
#pragma unroll
      for (int e = 0; e < 8; ++e) s += (float)__builtin_bit_cast(_Float16, (uint16_t)(vw[e >> 1] >> (16 * (e & 1))));
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) s += __shfl_xor(s, o, 16);
      lds[(m * tile_groups + gg) * kGroupStrideU4 + bb] = v;
      if (bb == 0) xsum[m * tile_groups + gg] = s;
    }
    __syncthreads();

    // 3. Dot products.
#pragma unroll
    for (int i = 0; i < kMaxGroupsPerLane; ++i) {
      const int gl = j + i * L;
      if (gl < tgn) {
        float acc[MT][4];
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
          for (int c = 0; c < 4; ++c) acc[m][c] = 0.0f;
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) {
          uint32_t w[BITS];
#pragma unroll
          for (int p = 0; p < BITS; ++p) {
            const u32x4 q = wv[i][p];
            w[p] = cc == 0 ? q.x : cc == 1 ? q.y : cc == 2 ? q.z : q.w;
          }
#pragma unroll
          for (int m = 0; m < MT; ++m) {
            const u32x4* xp4 = lds + (m * tile_groups + gl) * kGroupStrideU4 + cc * 4;
            uint32_t xp[16];
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              const u32x4 xv = xp4[v];
              xp[4 * v + 0] = xv.x;
              xp[4 * v + 1] = xv.y;
              xp[4 * v + 2] = xv.z;
              xp[4 * v + 3] = xv.w;
            }
            chunk_dot<BITS>(w, xp, acc[m]);
          }
        }
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          const float a = classes_to_value<BITS>(acc[m]);
          const float d = fmaf(-zv[i], xsum[m * tile_groups + gl], a);
          yacc[m] = fmaf(sv[i], d, yacc[m]);
        }
      }
    }
    if (tg0 + tile_groups < G) __syncthreads();  // LDS is restaged for the next tile
  }

  // 4. Combine the L lanes of each row (fixed butterfly) and store fp16.
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    float v = yacc[m];
    for (int o = L >> 1; o >= 1; o >>= 1) v += __shfl_xor(v, o, L);
    if (j == 0 && row_ok && m < M) y[(int64_t)m * N + n] = __builtin_bit_cast(uint16_t, (_Float16)v);
  }
}

// ---------------------------------------------------------------------------
// Flat-unit kernel (used when the block's activations fit in LDS).
//
// A block owns R consecutive rows and every (row, group) unit of them,
// dealt out flat over its 256 threads (unit u = r*G + g goes to thread
// u mod 256), so lanes are balanced for any group count.  Activations are
// loaded first (they are needed first and sit in L2), then the weights of
// the thread's units; the activation tile is written to LDS together with
// each group's sum.  Every unit writes its partial to LDS, and each row's
// partials are added in a fixed order (16 lanes per row, then a DPP tree).
// All global reads are buffer loads against per-block extents: addresses
// are 32-bit offsets from scalar bases, and an offset past the extent reads
// zero, so the tail of the last block needs no extra guards.
// ---------------------------------------------------------------------------
constexpr uint32_t kOnesPair = 0x3C003C00u;  // fp16 (1.0, 1.0)
constexpr int kBufferFlags = 0x00020000;     // raw buffer, 32-bit data
// Cache policy of the weight stream: non-temporal, read once, so it does not
// evict the activations every block re-reads from L2.
constexpr int kStreamPolicy = 2;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kBufferFlags);
}

// Loads of one unit.  A unit past the block's rows (r >= rows) has offsets
// past each buffer's extent, so it reads zeros with no condition: a branch
// or select around a load makes the compiler wait for the load at the
// join, which would serialize the whole batch of loads.
template <int BITS>
__device__ __forceinline__ void load_flat_unit(__amdgpu_buffer_rsrc_t qr, __amdgpu_buffer_rsrc_t sr,
                                               __amdgpu_buffer_rsrc_t zr, int r, int g, int G,
                                               u32x4 (&w)[BITS], float& s, float& z) {
  const uint32_t unit = (uint32_t)(r * G + g);
#pragma unroll
  for (int p = 0; p < BITS; ++p)
    w[p] = __builtin_amdgcn_raw_buffer_load_b128(qr, ((uint32_t)(r * BITS + p) * G + g) * 16, 0, kStreamPolicy);
  s = (float)__builtin_bit_cast(_Float16, __builtin_amdgcn_raw_buffer_load_b16(sr, unit * 2, 0, 0));
  z = (float)__builtin_amdgcn_raw_buffer_load_b8(zr, unit, 0, 0);
}

// Sum over the 16 lanes of a DPP row; every lane receives the same total
// (each step adds a lane's value to its partner's, a commutative pairing).
__device__ __forceinline__ float row16_sum(float v) {
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false));   // quad_perm [1,0,3,2]
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, false));   // quad_perm [2,3,0,1]
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x141, 0xF, 0xF, false));  // row_half_mirror
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x140, 0xF, 0xF, false));  // row_mirror
  return v;
}

// One staging pass: activation units base + t + i*NT (16 bytes each, the
// 16 lanes of a DPP row holding one 128-group) go to LDS, and the group's
// sum of activations to xsum.
template <int MT, int NT, int XB>
__device__ __forceinline__ void stage_x_pass(const u32x4 (&xv)[XB], int base, int t, int XU,
                                             u32x4* xl, float* xsum) {
#pragma unroll
  for (int i = 0; i < XB; ++i) {
    const int idx = base + t + i * NT;
    float ps = dot2(xv[i].x, kOnesPair, 0.0f);
    ps = dot2(xv[i].y, kOnesPair, ps);
    ps = dot2(xv[i].z, kOnesPair, ps);
    ps = dot2(xv[i].w, kOnesPair, ps);
    ps = row16_sum(ps);
    if (idx < XU) {
      const int mg = idx >> 4;  // m*G + g
      const int b = idx & 15;
      xl[mg * kGroupStrideU4 + b] = xv[i];
      if (b == 0) xsum[mg] = ps;
    }
  }
}

// Sum over the 64 lanes of a wave in a fixed order (every lane receives it):
// DPP sums of the four 16-lane rows, then the rows in order (lane reads; no
// LDS round trips).
__device__ __forceinline__ float wave_sum64(float v) {
  v = row16_sum(v);
  const int b = __builtin_bit_cast(int, v);
  return ((__builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 0)) +
           __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 16))) +
          __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 32))) +
         __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 48));
}

// Norm prologue, loads: this thread's activation units t + i*NT (8 values
// each) of the residual, the delta and the norm weight.  Units past the row
// (and the delta when there is none) read zeros.
template <int XB>
struct NormLoads {
  u32x4 r0[XB], r1[XB], d[XB], w[XB];
};

template <int XB, int NT>
__device__ __forceinline__ NormLoads<XB> norm_issue(const NormPrologue& np, int K, int t) {
  NormLoads<XB> L;
  const __amdgpu_buffer_rsrc_t rr = make_rsrc(np.res_in, (uint32_t)K * 4);
  const __amdgpu_buffer_rsrc_t dr = make_rsrc(np.delta, np.delta ? (uint32_t)K * 2 : 0u);
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(np.weight, (uint32_t)K * 2);
#pragma unroll
  for (int i = 0; i < XB; ++i) {
    const uint32_t u = (uint32_t)(t + i * NT);
    L.r0[i] = __builtin_amdgcn_raw_buffer_load_b128(rr, u * 32, 0, 0);
    L.r1[i] = __builtin_amdgcn_raw_buffer_load_b128(rr, u * 32 + 16, 0, 0);
    L.d[i] = __builtin_amdgcn_raw_buffer_load_b128(dr, u * 16, 0, 0);
    L.w[i] = __builtin_amdgcn_raw_buffer_load_b128(wr, u * 16, 0, 0);
  }
  return L;
}

__device__ __forceinline__ float u2f(uint32_t u) { return __builtin_bit_cast(float, u); }
__device__ __forceinline__ float lo_h(uint32_t u) { return (float)__builtin_bit_cast(_Float16, (uint16_t)(u & 0xFFFFu)); }
__device__ __forceinline__ float hi_h(uint32_t u) { return (float)__builtin_bit_cast(_Float16, (uint16_t)(u >> 16)); }
__device__ __forceinline__ uint32_t pack_h2(float a, float b) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)a) | ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)b) << 16);
}

// Norm prologue, arithmetic: v = res + delta, the row's sum of squares over
// the block (thread partials in unit order, wave sums, waves in order),
// x = fp16(v / sqrt(mean(v^2) + eps) * weight) into xv (the activation units
// the staging pass writes to LDS).  The writer block stores v to res_out.
// Every thread of the block calls it (one barrier).  The whole row is this
// thread's XB units: K <= 8 * XB * NT.
template <int XB, int NT>
__device__ __forceinline__ void norm_finish(const NormLoads<XB>& L, const NormPrologue& np, int K, int t,
                                            bool writer, u32x4 (&xv)[XB]) {
  __shared__ float red[NT / 64];
  float v[XB][8];
  float ss = 0.0f;
#pragma unroll
  for (int i = 0; i < XB; ++i) {
    // (elements are copied to scalars first: a bit cast of a vector element
    // expression was compiled as a cast of element 0)
    const float r[8] = {u2f(L.r0[i].x), u2f(L.r0[i].y), u2f(L.r0[i].z), u2f(L.r0[i].w),
                        u2f(L.r1[i].x), u2f(L.r1[i].y), u2f(L.r1[i].z), u2f(L.r1[i].w)};
    const uint32_t d[4] = {L.d[i].x, L.d[i].y, L.d[i].z, L.d[i].w};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      v[i][e] = r[e] + ((e & 1) ? hi_h(d[e >> 1]) : lo_h(d[e >> 1]));
      ss = fmaf(v[i][e], v[i][e], ss);
    }
  }
  ss = wave_sum64(ss);
  if ((t & 63) == 0) red[t >> 6] = ss;
  __syncthreads();
  float tot = 0.0f;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) tot += red[w];
  const float inv = 1.0f / sqrtf(tot / (float)K + np.eps);
#pragma unroll
  for (int i = 0; i < XB; ++i) {
    const uint32_t w[4] = {L.w[i].x, L.w[i].y, L.w[i].z, L.w[i].w};
    uint32_t x[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      x[e] = pack_h2(v[i][2 * e] * inv * lo_h(w[e]), v[i][2 * e + 1] * inv * hi_h(w[e]));
    xv[i] = u32x4{x[0], x[1], x[2], x[3]};
  }
  if (writer && np.res_out != nullptr) {
#pragma unroll
    for (int i = 0; i < XB; ++i) {
      const int u = t + i * NT;
      if (8 * u < K) {
        float4* o = reinterpret_cast<float4*>(np.res_out + 8 * u);
        o[0] = float4{v[i][0], v[i][1], v[i][2], v[i][3]};
        o[1] = float4{v[i][4], v[i][5], v[i][6], v[i][7]};
      }
    }
  }
}

// Dot products of RPL units that share group g (rows of one lane): the
// group's activations are read from LDS once per chunk and used for every
// row, so LDS reads per weight fall by RPL.
template <int BITS, int MT, int RPL>
__device__ __forceinline__ void units_dot(const u32x4 (&wv)[RPL][BITS], const u32x4* xl, int G, int g,
                                          float (&acc)[RPL][MT][4]) {
#pragma unroll
  for (int i = 0; i < RPL; ++i)
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[i][m][c] = 0.0f;
#pragma unroll
  for (int cc = 0; cc < 4; ++cc) {
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const u32x4* xp4 = xl + (m * G + g) * kGroupStrideU4 + cc * 4;
      uint32_t xp[16];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const u32x4 q = xp4[v];
        xp[4 * v + 0] = q.x;
        xp[4 * v + 1] = q.y;
        xp[4 * v + 2] = q.z;
        xp[4 * v + 3] = q.w;
      }
#pragma unroll
      for (int i = 0; i < RPL; ++i) {
        uint32_t w[BITS];
#pragma unroll
        for (int p = 0; p < BITS; ++p) w[p] = wv[i][p][cc];
        chunk_dot<BITS>(w, xp, acc[i][m]);
      }
    }
  }
}

// Output stage of the fused gate|up + SiLU-and-multiply linear: the weight
// rows come in (gate, up) pairs, rows 2j and 2j + 1, and output column
// (row0 + 2j) / 2 of the N / 2 columns is silu(gate) * up of the two rows'
// fp32 sums, rounded once to fp16.  R, row0 and rows are even.
template <int MT, int NT>
__device__ __forceinline__ void swiglu_rows(const float* part, int R, int G, int rows, int M, int N, int64_t row0,
                                            uint16_t* __restrict__ y, int t) {
  const int l = t & 15;
  for (int pr = t >> 4; 2 * pr < rows; pr += NT / 16) {
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      float ag = 0.0f, au = 0.0f;
      for (int g = l; g < G; g += 16) {
        ag += part[m * R * G + (2 * pr) * G + g];
        au += part[m * R * G + (2 * pr + 1) * G + g];
      }
      ag = row16_sum(ag);
      au = row16_sum(au);
      if (l == 0 && m < M)
        y[(int64_t)m * (N / 2) + row0 / 2 + pr] = __builtin_bit_cast(uint16_t, (_Float16)(ag / (1.0f + expf(-ag)) * au));
    }
  }
}

// A value held in scalar registers from the point of the call on: the "+s"
// operand keeps the compiler from re-reading a kernel argument where it is
// used.  Arguments past the preloaded ones (the output pointer, the norm's
// eps and residual output) are pinned right after a block issues its loads,
// so their scalar round trip overlaps the loads instead of sitting at the
// end of the block's critical path.
template <typename T>
__device__ __forceinline__ void pin_sgpr(T& v) {
  asm volatile("" : "+s"(v));
}

// One block of the flat kernel: rows block*R .. block*R + R - 1 of one call.
// Thread t takes units t + i*NT (i < UPT) of each pass over the block's
// units; every launch uses UPT = 1 (more units per thread measured slower).
// SW: the fused gate|up + SiLU-and-multiply output stage (swiglu_rows).
template <int BITS, int MT, int NT, int UPT, int XB, bool SW = false, bool NORM = false, bool RES = false>
__device__ __forceinline__ void flat_block(
    const uint16_t* __restrict__ x, const uint32_t* __restrict__ qw, const uint16_t* __restrict__ scales,
    const uint8_t* __restrict__ zeros, uint16_t* __restrict__ y, int M, int N, int G, int R, float inv_g,
    int block, const NormPrologue& np = NormPrologue{}, const ResidualEpilogue& re = ResidualEpilogue{}) {
  extern __shared__ u32x4 lds[];
  u32x4* xl = lds;                                                                // [MT][G][17]
  float* xsum = reinterpret_cast<float*>(lds + (size_t)MT * G * kGroupStrideU4);  // [MT][G]
  float* part = xsum + MT * G;                                                    // [MT][R*G]

  const int t = threadIdx.x;
  // An idle block (an XCD-rounding slot past the last row) has rows = 0: every
  // buffer extent is zero, so it loads and stores nothing.  (32-bit unsigned
  // scalar arithmetic: block * R < N + 8R < 2^32.)
  const uint32_t r0u = (uint32_t)block * (uint32_t)R;
  const int rows = r0u < (uint32_t)N ? (int)min((uint32_t)R, (uint32_t)N - r0u) : 0;
  const int64_t row0 = (int64_t)r0u;
  const int U = rows * G;
  const int XU = MT * G * 16;  // activation tile in 16-byte units (rows m >= M read as zero)

  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, (uint32_t)M * G * 256);
  const __amdgpu_buffer_rsrc_t qr = make_rsrc(qw + row0 * BITS * G * 4, (uint32_t)rows * BITS * G * 16);
  const __amdgpu_buffer_rsrc_t sr = make_rsrc(scales + row0 * G, (uint32_t)U * 2);
  const __amdgpu_buffer_rsrc_t zr = make_rsrc(zeros + row0 * G, (uint32_t)U);

  // Unit t + i*NT is (row r, group g).  Computed before any load so that no
  // load waits on it.  t / G as trunc((t + 0.5) * fl(1/G)): the quotient's
  // fractional part is at least 0.5/G away from an integer and the float
  // error is below 1025 * 2^-23 / G, so the truncation is exact for every
  // t < 1024 and G >= 1.
  const int r0 = (int)(((float)t + 0.5f) * inv_g);
  const int g0 = t - r0 * G;
  __builtin_amdgcn_sched_barrier(0);

  // 1. First pass of activation loads (needed first: they are staged while
  //    the weights stream in), then at once the weights of this thread's
  //    units.  The scheduling barrier keeps the activation processing below
  //    from being hoisted between the two batches of loads, which would make
  //    the weight stream wait for an activation round trip.
  //    Index XM = M*G*16 is the end of x's extent: loads past it read zero.
  u32x4 xv[XB];
  NormLoads<NORM ? XB : 1> nl_;  // the norm prologue's loads (NORM: the row's residual, delta, weight)
  if constexpr (NORM) {
    nl_ = norm_issue<XB, NT>(np, 128 * G, t);
  } else {
#pragma unroll
    for (int i = 0; i < XB; ++i)
      xv[i] = __builtin_amdgcn_raw_buffer_load_b128(xr, (uint32_t)(t + i * NT) * 16, 0, 0);
  }
  u32x4 wv[UPT][BITS];
  float sv[UPT], zv[UPT];
  int gi[UPT];
  {
    int r = r0, g = g0;
#pragma unroll
    for (int i = 0; i < UPT; ++i) {
      load_flat_unit<BITS>(qr, sr, zr, r, g, G, wv[i], sv[i], zv[i]);
      gi[i] = g;
      if (i + 1 < UPT) {  // (r, g) advance by (NT / G, NT % G)
        g += NT % G;
        r += NT / G;
        if (g >= G) { g -= G; r += 1; }
      }
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  uint16_t* const yo = [&] { uint16_t* p = y; pin_sgpr(p); return p; }();
  NormPrologue npl = np;
  if constexpr (NORM) {
    pin_sgpr(npl.eps);
    pin_sgpr(npl.res_out);
  }
  // RES: the residual of row t / 16, read now by the lane that will write
  // that row's output (every launch has rows <= NT / 16: one row per group
  // of 16 lanes); rows past the block's read zero.
  float rres = 0.0f;
  float* res_out = re.res_out;
  if constexpr (RES) {
    pin_sgpr(res_out);
    const __amdgpu_buffer_rsrc_t rr = make_rsrc(re.res_in + row0, (uint32_t)rows * 4);
    rres = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rr, (uint32_t)(t >> 4) * 4, 0, 0));
  }

  // 3. Stage activations and per-group sums (first pass from the loads above).
  if constexpr (NORM) norm_finish<XB, NT>(nl_, npl, 128 * G, t, block == 0, xv);
  stage_x_pass<MT, NT, XB>(xv, 0, t, XU, xl, xsum);
  for (int base = XB * NT; !NORM && base < XU; base += XB * NT) {
#pragma unroll
    for (int i = 0; i < XB; ++i)
      xv[i] = __builtin_amdgcn_raw_buffer_load_b128(xr, (uint32_t)(base + t + i * NT) * 16, 0, 0);
    stage_x_pass<MT, NT, XB>(xv, base, t, XU, xl, xsum);
  }
  __syncthreads();

  // 4. Units: one 128-group of one row each ((r, g) advance by (NT / G,
  //    NT % G) per unit step; every launch has R * G <= NT, one pass).
  const int dr = NT / G, dg = NT - (NT / G) * G;
  int ur = r0, ug = g0;
  for (int ub = 0; ub < U; ub += UPT * NT) {
    if (ub > 0) {
      int r = ur, g = ug;
#pragma unroll
      for (int i = 0; i < UPT; ++i) {
        load_flat_unit<BITS>(qr, sr, zr, r, g, G, wv[i], sv[i], zv[i]);
        gi[i] = g;
        g += dg;
        r += dr;
        if (g >= G) { g -= G; r += 1; }
      }
    }
#pragma unroll
    for (int i = 0; i < UPT; ++i) {
      const int u = ub + t + i * NT;
      if (u < U) {
        const int g = gi[i];
        float acc[MT][4];
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
          for (int c = 0; c < 4; ++c) acc[m][c] = 0.0f;
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) {
          uint32_t w[BITS];
#pragma unroll
          for (int p = 0; p < BITS; ++p) w[p] = wv[i][p][cc];
#pragma unroll
          for (int m = 0; m < MT; ++m) {
            const u32x4* xp4 = xl + (m * G + g) * kGroupStrideU4 + cc * 4;
            uint32_t xp[16];
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              const u32x4 q = xp4[v];
              xp[4 * v + 0] = q.x;
              xp[4 * v + 1] = q.y;
              xp[4 * v + 2] = q.z;
              xp[4 * v + 3] = q.w;
            }
            chunk_dot<BITS>(w, xp, acc[m]);
          }
        }
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          const float a = classes_to_value<BITS>(acc[m]);
          part[m * R * G + u] = sv[i] * fmaf(-zv[i], xsum[m * G + g], a);
        }
      }
    }
    // advance this thread's unit cursor by one batch
#pragma unroll
    for (int i = 0; i < UPT; ++i) {
      ug += dg;
      ur += dr;
      if (ug >= G) { ug -= G; ur += 1; }
    }
  }
  __syncthreads();

  // 5. Row sums in a fixed order: lane l of a row's 16 adds groups l, l+16, ...
  const int l = t & 15;
  if constexpr (SW) {
    swiglu_rows<MT, NT>(part, R, G, rows, M, N, row0, yo, t);
  } else {
    for (int rr = t >> 4; rr < rows; rr += NT / 16) {
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        float acc = 0.0f;
        for (int g = l; g < G; g += 16) acc += part[m * R * G + rr * G + g];
        acc = row16_sum(acc);
        if (l == 0 && m < M) {
          const _Float16 yh = (_Float16)acc;
          if (!RES || yo != nullptr) yo[(int64_t)m * N + row0 + rr] = __builtin_bit_cast(uint16_t, yh);
          if constexpr (RES) res_out[row0 + rr] = rres + (float)yh;
        }
      }
    }
  }
}

// One block of the flat kernel with RPL rows per lane: the block's R rows
// form RPL layers of R1 = R / RPL rows (R1 * G <= NT), and thread
// t = r*G + g of the first layer takes group g of rows r, r + R1, r + 2*R1,
// ...  Loads, staging and the row sums are those of flat_block.
template <int BITS, int MT, int NT, int RPL, int XB, bool SW = false, bool NORM = false, bool RES = false>
__device__ __forceinline__ void flat_block_rpl(
    const uint16_t* __restrict__ x, const uint32_t* __restrict__ qw, const uint16_t* __restrict__ scales,
    const uint8_t* __restrict__ zeros, uint16_t* __restrict__ y, int M, int N, int G, int R, float inv_g,
    int block, const NormPrologue& np = NormPrologue{}, const ResidualEpilogue& re = ResidualEpilogue{}) {
  extern __shared__ u32x4 lds[];
  u32x4* xl = lds;                                                                // [MT][G][17]
  float* xsum = reinterpret_cast<float*>(lds + (size_t)MT * G * kGroupStrideU4);  // [MT][G]
  float* part = xsum + MT * G;                                                    // [MT][R*G]

  const int t = threadIdx.x;
  // An idle block (an XCD-rounding slot past the last row) has rows = 0: every
  // buffer extent is zero, so it loads and stores nothing.  (32-bit unsigned
  // scalar arithmetic: block * R < N + 8R < 2^32.)
  const uint32_t r0u = (uint32_t)block * (uint32_t)R;
  const int rows = r0u < (uint32_t)N ? (int)min((uint32_t)R, (uint32_t)N - r0u) : 0;
  const int64_t row0 = (int64_t)r0u;
  const int U = rows * G;
  const int XU = MT * G * 16;  // activation tile in 16-byte units (rows m >= M read as zero)
  const int R1 = R / RPL;

  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, (uint32_t)M * G * 256);
  const __amdgpu_buffer_rsrc_t qr = make_rsrc(qw + row0 * BITS * G * 4, (uint32_t)rows * BITS * G * 16);
  const __amdgpu_buffer_rsrc_t sr = make_rsrc(scales + row0 * G, (uint32_t)U * 2);
  const __amdgpu_buffer_rsrc_t zr = make_rsrc(zeros + row0 * G, (uint32_t)U);

  // Thread t = r0*G + g0 (t / G computed as in flat_block).  Threads past
  // the first layer (r0 >= R1) own no unit: their loads start at row R,
  // past every extent, and read zeros.
  const int r0 = (int)(((float)t + 0.5f) * inv_g);
  const int g0 = t - r0 * G;
  const int rb = r0 < R1 ? r0 : R;
  __builtin_amdgcn_sched_barrier(0);

  // 1. First pass of activation loads (needed first: they are staged while
  //    the weights stream in), then at once the weights of this thread's
  //    units.  The scheduling barrier keeps the activation processing below
  //    from being hoisted between the two batches of loads, which would make
  //    the weight stream wait for an activation round trip.
  //    Index XM = M*G*16 is the end of x's extent: loads past it read zero.
  u32x4 xv[XB];
  NormLoads<NORM ? XB : 1> nl_;  // the norm prologue's loads (NORM: the row's residual, delta, weight)
  if constexpr (NORM) {
    nl_ = norm_issue<XB, NT>(np, 128 * G, t);
  } else {
#pragma unroll
    for (int i = 0; i < XB; ++i)
      xv[i] = __builtin_amdgcn_raw_buffer_load_b128(xr, (uint32_t)(t + i * NT) * 16, 0, 0);
  }
  u32x4 wv[RPL][BITS];
  float sv[RPL], zv[RPL];
#pragma unroll
  for (int i = 0; i < RPL; ++i) load_flat_unit<BITS>(qr, sr, zr, rb + i * R1, g0, G, wv[i], sv[i], zv[i]);
  __builtin_amdgcn_sched_barrier(0);
  uint16_t* const yo = [&] { uint16_t* p = y; pin_sgpr(p); return p; }();
  NormPrologue npl = np;
  if constexpr (NORM) {
    pin_sgpr(npl.eps);
    pin_sgpr(npl.res_out);
  }
  // RES: the residual of row t / 16, read now by the lane that will write
  // that row's output (every launch has rows <= NT / 16: one row per group
  // of 16 lanes); rows past the block's read zero.
  float rres = 0.0f;
  float* res_out = re.res_out;
  if constexpr (RES) {
    pin_sgpr(res_out);
    const __amdgpu_buffer_rsrc_t rr = make_rsrc(re.res_in + row0, (uint32_t)rows * 4);
    rres = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rr, (uint32_t)(t >> 4) * 4, 0, 0));
  }

  // 2. Stage activations and per-group sums (first pass from the loads above).
  if constexpr (NORM) norm_finish<XB, NT>(nl_, npl, 128 * G, t, block == 0, xv);
  stage_x_pass<MT, NT, XB>(xv, 0, t, XU, xl, xsum);
  for (int base = XB * NT; !NORM && base < XU; base += XB * NT) {
#pragma unroll
    for (int i = 0; i < XB; ++i)
      xv[i] = __builtin_amdgcn_raw_buffer_load_b128(xr, (uint32_t)(base + t + i * NT) * 16, 0, 0);
    stage_x_pass<MT, NT, XB>(xv, base, t, XU, xl, xsum);
  }
  __syncthreads();

  // 3. Units: the partial of unit (r, g) goes to part[m][r*G + g].
  // Rows past `rows` read zero weights, scales and zero points, so their
  // partials are zero (and never summed).
  if (r0 < R1) {
    float acc[RPL][MT][4];
    units_dot<BITS, MT, RPL>(wv, xl, G, g0, acc);
#pragma unroll
    for (int i = 0; i < RPL; ++i)
#pragma unroll
      for (int m = 0; m < MT; ++m)
        part[m * R * G + (r0 + i * R1) * G + g0] =
            sv[i] * fmaf(-zv[i], xsum[m * G + g0], classes_to_value<BITS>(acc[i][m]));
  }
  __syncthreads();

  // 4. Row sums in a fixed order: lane l of a row's 16 adds groups l, l+16, ...
  const int l = t & 15;
  if constexpr (SW) {
    swiglu_rows<MT, NT>(part, R, G, rows, M, N, row0, yo, t);
  } else {
    for (int rr = t >> 4; rr < rows; rr += NT / 16) {
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        float acc = 0.0f;
        for (int g = l; g < G; g += 16) acc += part[m * R * G + rr * G + g];
        acc = row16_sum(acc);
        if (l == 0 && m < M) {
          const _Float16 yh = (_Float16)acc;
          if (!RES || yo != nullptr) yo[(int64_t)m * N + row0 + rr] = __builtin_bit_cast(uint16_t, yh);
          if constexpr (RES) res_out[row0 + rr] = rres + (float)yh;
        }
      }
    }
  }
}

// The arguments every wave needs before its first memory request come first
// (they arrive preloaded in scalar registers); y, needed only at the end,
// comes last.
template <int BITS, int MT, int NT, int RPL, int XB, bool SW>
__global__ __launch_bounds__(NT) void linear_flat_kernel(
    const uint16_t* __restrict__ x, const uint32_t* __restrict__ qw, const uint16_t* __restrict__ scales,
    const uint8_t* __restrict__ zeros, int M, int N, int G, int R, float inv_g, int nblocks,
    uint16_t* __restrict__ y) {
  // Slots of the XCD-rounded grid past nblocks get rows = 0 in flat_block (no
  // early return).
  if constexpr (RPL == 1)
    flat_block<BITS, MT, NT, 1, XB, SW>(x, qw, scales, zeros, y, M, N, G, R, inv_g, xcd_block(nblocks));
  else
    flat_block_rpl<BITS, MT, NT, RPL, XB, SW>(x, qw, scales, zeros, y, M, N, G, R, inv_g, xcd_block(nblocks));
}

// Batch-1 linear with the residual output stage: y = x w_hat^T as
// linear_flat_kernel computes it, and res_out[n] = res_in[n] + y[n]; y may be
// null, and then only res_out is written (one output stream less).  The
// first fourteen dwords of arguments (preloaded) are what a wave needs before
// its first requests, res_in included; fl(1/G) comes from v_rcp_f32, whose
// error (one ulp) leaves trunc((t + 0.5) / G) exact for t < 1024 as in
// flat_block.
template <int BITS, int NT, int RPL, int XB>
__global__ __launch_bounds__(NT) void linear_flat_res_kernel(
    const uint16_t* __restrict__ x, const uint32_t* __restrict__ qw, const uint16_t* __restrict__ scales,
    const uint8_t* __restrict__ zeros, int N, int G, int R, int nblocks, const float* __restrict__ res_in,
    uint16_t* __restrict__ y, float* __restrict__ res_out) {
  const float inv_g = __builtin_amdgcn_rcpf((float)G);
  ResidualEpilogue re;
  re.res_in = res_in;
  re.res_out = res_out;
  if constexpr (RPL == 1)
    flat_block<BITS, 1, NT, 1, XB, false, false, true>(x, qw, scales, zeros, y, 1, N, G, R, inv_g,
                                                       xcd_block(nblocks), NormPrologue{}, re);
  else
    flat_block_rpl<BITS, 1, NT, RPL, XB, false, false, true>(x, qw, scales, zeros, y, 1, N, G, R, inv_g,
                                                             xcd_block(nblocks), NormPrologue{}, re);
}

// The same with the residual add + RMSNorm prologue (M = 1; no activation
// pointer: the row is formed from np, XB units of 8 elements per thread).
// The first fourteen dwords of arguments (preloaded in scalar registers) are
// what a wave needs before its first requests: the three prologue rows, the
// weights, N and the packed shape gr = G | R << 8 (G <= 64, R <= 512); the
// block count and fl(1/G) are derived from them.
template <int NT, int RPL, bool SW, int BITS, int XB>
__global__ __launch_bounds__(NT) void linear_flat_norm_kernel(
    const float* __restrict__ res_in, const uint16_t* __restrict__ delta, const uint16_t* __restrict__ weight,
    const uint32_t* __restrict__ qw, const uint16_t* __restrict__ scales, const uint8_t* __restrict__ zeros, int N,
    int gr, uint16_t* __restrict__ y, float* __restrict__ res_out, float eps) {
  const int G = gr & 0xFF, R = gr >> 8;
  const float inv_g = 1.0f / (float)G;  // correctly rounded, as the host's
  const int nblocks = (N - 1) / R + 1;
  NormPrologue np;
  np.res_in = res_in;
  np.delta = delta;
  np.weight = weight;
  np.res_out = res_out;
  np.eps = eps;
  if constexpr (RPL == 1)
    flat_block<BITS, 1, NT, 1, XB, SW, true>(nullptr, qw, scales, zeros, y, 1, N, G, R, inv_g, xcd_block(nblocks), np);
  else
    flat_block_rpl<BITS, 1, NT, RPL, XB, SW, true>(nullptr, qw, scales, zeros, y, 1, N, G, R, inv_g,
                                                  xcd_block(nblocks), np);
}

// Several independent calls in one launch: block b belongs to the last call
// whose first block is <= b.  The call's fields are picked with constant
// indices (uniform selects), so the argument block is never indexed at run
// time.
template <int BITS, int MT, int NT, int XB>
__global__ __launch_bounds__(NT) void linear_flat_group_kernel(const LinearGroup grp, int M) {
  // Slots past the last call's blocks fall to that call with rows = 0.
  const int b = xcd_block(grp.blocks);
  LinearCall c = grp.call[0];
#pragma unroll
  for (int j = 1; j < kMaxGroup; ++j)
    if (j < grp.count && b >= grp.call[j].first_block) c = grp.call[j];
  flat_block<BITS, MT, NT, 1, XB>(c.x, c.qw, c.scales, c.zeros, c.y, M, c.N, c.G, c.R, c.inv_g, b - c.first_block);
}

// ---------------------------------------------------------------------------
// The SwiGLU MLP block of one token in one launch: residual add + RMSNorm,
// the gate|up linear with SiLU-and-multiply, and the down linear (the
// decode step's post-attention half of a decoder layer, Sec. 5 / Table 3
// setting, with every weight W3G128 or W4G128 under Eq. 1).
//
// The down linear is split over the intermediate dimension I: slice b
// (logical block b) owns intermediates [128b, 128b + 128), which are the
// 256 interleaved gate|up rows 256b .. 256b + 255 and group b of every down
// row.  The block
//   1. loads everything it needs at once: the residual row, the norm weight
//      and the delta (registers), its gate|up units (registers, UA per
//      thread), the scales and zero points of its down group (registers)
//      and the down codes of its group, D * BITS 16-byte pieces, straight
//      into LDS;
//   2. forms x = RMSNorm(residual + delta) as the norm-prologue linear does
//      and stages it with its group sums;
//   3. computes its 256 x G1 gate|up unit partials, then h = fp16(silu(gate)
//      * up) of its 128 intermediates (the fused gate|up linear's output
//      stage and rounding) and their sum;
//   4. computes its D down partials s * (sum_k q h - z sum_k h) and writes
//      them to part[b][0..D).
// The partials are added in a fixed order without any block waiting on
// another: slices form teams of team_size consecutive slices; the last block
// of a team to finish (an atomic counter per team) adds its team's partials
// in slice order into team[k], and the last of those adders adds the team
// sums in team order and writes y in fp16.  Each adder resets its counter,
// so the counters are zero whenever no launch is in flight.
// ---------------------------------------------------------------------------
constexpr int kMlpThreads = 1024;
constexpr int kMlpDownUnits = 3;  // down rows per thread: D <= 3 * 1024

struct MlpArgs {
  NormPrologue np;
  const uint32_t* gu_qw;
  const uint16_t* gu_s;
  const uint8_t* gu_z;
  const uint32_t* dn_qw;
  const uint16_t* dn_s;
  const uint8_t* dn_z;
  uint16_t* y;
  float* part;      // [S][D]
  float* team;      // [T][D]
  uint32_t* count;  // [T + 1]
  int D, G1, S, team_size, T;
  float inv_g1;
};

// sum_{j < count} p[j * stride], added in order j = 0, 1, ...; the loads of
// up to kMlpSumBatch terms are issued together (each is a round trip to
// memory: one at a time they would serialize).
constexpr int kMlpSumBatch = 16;
__device__ __forceinline__ float ordered_sum(const float* p, int stride, int count) {
  float sum = 0.0f;
  for (int j0 = 0; j0 < count; j0 += kMlpSumBatch) {
    float v[kMlpSumBatch];
#pragma unroll
    for (int j = 0; j < kMlpSumBatch; ++j) v[j] = p[(size_t)min(j0 + j, count - 1) * stride];
#pragma unroll
    for (int j = 0; j < kMlpSumBatch; ++j)
      if (j0 + j < count) sum += v[j];
  }
  return sum;
}

template <int BITS, int UA>
__global__ __launch_bounds__(kMlpThreads) void mlp_block_kernel(const MlpArgs a) {
  typedef __attribute__((address_space(3))) void lds_void;
  extern __shared__ u32x4 lds[];
  __shared__ int last;
  const int D = a.D, G1 = a.G1, G2 = a.S;
  u32x4* dl = lds;                                        // [D * BITS] down codes of group b
  u32x4* xl = dl + (size_t)D * BITS;                      // [G1][17] x
  u32x4* hl = xl + (size_t)G1 * kGroupStrideU4;           // [16] h of the slice
  float* xsum = reinterpret_cast<float*>(hl + 16);        // [G1]
  float* pa = xsum + G1;                                  // [256 * G1] gate|up unit partials
  float* hsum = pa + 256 * G1;                            // [1]

  const int b = xcd_block(G2);
  if (b >= G2) return;  // XCD-rounding slot
  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;

  const __amdgpu_buffer_rsrc_t qa = make_rsrc(a.gu_qw + (size_t)b * 256 * BITS * G1 * 4, 256u * BITS * G1 * 16);
  const __amdgpu_buffer_rsrc_t sa = make_rsrc(a.gu_s + (size_t)b * 256 * G1, 256u * G1 * 2);
  const __amdgpu_buffer_rsrc_t za = make_rsrc(a.gu_z + (size_t)b * 256 * G1, 256u * G1);
  const __amdgpu_buffer_rsrc_t qd = make_rsrc(a.dn_qw, (uint32_t)D * BITS * G2 * 16);
  const __amdgpu_buffer_rsrc_t sd = make_rsrc(a.dn_s, (uint32_t)D * G2 * 2);
  const __amdgpu_buffer_rsrc_t zd = make_rsrc(a.dn_z, (uint32_t)D * G2);
  const int dr = kMlpThreads / G1, dg = kMlpThreads - (kMlpThreads / G1) * G1;
  const int r0 = (int)(((float)t + 0.5f) * a.inv_g1);  // t / G1, exact for t < 1024 (see flat_block)
  const int g0 = t - r0 * G1;
  __builtin_amdgcn_sched_barrier(0);

  // 1. Loads.  Units past the slice's 256 rows and down rows past D read
  //    zeros (offsets past the extents).
  NormLoads<1> nl = norm_issue<1, kMlpThreads>(a.np, D, t);
  u32x4 wa[UA][BITS];
  float sva[UA], zva[UA];
  int ga[UA];
  {
    int r = r0, g = g0;
#pragma unroll
    for (int i = 0; i < UA; ++i) {
      load_flat_unit<BITS>(qa, sa, za, r, g, G1, wa[i], sva[i], zva[i]);
      ga[i] = g;
      g += dg;
      r += dr;
      if (g >= G1) { g -= G1; r += 1; }
    }
  }
  float svd[kMlpDownUnits], zvd[kMlpDownUnits];
#pragma unroll
  for (int i = 0; i < kMlpDownUnits; ++i) {
    const uint32_t u = (uint32_t)(t + i * kMlpThreads) * G2 + b;
    svd[i] = (float)__builtin_bit_cast(_Float16, __builtin_amdgcn_raw_buffer_load_b16(sd, u * 2, 0, 0));
    zvd[i] = (float)__builtin_amdgcn_raw_buffer_load_b8(zd, u, 0, 0);
  }
  // Down codes: piece k = n * BITS + p (row n, plane p) of group b to
  // dl[k]; one instruction moves 64 pieces.  D * BITS is a multiple of 64.
  for (int j = wave; 64 * j < D * BITS; j += kMlpThreads / 64) {
    const uint32_t k = (uint32_t)(64 * j + lane);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(qd, (lds_void*)(dl + 64 * j), 16, (k * G2 + b) * 16, 0, 0, 0);
  }
  __builtin_amdgcn_sched_barrier(0);

  // 2. x = RMSNorm(residual + delta) * weight, staged with its group sums.
  u32x4 xv[1];
  norm_finish<1, kMlpThreads>(nl, a.np, D, t, b == 0, xv);
  stage_x_pass<1, kMlpThreads, 1>(xv, 0, t, G1 * 16, xl, xsum);
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's down pieces are in LDS
  __syncthreads();

  // 3. Gate|up unit partials, then h and its sum.
#pragma unroll
  for (int i = 0; i < UA; ++i) {
    const int u = t + i * kMlpThreads;
    if (u < 256 * G1) {
      const int g = ga[i];
      float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int cc = 0; cc < 4; ++cc) {
        uint32_t w[BITS];
#pragma unroll
        for (int p = 0; p < BITS; ++p) w[p] = wa[i][p][cc];
        const u32x4* xp4 = xl + g * kGroupStrideU4 + cc * 4;
        uint32_t xp[16];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const u32x4 q = xp4[v];
          xp[4 * v + 0] = q.x;
          xp[4 * v + 1] = q.y;
          xp[4 * v + 2] = q.z;
          xp[4 * v + 3] = q.w;
        }
        chunk_dot<BITS>(w, xp, acc);
      }
      pa[u] = sva[i] * fmaf(-zva[i], xsum[g], classes_to_value<BITS>(acc));
    }
  }
  __syncthreads();
  {
    uint16_t* hh = reinterpret_cast<uint16_t*>(hl);
    const int l = t & 15;
    for (int pr = t >> 4; pr < 128; pr += kMlpThreads / 16) {
      float ag = 0.0f, au = 0.0f;
      for (int g = l; g < G1; g += 16) {
        ag += pa[(2 * pr) * G1 + g];
        au += pa[(2 * pr + 1) * G1 + g];
      }
      ag = row16_sum(ag);
      au = row16_sum(au);
      if (l == 0) hh[pr] = __builtin_bit_cast(uint16_t, (_Float16)(ag / (1.0f + expf(-ag)) * au));
    }
  }
  __syncthreads();
  if (t < 16) {
    const u32x4 hv = hl[t];
    float ps = dot2(hv.x, kOnesPair, 0.0f);
    ps = dot2(hv.y, kOnesPair, ps);
    ps = dot2(hv.z, kOnesPair, ps);
    ps = dot2(hv.w, kOnesPair, ps);
    ps = row16_sum(ps);
    if (t == 0) *hsum = ps;
  }
  __syncthreads();

  // 4. Down partials of group b.
  const float hs = *hsum;
#pragma unroll
  for (int i = 0; i < kMlpDownUnits; ++i) {
    const int n = t + i * kMlpThreads;
    if (n < D) {
      u32x4 wv[BITS];
#pragma unroll
      for (int p = 0; p < BITS; ++p) wv[p] = dl[n * BITS + p];
      float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int cc = 0; cc < 4; ++cc) {
        uint32_t w[BITS];
#pragma unroll
        for (int p = 0; p < BITS; ++p) w[p] = wv[p][cc];
        uint32_t xp[16];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const u32x4 q = hl[cc * 4 + v];
          xp[4 * v + 0] = q.x;
          xp[4 * v + 1] = q.y;
          xp[4 * v + 2] = q.z;
          xp[4 * v + 3] = q.w;
        }
        chunk_dot<BITS>(w, xp, acc);
      }
      a.part[(size_t)b * D + n] = svd[i] * fmaf(-zvd[i], hs, classes_to_value<BITS>(acc));
    }
  }
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's partial stores are done

  // 5. Fixed-order sums by the last-arriving blocks.  Every wave waits for
  //    its own partial stores to complete (the workgroup barrier alone does
  //    not wait for global stores), so after the barrier they are all in
  //    this XCD's L2, and thread 0's device-scope release fence writes them
  //    back before its counter increment; the adder's thread 0 acquires, and
  //    the next barrier orders the other waves' loads after it.  (One fence
  //    per block: a device-scope fence writes back and invalidates the L2, and
  //    one in every wave measured several times slower.)
  __syncthreads();
  const int k = b / a.team_size;
  const int k0 = k * a.team_size;
  const int kn = min(a.team_size, G2 - k0);
  if (t == 0) {
    __threadfence();
    const bool l = atomicAdd(&a.count[k], 1u) == (uint32_t)(kn - 1);
    if (l) __threadfence();
    last = l;
  }
  __syncthreads();
  if (!last) return;
  for (int n = t; n < D; n += kMlpThreads)
    a.team[(size_t)k * D + n] = ordered_sum(a.part + (size_t)k0 * D + n, D, kn);
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's team-sum stores are done
  __syncthreads();
  if (t == 0) {
    atomicExch(&a.count[k], 0u);
    __threadfence();
    const bool l = atomicAdd(&a.count[a.T], 1u) == (uint32_t)(a.T - 1);
    if (l) __threadfence();
    last = l;
  }
  __syncthreads();
  if (!last) return;
  for (int n = t; n < D; n += kMlpThreads)
    a.y[n] = __builtin_bit_cast(uint16_t, (_Float16)ordered_sum(a.team + n, D, a.T));
  if (t == 0) atomicExch(&a.count[a.T], 0u);
}

int ceil_pow2(int v) {
  int p = 1;
  while (p < v) p <<= 1;
  return p;
}

}  // namespace

// Flat-unit kernel configuration for MT activation rows (1, 2, 4) and rows
// of G groups: one (row, group) unit per thread (fewest loads per lane
// measured best on every shape) and whole rows per block, so the reduction
// stays inside the block.  The caller uses it when lds fits the 64 KB budget.
//  - Threads per block: every block stages the whole activation row, so
//    longer rows want more rows per block (about 8 or more) to amortize it;
//    short rows with few of them use smaller blocks so that the grid still
//    covers the compute units.  Rows of 65..128 groups use 256 threads at one
//    activation row and 512 at two, with two rows per lane (below).
//  - Rows per lane: a thread takes group g of RPL rows, so every activation
//    group read from LDS serves RPL rows and each block's activation tile
//    serves RPL times as many rows; the lane's dot products get RPL times
//    longer.  Measured on MI355X, two rows per lane pay off when
//     - one activation row has 65..128 groups,
//     - the grid at one row per lane holds more waves than the chip keeps
//       resident (32 per compute unit), so waves would run in several rounds,
//     - two activation rows meet rows of 32..128 groups (twice the LDS
//       reads per unit);
//    elsewhere one row per lane is faster (the lanes' own latency decides).
FlatPlan flat_plan(int MT, int64_t N, int G) {
  FlatPlan p;
  int NT = G <= 32 ? 256 : G <= 64 ? 512 : G <= 128 ? (MT == 1 ? 256 : 512) : 1024;
  if (MT == 1)
    while (NT > 64 && G <= 16 && NT / 2 >= G && (N + NT / G - 1) / (NT / G) < 256) NT /= 2;
  const int XB = (MT * G * 16 <= 2 * NT) ? 2 : 5;
  auto lds_bytes = [&](int rows) { return (size_t)MT * G * (kGroupStrideU4 * 16 + 4) + (size_t)MT * rows * G * 4; };
  int R = max(1, NT / G);
  R = max(1, min(R, 4096 / (G * MT)));  // partials: at most 16 KB
  int want;
  {
    const int64_t waves1 = (N + R - 1) / R * (NT / 64);
    if (MT == 1)
      want = (G > 64 && G <= 128) || (G <= 64 && waves1 > kResidentWaves) ? 2 : 1;
    else
      want = (MT == 2 && G >= 32 && G <= 128) ? 2 : 1;
  }
  int RPL = 1;
  if (want > 1 && NT >= 256 && G <= NT) {
    const int r1 = min(NT / G, 4096 / (G * MT * want));
    if (r1 >= 1 && lds_bytes(want * r1) <= 64 * 1024) {
      RPL = want;
      R = want * r1;
    }
  }
  p.NT = NT;
  p.XB = XB;
  p.R = R;
  p.RPL = RPL;
  p.lds = lds_bytes(R);
  return p;
}

template <int BITS>
hipError_t launch_linear(const uint16_t* x, const uint32_t* qweight, const uint16_t* scales,
                         const uint8_t* zeros, uint16_t* y, int M, int64_t N, int64_t K,
                         hipStream_t stream, const LaunchEvents& ev, float* workspace,
                         size_t workspace_bytes) {
  const int G = (int)(K / 128);
  const int MT = ceil_pow2(M);
  // Matrix cores from kMfmaMinM activation rows on.
  if (M >= kMfmaMinM)
    return launch_linear_mfma<BITS>(x, qweight, scales, zeros, y, M, N, K, stream, ev, workspace, workspace_bytes);
  const u32x4* x4 = reinterpret_cast<const u32x4*>(x);
  const u32x4* q4 = reinterpret_cast<const u32x4*>(qweight);
  {
    const FlatPlan fp = flat_plan(MT, N, G);
    const int NT = fp.NT, XB = fp.XB, R = fp.R, RPL = fp.RPL;
    const size_t lds = fp.lds;
    if (MT <= 4 && lds <= 64 * 1024) {
      const int nblocks = (int)((N + R - 1) / R);
      const unsigned blocks = xcd_grid(nblocks);
#define LAQ_FLAT_K(MTV, XBV, NTV, RPLV)                                                                     \
  launch(linear_flat_kernel<BITS, MTV, NTV, RPLV, XBV, false>, dim3(blocks), dim3(NTV), (uint32_t)lds, stream, \
         ev, x, qweight, scales, zeros, M, (int)N, G, R, 1.0f / (float)G, nblocks, y)
#define LAQ_FLAT_NT(MTV, XBV, NTV)                       \
  do {                                                   \
    if (RPL == 2) LAQ_FLAT_K(MTV, XBV, NTV, 2);          \
    else LAQ_FLAT_K(MTV, XBV, NTV, 1);                   \
  } while (0)
#define LAQ_FLAT(MTV, XBV)                              \
  do {                                                  \
    if (NT == 1024) LAQ_FLAT_NT(MTV, XBV, 1024);        \
    else if (NT == 512) LAQ_FLAT_NT(MTV, XBV, 512);     \
    else if constexpr (MTV > 1) LAQ_FLAT_NT(MTV, XBV, 256); \
    else if (NT == 256) LAQ_FLAT_NT(MTV, XBV, 256);     \
    else if (NT == 128) LAQ_FLAT_K(MTV, XBV, 128, 1);   \
    else LAQ_FLAT_K(MTV, XBV, 64, 1);                   \
  } while (0)
#define LAQ_FLAT_XB(MTV)          \
  if (XB == 2) LAQ_FLAT(MTV, 2);  \
  else LAQ_FLAT(MTV, 5);
      switch (MT) {
        case 1: LAQ_FLAT_XB(1); break;
        case 2: LAQ_FLAT_XB(2); break;
        default: LAQ_FLAT_XB(4); break;
      }
#undef LAQ_FLAT_XB
#undef LAQ_FLAT
#undef LAQ_FLAT_NT
#undef LAQ_FLAT_K
      return hipGetLastError();
    }
  }
  // Activation tile too large for the flat kernel's LDS: matrix cores for
  // several rows, the K-tiled kernel below for one.
  if (M >= 2)
    return launch_linear_mfma<BITS>(x, qweight, scales, zeros, y, M, N, K, stream, ev, workspace, workspace_bytes);
  // Lanes per row: enough that one K tile covers the row in a few groups per
  // lane, then more while the grid is small, capped by the row's group count.
  int L = 4;
  while (L < 64 && L * kMaxGroupsPerLane < G) L <<= 1;
  while (L < 64 && L < G && (N + (kThreads / L) - 1) / (kThreads / L) < 512) L <<= 1;
  int lpr_log2 = 0;
  while ((1 << lpr_log2) < L) ++lpr_log2;
  const int per_group_bytes = kGroupStrideU4 * 16 + 4;
  int tile = kLdsBudget / (MT * per_group_bytes);
  tile = min(tile, L * kMaxGroupsPerLane);
  tile = min(tile, G);
  const size_t lds = (size_t)MT * tile * per_group_bytes;
  const int rows_per_block = kThreads / L;
  const unsigned blocks = (unsigned)((N + rows_per_block - 1) / rows_per_block);
#define LAQ_LAUNCH(MTV)                                                                              \
  launch(linear_kernel<BITS, MTV>, dim3(blocks), dim3(kThreads), (uint32_t)lds, stream, ev, x4, q4, \
         scales, zeros, y, M, (int)N, G, lpr_log2, tile)
  switch (MT) {
    case 1: LAQ_LAUNCH(1); break;
    case 2: LAQ_LAUNCH(2); break;
    case 4: LAQ_LAUNCH(4); break;
    case 8: LAQ_LAUNCH(8); break;
    default: LAQ_LAUNCH(16); break;
  }
#undef LAQ_LAUNCH
  return hipGetLastError();
}

bool swiglu_fits(int M, int64_t K) { return M >= 1 && M <= 4 && K >= 128 && K % 128 == 0 && ceil_pow2(M) * K <= 16384; }

template <int BITS>
hipError_t launch_linear_swiglu(const uint16_t* x, const uint32_t* qweight, const uint16_t* scales,
                                const uint8_t* zeros, uint16_t* y, int M, int64_t N, int64_t K, hipStream_t stream,
                                const LaunchEvents& ev) {
  // The flat kernel at one row per lane with an even number of rows per
  // block, so that every (gate, up) pair of rows meets in one block's
  // partials.  MT * G <= 128 keeps the activation tile and the partials
  // within 52 KB of LDS.
  if (!swiglu_fits(M, K) || N % 2 != 0) return hipErrorInvalidValue;
  const int G = (int)(K / 128);
  const int MT = ceil_pow2(M);
  const int NT = G <= 32 ? 256 : G <= 64 ? 512 : (MT == 1 ? 256 : 512);
  const int XB = (MT * G * 16 <= 2 * NT) ? 2 : 5;
  int R = max(1, min(NT / G, 4096 / (G * MT)));
  R = max(2, R & ~1);
  const size_t lds = (size_t)MT * G * (kGroupStrideU4 * 16 + 4) + (size_t)MT * R * G * 4;
  const int nblocks = (int)((N + R - 1) / R);
  const unsigned blocks = xcd_grid(nblocks);
#define LAQ_SW_K(MTV, XBV, NTV)                                                                                   \
  launch(linear_flat_kernel<BITS, MTV, NTV, 1, XBV, true>, dim3(blocks), dim3(NTV), (uint32_t)lds, stream, ev, x, \
         qweight, scales, zeros, M, (int)N, G, R, 1.0f / (float)G, nblocks, y)
#define LAQ_SW_NT(MTV, XBV)                 \
  do {                                      \
    if (NT == 512) LAQ_SW_K(MTV, XBV, 512); \
    else LAQ_SW_K(MTV, XBV, 256);           \
  } while (0)
#define LAQ_SW_XB(MTV)              \
  if (XB == 2) LAQ_SW_NT(MTV, 2);   \
  else LAQ_SW_NT(MTV, 5);
  switch (MT) {
    case 1: LAQ_SW_XB(1); break;
    case 2: LAQ_SW_XB(2); break;
    default: LAQ_SW_XB(4); break;
  }
#undef LAQ_SW_XB
#undef LAQ_SW_NT
#undef LAQ_SW_K
  return hipGetLastError();
}

bool norm_linear_fits(int64_t K) { return K >= 128 && K % 128 == 0 && K <= 8192; }

template <int BITS>
hipError_t launch_linear_norm(const NormPrologue& np, const uint32_t* qweight, const uint16_t* scales,
                              const uint8_t* zeros, uint16_t* y, int64_t N, int64_t K, bool swiglu,
                              hipStream_t stream, const LaunchEvents& ev) {
  // The M = 1 flat kernel's configuration (rows per block, rows per lane as
  // launch_linear chooses them).  The prologue needs the whole row in
  // registers before its one reduction, XB units of 8 elements per thread:
  // blocks of 256 threads up to 16 groups and 512 up to 64, so that one unit
  // per thread covers rows up to 32 groups and two up to 64.  (Measured on
  // MI355X, Qwen3-4B decode step: 512-thread blocks with one prologue unit
  // per thread for the 20-group q|k|v and gate|up rows instead of 256 with
  // two, 1005-1008 -> 996-997 us per token; the prologue's loads and its
  // row reads are per block, so fewer, larger blocks issue fewer of them.)
  if (!norm_linear_fits(K) || (swiglu && N % 2 != 0)) return hipErrorInvalidValue;
  const int G = (int)(K / 128);
  const int NT = G <= 16 ? 256 : 512;
  const bool one_unit = K <= 8 * NT;
  auto lds_bytes = [&](int rows) { return (size_t)G * (kGroupStrideU4 * 16 + 4) + (size_t)rows * G * 4; };
  int R = max(1, min(NT / G, 4096 / G));
  int RPL = 1;
  if (swiglu) {
    R = max(2, R & ~1);
  } else if ((N + R - 1) / R * (NT / 64) > kResidentWaves) {
    const int r1 = min(NT / G, 4096 / (G * 2));
    if (r1 >= 1 && lds_bytes(2 * r1) <= 64 * 1024) {
      RPL = 2;
      R = 2 * r1;
    }
  }
  const size_t lds = lds_bytes(R);
  const int nblocks = (int)((N + R - 1) / R);
  const dim3 grid(xcd_grid(nblocks));
#define LAQ_NORM_K(NTV, RPLV, SWV, XBV)                                                                           \
  launch(linear_flat_norm_kernel<NTV, RPLV, SWV, BITS, XBV>, grid, dim3(NTV), (uint32_t)lds, stream, ev, np.res_in, \
         np.delta, np.weight, qweight, scales, zeros, (int)N, G | R << 8, y, np.res_out, np.eps)
  if (NT == 256) {  // K <= 2048: one unit per thread
    if (swiglu) LAQ_NORM_K(256, 1, true, 1);
    else if (RPL == 2) LAQ_NORM_K(256, 2, false, 1);
    else LAQ_NORM_K(256, 1, false, 1);
  } else if (one_unit) {
    if (swiglu) LAQ_NORM_K(512, 1, true, 1);
    else if (RPL == 2) LAQ_NORM_K(512, 2, false, 1);
    else LAQ_NORM_K(512, 1, false, 1);
  } else {
    if (swiglu) LAQ_NORM_K(512, 1, true, 2);
    else if (RPL == 2) LAQ_NORM_K(512, 2, false, 2);
    else LAQ_NORM_K(512, 1, false, 2);
  }
#undef LAQ_NORM_K
  return hipGetLastError();
}

bool residual_linear_fits(int64_t N, int64_t K) {
  // At least 16 groups: a block's rows then fit one row per 16 lanes.
  if (N < 1 || K < 2048 || K % 128 != 0) return false;
  const FlatPlan fp = flat_plan(1, N, (int)(K / 128));
  return fp.lds <= 64 * 1024 && fp.R <= fp.NT / 16;
}

template <int BITS>
hipError_t launch_linear_residual(const uint16_t* x, const uint32_t* qweight, const uint16_t* scales,
                                  const uint8_t* zeros, uint16_t* y, const float* res_in, float* res_out, int64_t N,
                                  int64_t K, hipStream_t stream, const LaunchEvents& ev) {
  // The M = 1 flat kernel's configuration, so y is the plain call's, bit for bit.
  if (!residual_linear_fits(N, K)) return hipErrorInvalidValue;
  const int G = (int)(K / 128);
  const FlatPlan fp = flat_plan(1, N, G);
  const int nblocks = (int)((N + fp.R - 1) / fp.R);
  const dim3 grid(xcd_grid(nblocks));
#define LAQ_RES_K(NTV, RPLV, XBV)                                                                                 \
  launch(linear_flat_res_kernel<BITS, NTV, RPLV, XBV>, grid, dim3(NTV), (uint32_t)fp.lds, stream, ev, x, qweight, \
         scales, zeros, (int)N, G, fp.R, nblocks, res_in, y, res_out)
#define LAQ_RES_RPL(NTV, XBV)                   \
  do {                                          \
    if (fp.RPL == 2) LAQ_RES_K(NTV, 2, XBV);    \
    else LAQ_RES_K(NTV, 1, XBV);                \
  } while (0)
  if (fp.NT == 256 && fp.XB == 2) LAQ_RES_RPL(256, 2);
  else if (fp.NT == 256) LAQ_RES_RPL(256, 5);
  else if (fp.NT == 512) LAQ_RES_RPL(512, 2);
  else if (fp.NT == 1024) LAQ_RES_RPL(1024, 5);
  else if (fp.NT == 128) LAQ_RES_K(128, 1, 2);
  else if (fp.NT == 64) LAQ_RES_K(64, 1, 2);
  else return hipErrorInvalidValue;
#undef LAQ_RES_RPL
#undef LAQ_RES_K
  return hipGetLastError();
}

MlpPlan mlp_plan(int64_t D, int64_t I, int bits) {
  MlpPlan p;
  if (D < 128 || D % 128 != 0 || D > kMlpMaxHidden || I < 128 || I % 128 != 0 || I > kMlpMaxInter) return p;
  const int G1 = (int)(D / 128);
  const size_t lds = ((size_t)D * bits + (size_t)G1 * kGroupStrideU4 + 16) * 16 + ((size_t)G1 * 257 + 1) * 4;
  if (lds > kMlpLdsBytes) return p;
  p.S = (int)(I / 128);
  p.T = 1;
  while (p.T * p.T < p.S) ++p.T;  // about sqrt(S) teams of about sqrt(S) slices
  p.team_size = (p.S + p.T - 1) / p.T;
  p.T = (p.S + p.team_size - 1) / p.team_size;
  p.lds = lds;
  return p;
}

size_t mlp_workspace_bytes(const MlpPlan& p, int64_t D) {
  if (p.S == 0) return 0;
  return ((size_t)(p.S + p.T) * (size_t)D * 4 + (size_t)(p.T + 1) * 4 + 15) / 16 * 16;
}

template <int BITS>
hipError_t launch_mlp(const NormPrologue& np, const uint32_t* gu_qw, const uint16_t* gu_s, const uint8_t* gu_z,
                      const uint32_t* dn_qw, const uint16_t* dn_s, const uint8_t* dn_z, uint16_t* y, int64_t D,
                      int64_t I, void* workspace, hipStream_t stream, const LaunchEvents& ev) {
  const MlpPlan p = mlp_plan(D, I, BITS);
  if (p.S == 0) return hipErrorInvalidValue;
  MlpArgs a;
  a.np = np;
  a.gu_qw = gu_qw;
  a.gu_s = gu_s;
  a.gu_z = gu_z;
  a.dn_qw = dn_qw;
  a.dn_s = dn_s;
  a.dn_z = dn_z;
  a.y = y;
  a.part = static_cast<float*>(workspace);
  a.team = a.part + (size_t)p.S * D;
  a.count = reinterpret_cast<uint32_t*>(a.team + (size_t)p.T * D);
  a.D = (int)D;
  a.G1 = (int)(D / 128);
  a.S = p.S;
  a.team_size = p.team_size;
  a.T = p.T;
  a.inv_g1 = 1.0f / (float)a.G1;
  const int UA = (a.G1 + 3) / 4;  // 256 rows x G1 groups over 1024 threads
  const dim3 grid(xcd_grid(p.S)), blk(kMlpThreads);
  switch (UA) {
    case 1: launch(mlp_block_kernel<BITS, 1>, grid, blk, (uint32_t)p.lds, stream, ev, a); break;
    case 2: launch(mlp_block_kernel<BITS, 2>, grid, blk, (uint32_t)p.lds, stream, ev, a); break;
    case 3: launch(mlp_block_kernel<BITS, 3>, grid, blk, (uint32_t)p.lds, stream, ev, a); break;
    case 4: launch(mlp_block_kernel<BITS, 4>, grid, blk, (uint32_t)p.lds, stream, ev, a); break;
    default: launch(mlp_block_kernel<BITS, 5>, grid, blk, (uint32_t)p.lds, stream, ev, a); break;
  }
  return hipGetLastError();
}

template <int BITS>
hipError_t launch_linear_group(LinearCall* calls, int count, int M, hipStream_t stream, const LaunchEvents& ev) {
  int G_max = 1;
  for (int i = 0; i < count; ++i) G_max = max(G_max, calls[i].G);
  const int MT = ceil_pow2(M);
  // Matrix cores from kMfmaMinM activation rows on, except that the VALU
  // kernel stays ahead up to 4 rows when the group's rows are short (measured
  // on MI355X: it re-reads the activations from LDS per unit, which costs more
  // as rows get longer; the grouped matrix-core kernel has no one-wave-per-quad
  // form).
  if (M >= kMfmaMinM && !(M <= 4 && G_max <= 24))
    return launch_linear_mfma_group<BITS>(calls, count, M, stream, ev);
  const int NT = G_max <= 32 ? 256 : (G_max <= 64 ? 512 : 1024);
  const int XB = (MT * G_max * 16 <= 2 * NT) ? 2 : 5;
  size_t lds = 0;
  int64_t blocks = 0;
  LinearGroup grp{};
  for (int i = 0; i < count; ++i) {
    LinearCall& c = calls[i];
    c.R = max(1, min(max(1, NT / c.G), 4096 / (c.G * MT)));
    c.inv_g = 1.0f / (float)c.G;
    lds = std::max(lds, (size_t)MT * c.G * (kGroupStrideU4 * 16 + 4) + (size_t)MT * c.R * c.G * 4);
    c.first_block = (int)blocks;
    blocks += (c.N + c.R - 1) / c.R;
    grp.call[i] = c;
  }
  grp.count = count;
  grp.blocks = (int)blocks;
  if (MT > 4 || lds > 64 * 1024) {
    if (M >= 2) return launch_linear_mfma_group<BITS>(calls, count, M, stream, ev);
    // One activation row too long for LDS: one launch per call.
    for (int i = 0; i < count; ++i) {
      const LinearCall& c = calls[i];
      LaunchEvents e_i;  // the measurement hook spans the whole sequence
      e_i.start = i == 0 ? ev.start : nullptr;
      e_i.stop = i == count - 1 ? ev.stop : nullptr;
      const hipError_t e = launch_linear<BITS>(c.x, c.qw, c.scales, c.zeros, c.y, M, c.N, (int64_t)c.G * 128,
                                               stream, e_i);
      if (e != hipSuccess) return e;
    }
    return hipSuccess;
  }
#define LAQ_FLAT_G(MTV, XBV, NTV)                                                                         \
  launch(linear_flat_group_kernel<BITS, MTV, NTV, XBV>, dim3(xcd_grid(blocks)), dim3(NTV), (uint32_t)lds, \
         stream, ev, grp, M)
#define LAQ_FLAT_GN(MTV, XBV)                              \
  do {                                                     \
    if (NT == 1024) LAQ_FLAT_G(MTV, XBV, 1024);            \
    else if (NT == 512) LAQ_FLAT_G(MTV, XBV, 512);         \
    else LAQ_FLAT_G(MTV, XBV, 256);                        \
  } while (0)
#define LAQ_FLAT_GX(MTV)           \
  if (XB == 2) LAQ_FLAT_GN(MTV, 2); \
  else LAQ_FLAT_GN(MTV, 5);
  switch (MT) {
    case 1: LAQ_FLAT_GX(1); break;
    case 2: LAQ_FLAT_GX(2); break;
    default: LAQ_FLAT_GX(4); break;
  }
#undef LAQ_FLAT_GX
#undef LAQ_FLAT_GN
#undef LAQ_FLAT_G
  return hipGetLastError();
}

template hipError_t launch_linear_swiglu<3>(const uint16_t*, const uint32_t*, const uint16_t*, const uint8_t*,
                                            uint16_t*, int, int64_t, int64_t, hipStream_t, const LaunchEvents&);
template hipError_t launch_linear_swiglu<4>(const uint16_t*, const uint32_t*, const uint16_t*, const uint8_t*,
                                            uint16_t*, int, int64_t, int64_t, hipStream_t, const LaunchEvents&);
template hipError_t launch_linear_norm<3>(const NormPrologue&, const uint32_t*, const uint16_t*, const uint8_t*,
                                          uint16_t*, int64_t, int64_t, bool, hipStream_t, const LaunchEvents&);
template hipError_t launch_linear_norm<4>(const NormPrologue&, const uint32_t*, const uint16_t*, const uint8_t*,
                                          uint16_t*, int64_t, int64_t, bool, hipStream_t, const LaunchEvents&);
template hipError_t launch_linear_residual<3>(const uint16_t*, const uint32_t*, const uint16_t*, const uint8_t*,
                                              uint16_t*, const float*, float*, int64_t, int64_t, hipStream_t,
                                              const LaunchEvents&);
template hipError_t launch_linear_residual<4>(const uint16_t*, const uint32_t*, const uint16_t*, const uint8_t*,
                                              uint16_t*, const float*, float*, int64_t, int64_t, hipStream_t,
                                              const LaunchEvents&);
template hipError_t launch_mlp<3>(const NormPrologue&, const uint32_t*, const uint16_t*, const uint8_t*,
                                  const uint32_t*, const uint16_t*, const uint8_t*, uint16_t*, int64_t, int64_t,
                                  void*, hipStream_t, const LaunchEvents&);
template hipError_t launch_linear_group<3>(LinearCall*, int, int, hipStream_t, const LaunchEvents&);
template hipError_t launch_linear_group<4>(LinearCall*, int, int, hipStream_t, const LaunchEvents&);
template hipError_t launch_linear<3>(const uint16_t*, const uint32_t*, const uint16_t*, const uint8_t*,
                                     uint16_t*, int, int64_t, int64_t, hipStream_t,
                                     const LaunchEvents&, float*, size_t);
template hipError_t launch_linear<4>(const uint16_t*, const uint32_t*, const uint16_t*, const uint8_t*,
                                     uint16_t*, int, int64_t, int64_t, hipStream_t,
                                     const LaunchEvents&, float*, size_t);

}  // namespace laq
