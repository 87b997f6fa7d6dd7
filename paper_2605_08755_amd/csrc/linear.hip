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

int ceil_pow2(int v) {
  int p = 1;
  while (p < v) p <<= 1;
  return p;
}

}  // namespace

template <int BITS>
hipError_t launch_linear(const uint16_t* x, const uint32_t* qweight, const uint16_t* scales,
                         const uint8_t* zeros, uint16_t* y, int M, int64_t N, int64_t K,
                         hipStream_t stream, const LaunchEvents& ev) {
  const int G = (int)(K / 128);
  const int MT = ceil_pow2(M);
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
  const u32x4* x4 = reinterpret_cast<const u32x4*>(x);
  const u32x4* q4 = reinterpret_cast<const u32x4*>(qweight);
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

template hipError_t launch_linear<3>(const uint16_t*, const uint32_t*, const uint16_t*, const uint8_t*,
                                     uint16_t*, int, int64_t, int64_t, hipStream_t,
                                     const LaunchEvents&);
template hipError_t launch_linear<4>(const uint16_t*, const uint32_t*, const uint16_t*, const uint8_t*,
                                     uint16_t*, int, int64_t, int64_t, hipStream_t,
                                     const LaunchEvents&);

}  // namespace laq
