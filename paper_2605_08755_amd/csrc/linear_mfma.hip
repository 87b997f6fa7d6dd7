// Skinny-GEMM path (M = 2..16 activation rows) on the matrix cores.
//
// y[m][n] = sum_g s[n][g] * sum_{k in g} x[m][k] * (q[n][k] - z[n][g])   (Eq. 1)
//
// One v_mfma_f32_16x16x32_f16 multiplies a 16 x 32 activation tile (rows m,
// zero past M) by a 32 x 16 tile of exact (q - z) values of 16 weight rows.
// Lane l of a wave owns weight row n = l % 16 of the current 16-row tile and
// chunk q = l / 16 of the current 128-group, so the four chunks of a group
// are spread over the four 16-lane quarters and every MFMA's 32-element K
// window stays inside one group (one scale and zero point per row).  The
// MFMA result fragment of lane l is column n = l % 16 (rows m = 4(l/16)..+3),
// i.e. the lane's own weight row, so each lane scales its accumulator by its
// own s[n][g] with no data exchange.
//
// Unpack to exact fp16 (q - z): OR-ing a 3-bit (or 4-bit) code field at
// mantissa bits [p, p+b) with the bits of 2^(10-p) gives the fp16 value
// 2^(10-p) + q exactly; one packed fp16 add of -(2^(10-p) + z) leaves q - z
// exactly.  One v_and_or_b32 + one v_pk_add_f16 per two codes.
//
// The four waves of a block split the groups of the block's rows; their
// partial sums are added in a fixed order through LDS (deterministic).
#include "laq_internal.h"

namespace laq {

namespace {

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float float4_t __attribute__((ext_vector_type(4)));

constexpr int kMfmaThreads = 256;  // 4 waves
constexpr int kBufferFlagsM = 0x00020000;
constexpr int kStreamPolicyM = 2;  // non-temporal weight stream

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kBufferFlagsM);
}

__device__ __forceinline__ uint32_t pk_add_f16(uint32_t a, uint32_t b) {
  return __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2_t, a) + __builtin_bit_cast(half2_t, b));
}

// fp16 bit patterns of -(2^(10-p) + z) in both halves, for the field
// offsets used by the layouts (ulp of 2^(10-p) is 2^-p, so + z is + z*2^p ulps).
__device__ __forceinline__ uint32_t neg_magic(uint32_t base_bits, uint32_t z, uint32_t shift) {
  const uint32_t h = base_bits + (z << shift);
  return h | (h << 16);
}

// Exact (q - z) pairs of one 32-code chunk, in natural order: pair t holds
// codes 2t (low half) and 2t+1 (high half).
template <int BITS>
__device__ __forceinline__ void unpack_chunk_exact(const uint32_t (&w)[BITS], uint32_t z, uint32_t (&pr)[16]) {
  if constexpr (BITS == 3) {
    const uint32_t n0 = neg_magic(0xE400u, z, 0);  // -(1024 + z): fields at bits 0-2
    const uint32_t n3 = neg_magic(0xD800u, z, 3);  // -(128 + z):  bits 3-5
    const uint32_t n6 = neg_magic(0xCC00u, z, 6);  // -(16 + z):   bits 6-8
    const uint32_t n7 = neg_magic(0xC800u, z, 7);  // -(8 + z):    bits 7-9
#pragma unroll
    for (int p = 0; p < 3; ++p) {
      const uint32_t t = w[p] >> 10;
      pr[5 * p + 0] = pk_add_f16((w[p] & 0x00070007u) | 0x64006400u, n0);
      pr[5 * p + 1] = pk_add_f16((w[p] & 0x00380038u) | 0x58005800u, n3);
      pr[5 * p + 2] = pk_add_f16((w[p] & 0x01C001C0u) | 0x4C004C00u, n6);
      pr[5 * p + 3] = pk_add_f16((t & 0x00070007u) | 0x64006400u, n0);
      pr[5 * p + 4] = pk_add_f16((t & 0x00380038u) | 0x58005800u, n3);
    }
    // codes 30/31: code bit j is bit 9 / bit 25 of plane j -> field at bits 7-9
    const uint32_t spare = ((w[0] >> 2) & 0x00800080u) | ((w[1] >> 1) & 0x01000100u) | (w[2] & 0x02000200u);
    pr[15] = pk_add_f16(spare | 0x48004800u, n7);
  } else {
    const uint32_t n0 = neg_magic(0xE400u, z, 0);  // -(1024 + z): nibbles at bits 0-3
    const uint32_t n4 = neg_magic(0xD400u, z, 4);  // -(64 + z):   bits 4-7
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const uint32_t t = w[p] >> 8;
      pr[4 * p + 0] = pk_add_f16((w[p] & 0x000F000Fu) | 0x64006400u, n0);
      pr[4 * p + 1] = pk_add_f16((w[p] & 0x00F000F0u) | 0x54005400u, n4);
      pr[4 * p + 2] = pk_add_f16((t & 0x000F000Fu) | 0x64006400u, n0);
      pr[4 * p + 3] = pk_add_f16((t & 0x00F000F0u) | 0x54005400u, n4);
    }
  }
}

__device__ __forceinline__ half8_t frag(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
  return __builtin_bit_cast(half8_t, u32x4v{a, b, c, d});
}

// Loads of one (tile, group) for this lane: the chunk's BITS plane words,
// the row's scale and zero point.  Rows past the block's extent read zeros.
template <int BITS>
struct TileLoad {
  uint32_t w[BITS];
  uint32_t s;
  uint32_t z;
};

template <int BITS, int TW>
__global__ __launch_bounds__(kMfmaThreads) void linear_mfma_kernel(
    const uint16_t* __restrict__ x, const uint32_t* __restrict__ qw, const uint16_t* __restrict__ scales,
    const uint8_t* __restrict__ zeros, uint16_t* __restrict__ y, int M, int N, int G, int K) {
  __shared__ float red[4][TW][4][64];  // per-wave partial results, [wave][tile][r][lane]

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int nl = lane & 15;  // weight row within a tile / result column
  const int q = lane >> 4;   // chunk of the group / activation row block
  const int64_t row0 = (int64_t)blockIdx.x * (16 * TW);
  const int rows = (int)min((int64_t)16 * TW, (int64_t)N - row0);
  const int C = 4 * G;

  const __amdgpu_buffer_rsrc_t xr = rsrc(x, (uint32_t)M * K * 2);
  const __amdgpu_buffer_rsrc_t qr = rsrc(qw + row0 * BITS * C, (uint32_t)rows * BITS * C * 4);
  const __amdgpu_buffer_rsrc_t sr = rsrc(scales + row0 * G, (uint32_t)rows * G * 2);
  const __amdgpu_buffer_rsrc_t zr = rsrc(zeros + row0 * G, (uint32_t)rows * G);

  // this wave's share of the groups
  const int g_begin = (G * wave) / 4;
  const int g_end = (G * (wave + 1)) / 4;

  float4_t yacc[TW];
#pragma unroll
  for (int t = 0; t < TW; ++t) yacc[t] = float4_t{0.f, 0.f, 0.f, 0.f};

  // activation fragment source: row m = lane % 16, bytes of chunk (4g + q)
  const uint32_t xrow = (uint32_t)(lane & 15) * (uint32_t)K * 2;

  auto load_group = [&](int g, u32x4 (&xa)[4], TileLoad<BITS> (&tl)[TW]) {
    const uint32_t xo = xrow + (uint32_t)(128 * g + 32 * q) * 2;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) xa[jj] = __builtin_amdgcn_raw_buffer_load_b128(xr, xo + 16 * jj, 0, 0);
#pragma unroll
    for (int t = 0; t < TW; ++t) {
      const uint32_t nloc = (uint32_t)(16 * t + nl);
#pragma unroll
      for (int p = 0; p < BITS; ++p)
        tl[t].w[p] = __builtin_amdgcn_raw_buffer_load_b32(qr, ((nloc * BITS + p) * C + 4 * g + q) * 4, 0, kStreamPolicyM);
      tl[t].s = __builtin_amdgcn_raw_buffer_load_b16(sr, (nloc * G + g) * 2, 0, 0);
      tl[t].z = __builtin_amdgcn_raw_buffer_load_b8(zr, nloc * G + g, 0, 0);
    }
  };

  auto compute_group = [&](const u32x4 (&xc)[4], const TileLoad<BITS> (&tc)[TW]) {
#pragma unroll
    for (int t = 0; t < TW; ++t) {
      uint32_t pr[16];
      unpack_chunk_exact<BITS>(tc[t].w, tc[t].z, pr);
      float4_t c = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const half8_t a = __builtin_bit_cast(half8_t, xc[jj]);
        const half8_t b = frag(pr[4 * jj + 0], pr[4 * jj + 1], pr[4 * jj + 2], pr[4 * jj + 3]);
        c = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
      }
      const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)tc[t].s);
      yacc[t] += s * c;
    }
  };

  // Two-deep pipeline: the loads of the next group are in flight while the
  // current one is unpacked and multiplied.
  if (g_begin < g_end) {
    u32x4 xa0[4], xa1[4];
    TileLoad<BITS> tl0[TW], tl1[TW];
    load_group(g_begin, xa0, tl0);
    for (int g = g_begin; g < g_end; g += 2) {
      if (g + 1 < g_end) load_group(g + 1, xa1, tl1);
      compute_group(xa0, tl0);
      if (g + 1 < g_end) {
        if (g + 2 < g_end) load_group(g + 2, xa0, tl0);
        compute_group(xa1, tl1);
      }
    }
  }

  // fixed-order reduction of the four waves' partials
#pragma unroll
  for (int t = 0; t < TW; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) red[wave][t][r][lane] = yacc[t][r];
  __syncthreads();
  for (int idx = threadIdx.x; idx < TW * 4 * 64; idx += kMfmaThreads) {
    const int t = idx / 256;
    const int r = (idx >> 6) & 3;
    const int ln = idx & 63;
    const float v = ((red[0][t][r][ln] + red[1][t][r][ln]) + red[2][t][r][ln]) + red[3][t][r][ln];
    const int m = 4 * (ln >> 4) + r;
    const int nloc = 16 * t + (ln & 15);
    if (m < M && nloc < rows) y[(int64_t)m * N + row0 + nloc] = __builtin_bit_cast(uint16_t, (_Float16)v);
  }
}

}  // namespace

template <int BITS>
hipError_t launch_linear_mfma(const uint16_t* x, const uint32_t* qweight, const uint16_t* scales,
                              const uint8_t* zeros, uint16_t* y, int M, int64_t N, int64_t K,
                              hipStream_t stream, const LaunchEvents& ev) {
  const int G = (int)(K / 128);
  // Two tiles per wave when that still leaves a couple of blocks per CU.
  const int tiles = (int)((N + 15) / 16);
  const int TW = tiles >= 1024 ? 2 : 1;
  const unsigned blocks = (unsigned)((N + 16 * TW - 1) / (16 * TW));
  if (TW == 2)
    launch(linear_mfma_kernel<BITS, 2>, dim3(blocks), dim3(kMfmaThreads), 0, stream, ev, x, qweight, scales, zeros,
           y, M, (int)N, G, (int)K);
  else
    launch(linear_mfma_kernel<BITS, 1>, dim3(blocks), dim3(kMfmaThreads), 0, stream, ev, x, qweight, scales, zeros,
           y, M, (int)N, G, (int)K);
  return hipGetLastError();
}

template hipError_t launch_linear_mfma<3>(const uint16_t*, const uint32_t*, const uint16_t*, const uint8_t*,
                                          uint16_t*, int, int64_t, int64_t, hipStream_t, const LaunchEvents&);
template hipError_t launch_linear_mfma<4>(const uint16_t*, const uint32_t*, const uint16_t*, const uint8_t*,
                                          uint16_t*, int, int64_t, int64_t, hipStream_t, const LaunchEvents&);

}  // namespace laq
