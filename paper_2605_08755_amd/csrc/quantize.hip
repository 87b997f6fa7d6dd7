// Quantize + pack kernel: Eq. 1 (Sec. 2) with round-to-nearest min-max
// scale and zero point per group of 128 consecutive weights of a row, packed
// into the plane layout of include/laq.h (32 codes in three 32-bit words for
// W3, as App. G keeps; eight 4-bit codes per word for W4).
//
// Mapping: 16 lanes per group (one DPP row), each lane owns 8 consecutive
// weights (one 16-byte load; a group is 256 contiguous bytes, so a wave reads
// 1 KB contiguous).  The group range is reduced across the 16 lanes with DPP
// (min/max are exact in any order), every lane derives the same (s, z) with IEEE fp32
// arithmetic, quantizes its 8 weights with the IEEE quotient (formed from a
// reciprocal and two fused multiply-adds, see below) and round-half-even,
// and the 4 lanes of each 32-code chunk OR their bits into the plane words.
//
// The same kernel also packs with caller-supplied parameters (GIVEN): Eq. 1
// with the scale and zero point read from memory (e.g. the ones LAQuant's
// QAT learned) instead of the min-max ones.
#include "laq_internal.h"

namespace laq {

namespace {

__device__ __forceinline__ float half_bits_to_float(uint32_t h) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
}

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

template <int CTRL>
__device__ __forceinline__ void minmax_step(float& lo, float& hi) {
  lo = fminf(lo, dpp<CTRL>(lo));
  hi = fmaxf(hi, dpp<CTRL>(hi));
}

// Minimum and maximum over the 16 lanes of a DPP row (a group's lanes);
// every lane receives both.  Exact in any order.
__device__ __forceinline__ void row16_minmax(float& lo, float& hi) {
  minmax_step<0xB1>(lo, hi);   // quad_perm [1,0,3,2]
  minmax_step<0x4E>(lo, hi);   // quad_perm [2,3,0,1]
  minmax_step<0x141>(lo, hi);  // row_half_mirror
  minmax_step<0x140>(lo, hi);  // row_mirror
}

template <int BITS, bool GIVEN>
__global__ __launch_bounds__(256) void quantize_kernel(const u32x4* __restrict__ w, int64_t n_groups,
                                                       int G, uint32_t* __restrict__ qweight,
                                                       uint16_t* __restrict__ scales,
                                                       uint8_t* __restrict__ zeros) {
#pragma clang fp contract(off)
  const int64_t grp = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 4;  // flat n*G + g
  const int b = threadIdx.x & 15;                                       // 8-weight slice
  if (grp >= n_groups) return;  // whole 16-lane segments leave together

  const u32x4 raw = __builtin_nontemporal_load(w + grp * 16 + b);
  const uint32_t words[4] = {raw.x, raw.y, raw.z, raw.w};
  float v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = half_bits_to_float((words[e >> 1] >> (16 * (e & 1))) & 0xFFFFu);

  constexpr float qmax = (float)((1 << BITS) - 1);
  uint32_t s16;
  float s, z;
  if constexpr (GIVEN) {
    s16 = scales[grp];
    s = half_bits_to_float(s16);
    z = (float)zeros[grp];
  } else {
    // Group range, widened to contain 0.
    float lo = 0.0f, hi = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      lo = fminf(lo, v[e]);
      hi = fmaxf(hi, v[e]);
    }
    row16_minmax(lo, hi);
    const float s32 = (hi - lo) / qmax;  // IEEE division (no fast-math)
    s16 = __builtin_bit_cast(uint16_t, (_Float16)s32);  // round-to-nearest-even
    if (s16 == 0) s16 = 1;                              // 2^-24 when the range underflows
    s = half_bits_to_float(s16);
    z = fminf(fmaxf(rintf(-lo / s), 0.0f), qmax);
  }

  // Codes: the clip is taken on the real value (a quotient that is not a
  // number gives 0), so no out-of-range value reaches the integer conversion.
  //
  // The quotient v / s is formed without a per-weight division: with
  // y = RN(1/s) (one IEEE division per group), q = RN(v*y), r = v - q*s
  // (exact, fused) and q' = RN(q + r*y) (fused), q' equals the IEEE binary32
  // quotient RN(v/s) for every finite fp16 v and every finite positive fp16
  // s -- checked exhaustively over all 2.0e9 such pairs
  // (tests/native/fp16_quotient_check.c).  The min-max scale is always in
  // that domain; a caller-supplied scale outside it (zero, infinite or not
  // a number) takes the true division.
  uint32_t q[8];
  if (!GIVEN || (s > 0.0f && s <= 65504.0f)) {
    const float y = 1.0f / s;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float q0 = v[e] * y;
      const float r = fmaf(-q0, s, v[e]);
      const float qt = fmaf(r, y, q0);
      q[e] = (uint32_t)fminf(fmaxf(rintf(qt) + z, 0.0f), qmax);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) q[e] = (uint32_t)fminf(fmaxf(rintf(v[e] / s) + z, 0.0f), qmax);
  }

  // (row, group) of this lane: the block's first group splits on the scalar
  // unit; a lane's group is at most 15 further, i.e. one row wrap when G >= 16.
  const int64_t base = (int64_t)blockIdx.x * 16;
  const int64_t n0 = base / G;
  const int g0 = (int)(base - n0 * G);
  int g = g0 + (int)(threadIdx.x >> 4);
  int64_t n = n0;
  if (G >= 16) {
    if (g >= G) {
      g -= G;
      n += 1;
    }
  } else {
    n += g / G;
    g = g % G;
  }
  const int chunk = b >> 2;  // 32-code chunk of the group this lane belongs to
  const int sub = b & 3;     // which 8 codes of the chunk (codes 8*sub .. 8*sub+7)
  const int64_t C = 4 * (int64_t)G;
  const int64_t c = 4 * (int64_t)g + chunk;

  if constexpr (BITS == 4) {
    // Plane `sub` holds codes 8*sub..8*sub+7: pair t of the plane at bit 4t of
    // each 16-bit half (even code low half, odd code high half).
    uint32_t word = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) word |= q[e] << (((e & 1) << 4) + ((e >> 1) << 2));
    qweight[(n * 4 + sub) * C + c] = word;
  } else {
    // The chunk's 32 codes in natural order (code i at bits 3i of a 96-bit
    // string W2:W1:W0), assembled in every lane of the chunk's quad from the
    // four lanes' 24-bit pieces.  Lane `sub` < 3 then builds plane `sub`:
    // codes 10*sub .. 10*sub+9 are the 30 bits starting at bit 30*sub, placed
    // into the five 3-bit fields of each 16-bit half, plus bit `sub` of codes
    // 30 and 31 at bits 9 and 25.
    uint32_t nat = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) nat |= q[e] << (3 * e);
    const uint32_t n0w = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)nat, 0x00, 0xF, 0xF, false);  // quad_perm [0,0,0,0]
    const uint32_t n1w = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)nat, 0x55, 0xF, 0xF, false);  // quad_perm [1,1,1,1]
    const uint32_t n2w = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)nat, 0xAA, 0xF, 0xF, false);  // quad_perm [2,2,2,2]
    const uint32_t n3w = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)nat, 0xFF, 0xF, 0xF, false);  // quad_perm [3,3,3,3]
    const uint32_t W0 = n0w | (n1w << 24);
    const uint32_t W1 = (n1w >> 8) | (n2w << 16);
    const uint32_t W2 = (n2w >> 16) | (n3w << 8);
    const uint32_t win1 = __builtin_amdgcn_alignbit(W1, W0, 30);  // bits 30..61
    const uint32_t win2 = __builtin_amdgcn_alignbit(W2, W1, 28);  // bits 60..91
    const uint32_t win = sub == 0 ? W0 : (sub == 1 ? win1 : win2);
    uint32_t pw = 0;
#pragma unroll
    for (int j = 0; j < 10; ++j) {
      const int field = j >> 1;
      const int shift = ((j & 1) << 4) + 3 * field + (field >= 3 ? 1 : 0);
      pw |= ((win >> (3 * j)) & 7u) << shift;
    }
    const uint32_t spare = W2 >> (26 + sub);  // bit 0: bit `sub` of code 30; bit 3: of code 31
    pw |= ((spare & 1u) << 9) | (((spare >> 3) & 1u) << 25);
    if (sub < 3) qweight[(n * 3 + sub) * C + c] = pw;
  }
  if (!GIVEN && b == 0) {
    scales[grp] = (uint16_t)s16;
    zeros[grp] = (uint8_t)z;
  }
}

}  // namespace

template <int BITS>
hipError_t launch_quantize(const uint16_t* w, int64_t N, int64_t K, uint32_t* qweight,
                           uint16_t* scales, uint8_t* zeros, hipStream_t stream,
                           const LaunchEvents& ev) {
  const int64_t G = K / 128;
  const int64_t n_groups = N * G;
  const int64_t blocks = (n_groups + 15) / 16;  // 16 groups per 256-thread block
  launch(quantize_kernel<BITS, false>, dim3((unsigned)blocks), dim3(256), 0, stream, ev,
         reinterpret_cast<const u32x4*>(w), n_groups, (int)G, qweight, scales, zeros);
  return hipGetLastError();
}

template <int BITS>
hipError_t launch_pack(const uint16_t* w, const uint16_t* scales, const uint8_t* zeros, int64_t N,
                       int64_t K, uint32_t* qweight, hipStream_t stream, const LaunchEvents& ev) {
  const int64_t G = K / 128;
  const int64_t n_groups = N * G;
  const int64_t blocks = (n_groups + 15) / 16;
  // The GIVEN kernel only reads scales and zeros.
  launch(quantize_kernel<BITS, true>, dim3((unsigned)blocks), dim3(256), 0, stream, ev,
         reinterpret_cast<const u32x4*>(w), n_groups, (int)G, qweight, const_cast<uint16_t*>(scales),
         const_cast<uint8_t*>(zeros));
  return hipGetLastError();
}

template hipError_t launch_quantize<3>(const uint16_t*, int64_t, int64_t, uint32_t*, uint16_t*,
                                       uint8_t*, hipStream_t, const LaunchEvents&);
template hipError_t launch_quantize<4>(const uint16_t*, int64_t, int64_t, uint32_t*, uint16_t*,
                                       uint8_t*, hipStream_t, const LaunchEvents&);
template hipError_t launch_pack<3>(const uint16_t*, const uint16_t*, const uint8_t*, int64_t, int64_t,
                                   uint32_t*, hipStream_t, const LaunchEvents&);
template hipError_t launch_pack<4>(const uint16_t*, const uint16_t*, const uint8_t*, int64_t, int64_t,
                                   uint32_t*, hipStream_t, const LaunchEvents&);

}  // namespace laq
