// Quantize + pack kernel: Eq. 1 (Sec. 2) with round-to-nearest min-max
// scale and zero point per group of 128 consecutive weights of a row, packed
// into the plane layout of include/laq.h (32 codes in three 32-bit words for
// W3, as App. G keeps; eight 4-bit codes per word for W4).
//
// Mapping: 16 lanes per group, each lane owns 8 consecutive weights (one
// 16-byte load; a group is 256 contiguous bytes, so a wave reads 1 KB
// contiguous).  The group range is reduced across the 16 lanes (min/max are
// exact in any order), every lane derives the same (s, z) with IEEE fp32
// arithmetic, quantizes its 8 weights with true division and round-half-even,
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
#pragma unroll
    for (int o = 8; o >= 1; o >>= 1) {
      lo = fminf(lo, __shfl_xor(lo, o, 16));
      hi = fmaxf(hi, __shfl_xor(hi, o, 16));
    }
    const float s32 = (hi - lo) / qmax;  // IEEE division (no fast-math)
    s16 = __builtin_bit_cast(uint16_t, (_Float16)s32);  // round-to-nearest-even
    if (s16 == 0) s16 = 1;                              // 2^-24 when the range underflows
    s = half_bits_to_float(s16);
    z = fminf(fmaxf(rintf(-lo / s), 0.0f), qmax);
  }

  // Codes: the clip is taken on the real value (a quotient that is not a
  // number gives 0), so no out-of-range value reaches the integer conversion.
  uint32_t q[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float t = fminf(fmaxf(rintf(v[e] / s) + z, 0.0f), qmax);
    q[e] = (uint32_t)t;
  }

  const int64_t n = grp / G;
  const int g = (int)(grp - n * G);
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
    // Three planes, each holding ten codes in five 3-bit fields per 16-bit
    // half; the last two codes of the chunk are spread one bit per plane.
    uint32_t pw[3] = {0u, 0u, 0u};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int i = 8 * sub + e;  // code index in the chunk
      if (i < 30) {
        const int plane = i / 10;
        const int r = i - 10 * plane;
        const int field = r >> 1;
        const int shift = ((r & 1) << 4) + 3 * field + (field >= 3 ? 1 : 0);
        const uint32_t bits = q[e] << shift;
        pw[0] |= plane == 0 ? bits : 0u;
        pw[1] |= plane == 1 ? bits : 0u;
        pw[2] |= plane == 2 ? bits : 0u;
      } else {
        const int pos = (i == 30) ? 9 : 25;
#pragma unroll
        for (int p = 0; p < 3; ++p) pw[p] |= ((q[e] >> p) & 1u) << pos;
      }
    }
#pragma unroll
    for (int p = 0; p < 3; ++p) {
      pw[p] |= __shfl_xor(pw[p], 1, 4);
      pw[p] |= __shfl_xor(pw[p], 2, 4);
    }
    if (sub == 0) {
#pragma unroll
      for (int p = 0; p < 3; ++p) qweight[(n * 3 + p) * C + c] = pw[p];
    }
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
