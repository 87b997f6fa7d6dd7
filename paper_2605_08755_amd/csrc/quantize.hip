// Quantize + pack kernel: Eq. 1 (Sec. 2) with round-to-nearest min-max
// scale and zero point per group of 128 consecutive weights of a row, packed
// into the plane layout of include/laq.h (32 codes in three 32-bit words for
// W3, as App. H keeps; eight 4-bit codes per word for W4).
//
// Mapping: a wave takes 16 consecutive groups (4 KiB of fp16, read as four
// fully coalesced 1 KiB direct-to-LDS loads) and 4 lanes per group (a
// quad), lane j owning the group's 32-code chunk j, so each lane packs its
// chunk's plane words by itself.  The group range is reduced on packed fp16
// pairs in the lane and across the quad with DPP (min/max are exact in any
// order); every lane derives the same (s, z) with IEEE fp32 arithmetic and
// quantizes its 32 weights with the IEEE quotient (formed from a reciprocal
// and two fused multiply-adds, see below) and round-half-even.
//
// The same kernel also packs with caller-supplied parameters (GIVEN): Eq. 1
// with the scale and zero point read from memory (e.g. the ones LAQuant's
// QAT learned) instead of the min-max ones.
#include "laq_internal.h"

namespace laq {

namespace {

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

// Minimum and maximum over the 4 lanes of a quad; every lane receives both.
__device__ __forceinline__ void quad_minmax(float& lo, float& hi) {
  lo = fminf(lo, dpp<0xB1>(lo));  // quad_perm [1,0,3,2]
  hi = fmaxf(hi, dpp<0xB1>(hi));
  lo = fminf(lo, dpp<0x4E>(lo));  // quad_perm [2,3,0,1]
  hi = fmaxf(hi, dpp<0x4E>(hi));
}

// Codes are carried as the bit patterns of floats: for |t| < 2^22, the sum
// 1.5 * 2^23 + t rounds t to an integer, half to even (the rounding of
// Eq. 1's round()), and its bit pattern is kCodeBits + round(t).  With the
// zero point folded into the clip bounds, a code is
//   c = clamp(bits(t + 1.5 * 2^23), kCodeBits - z, kCodeBits + qmax - z)
//     = kCodeBits - z + clip(round(t) + z, 0, qmax)
// as a signed 32-bit integer; a quotient beyond 2^22 in magnitude still
// lands on the right bound (positive floats order like their bit patterns,
// negative ones are negative integers).  Packing adds each c shifted to its
// field and subtracts (kCodeBits - z) times the sum of the fields' unit
// values once per word (all modulo 2^32), which leaves the OR of the codes.
constexpr float kCodeBase = 12582912.0f;  // 1.5 * 2^23
constexpr int kCodeBits = 0x4B400000;

// W3 plane p of a chunk holds codes 10p .. 10p+9: code 10p + f at bit kW3Shift[f]
// (five 3-bit fields per 16-bit half, even codes in the low half), and bit p
// of codes 30 and 31 at bits 9 and 25.
constexpr int kW3Shift[10] = {0, 16, 3, 19, 6, 22, 10, 26, 13, 29};
constexpr uint32_t kW3Units = 0x24492449u;  // sum of 1 << kW3Shift[f]
// W4 plane p holds codes 8p .. 8p+7: code 8p + e at bit 16 (e % 2) + 4 (e / 2).
constexpr int kW4Shift[8] = {0, 16, 4, 20, 8, 24, 12, 28};
constexpr uint32_t kW4Units = 0x11111111u;  // sum of 1 << kW4Shift[e]

__device__ __forceinline__ uint32_t shl_add(uint32_t a, int sh, uint32_t b) { return (a << sh) + b; }

// Median of three signed integers: clamp(x, lo, hi) for lo <= hi (one
// instruction; the compiler forms it only for constant bounds).
__device__ __forceinline__ int med3_i32(int x, int lo, int hi) {
  int r;
  asm("v_med3_i32 %0, %1, %2, %3" : "=v"(r) : "v"(x), "v"(lo), "v"(hi));
  return r;
}

// The group's codes.  The quotient v / s is formed without a per-weight
// division: with y = RN(1/s) (one IEEE division per group), q = RN(v*y),
// r = v - q*s (exact, fused) and q' = RN(q + r*y) (fused), q' equals the
// IEEE binary32 quotient RN(v/s) for every finite fp16 v and every finite
// positive fp16 s -- checked exhaustively over all 2.0e9 such pairs
// (tests/native/fp16_quotient_check.c, which uses the same operations).  q
// is written as fma(v, y, +0), which differs from RN(v*y) only in the sign
// of a zero and gives the same q'.  For a scale outside that domain (one the
// interface excludes) the codes are unspecified.
template <int BITS>
__device__ __forceinline__ void group_codes(const uint32_t (&h)[16], float s, int z, int (&c)[32]) {
#pragma clang fp contract(off)
  const float y = 1.0f / s;  // IEEE division (no fast-math)
  const int lo = kCodeBits - z;
  const int hi = lo + (1 << BITS) - 1;
#pragma unroll
  for (int e = 0; e < 32; ++e) {
    const float v = (float)__builtin_bit_cast(half2_t, h[e >> 1])[e & 1];  // exact
    const float q0 = fmaf(v, y, 0.0f);
    const float r = fmaf(-q0, s, v);
    const float qt = fmaf(r, y, q0);
    c[e] = med3_i32(__builtin_bit_cast(int, qt + kCodeBase), lo, hi);
  }
}

// Staging of a wave's 16 groups (4 KiB): four direct-to-LDS loads, each
// 1 KiB of consecutive bytes (lane l of load i fills stage position 64 i + l),
// then lane 4q + j reads chunk j of group q, its four 16-byte pieces
// 16q + 4j + k.  Piece P is stored at position P ^ ((P >> 4) & 3), so the
// 16 lanes of one LDS read cycle hit 16 different bank quads.
constexpr int kWaveGroups = 16;
__device__ __forceinline__ int stage_slot(int piece) { return piece ^ ((piece >> 4) & 3); }

template <int BITS, bool GIVEN>
__global__ __launch_bounds__(256) void quantize_kernel(const u32x4* __restrict__ w, int64_t n_groups,
                                                       int G, float inv_g, uint32_t* __restrict__ qweight,
                                                       uint16_t* __restrict__ scales,
                                                       uint8_t* __restrict__ zeros) {
#pragma clang fp contract(off)
  typedef __attribute__((address_space(3))) void lds_void;
  __shared__ u32x4 stage[4][64 * 4];
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);          // wave-uniform: scalar descriptor
  const int64_t wg0 = (int64_t)blockIdx.x * 64 + wave * kWaveGroups;  // first group (flat n*G + g) of the wave
  const int64_t wgn = n_groups - wg0;
  if (wgn <= 0) return;
  const int64_t grp = wg0 + (lane >> 2);  // this lane's group
  const int j = lane & 3;                 // and its chunk
  const bool live = grp < n_groups;

  // Loads past the wave's last group read zeros (buffer extent).
  const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<u32x4*>(w + wg0 * 16), (short)0, (int)((wgn < kWaveGroups ? wgn : kWaveGroups) * 256),
      0x00020000);
#pragma unroll
  for (int i = 0; i < 4; ++i)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (lds_void*)&stage[wave][64 * i], 16,
                                             (uint32_t)stage_slot(64 * i + lane) * 16, 0, 0,
                                             2 /* non-temporal: read once */);
  uint32_t s16 = 0;
  int zi = 0;
  if constexpr (GIVEN) {  // issued with the weight loads (same wait)
    const int64_t gl = live ? grp : wg0;
    s16 = scales[gl];
    zi = zeros[gl];
  }
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): the stage is written
  __builtin_amdgcn_sched_barrier(0);
  // Lanes past the last group (in the grid's last wave only) compute on zeros
  // and store nothing: no branch here, so the parameter loads above are not
  // moved behind the wait.

  uint32_t h[16];  // fp16 pairs: pair e holds codes 2e (low half) and 2e + 1 of the chunk
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const u32x4 v = stage[wave][stage_slot(4 * lane + k)];
    h[4 * k + 0] = v.x;
    h[4 * k + 1] = v.y;
    h[4 * k + 2] = v.z;
    h[4 * k + 3] = v.w;
  }

  constexpr int qmax = (1 << BITS) - 1;
  if constexpr (!GIVEN) {
    // Group range, widened to contain 0: fp16 pairs reduced in the lane
    // (exact in any order), then across the quad.
    half2_t mn = __builtin_bit_cast(half2_t, h[0]), mx = mn;
#pragma unroll
    for (int e = 1; e < 16; ++e) {
      mn = __builtin_elementwise_minimum(mn, __builtin_bit_cast(half2_t, h[e]));
      mx = __builtin_elementwise_maximum(mx, __builtin_bit_cast(half2_t, h[e]));
    }
    float lo = fminf(0.0f, fminf((float)mn[0], (float)mn[1]));
    float hi = fmaxf(0.0f, fmaxf((float)mx[0], (float)mx[1]));
    quad_minmax(lo, hi);
    const float s32 = (hi - lo) / (float)qmax;          // IEEE division (no fast-math)
    s16 = __builtin_bit_cast(uint16_t, (_Float16)s32);  // round-to-nearest-even
    if (s16 == 0) s16 = 1;                              // 2^-24 when the range underflows
    const float sh = (float)__builtin_bit_cast(_Float16, (uint16_t)s16);
    zi = (int)fminf(fmaxf(rintf(-lo / sh), 0.0f), (float)qmax);
  }
  const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)s16);
  int c[32];
  group_codes<BITS>(h, s, zi, c);
  const uint32_t base = 0u - (uint32_t)(kCodeBits - zi) * (BITS == 4 ? kW4Units : kW3Units);

  // (row, group) of this lane: the block's first group splits on the scalar
  // unit; a lane's group is at most 63 further, i.e. at most one row wrap when
  // G >= 64, and otherwise (d + g0 < 128) the quotient is trunc((d + g0 +
  // 0.5) * fl(1/G)), exact for numerators below 1024.
  const int64_t gbase = (int64_t)blockIdx.x * 64;
  const int64_t n0 = gbase / G;
  const int g0 = (int)(gbase - n0 * G);
  const int num = g0 + (t >> 2);
  const int wrap = G >= 64 ? (num >= G ? 1 : 0) : (int)(((float)num + 0.5f) * inv_g);
  const int64_t n = n0 + wrap;
  const int g = num - wrap * G;
  const int64_t C = 4 * (int64_t)G;
  const int64_t cw = 4 * (int64_t)g + j;

  if constexpr (BITS == 4) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      uint32_t word = base;
#pragma unroll
      for (int e = 0; e < 8; ++e) word = shl_add((uint32_t)c[8 * p + e], kW4Shift[e], word);
      if (live) qweight[(n * 4 + p) * C + cw] = word;
    }
  } else {
    // bit p of codes 30 and 31 sits at bit 9 + p and 25 + p of `spare`
    const uint32_t spare = (((uint32_t)(c[30] - (kCodeBits - zi))) << 9) | (((uint32_t)(c[31] - (kCodeBits - zi))) << 25);
#pragma unroll
    for (int p = 0; p < 3; ++p) {
      uint32_t word = base;
#pragma unroll
      for (int f = 0; f < 10; ++f) word = shl_add((uint32_t)c[10 * p + f], kW3Shift[f], word);
      word |= (spare >> p) & 0x02000200u;
      if (live) qweight[(n * 3 + p) * C + cw] = word;
    }
  }
  if (!GIVEN && live && j == 0) {
    scales[grp] = (uint16_t)s16;
    zeros[grp] = (uint8_t)zi;
  }
}

}  // namespace

template <int BITS>
hipError_t launch_quantize(const uint16_t* w, int64_t N, int64_t K, uint32_t* qweight,
                           uint16_t* scales, uint8_t* zeros, hipStream_t stream,
                           const LaunchEvents& ev) {
  const int64_t G = K / 128;
  const int64_t n_groups = N * G;
  const int64_t blocks = (n_groups + 63) / 64;  // 64 groups per 256-thread block
  launch(quantize_kernel<BITS, false>, dim3((unsigned)blocks), dim3(256), 0, stream, ev,
         reinterpret_cast<const u32x4*>(w), n_groups, (int)G, 1.0f / (float)G, qweight, scales, zeros);
  return hipGetLastError();
}

template <int BITS>
hipError_t launch_pack(const uint16_t* w, const uint16_t* scales, const uint8_t* zeros, int64_t N,
                       int64_t K, uint32_t* qweight, hipStream_t stream, const LaunchEvents& ev) {
  const int64_t G = K / 128;
  const int64_t n_groups = N * G;
  const int64_t blocks = (n_groups + 63) / 64;
  // The GIVEN kernel only reads scales and zeros.
  launch(quantize_kernel<BITS, true>, dim3((unsigned)blocks), dim3(256), 0, stream, ev,
         reinterpret_cast<const u32x4*>(w), n_groups, (int)G, 1.0f / (float)G, qweight,
         const_cast<uint16_t*>(scales), const_cast<uint8_t*>(zeros));
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
