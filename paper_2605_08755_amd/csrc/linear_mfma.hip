// Skinny-GEMM path (several activation rows) on the matrix cores.
//
// y[m][n] = sum_g s[n][g] * sum_{k in g} x[m][k] * (q[n][k] - z[n][g])   (Eq. 1)
//
// One v_mfma_f32_16x16x32_f16 multiplies a 16 x 32 activation tile (rows m,
// zero past M) by a 32 x 16 tile of exact (q - z) values of 16 weight rows.
// Lane l supplies weight row n = l % 16 and, within the 32-wide K window,
// the 8 codes of chunk l / 16 of the current 128-group, so every window stays
// inside one group (one scale and zero point per row).  The result fragment
// of lane l is column n = l % 16 (rows m = 4(l/16)..+3), i.e. the lane's own
// weight row, so each lane scales by its own row's s[n][g].
//
// Unpack to exact fp16 (q - z): OR-ing a 3-bit (or 4-bit) code field at
// mantissa bits [p, p+b) with the bits of 2^(10-p) gives the fp16 value
// 2^(10-p) + q exactly; one packed fp16 add of -(2^(10-p) + z) leaves q - z
// exactly.  One v_and_or_b32 + one v_pk_add_f16 per two codes.
//
// Kernels: one wave per quad of a 16-row tile, every load issued at once
// (rows of at most ten quads: fewer than 1024 tiles, or M <= 4); the same
// with three tiles per block sharing the quads' slabs (many tiles, rows of at
// most five quads, M > 4); one or two 16-row tiles per block, its waves
// splitting the row's quads (fewer tiles, longer rows); four tiles per block
// over a K range, one quad ahead (split K, whose fp32 partials a second
// kernel adds in order); four or eight tiles per block walking K one quad at
// a time, two quads ahead (many tiles, longer rows).  Every reduction order
// is fixed, so results are deterministic.
#include <type_traits>
#include <utility>

#include "laq_internal.h"

namespace laq {

namespace {

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float float4_t __attribute__((ext_vector_type(4)));

constexpr int kBufferFlagsM = 0x00020000;
// Cache policy of the weight loads.  A lane's 16-byte load covers four groups
// of one row and plane, so one load instruction uses half of each 128-byte
// line it touches and the next quad's load uses the other half.  With the
// non-temporal hint that second half was read again from memory when the
// loads of the two quads were a quad's compute apart (the one-tile and
// quad-walking kernels: Qwen3-32B gate|up 44.8 -> 39.4 us, down 36.1 -> 33.1
// us at M = 16 with plain loads); the kernel that requests all quads at once
// keeps the hint.
constexpr int kWeightPolicy = 0;    // plain
constexpr int kWeightPolicyNT = 2;  // non-temporal

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kBufferFlagsM);
}

__device__ __forceinline__ uint32_t pk_add_f16(uint32_t a, uint32_t b) {
  return __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2_t, a) + __builtin_bit_cast(half2_t, b));
}

// (a & m) | c in one v_and_or_b32.  The mask lives in a scalar register and
// the magic constant in a vector register (a VOP3 instruction takes no
// literal on this target, and at most one scalar operand); left to itself the
// compiler emits a v_and_b32 and a v_or_b32 with literals instead.
__device__ __forceinline__ uint32_t and_or(uint32_t a, uint32_t m, uint32_t c) {
  uint32_t r;
  asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "s"(m), "v"(c));  // mask from a scalar register
  return r;
}

// fp16 bit patterns of -(2^(10-p) + z) in both halves, for the field
// offsets used by the layouts (ulp of 2^(10-p) is 2^-p, so + z is + z*2^p
// ulps).  zz holds z in both 16-bit halves; z << shift < 2^11, so no carry
// crosses between the halves.
__device__ __forceinline__ uint32_t neg_magic(uint32_t base_bits, uint32_t zz, uint32_t shift) {
  return (base_bits | (base_bits << 16)) + (zz << shift);
}

// Exact (q - z) pairs of one 32-code chunk, in natural order: pair t holds
// codes 2t (low half) and 2t+1 (high half).
template <int BITS>
__device__ __forceinline__ void unpack_chunk_exact(const uint32_t (&w)[BITS], uint32_t z1, uint32_t (&pr)[16]) {
  const uint32_t z = z1 | (z1 << 16);
  if constexpr (BITS == 3) {
    const uint32_t n0 = neg_magic(0xE400u, z, 0);  // -(1024 + z): fields at bits 0-2
    const uint32_t n3 = neg_magic(0xD800u, z, 3);  // -(128 + z):  bits 3-5
    const uint32_t n6 = neg_magic(0xCC00u, z, 6);  // -(16 + z):   bits 6-8
    const uint32_t n7 = neg_magic(0xC800u, z, 7);  // -(8 + z):    bits 7-9
#pragma unroll
    for (int p = 0; p < 3; ++p) {
      const uint32_t t = w[p] >> 10;
      pr[5 * p + 0] = pk_add_f16(and_or(w[p], 0x00070007u, 0x64006400u), n0);
      pr[5 * p + 1] = pk_add_f16(and_or(w[p], 0x00380038u, 0x58005800u), n3);
      pr[5 * p + 2] = pk_add_f16(and_or(w[p], 0x01C001C0u, 0x4C004C00u), n6);
      pr[5 * p + 3] = pk_add_f16(and_or(t, 0x00070007u, 0x64006400u), n0);
      pr[5 * p + 4] = pk_add_f16(and_or(t, 0x00380038u, 0x58005800u), n3);
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
      pr[4 * p + 0] = pk_add_f16(and_or(w[p], 0x000F000Fu, 0x64006400u), n0);
      pr[4 * p + 1] = pk_add_f16(and_or(w[p], 0x00F000F0u, 0x54005400u), n4);
      pr[4 * p + 2] = pk_add_f16(and_or(t, 0x000F000Fu, 0x64006400u), n0);
      pr[4 * p + 3] = pk_add_f16(and_or(t, 0x00F000F0u, 0x54005400u), n4);
    }
  }
}

__device__ __forceinline__ half8_t frag(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
  return __builtin_bit_cast(half8_t, u32x4v{a, b, c, d});
}

// Fragment reads from an LDS slab that direct-to-LDS loads fill, written as
// inline assembly on purpose: the compiler's wait insertion treats any LDS
// read that follows a direct-to-LDS load as dependent on every such load in
// flight, so it would wait for the loads of later quads too.  The waits the
// data flow needs are explicit instead: vmcnt before the barrier that
// publishes a slab, lgkmcnt (lds_wait) before the fragments are used.
__device__ __forceinline__ uint32_t lds_addr(const u32x4* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) u32x4*)p;
}
__device__ __forceinline__ u32x4 lds_read_b128(uint32_t addr) {
  u32x4 r;
  asm volatile("ds_read_b128 %0, %1" : "=v"(r) : "v"(addr));
  return r;
}
// Waits for the outstanding LDS reads; the fragments pass through the
// statement, so no use of them is scheduled before the wait.
__device__ __forceinline__ void lds_wait(u32x4 (&f)[4]) {
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3]));
}

// s_waitcnt vmcnt(N) (other counters unconstrained), N a compile-time constant <= 63.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | (((N >> 4) & 3) << 14));
}

// f(std::integral_constant<int, I>{}) for I = 0 .. N-1, in order.
template <typename F, int... Is>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, Is...>) {
  (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Loads of dead lanes (rows past M, columns past K, groups past G) OR bit
// 31 into their offsets: that is past every buffer extent, so the load
// returns zero and moves no data.

// 4 x 4 transpose across the four 16-lane quarters of a wave: on entry
// register c of quarter j holds element (j, c); on exit register j of
// quarter c holds it.  Two rounds of lane-half swaps (32 lanes, then 16).
__device__ __forceinline__ void transpose_quarters(uint32_t& r0, uint32_t& r1, uint32_t& r2, uint32_t& r3) {
  auto a = __builtin_amdgcn_permlane32_swap(r0, r2, false, false);
  auto b = __builtin_amdgcn_permlane32_swap(r1, r3, false, false);
  auto c = __builtin_amdgcn_permlane16_swap(a[0], b[0], false, false);
  auto d = __builtin_amdgcn_permlane16_swap(a[1], b[1], false, false);
  r0 = c[0];
  r1 = c[1];
  r2 = d[0];
  r3 = d[1];
}

// Block: TW tiles of 16 weight rows and every group of them.  Work item of a
// wave: the four consecutive groups 4Q..4Q+3 (a "quad") of all TW tiles; the
// W waves of the block take quads wave, wave + W, ...
//
// Loads of a quad, lane (n = lane % 16, j = lane / 16): per tile, one 16-byte
// load per plane of row n, group 4Q + j (four chunks), so each row of a tile
// reads 64 contiguous bytes per plane, and the scale and zero point of that
// (row, group).  The quad's activations x[0..M-1][512Q .. 512Q+511] go into
// the wave's own LDS slab of M rows with 16-byte direct-to-LDS loads, one
// fully coalesced 1 KiB row piece per instruction (fragment loads straight
// from memory would touch 64 separate cache lines per instruction); lanes of
// activation rows m >= M read row M - 1, which feeds only result rows that
// are not stored.  A slab of M rows (not 16) lets small M keep more waves
// resident.  A
// quarter transpose then gives quarter q chunk q of every group of the quad,
// the layout the matrix core wants (lane (n, q) supplies row n's codes 32q ..
// 32q+31 of the group).  Slots past the last group read zeros.
constexpr int kSlabRowU4 = 64;          // one slab row: 64 pieces of 16 bytes
constexpr int kBlockLdsU4 = 160 * 64;   // 160 KiB of LDS per block

// Waves of a linear_mfma_kernel block: one per quad of the row, at most 8
// (more waves per block measured slower: Qwen3-4B down, 19 quads, at M = 16
// 10.3 us with 10 waves, 10.0 with 8) and as many M-row activation slabs
// (M KiB each) as fit in 160 KiB; longer rows loop.  The host sizes the
// block with it and the kernel derives its wave count from it.
__host__ __device__ constexpr int mfma_block_waves(int M, int nq) {
  const int wmax = 8 < kBlockLdsU4 / (M * kSlabRowU4) ? 8 : kBlockLdsU4 / (M * kSlabRowU4);
  return wmax < nq ? wmax : nq;
}

template <int BITS, int TW>
__device__ __forceinline__ void mfma_block(
    const uint16_t* __restrict__ x, const uint32_t* __restrict__ qw, const uint16_t* __restrict__ scales,
    const uint8_t* __restrict__ zeros, uint16_t* __restrict__ y, int M, int N, int G, int block, int W) {
  typedef __attribute__((address_space(3))) void lds_void;
  extern __shared__ u32x4 wslabs[];  // [W][M rows][64 pieces]; afterwards the wave's partials

  const int K = 128 * G;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform: scalar loop
  const int nl = lane & 15;  // weight row of a tile / activation row / result column
  const int q = lane >> 4;   // load: group of the quad; compute: chunk of the group
  // Row range in 32-bit unsigned scalar arithmetic (row0 < N + 2^10 < 2^32):
  // 64-bit compares would run on the vector unit ahead of the first load.
  const uint32_t r0u = (uint32_t)block * (16u * TW);
  const int64_t row0 = (int64_t)r0u;
  const int rows = r0u < (uint32_t)N ? (int)min(16u * TW, (uint32_t)N - r0u) : 0;
  const int C = 4 * G;
  const int nq = (G + 3) >> 2;
  u32x4* const sl = wslabs + wave * (M * kSlabRowU4);
  const int swz = nl & 7;
  const int arow = min(nl, M - 1);  // activation row read by this lane

  const __amdgpu_buffer_rsrc_t xr = rsrc(x, (uint32_t)M * K * 2);
  const __amdgpu_buffer_rsrc_t qr = rsrc(qw + row0 * BITS * C, (uint32_t)rows * BITS * C * 4);
  const __amdgpu_buffer_rsrc_t sr = rsrc(scales + row0 * G, (uint32_t)rows * G * 2);
  const __amdgpu_buffer_rsrc_t zr = rsrc(zeros + row0 * G, (uint32_t)rows * G);

  float4_t yacc[TW];
#pragma unroll
  for (int t = 0; t < TW; ++t) yacc[t] = float4_t{0.f, 0.f, 0.f, 0.f};

  for (int Q = wave; Q < nq; Q += W) {
    // 1. Loads.  Rows past the block are past their extents.  The slab is
    //    rewritten only after the previous quad's fragment reads returned.
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
    // Groups past G get bit 31 set in their offsets (past every extent):
    // arithmetic, not a select, which the compiler may turn into a branch
    // that waits for the loads before it.
    const int gq = 4 * Q + q;
    const uint32_t dead = (uint32_t)(gq >= G) << 31;
    u32x4 wv[TW][BITS];
    uint32_t sraw[TW], zraw[TW];
#pragma unroll
    for (int t = 0; t < TW; ++t) {
      const int nrow = 16 * t + nl;
#pragma unroll
      for (int p = 0; p < BITS; ++p)
        wv[t][p] = __builtin_amdgcn_raw_buffer_load_b128(
            qr, (uint32_t)(((nrow * BITS + p) * C + 4 * gq) * 4) | dead, 0, kWeightPolicy);
      sraw[t] = __builtin_amdgcn_raw_buffer_load_b16(sr, (uint32_t)(nrow * G + gq) * 2 | dead, 0, 0);
      zraw[t] = __builtin_amdgcn_raw_buffer_load_b8(zr, (uint32_t)(nrow * G + gq) | dead, 0, 0);
    }
    // Slab row m: lane l fetches piece l ^ (m & 7) (8 columns) into position
    // l; columns past K read zero.
    for (int m = 0; m < M; ++m) {
      const int col = 512 * Q + 8 * (lane ^ (m & 7));
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void*)(sl + m * 64), 16,
                                               (uint32_t)(m * K + col) * 2 | (uint32_t)!(col < K) << 31, 0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): weights and slab
    __builtin_amdgcn_sched_barrier(0);

    // 2. Quarter transposes: plane words (chunk q of group 4Q + j now in
    //    component j) and the four groups' scale | zero << 16 in every quarter.
    uint32_t wt[TW][BITS][4];
    uint32_t szj[TW][4];
#pragma unroll
    for (int t = 0; t < TW; ++t) {
#pragma unroll
      for (int p = 0; p < BITS; ++p) {
        wt[t][p][0] = wv[t][p][0];
        wt[t][p][1] = wv[t][p][1];
        wt[t][p][2] = wv[t][p][2];
        wt[t][p][3] = wv[t][p][3];
        transpose_quarters(wt[t][p][0], wt[t][p][1], wt[t][p][2], wt[t][p][3]);
      }
      const uint32_t sz = sraw[t] | (zraw[t] << 16);
      szj[t][0] = szj[t][1] = szj[t][2] = szj[t][3] = sz;
      transpose_quarters(szj[t][0], szj[t][1], szj[t][2], szj[t][3]);
    }

    // 3. Per group and tile: exact (q - z) pairs, four MFMAs, scale.
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      half8_t a[4];
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) a[jj] = __builtin_bit_cast(half8_t, sl[arow * 64 + ((16 * j + 4 * q + jj) ^ swz)]);
#pragma unroll
      for (int t = 0; t < TW; ++t) {
        uint32_t w[BITS];
#pragma unroll
        for (int p = 0; p < BITS; ++p) w[p] = wt[t][p][j];
        uint32_t pr[16];
        unpack_chunk_exact<BITS>(w, szj[t][j] >> 16, pr);
        float4_t c = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const half8_t b = frag(pr[4 * jj + 0], pr[4 * jj + 1], pr[4 * jj + 2], pr[4 * jj + 3]);
          c = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[jj], b, c, 0, 0, 0);
        }
        const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)(szj[t][j] & 0xFFFFu));
        yacc[t] += s * c;
      }
    }
  }

  // 4. Fixed-order reduction of the W waves' partials (each wave's partials,
  //    TW KiB, go into its own slab of M >= TW KiB, whose reads have all
  //    returned).
  float* red = reinterpret_cast<float*>(wslabs);
  const int kWaveSlabF = M * kSlabRowU4 * 4;
#pragma unroll
  for (int t = 0; t < TW; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r) red[wave * kWaveSlabF + (t * 4 + r) * 64 + lane] = yacc[t][r];
  __syncthreads();
  for (int idx = threadIdx.x; idx < TW * 4 * 64; idx += 64 * W) {
    const int t = idx >> 8;
    const int r = (idx >> 6) & 3;
    const int ln = idx & 63;
    float v = 0.0f;
    for (int w = 0; w < W; ++w) v += red[w * kWaveSlabF + (t * 4 + r) * 64 + ln];
    const int m = 4 * (ln >> 4) + r;
    const int n = 16 * t + (ln & 15);
    if (m < M && n < rows) y[(int64_t)m * N + row0 + n] = __builtin_bit_cast(uint16_t, (_Float16)v);
  }
}

// ---------------------------------------------------------------------------
// Activation-sharing variant for many row tiles and rows longer than five
// quads (K > 2560).  A block of TB waves owns TB
// consecutive 16-row tiles, one per wave, and walks K one quad (4 groups =
// 512 columns) at a time.  The quad's activation slab x[0..15][512q ..
// 512q+511] (rows past M read as zero) goes straight from memory into LDS
// (16-byte direct-to-LDS buffer loads, no registers), once per block for its
// TB tiles, into one of three buffers.  The slab and the wave's weights of
// quad q+2 are requested while quad q is computed; per lane and quad the
// weights are the loads of mfma_block (row n, group 4q + j, one 16-byte load
// per plane), in one of three register sets in turn.  One barrier per quad.
//
// Slab rows are 64 pieces of 16 bytes; piece p of row m sits at position
// p ^ (m & 7), so the A-fragment reads of a wave (16 rows x 4 pieces) spread
// over all LDS banks.  Lane l of a direct load writes position l, so it
// fetches piece l ^ (m & 7).
// ---------------------------------------------------------------------------
constexpr int kSlabBuffers = 3;
constexpr uint32_t kSlabBytes = 16 * 64 * 16;
constexpr uint32_t kSlabLdsBytes = kSlabBuffers * kSlabBytes;

struct QuadWeights3 {
  u32x4 w[3];
  uint32_t s, z;
};
struct QuadWeights4 {
  u32x4 w[4];
  uint32_t s, z;
};
template <int BITS>
using QuadWeights = typename std::conditional<BITS == 3, QuadWeights3, QuadWeights4>::type;

// Loads of one quad for lane (n, j); groups past G (and idle tiles, whose
// extents are zero) read zeros.  BITS + 2 vector-memory instructions; AUX is
// the cache policy of the code loads.
template <int BITS, int AUX>
__device__ __forceinline__ QuadWeights<BITS> load_quad(__amdgpu_buffer_rsrc_t qr, __amdgpu_buffer_rsrc_t sr,
                                                       __amdgpu_buffer_rsrc_t zr, int n, int j, int q, int G,
                                                       bool live) {
  QuadWeights<BITS> r;
  const int C = 4 * G;
  const int gq = 4 * q + j;
  // A dead lane's offsets get bit 31 (past every extent) by an OR: a select
  // between offsets was compiled into branches that wait at their join.
  const uint32_t dead = (uint32_t)!(live && gq < G) << 31;
#pragma unroll
  for (int p = 0; p < BITS; ++p)
    r.w[p] = __builtin_amdgcn_raw_buffer_load_b128(qr, (uint32_t)(((n * BITS + p) * C + 4 * gq) * 4) | dead, 0, AUX);
  r.s = __builtin_amdgcn_raw_buffer_load_b16(sr, (uint32_t)(n * G + gq) * 2 | dead, 0, 0);
  r.z = __builtin_amdgcn_raw_buffer_load_b8(zr, (uint32_t)(n * G + gq) | dead, 0, 0);
  return r;
}

template <int BITS, int TB>
__device__ __forceinline__ void mfma_tiles_block(
    const uint16_t* __restrict__ x, const uint32_t* __restrict__ qw, const uint16_t* __restrict__ scales,
    const uint8_t* __restrict__ zeros, uint16_t* __restrict__ y, int M, int N, int G, int block) {
  extern __shared__ u32x4 slab[];  // [kSlabBuffers][16 rows][64 pieces]
  constexpr int XL = 16 / TB;      // slab rows (direct loads) per wave and quad
  constexpr int WL = BITS + 2;     // weight loads per lane and quad
  const int K = 128 * G;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform: scalar descriptors
  const int nl = lane & 15;  // weight row / activation row / result column
  const int j = lane >> 4;   // load: group of the quad; compute: chunk of the group
  const int nq = (G + 3) >> 2;
  const uint32_t r0u = ((uint32_t)block * TB + (uint32_t)wave) * 16u;  // 32-bit: see mfma_block
  const int64_t row0 = (int64_t)r0u;
  const int rows = r0u < (uint32_t)N ? (int)min(16u, (uint32_t)N - r0u) : 0;

  const __amdgpu_buffer_rsrc_t xr = rsrc(x, (uint32_t)M * K * 2);
  const __amdgpu_buffer_rsrc_t qr = rsrc(qw + row0 * BITS * 4 * G, (uint32_t)rows * BITS * G * 16);  // 16 B per plane-group
  const __amdgpu_buffer_rsrc_t sr = rsrc(scales + row0 * G, (uint32_t)rows * G * 2);
  const __amdgpu_buffer_rsrc_t zr = rsrc(zeros + row0 * G, (uint32_t)rows * G);

  // Slab of quad qq into buffer qq % 3: wave w fetches rows w, w + TB, ...;
  // rows m >= M, columns past K and quads past the last read zeros.
  auto fetch_slab = [&](int qq) {
    typedef __attribute__((address_space(3))) void lds_void;
    const int buf = qq % kSlabBuffers;
#pragma unroll
    for (int i = 0; i < XL; ++i) {
      const int m = wave + i * TB;
      const int piece = lane ^ (m & 7);
      const int col = 512 * qq + 8 * piece;
      const uint32_t dead = (uint32_t)!(m < M && qq < nq && col < K) << 31;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void*)(slab + (buf * 16 + m) * 64), 16,
                                               (uint32_t)(m * K + col) * 2 | dead, 0, 0, 0);
    }
  };

  float4_t yacc = float4_t{0.f, 0.f, 0.f, 0.f};
  // Quad q's products from its weights and slab buffer q % 3.
  auto compute = [&](const QuadWeights<BITS>& cur, int q) {
    // Quarter transposes: chunk j of group 4q + gi in component gi.
    uint32_t wt[BITS][4];
#pragma unroll
    for (int p = 0; p < BITS; ++p) {
      wt[p][0] = cur.w[p][0];
      wt[p][1] = cur.w[p][1];
      wt[p][2] = cur.w[p][2];
      wt[p][3] = cur.w[p][3];
      transpose_quarters(wt[p][0], wt[p][1], wt[p][2], wt[p][3]);
    }
    uint32_t szj[4];
    szj[0] = szj[1] = szj[2] = szj[3] = cur.s | (cur.z << 16);
    transpose_quarters(szj[0], szj[1], szj[2], szj[3]);

    const u32x4* sl = slab + ((q % kSlabBuffers) * 16 + nl) * 64;
    const int swz = nl & 7;
#pragma unroll
    for (int gi = 0; gi < 4; ++gi) {
      uint32_t w[BITS];
#pragma unroll
      for (int p = 0; p < BITS; ++p) w[p] = wt[p][gi];
      uint32_t pr[16];
      unpack_chunk_exact<BITS>(w, szj[gi] >> 16, pr);
      float4_t c = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const half8_t a = __builtin_bit_cast(half8_t, sl[(16 * gi + 4 * j + jj) ^ swz]);
        const half8_t b = frag(pr[4 * jj + 0], pr[4 * jj + 1], pr[4 * jj + 2], pr[4 * jj + 3]);
        c = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
      }
      const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)(szj[gi] & 0xFFFFu));
      yacc += s * c;
    }
  };
  // One quad of the walk: request quad q + 2's slab and weights (into the
  // register set quad q - 1 used; loads past the last quad read zeros, and
  // the slab buffer written was last read in quad q - 1), compute quad q,
  // then wait until only quad q + 2's loads are outstanding, which completes
  // quad q + 1's, and publish its slab with the barrier.
  auto step = [&](int q, const QuadWeights<BITS>& cur, QuadWeights<BITS>& ahead) {
    fetch_slab(q + 2);
    ahead = load_quad<BITS, kWeightPolicy>(qr, sr, zr, nl, j, q + 2, G, q + 2 < nq);
    __builtin_amdgcn_sched_barrier(0);
    compute(cur, q);
    __builtin_amdgcn_sched_barrier(0);
    wait_vmcnt<XL + WL>();
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
  };

  // Three register sets of quad weights in turn, so that no load waits for
  // a register copy: the loop is unrolled by three.  Issue order X0, W0,
  // X1, W1: waiting until only X1 and W1 are outstanding completes X0 (this
  // wave's part of the slab) and W0.
  QuadWeights<BITS> wa, wb, wc;
  fetch_slab(0);
  wa = load_quad<BITS, kWeightPolicy>(qr, sr, zr, nl, j, 0, G, true);
  __builtin_amdgcn_sched_barrier(0);
  fetch_slab(1);
  wb = load_quad<BITS, kWeightPolicy>(qr, sr, zr, nl, j, 1, G, 1 < nq);
  __builtin_amdgcn_sched_barrier(0);
  wait_vmcnt<XL + WL>();
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  int q = 0;
  for (; q + 3 <= nq; q += 3) {
    step(q, wa, wc);
    step(q + 1, wb, wa);
    step(q + 2, wc, wb);
  }
  // The last one or two quads: their loads are in flight already.
  if (q < nq) {
    compute(wa, q);
    if (q + 1 < nq) {
      __builtin_amdgcn_sched_barrier(0);
      wait_vmcnt<0>();
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      compute(wb, q + 1);
    }
  }

  // Lane (n, j) holds rows m = 4j .. 4j+3 of column n.
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int m = 4 * j + r;
    if (m < M && nl < rows) y[(int64_t)m * N + row0 + nl] = __builtin_bit_cast(uint16_t, (_Float16)yacc[r]);
  }
}

template <int BITS, int TB>
__global__ __launch_bounds__(64 * TB) void linear_mfma_tiles_kernel(
    const uint16_t* __restrict__ x, const uint32_t* __restrict__ qw, const uint16_t* __restrict__ scales,
    const uint8_t* __restrict__ zeros, uint16_t* __restrict__ y, int M, int N, int G, int nblocks) {
  const int block = xcd_block(nblocks);
  if (block >= nblocks) return;  // idle slot of the XCD-rounded grid (the whole block leaves)
  mfma_tiles_block<BITS, TB>(x, qw, scales, zeros, y, M, N, G, block);
}

// ---------------------------------------------------------------------------
// The K ranges of split K (rows of many quads, fewer than 1024 tiles).  A
// block of four waves owns four 16-row tiles, one per wave, over a range of
// NQ quads, and keeps the activation slabs of all its NQ quads (each slab once
// per block, x[0..M-1][512q .. 512q+511] into LDS by direct-to-LDS loads, four
// rows per wave; rows past M read zeros) and the wave's weights of all NQ
// quads (registers).  Quad q + 1 is requested before quad q is computed, so
// its loads land during that compute; requesting everything first kept each
// wave in the issue of its last loads, with nothing to compute, for most of
// the time the data took to arrive.
// ---------------------------------------------------------------------------
constexpr int kFullTiles = 4;
constexpr int kFullAhead = 1;  // quads requested ahead of the one computed (1 measured best; 2, 3 slower)

// Quads q0 .. q0+NQ-1 (those past the row read zeros).  part == nullptr: the
// result goes to y as fp16; otherwise the fp32 partial sums go to
// part[m][n] (split K).
template <int BITS, int NQ>
__device__ __forceinline__ void mfma_full_block(
    const uint16_t* __restrict__ x, const uint32_t* __restrict__ qw, const uint16_t* __restrict__ scales,
    const uint8_t* __restrict__ zeros, uint16_t* __restrict__ y, int M, int N, int G, int block, int q0,
    float* __restrict__ part) {
  typedef __attribute__((address_space(3))) void lds_void;
  extern __shared__ u32x4 slab[];  // [NQ][16 rows][64 pieces]
  const int K = 128 * G;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform: scalar descriptors
  const int nl = lane & 15;  // weight row / activation row / result column
  const int j = lane >> 4;   // load: group of the quad; compute: chunk of the group
  const uint32_t r0u = ((uint32_t)block * kFullTiles + (uint32_t)wave) * 16u;  // 32-bit: see mfma_block
  const int64_t row0 = (int64_t)r0u;
  const int rows = r0u < (uint32_t)N ? (int)min(16u, (uint32_t)N - r0u) : 0;

  const __amdgpu_buffer_rsrc_t xr = rsrc(x, (uint32_t)M * K * 2);
  const __amdgpu_buffer_rsrc_t qr = rsrc(qw + row0 * BITS * 4 * G, (uint32_t)rows * BITS * G * 16);
  const __amdgpu_buffer_rsrc_t sr = rsrc(scales + row0 * G, (uint32_t)rows * G * 2);
  const __amdgpu_buffer_rsrc_t zr = rsrc(zeros + row0 * G, (uint32_t)rows * G);

  // 1. Loads, quad by quad: the wave's four slab rows (wave, wave + 4,
  //    wave + 8, wave + 12; rows >= M, columns past K and groups past G read
  //    zeros), then its weights of the quad: XL + WL loads per quad, issued in
  //    this order (scheduling barriers), so that a wait for quad q can leave
  //    the later quads' loads in flight.  Quads are requested kFullAhead ahead
  //    of the one computed: a wave that requested everything first would sit
  //    in the issue of its last loads (the vector-memory pipe is the slow
  //    part) before it could start computing.
  constexpr int XL = 16 / kFullTiles;
  constexpr int WL = BITS + 2;
  constexpr int D = NQ < kFullAhead ? NQ : kFullAhead;
  static_assert(D * (XL + WL) <= 63, "outstanding loads exceed the vmcnt range");
  QuadWeights<BITS> wq[NQ];
  auto issue = [&](auto qc) {
    constexpr int q = decltype(qc)::value;
#pragma unroll
    for (int i = 0; i < XL; ++i) {
      const int m = wave + i * kFullTiles;
      const int col = 512 * (q0 + q) + 8 * (lane ^ (m & 7));
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void*)(slab + (q * 16 + m) * 64), 16,
                                               (uint32_t)(m * K + col) * 2 | (uint32_t)!(m < M && col < K) << 31,
                                               0, 0, 0);
    }
    wq[q] = load_quad<BITS, kWeightPolicyNT>(qr, sr, zr, nl, j, q0 + q, G, true);
    __builtin_amdgcn_sched_barrier(0);
  };
  static_for<D>(issue);
  asm volatile("" : "+s"(part));  // an argument past the preloaded ones: read it now, not at the end

  // 2. Quad by quad: wait until only the later quads' loads are outstanding,
  //    a bare barrier (the other waves' slab rows; a __syncthreads() fence
  //    would wait for every load in flight), request quad q + D, compute.
  float4_t yacc = float4_t{0.f, 0.f, 0.f, 0.f};
  const int swz = nl & 7;
  static_for<NQ>([&](auto qc) {
    constexpr int q = decltype(qc)::value;
    constexpr int issued = q + D < NQ ? q + D : NQ;  // quads requested so far
    wait_vmcnt<(issued - q - 1) * (XL + WL)>();
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (q + D < NQ) issue(std::integral_constant<int, q + D>{});
    // Quarter transposes: chunk j of group 4q + gi in component gi.
    uint32_t wt[BITS][4];
#pragma unroll
    for (int p = 0; p < BITS; ++p) {
      wt[p][0] = wq[q].w[p][0];
      wt[p][1] = wq[q].w[p][1];
      wt[p][2] = wq[q].w[p][2];
      wt[p][3] = wq[q].w[p][3];
      transpose_quarters(wt[p][0], wt[p][1], wt[p][2], wt[p][3]);
    }
    uint32_t szj[4];
    szj[0] = szj[1] = szj[2] = szj[3] = wq[q].s | (wq[q].z << 16);
    transpose_quarters(szj[0], szj[1], szj[2], szj[3]);

    const uint32_t sa = lds_addr(slab + (q * 16 + nl) * 64);
#pragma unroll
    for (int gi = 0; gi < 4; ++gi) {
      u32x4 fr[4];
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) fr[jj] = lds_read_b128(sa + 16 * ((16 * gi + 4 * j + jj) ^ swz));
      uint32_t w[BITS];
#pragma unroll
      for (int p = 0; p < BITS; ++p) w[p] = wt[p][gi];
      uint32_t pr[16];
      unpack_chunk_exact<BITS>(w, szj[gi] >> 16, pr);
      lds_wait(fr);
      float4_t c = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const half8_t b = frag(pr[4 * jj + 0], pr[4 * jj + 1], pr[4 * jj + 2], pr[4 * jj + 3]);
        c = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8_t, fr[jj]), b, c, 0, 0, 0);
      }
      const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)(szj[gi] & 0xFFFFu));
      yacc += s * c;
    }
  });

  // 3. Lane (n, j) holds rows m = 4j .. 4j+3 of column n.
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int m = 4 * j + r;
    if (m < M && nl < rows) {
      if (part) part[(int64_t)m * N + row0 + nl] = yacc[r];
      else y[(int64_t)m * N + row0 + nl] = __builtin_bit_cast(uint16_t, (_Float16)yacc[r]);
    }
  }
}

// Split K: logical block b = s * tile_blocks + t takes tile block t over the
// quads s * NQ .. s * NQ + NQ - 1 and writes its partial sums to part[s][M][N]
// (consecutive blocks share a K range, i.e. the activation columns, in L2).
template <int BITS, int NQ>
__global__ __launch_bounds__(64 * kFullTiles) void linear_mfma_split_kernel(
    const uint16_t* __restrict__ x, const uint32_t* __restrict__ qw, const uint16_t* __restrict__ scales,
    const uint8_t* __restrict__ zeros, int M, int N, int G, int tile_blocks, int nblocks,
    float* __restrict__ part) {
  const int b = xcd_block(nblocks);
  if (b >= nblocks) return;  // idle slot of the XCD-rounded grid (the whole block leaves)
  const int sidx = b / tile_blocks;
  mfma_full_block<BITS, NQ>(x, qw, scales, zeros, nullptr, M, N, G, b - sidx * tile_blocks, sidx * NQ,
                            part + (int64_t)sidx * M * N);
}

// y[i] = fp16 of the sum of the S partials part[s][i], s = 0 .. S-1 in order.
// Each thread owns four consecutive outputs (16-byte partial loads when
// M*N is a multiple of 4) and requests eight partials at a time before adding
// them in order, so the loads of a thread overlap.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part,
                                                            uint16_t* __restrict__ y, int S, int64_t MN) {
  const int64_t i0 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (i0 >= MN) return;
  float4_t acc;
  if ((MN & 3) == 0) {
    const float4_t* p4 = reinterpret_cast<const float4_t*>(part) + (i0 >> 2);
    const int64_t stride = MN >> 2;
    acc = p4[0];
    int s = 1;
    for (; s + 8 <= S; s += 8) {
      float4_t v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = p4[(int64_t)(s + k) * stride];
#pragma unroll
      for (int k = 0; k < 8; ++k) acc += v[k];
    }
    for (; s < S; ++s) acc += p4[(int64_t)s * stride];
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] = i0 + e < MN ? part[i0 + e] : 0.0f;
    for (int s = 1; s < S; ++s) {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (i0 + e < MN) acc[e] += part[(int64_t)s * MN + i0 + e];
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e)
    if (i0 + e < MN) y[i0 + e] = __builtin_bit_cast(uint16_t, (_Float16)acc[e]);
}

template <int BITS, int TW>
__global__ __launch_bounds__(1024 / TW) void linear_mfma_kernel(
    const uint16_t* __restrict__ x, const uint32_t* __restrict__ qw, const uint16_t* __restrict__ scales,
    const uint8_t* __restrict__ zeros, uint16_t* __restrict__ y, int M, int N, int G, int nblocks) {
  const int block = xcd_block(nblocks);
  if (block >= nblocks) return;  // idle slot of the XCD-rounded grid
  mfma_block<BITS, TW>(x, qw, scales, zeros, y, M, N, G, block, mfma_block_waves(M, (G + 3) >> 2));
}

// Several independent calls in one launch (one 16-row tile per block); the
// call of block b is picked with constant indices, as in the flat kernel.
template <int BITS>
__global__ __launch_bounds__(1024) void linear_mfma_group_kernel(const LinearGroup grp, int M) {
  const int b = xcd_block(grp.blocks);
  if (b >= grp.blocks) return;  // idle slot of the XCD-rounded grid
  LinearCall c = grp.call[0];
#pragma unroll
  for (int j = 1; j < kMaxGroup; ++j)
    if (j < grp.count && b >= grp.call[j].first_block) c = grp.call[j];
  mfma_block<BITS, 1>(c.x, c.qw, c.scales, c.zeros, c.y, M, c.N, c.G, b - c.first_block, grp.waves);
}

// ---------------------------------------------------------------------------
// One 16-row tile per block and one wave per quad (512 columns) of the row,
// for rows of at most kQuadWaveMax quads whose activations fit in LDS.  Every
// wave issues all its loads at once: its quad's activations
// x[0..MT-1][512q, 512q+512) into its own LDS slab (direct-to-LDS; rows past M
// and columns past K read zeros; no other wave reads it, so no barrier), then
// the quad's weights (one register set).  It reads its sixteen A fragments
// (4 groups x 4 MFMAs) from the slab as soon as the slab has arrived, then
// multiplies by the weights, scales per group and writes its four
// accumulators over its slab.  After one barrier the waves' partials are
// added in wave order and rounded.  Compared with waves that each walk
// several quads, every load of the tile is in flight at once and every wave
// pays one memory round trip.
// ---------------------------------------------------------------------------
constexpr int kQuadWaveMax = 10;  // quads per row (waves per block) the kernel takes
constexpr int kQuadWaveResident = 256 * 20;  // waves resident at the up-front form's 5 per SIMD

// ds_read_b128 at a register address plus a compile-time byte offset (inline
// assembly for the reason given at lds_read_b128).
template <int OFF>
__device__ __forceinline__ u32x4 lds_read_b128_off(uint32_t addr) {
  u32x4 r;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
  return r;
}

template <int BITS, int MT, bool LOWREG>
__global__ __launch_bounds__(64 * kQuadWaveMax) __attribute__((amdgpu_waves_per_eu(LOWREG ? 8 : 1))) void
linear_mfma_quad_wave_kernel(
    const uint16_t* __restrict__ x, const uint32_t* __restrict__ qw, const uint16_t* __restrict__ scales,
    const uint8_t* __restrict__ zeros, uint16_t* __restrict__ y, int M, int N, int G, int nblocks) {
  static_assert(MT == 4 || MT == 8 || MT == 16, "slab rows");
  typedef __attribute__((address_space(3))) void lds_void;
  extern __shared__ u32x4 wslab[];  // [W][MT rows][64 pieces]; afterwards [W][4][64] fp32 partials
  constexpr int WL = BITS + 2;      // weight loads per lane
  const int b = xcd_block(nblocks);
  if (b >= nblocks) return;  // idle slot of the XCD-rounded grid (the whole block leaves)
  const int K = 128 * G;
  const int W = (G + 3) >> 2;  // one wave per quad (the block size)
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // this wave's quad
  const int nl = lane & 15;  // weight row / activation row / result column
  const int j = lane >> 4;   // load: group of the quad; compute: chunk of the group
  const uint32_t r0u = (uint32_t)b * 16u;  // 32-bit: see mfma_block
  const int64_t row0 = (int64_t)r0u;
  const int rows = r0u < (uint32_t)N ? (int)min(16u, (uint32_t)N - r0u) : 0;
  u32x4* const sl = wslab + wave * (MT * 64);

  const __amdgpu_buffer_rsrc_t xr = rsrc(x, (uint32_t)M * K * 2);
  const __amdgpu_buffer_rsrc_t qr = rsrc(qw + row0 * BITS * 4 * G, (uint32_t)rows * BITS * G * 16);
  const __amdgpu_buffer_rsrc_t sr = rsrc(scales + row0 * G, (uint32_t)rows * G * 2);
  const __amdgpu_buffer_rsrc_t zr = rsrc(zeros + row0 * G, (uint32_t)rows * G);

  // 1. The slab (MT direct loads), then the weights.  The waits below count
  //    outstanding loads in this issue order (scheduling barriers).
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    const int col = 512 * wave + 8 * (lane ^ (m & 7));
    __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void*)(sl + m * 64), 16,
                                             (uint32_t)(m * K + col) * 2 | (uint32_t)!(m < M && col < K) << 31, 0,
                                             0, 0);
  }
  __builtin_amdgcn_sched_barrier(0);
  const QuadWeights<BITS> qwt = load_quad<BITS, kWeightPolicy>(qr, sr, zr, nl, j, wave, G, true);
  __builtin_amdgcn_sched_barrier(0);

  // 2. The A fragments: group gi, MFMA jj reads piece 16 gi + 4 j + jj of the
  //    lane's activation row (stored at position piece ^ (row & 7)).
  wait_vmcnt<WL>();
  __builtin_amdgcn_sched_barrier(0);
  const int arow = nl & (MT - 1);
  const uint32_t abase = lds_addr(sl + arow * 64);
  const int swz = arow & 7;
  uint32_t aoff[4];
#pragma unroll
  for (int jj = 0; jj < 4; ++jj) aoff[jj] = abase + 16 * ((4 * j + jj) ^ swz);
  //    Read up front (64 registers) unless LOWREG, which reads each group's
  //    four fragments just before its MFMAs so the kernel fits in 64 VGPRs
  //    (8 waves per SIMD instead of 5).
  u32x4 af[4][4];
  if constexpr (!LOWREG) {
    static_for<4>([&](auto gc) {
      constexpr int gi = decltype(gc)::value;
      static_for<4>([&](auto jc) {
        constexpr int jj = decltype(jc)::value;
        af[gi][jj] = lds_read_b128_off<256 * gi>(aoff[jj]);
      });
    });
#pragma unroll
    for (int gi = 0; gi < 4; ++gi) lds_wait(af[gi]);
  }

  // 3. Quarter transposes (chunk j of group 4q + gi in component gi), exact
  //    (q - z) pairs, four MFMAs per group, scale.
  wait_vmcnt<0>();
  __builtin_amdgcn_sched_barrier(0);
  uint32_t wt[BITS][4];
#pragma unroll
  for (int p = 0; p < BITS; ++p) {
    wt[p][0] = qwt.w[p][0];
    wt[p][1] = qwt.w[p][1];
    wt[p][2] = qwt.w[p][2];
    wt[p][3] = qwt.w[p][3];
    transpose_quarters(wt[p][0], wt[p][1], wt[p][2], wt[p][3]);
  }
  uint32_t szj[4];
  szj[0] = szj[1] = szj[2] = szj[3] = qwt.s | (qwt.z << 16);
  transpose_quarters(szj[0], szj[1], szj[2], szj[3]);
  float4_t yacc = float4_t{0.f, 0.f, 0.f, 0.f};
  static_for<4>([&](auto gc) {
    constexpr int gi = decltype(gc)::value;
    if constexpr (LOWREG) {
      static_for<4>([&](auto jc) {
        constexpr int jj = decltype(jc)::value;
        af[gi][jj] = lds_read_b128_off<256 * gi>(aoff[jj]);
      });
    }
    uint32_t w[BITS];
#pragma unroll
    for (int p = 0; p < BITS; ++p) w[p] = wt[p][gi];
    uint32_t pr[16];
    unpack_chunk_exact<BITS>(w, szj[gi] >> 16, pr);
    if constexpr (LOWREG) lds_wait(af[gi]);
    float4_t c = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const half8_t bf = frag(pr[4 * jj + 0], pr[4 * jj + 1], pr[4 * jj + 2], pr[4 * jj + 3]);
      c = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8_t, af[gi][jj]), bf, c, 0, 0, 0);
    }
    const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)(szj[gi] & 0xFFFFu));
    yacc += s * c;
  });
  float* part = reinterpret_cast<float*>(sl);  // [4][64], over the slab just read
#pragma unroll
  for (int r = 0; r < 4; ++r) part[r * 64 + lane] = yacc[r];
  __syncthreads();

  // 4. Outputs (row n, activation row m): the W waves' partials in order.
  //    Lane (n, j) of a wave held rows m = 4j .. 4j+3 of column n.
  const float* red = reinterpret_cast<const float*>(wslab);
  const int wstride = MT * 64 * 4;  // floats per wave region
  for (int idx = threadIdx.x; idx < 256; idx += 64 * W) {
    const int r = idx >> 6;
    const int ln = idx & 63;
    float v = 0.0f;
    for (int w = 0; w < W; ++w) v += red[w * wstride + r * 64 + ln];
    const int m = 4 * (ln >> 4) + r;
    const int n = ln & 15;
    if (m < M && n < rows) y[(int64_t)m * N + row0 + n] = __builtin_bit_cast(uint16_t, (_Float16)v);
  }
}

// ---------------------------------------------------------------------------
// Many row tiles, rows of at most five quads, more than four activation rows:
// one wave per (tile, quad) as in the kernel above, with TPB tiles per block
// sharing the quads' activation slabs, so that a slab of 8 or 16 rows (8 or
// 16 KiB per quad) serves TPB waves and two blocks of 3 x 5 waves fit on a
// compute unit at 64 registers: every wave of the grid is resident and issues
// all its loads at once.  The waves of tile 0 bring slab q into LDS, one
// barrier publishes the slabs, every wave then reads its fragments group by
// group; a second barrier frees the slabs for the waves' partials, a third
// publishes them, and each tile's quads are added in order.  (Measured on
// MI355X: Qwen3-4B gate|up, 1216 tiles of 5 quads, M = 16 12.4 -> 11.2 us,
// M = 8 10.5 -> 10.0 us; at M <= 4 one tile per block stays faster, and two
// tiles per block left M = 16 at 12.8 us.)
// ---------------------------------------------------------------------------
template <int BITS, int MT, int TPB>
__global__ __launch_bounds__(1024) __attribute__((amdgpu_waves_per_eu(8))) void linear_mfma_quad_share_kernel(
    const uint16_t* __restrict__ x, const uint32_t* __restrict__ qw, const uint16_t* __restrict__ scales,
    const uint8_t* __restrict__ zeros, uint16_t* __restrict__ y, int M, int N, int G, int nblocks) {
  typedef __attribute__((address_space(3))) void lds_void;
  extern __shared__ u32x4 wslab[];  // [nq][MT rows][64 pieces]; afterwards [TPB * nq][4][64] fp32 partials
  constexpr int WL = BITS + 2;
  const int b = xcd_block(nblocks);
  if (b >= nblocks) return;  // idle slot of the XCD-rounded grid (the whole block leaves)
  const int K = 128 * G;
  const int nq = (G + 3) / 4;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int t = __builtin_amdgcn_readfirstlane(w / nq);  // tile of the block
  const int q = w - t * nq;                              // quad of the row
  const int nl = lane & 15;
  const int j = lane >> 4;
  const uint32_t r0u = ((uint32_t)b * TPB + (uint32_t)t) * 16u;  // 32-bit: see mfma_block
  const int64_t row0 = (int64_t)r0u;
  const int rows = r0u < (uint32_t)N ? (int)min(16u, (uint32_t)N - r0u) : 0;
  u32x4* const sl = wslab + q * (MT * 64);

  const __amdgpu_buffer_rsrc_t xr = rsrc(x, (uint32_t)M * K * 2);
  const __amdgpu_buffer_rsrc_t qr = rsrc(qw + row0 * BITS * 4 * G, (uint32_t)rows * BITS * G * 16);
  const __amdgpu_buffer_rsrc_t sr = rsrc(scales + row0 * G, (uint32_t)rows * G * 2);
  const __amdgpu_buffer_rsrc_t zr = rsrc(zeros + row0 * G, (uint32_t)rows * G);

  // 1. Tile 0's waves: the quad's slab (MT direct loads); then every wave its weights.
  if (t == 0) {
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const int col = 512 * q + 8 * (lane ^ (m & 7));
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void*)(sl + m * 64), 16,
                                               (uint32_t)(m * K + col) * 2 | (uint32_t)!(m < M && col < K) << 31, 0,
                                               0, 0);
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  const QuadWeights<BITS> qwt = load_quad<BITS, kWeightPolicy>(qr, sr, zr, nl, j, q, G, true);
  __builtin_amdgcn_sched_barrier(0);
  wait_vmcnt<WL>();  // tile 0: its slab (issued before the weights) has landed; others: nothing to wait for
  __builtin_amdgcn_sched_barrier(0);
  __syncthreads();               // every slab published

  const int arow = nl & (MT - 1);
  const uint32_t abase = lds_addr(sl + arow * 64);
  const int swz = arow & 7;
  uint32_t aoff[4];
#pragma unroll
  for (int jj = 0; jj < 4; ++jj) aoff[jj] = abase + 16 * ((4 * j + jj) ^ swz);

  // 2. Quarter transposes, exact (q - z) pairs, four MFMAs per group (each
  //    group's fragments read just before its MFMAs), scale.
  wait_vmcnt<0>();
  __builtin_amdgcn_sched_barrier(0);
  uint32_t wt[BITS][4];
#pragma unroll
  for (int p = 0; p < BITS; ++p) {
    wt[p][0] = qwt.w[p][0];
    wt[p][1] = qwt.w[p][1];
    wt[p][2] = qwt.w[p][2];
    wt[p][3] = qwt.w[p][3];
    transpose_quarters(wt[p][0], wt[p][1], wt[p][2], wt[p][3]);
  }
  uint32_t szj[4];
  szj[0] = szj[1] = szj[2] = szj[3] = qwt.s | (qwt.z << 16);
  transpose_quarters(szj[0], szj[1], szj[2], szj[3]);
  float4_t yacc = float4_t{0.f, 0.f, 0.f, 0.f};
  u32x4 af[4][4];
  static_for<4>([&](auto gc) {
    constexpr int gi = decltype(gc)::value;
    static_for<4>([&](auto jc) {
      constexpr int jj = decltype(jc)::value;
      af[gi][jj] = lds_read_b128_off<256 * gi>(aoff[jj]);
    });
    uint32_t wq[BITS];
#pragma unroll
    for (int p = 0; p < BITS; ++p) wq[p] = wt[p][gi];
    uint32_t pr[16];
    unpack_chunk_exact<BITS>(wq, szj[gi] >> 16, pr);
    lds_wait(af[gi]);
    float4_t c = float4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const half8_t bf = frag(pr[4 * jj + 0], pr[4 * jj + 1], pr[4 * jj + 2], pr[4 * jj + 3]);
      c = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8_t, af[gi][jj]), bf, c, 0, 0, 0);
    }
    const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)(szj[gi] & 0xFFFFu));
    yacc += s * c;
  });
  __syncthreads();  // every wave's fragment reads are done: the slabs are free
  float* part = reinterpret_cast<float*>(wslab) + w * 256;  // [4][64]
#pragma unroll
  for (int r = 0; r < 4; ++r) part[r * 64 + lane] = yacc[r];
  __syncthreads();

  // 3. Outputs of each tile: its nq waves' partials in quad order.
  const float* red = reinterpret_cast<const float*>(wslab);
  for (int idx = threadIdx.x; idx < 256 * TPB; idx += 64 * TPB * nq) {
    const int tt = idx >> 8;
    const int r = (idx >> 6) & 3;
    const int ln = idx & 63;
    float v = 0.0f;
    for (int qq = 0; qq < nq; ++qq) v += red[(tt * nq + qq) * 256 + r * 64 + ln];
    const int m = 4 * (ln >> 4) + r;
    const int n = ln & 15;
    const int64_t r0 = ((int64_t)b * TPB + tt) * 16;
    if (m < M && r0 + n < N) y[(int64_t)m * N + r0 + n] = __builtin_bit_cast(uint16_t, (_Float16)v);
  }
}

}  // namespace

SplitPlan mfma_split_plan(int M, int64_t N, int G) {
  SplitPlan p;
  const int64_t tiles = (N + 15) / 16;
  const int nq = (G + 3) / 4;
  if (M < 2 || tiles >= kMfmaShareMinTiles || nq < kSplitMinQuads) return p;
  // Blocks of four tiles over K ranges of qs quads: the longest ranges (the
  // fewest partial sums) that still give every compute unit a block.
  const int64_t tile_blocks = (tiles + kFullTiles - 1) / kFullTiles;
  const int64_t smin = (256 + tile_blocks - 1) / tile_blocks;
  p.qs = (int)min((int64_t)5, max((int64_t)1, (int64_t)nq / smin));
  p.S = (nq + p.qs - 1) / p.qs;
  p.tile_blocks = (int)tile_blocks;
  return p;
}

template <int BITS>
hipError_t launch_linear_mfma(const uint16_t* x, const uint32_t* qweight, const uint16_t* scales,
                              const uint8_t* zeros, uint16_t* y, int M, int64_t N, int64_t K,
                              hipStream_t stream, const LaunchEvents& ev, float* workspace,
                              size_t workspace_bytes) {
  const int G = (int)(K / 128);
  const int nq = (G + 3) / 4;
  const int64_t tiles = (N + 15) / 16;
  // Many tiles, rows of at most five quads, M > 4 (W4: M > 8; at M <= 8 the
  // one-tile blocks below are faster for W4): three tiles per block share
  // the quads' slabs, one wave per (tile, quad).
  if (tiles >= kMfmaShareMinTiles && nq <= 5 && M > (BITS == 4 ? 8 : 4)) {
    constexpr int TPB = 3;
    const int nblocks = (int)((tiles + TPB - 1) / TPB);
    const dim3 grid(xcd_grid(nblocks)), blk(64 * TPB * nq);
    if (M > 8)
      launch(linear_mfma_quad_share_kernel<BITS, 16, TPB>, grid, blk, (uint32_t)nq * 16 * 1024, stream, ev, x,
             qweight, scales, zeros, y, M, (int)N, G, nblocks);
    else
      launch(linear_mfma_quad_share_kernel<BITS, 8, TPB>, grid, blk, (uint32_t)nq * 8 * 1024, stream, ev, x,
             qweight, scales, zeros, y, M, (int)N, G, nblocks);
    return hipGetLastError();
  }
  // Rows of at most kQuadWaveMax quads whose activation slabs fit in LDS: one
  // tile per block, one wave per quad (measured on MI355X against the kernels
  // below: faster for every Qwen3-4B projection from M = 3 that the sharing
  // kernel above does not take).
  {
    const int MT = M <= 4 ? 4 : M <= 8 ? 8 : 16;
    const size_t lds = (size_t)nq * MT * 1024;
    if (nq <= kQuadWaveMax && lds <= (size_t)kBlockLdsU4 * 16 && (tiles < kMfmaShareMinTiles || M <= 8)) {
      const int nblocks = (int)tiles;
      const dim3 grid(xcd_grid(nblocks)), blk(64 * nq);
      // More waves than stay resident at 5 per SIMD (the up-front fragments'
      // register count): the 64-register form, 8 per SIMD (measured on
      // MI355X: Qwen3-4B gate|up at M = 4, 1216 tiles x 5 waves, 10.8 -> 8.6 us;
      // the smaller projections are 1-2 % faster with the fragments up front).
      const bool lowreg = tiles * nq > (int64_t)kQuadWaveResident;
#define LAQ_QW(MTV)                                                                                               \
  do {                                                                                                            \
    if (lowreg)                                                                                                   \
      launch(linear_mfma_quad_wave_kernel<BITS, MTV, true>, grid, blk, (uint32_t)lds, stream, ev, x, qweight,     \
             scales, zeros, y, M, (int)N, G, nblocks);                                                            \
    else                                                                                                          \
      launch(linear_mfma_quad_wave_kernel<BITS, MTV, false>, grid, blk, (uint32_t)lds, stream, ev, x, qweight,    \
             scales, zeros, y, M, (int)N, G, nblocks);                                                            \
  } while (0)
      if (MT == 4) LAQ_QW(4);
      else if (MT == 8) LAQ_QW(8);
      else LAQ_QW(16);
#undef LAQ_QW
      return hipGetLastError();
    }
  }
  // Many tiles, longer rows: blocks of four or eight tiles walking K share
  // each activation slab through LDS.
  if (tiles >= kMfmaShareMinTiles) {
    const int tb = tiles >= 3072 ? 8 : 4;
    const int nblocks = (int)((tiles + tb - 1) / tb);
    if (tb == 8)
      launch(linear_mfma_tiles_kernel<BITS, 8>, dim3(xcd_grid(nblocks)), dim3(512), kSlabLdsBytes, stream, ev, x,
             qweight, scales, zeros, y, M, (int)N, G, nblocks);
    else
      launch(linear_mfma_tiles_kernel<BITS, 4>, dim3(xcd_grid(nblocks)), dim3(256), kSlabLdsBytes, stream, ev, x,
             qweight, scales, zeros, y, M, (int)N, G, nblocks);
    return hipGetLastError();
  }
  // Fewer tiles, long rows, a workspace: split K over blocks of four tiles
  // that request their whole K range at once; a second kernel adds the
  // ranges' partial sums in order.
  const SplitPlan sp = mfma_split_plan(M, N, G);
  if (sp.S > 1 && workspace && workspace_bytes >= split_workspace_bytes(sp, M, N)) {
    const int nblocks = sp.tile_blocks * sp.S;
    LaunchEvents e1, e2;  // the measurement hook spans both kernels
    e1.start = ev.start;
    e2.stop = ev.stop;
    const dim3 grid(xcd_grid(nblocks)), blk(64 * kFullTiles);
    const uint32_t lds = (uint32_t)sp.qs * kSlabBytes;
    switch (sp.qs) {
      case 1: launch(linear_mfma_split_kernel<BITS, 1>, grid, blk, lds, stream, e1, x, qweight, scales, zeros, M, (int)N, G, sp.tile_blocks, nblocks, workspace); break;
      case 2: launch(linear_mfma_split_kernel<BITS, 2>, grid, blk, lds, stream, e1, x, qweight, scales, zeros, M, (int)N, G, sp.tile_blocks, nblocks, workspace); break;
      case 3: launch(linear_mfma_split_kernel<BITS, 3>, grid, blk, lds, stream, e1, x, qweight, scales, zeros, M, (int)N, G, sp.tile_blocks, nblocks, workspace); break;
      case 4: launch(linear_mfma_split_kernel<BITS, 4>, grid, blk, lds, stream, e1, x, qweight, scales, zeros, M, (int)N, G, sp.tile_blocks, nblocks, workspace); break;
      default: launch(linear_mfma_split_kernel<BITS, 5>, grid, blk, lds, stream, e1, x, qweight, scales, zeros, M, (int)N, G, sp.tile_blocks, nblocks, workspace); break;
    }
    const int64_t MN = (int64_t)M * N;
    launch(splitk_reduce_kernel, dim3((unsigned)((MN + 1023) / 1024)), dim3(256), 0, stream, e2,
           (const float*)workspace, y, sp.S, MN);
    return hipGetLastError();
  }
  // Two tiles per block share each activation fragment when rows are long
  // (the fragments then outweigh the weights) and there are enough tiles to
  // keep a block on every compute unit (measured on MI355X).  (At most M
  // tiles per wave: a wave's TW KiB of partials reuse its M KiB slab.)
  const int TW = min(M, (tiles >= 256 && G >= 32) ? 2 : 1);
  const int W = mfma_block_waves(M, nq);
  const int nblocks = (int)((tiles + TW - 1) / TW);
  const unsigned blocks = xcd_grid(nblocks);
  const uint32_t lds = (uint32_t)W * M * kSlabRowU4 * 16;
  if (TW == 2)
    launch(linear_mfma_kernel<BITS, 2>, dim3(blocks), dim3(64 * W), lds, stream, ev, x, qweight, scales, zeros, y, M,
           (int)N, G, nblocks);
  else
    launch(linear_mfma_kernel<BITS, 1>, dim3(blocks), dim3(64 * W), lds, stream, ev, x, qweight, scales, zeros, y, M,
           (int)N, G, nblocks);
  return hipGetLastError();
}

template <int BITS>
hipError_t launch_linear_mfma_group(LinearCall* calls, int count, int M, hipStream_t stream,
                                    const LaunchEvents& ev) {
  int nq_max = 1;
  int64_t blocks = 0;
  LinearGroup grp{};
  for (int i = 0; i < count; ++i) {
    LinearCall& c = calls[i];
    nq_max = max(nq_max, (c.G + 3) / 4);
    c.R = 1;
    c.first_block = (int)blocks;
    blocks += (c.N + 15) / 16;
    grp.call[i] = c;
  }
  grp.count = count;
  grp.blocks = (int)blocks;
  const int W = mfma_block_waves(M, nq_max);  // as for one call
  grp.waves = W;
  launch(linear_mfma_group_kernel<BITS>, dim3(xcd_grid(blocks)), dim3(64 * W), (uint32_t)W * M * kSlabRowU4 * 16,
         stream, ev, grp, M);
  return hipGetLastError();
}

template hipError_t launch_linear_mfma_group<3>(LinearCall*, int, int, hipStream_t, const LaunchEvents&);
template hipError_t launch_linear_mfma_group<4>(LinearCall*, int, int, hipStream_t, const LaunchEvents&);
template hipError_t launch_linear_mfma<3>(const uint16_t*, const uint32_t*, const uint16_t*, const uint8_t*,
                                          uint16_t*, int, int64_t, int64_t, hipStream_t, const LaunchEvents&, float*,
                                          size_t);
template hipError_t launch_linear_mfma<4>(const uint16_t*, const uint32_t*, const uint16_t*, const uint8_t*,
                                          uint16_t*, int, int64_t, int64_t, hipStream_t, const LaunchEvents&, float*,
                                          size_t);

}  // namespace laq
