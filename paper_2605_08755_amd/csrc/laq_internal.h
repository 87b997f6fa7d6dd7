// Internal declarations shared by the library's translation units (not part
// of the public ABI; the public contract is include/laq.h).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace laq {

// Native 128-bit vector (usable with the nontemporal load builtins).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// fp16 pair as the operand type of v_dot2_f32_f16.
typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ half2_t as_half2(uint32_t v) { return __builtin_bit_cast(half2_t, v); }

// XCD-aware block order.  MI355X deals consecutive workgroups of a launch to
// its eight XCDs in turn, and each XCD has its own L2.  A grid of
// xcd_grid(nblocks) workgroups (a multiple of 8) whose workgroup b takes
// logical block xcd_block(nblocks) = (b % 8) * (grid / 8) + b / 8 gives every
// XCD a contiguous range of logical blocks (rows); logical blocks >= nblocks
// are idle and return at once.  Any mapping of workgroups to XCDs gives the
// same results: this is a permutation of independent blocks.  The kernels
// take nblocks as an argument and derive grid / 8 = ceil(nblocks / 8) from
// it rather than reading the grid size: the explicit arguments arrive
// preloaded in scalar registers (the library is built with kernel-argument
// preloading), while the grid size would cost a memory round trip before a
// wave's first request.
inline unsigned xcd_grid(int64_t nblocks) { return (unsigned)(((nblocks + 7) / 8) * 8); }

__device__ __forceinline__ int xcd_block(int nblocks) {
  const int per = (nblocks + 7) >> 3;
  const int b = (int)blockIdx.x;
  return (b & 7) * per + (b >> 3);
}

// Optional events recorded at the kernel's execution start and end
// (hipExtLaunchKernelGGL); both null for an ordinary launch.
struct LaunchEvents {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};

template <typename F, typename... Args>
inline void launch(F kernel, dim3 grid, dim3 block, uint32_t lds, hipStream_t stream,
                   const LaunchEvents& ev, Args... args) {
  if (ev.start || ev.stop)
    hipExtLaunchKernelGGL(kernel, grid, block, lds, stream, ev.start, ev.stop, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, lds, stream, args...);
}

// Residual add + RMSNorm that a batch-1 linear applies to its activation row
// while staging it (the decode step's pre-attention and pre-MLP norms):
// v = res_in + delta (fp32), x = fp16(v / sqrt(mean(v^2) + eps) * weight).
struct NormPrologue {
  const float* res_in = nullptr;     // [K] fp32 residual stream
  const uint16_t* delta = nullptr;   // [K] fp16 added to it, or nullptr
  const uint16_t* weight = nullptr;  // [K] fp16 RMSNorm weight
  float* res_out = nullptr;          // [K] v, written by one block, or nullptr; never res_in
  float eps = 0.0f;
};

// Routing constants of the linear (measured on MI355X).  Every launch shape
// is a pure function of (M, N, K) and these constants: the library keeps no
// mutable state between calls.
constexpr int kMfmaMinM = 3;               // activation rows from which the matrix-core path is used
constexpr int kResidentWaves = 8192;       // waves the chip keeps resident (256 compute units x 32)
constexpr int kMfmaShareMinTiles = 1024;   // from this many 16-row tiles: tiles per block share the activations
constexpr int kSplitMinQuads = 40;         // fewer tiles: K is split (given a workspace) from rows of this many quads

// Several independent linears in one launch (kernel argument block, by value).
constexpr int kMaxGroup = 8;
struct LinearCall {
  const uint16_t* x;
  const uint32_t* qw;
  const uint16_t* scales;
  const uint8_t* zeros;
  uint16_t* y;
  int N, G;
  int R;            // rows per block (flat kernel) or 16-row tiles per block (matrix cores: 1)
  int first_block;  // first block of this call in the grid
  float inv_g;      // fl(1 / G) (flat kernel)
};
struct LinearGroup {
  LinearCall call[kMaxGroup];
  int count;
  int blocks;  // logical blocks of all calls (the grid is rounded up to a multiple of 8)
  int waves;   // matrix-core group: waves per block
};

// Residual output stage of a batch-1 linear: res_out[n] = res_in[n] + y[n]
// (fp32 plus the fp16 output) for every output row n.
struct ResidualEpilogue {
  const float* res_in = nullptr;
  float* res_out = nullptr;
};

// Launchers (return the HIP error of the launch; shapes already validated).
template <int BITS>
hipError_t launch_quantize(const uint16_t* w, int64_t N, int64_t K, uint32_t* qweight,
                           uint16_t* scales, uint8_t* zeros, hipStream_t stream,
                           const LaunchEvents& ev);

template <int BITS>
hipError_t launch_pack(const uint16_t* w, const uint16_t* scales, const uint8_t* zeros, int64_t N,
                       int64_t K, uint32_t* qweight, hipStream_t stream, const LaunchEvents& ev);

// Split K on the matrix-core path for fewer than kMfmaShareMinTiles row
// tiles and rows of at least kSplitMinQuads quads: S K ranges of qs quads,
// tile_blocks blocks of four tiles per range; S == 1 means no split.  A pure
// function of the shape.
struct SplitPlan {
  int S = 1;
  int qs = 0;
  int tile_blocks = 0;
};
SplitPlan mfma_split_plan(int M, int64_t N, int G);
// fp32 partial sums [S][M][N].
inline size_t split_workspace_bytes(const SplitPlan& p, int M, int64_t N) {
  return p.S > 1 ? (size_t)p.S * (size_t)M * (size_t)N * sizeof(float) : 0;
}

// workspace: device memory of workspace_bytes for the split-K partial sums,
// or null (then K is not split).
template <int BITS>
hipError_t launch_linear_mfma(const uint16_t* x, const uint32_t* qweight, const uint16_t* scales,
                              const uint8_t* zeros, uint16_t* y, int M, int64_t N, int64_t K,
                              hipStream_t stream, const LaunchEvents& ev, float* workspace,
                              size_t workspace_bytes);

// calls[i].{x, qw, scales, zeros, y, N, G} filled in by the caller; count in 1..kMaxGroup.
template <int BITS>
hipError_t launch_linear_group(LinearCall* calls, int count, int M, hipStream_t stream, const LaunchEvents& ev);

template <int BITS>
hipError_t launch_linear_mfma_group(LinearCall* calls, int count, int M, hipStream_t stream,
                                    const LaunchEvents& ev);

template <int BITS>
hipError_t launch_linear(const uint16_t* x, const uint32_t* qweight, const uint16_t* scales,
                         const uint8_t* zeros, uint16_t* y, int M, int64_t N, int64_t K,
                         hipStream_t stream, const LaunchEvents& ev, float* workspace = nullptr,
                         size_t workspace_bytes = 0);

// Configuration of the flat (VALU) kernel for MT = 1, 2 or 4 activation
// rows (linear.hip): threads per block, staging loads per thread, rows per
// block and per lane, LDS bytes.
struct FlatPlan {
  int NT = 256, XB = 2, R = 1, RPL = 1;
  size_t lds = 0;
};
FlatPlan flat_plan(int MT, int64_t N, int G);

// Gate|up linear with SiLU-and-multiply in its output stage: weight rows in
// (gate, up) pairs, y fp16 [M][N/2].  Shapes: swiglu_fits(M, K), N even.
bool swiglu_fits(int M, int64_t K);
template <int BITS>
hipError_t launch_linear_swiglu(const uint16_t* x, const uint32_t* qweight, const uint16_t* scales,
                                const uint8_t* zeros, uint16_t* y, int M, int64_t N, int64_t K, hipStream_t stream,
                                const LaunchEvents& ev);

// Batch-1 linear (gate|up + SiLU-and-multiply when swiglu) whose activation
// row is the residual add + RMSNorm of np, computed while the row is staged.
// Shapes: norm_linear_fits(K); N even when swiglu.
bool norm_linear_fits(int64_t K);
template <int BITS>
hipError_t launch_linear_norm(const NormPrologue& np, const uint32_t* qweight, const uint16_t* scales,
                              const uint8_t* zeros, uint16_t* y, int64_t N, int64_t K, bool swiglu,
                              hipStream_t stream, const LaunchEvents& ev);

// The SwiGLU MLP block of one token in one launch (linear.hip): norm
// prologue, gate|up + SiLU-and-multiply, down split over the intermediate
// dimension in S slices of 128, partials added by the last-arriving blocks
// in T teams.  S == 0: the shape is not supported.
constexpr int64_t kMlpMaxHidden = 2560;      // D: 256 x D/128 gate|up units over 1024 threads, <= 5 each
constexpr int64_t kMlpMaxInter = 1 << 20;    // I
constexpr size_t kMlpLdsBytes = 160 * 1024 - 256;  // LDS of one MI355X compute unit, less the static arrays
struct MlpPlan {
  int S = 0, T = 0, team_size = 0;
  size_t lds = 0;
};
MlpPlan mlp_plan(int64_t D, int64_t I, int bits);
// fp32 partials [S][D], team sums [T][D], then T + 1 uint32 counters.
size_t mlp_workspace_bytes(const MlpPlan& p, int64_t D);
template <int BITS>
hipError_t launch_mlp(const NormPrologue& np, const uint32_t* gu_qw, const uint16_t* gu_s, const uint8_t* gu_z,
                      const uint32_t* dn_qw, const uint16_t* dn_s, const uint8_t* dn_z, uint16_t* y, int64_t D,
                      int64_t I, void* workspace, hipStream_t stream, const LaunchEvents& ev);

// Batch-1 linear with the residual output stage (y = x w_hat^T, res_out =
// res_in + y).  Shapes: residual_linear_fits(N, K).
bool residual_linear_fits(int64_t N, int64_t K);
template <int BITS>
hipError_t launch_linear_residual(const uint16_t* x, const uint32_t* qweight, const uint16_t* scales,
                                  const uint8_t* zeros, uint16_t* y, const float* res_in, float* res_out, int64_t N,
                                  int64_t K, hipStream_t stream, const LaunchEvents& ev);

// Decode-step operations (decode.hip); head dimension 128.
int64_t decode_attention_tiles(int64_t L);
hipError_t launch_add_rmsnorm(float* res, const uint16_t* delta, const uint16_t* w, uint16_t* y, int64_t M,
                              int64_t D, float eps, hipStream_t stream, const LaunchEvents& ev);
hipError_t launch_qk_norm_rope(const uint16_t* qkv, const uint16_t* qw, const uint16_t* kw, const float* cos_sin,
                               int64_t pos, int64_t Hq, int64_t Hkv, float eps, uint16_t* q_out, uint16_t* kc,
                               uint16_t* vc, int64_t S_max, hipStream_t stream, const LaunchEvents& ev);
hipError_t launch_decode_attention(const uint16_t* q, const uint16_t* kc, const uint16_t* vc, int64_t Hq,
                                   int64_t Hkv, int64_t L, int64_t S_max, uint16_t* out, float* ws,
                                   hipStream_t stream, const LaunchEvents& ev);
int64_t decode_attention_qkv_tiles(int64_t Hkv, int64_t L);
hipError_t launch_decode_attention_qkv(const uint16_t* qkv, const uint16_t* qw, const uint16_t* kw,
                                       const float* cos_sin, int64_t pos, int64_t Hq, int64_t Hkv, float eps,
                                       uint16_t* kc, uint16_t* vc, int64_t S_max, uint16_t* out, float* ws,
                                       hipStream_t stream, const LaunchEvents& ev);
hipError_t launch_silu_mul(const uint16_t* gu, uint16_t* y, int64_t M, int64_t I, hipStream_t stream,
                           const LaunchEvents& ev);

}  // namespace laq
