// First-order head-to-neuron affinity on MI355X (gfx950): Section 3 of the paper,
// "Affinity scores", score FO, accumulated over a stream of calibration tokens.
//
// For token t with residual x (entering the FFN pre-norm), r = sqrt(mean(x^2) + eps),
// gain gamma, neuron k's pre-activations g_k = w^g_k . (gamma x / r) and u_k likewise,
// and head h's normalised piece p_h = gamma (a_h W_o^(h)) / r, the damage is
//   Delta_hk = silu'(g_k) u_k (p_h . w^g_k) + silu(g_k) (p_h . w^u_k)
// and the layer's raw score is A[g, k] = ||w^d_k||^2 sum_t sum_{h in g} Delta_hk^2.
//
// Re-association (exact up to rounding): p_h . w_k = (a_h . F_h[:, k]) / r with the folded
// matrix F_h = W_o^(h) diag(gamma) W^T of shape [dh, I].  So per token
//   Delta_hk = c1_k (a_h . Fg_h[:, k]) + c2_k (a_h . Fu_h[:, k]),
//   c1_k = silu'(g_k) u_k / r,   c2_k = silu(g_k) / r,
// and the whole layer is one long contraction per (token tile, neuron tile): first
// [x] x [gamma W_gate | gamma W_up]^T over d (operating point), then, for every head,
// [a_h] x [Fg_h | Fu_h] over dh, with a register epilogue after each head.
//
// Kernels of the bf16 path:
//   prep_gate_up_kernel   W' = W diag(gamma), gate and up rows interleaved per neuron tile
//   transpose_kernel      W_o^T, so both fold operands are K-contiguous
//   fold_kernel           F = W' W_o (MFMA)
//   down_norm_*_kernel    n_d[k] = ||w^d_k||^2 (row chunks, then their fixed-order sum)
//   rms_kernel            1/r per token
//   tile_tokens_kernel    [x | a] rewritten in MFMA fragment order, 1 KB per 32-row k-step
//   affinity_bf16_kernel  the fused operating point + per-head damage + token reduction
//   reduce_splits_kernel  deterministic fp64 sum of the per-split partials into A
// The bf16 weights of a neuron tile form one K-contiguous operand of 128 rows (64 gate,
// 64 up) and d + H*dh columns: [W' | F_0 | F_1 | ... | F_{H-1}].  The token operand is the
// matching concatenation [x | a_0 | ... | a_{H-1}] of the caller's x and attn, tiled once
// per slice so that every fragment load is contiguous; the fused kernel is one
// contraction over d + H*dh with epilogues at the operating-point and head boundaries.
// The fp32 path (dtype DTP_F32) runs the same decomposition with plain FMA kernels.
#include <atomic>
#include <cmath>
#include <vector>

#include "dtp_internal.h"
#include "tile_mfma.h"

namespace dtp {
namespace {

constexpr int kBM = 128;          // tokens per block tile: 4 waves x 32 rows
constexpr int kBN = 64;           // neurons per block tile
constexpr int kCols = 2 * kBN;    // MFMA columns per tile: 64 gate | 64 up
constexpr int kKC = 32;           // contraction depth per LDS stage of the fold
constexpr int kLdsRow = kKC + 8;  // bf16 per LDS row
constexpr int kThreads = 256;
constexpr int kSliceTokens = 1 << 18;  // tokens per internal slice (size of the 1/r buffer)
constexpr int kMaxSplits = 128;        // token splits per launch (size of the partials)
constexpr int kTileTokens = 1 << 15;   // tokens per bf16 slice (size of the tiled token buffer)
constexpr int kTargetBlocks = 768;     // bf16 kernel: aim for this many blocks per launch
constexpr int kTargetBlocksF32 = 768;  // fp32 kernel: the same, in blocks of 4 waves
constexpr size_t kLdsPerCu = 160 * 1024;  // LDS bytes per CU (gfx950)

template <typename T>
__device__ inline float load_f32(const T* p, int64_t i);
template <>
__device__ inline float load_f32<uint16_t>(const uint16_t* p, int64_t i) { return bf16_to_f32(p[i]); }
template <>
__device__ inline float load_f32<float>(const float* p, int64_t i) { return p[i]; }

// ------------------------------------------------------------------ weight preparation
// out[tile*128 + c][j] (row stride ld) = W[k][j] * gamma[j], k = tile*64 + c%64,
// W = gate for c < 64 else up; rows of padding neurons are zero.
template <typename T>
__global__ void prep_gate_up_kernel(const T* __restrict__ w_gate, const T* __restrict__ w_up,
                                    const T* __restrict__ gamma, int I, int d, int n_tiles,
                                    int64_t ld, T* __restrict__ out) {
  const int64_t total = (int64_t)n_tiles * kCols * d;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int j = (int)(idx % d);
    const int64_t rowi = idx / d;
    const int c = (int)(rowi % kCols);
    const int k = (int)(rowi / kCols) * kBN + (c % kBN);
    float v = 0.0f;
    if (k < I) v = load_f32(c < kBN ? w_gate : w_up, (int64_t)k * d + j) * load_f32(gamma, j);
    if constexpr (sizeof(T) == 2)
      out[rowi * ld + j] = f32_to_bf16(v);
    else
      out[rowi * ld + j] = v;
  }
}

// bf16 version of the above, eight columns per thread (d % 8 == 0): 16-byte loads and stores.
__global__ void prep_gate_up_bf16x8_kernel(const uint16_t* __restrict__ w_gate,
                                           const uint16_t* __restrict__ w_up,
                                           const uint16_t* __restrict__ gamma, int I, int d,
                                           int n_tiles, int64_t ld, uint16_t* __restrict__ out) {
  const int d8 = d / 8;
  const int64_t total = (int64_t)n_tiles * kCols * d8;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int j = (int)(idx % d8) * 8;
    const int64_t rowi = idx / d8;
    const int c = (int)(rowi % kCols);
    const int k = (int)(rowi / kCols) * kBN + (c % kBN);
    u32x4 o = {0u, 0u, 0u, 0u};
    if (k < I) {
      const u32x4 w = *reinterpret_cast<const u32x4*>((c < kBN ? w_gate : w_up) + (int64_t)k * d + j);
      const u32x4 g = *reinterpret_cast<const u32x4*>(gamma + j);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float lo = __uint_as_float(w[e] << 16) * __uint_as_float(g[e] << 16);
        const float hi = __uint_as_float(w[e] & 0xffff0000u) * __uint_as_float(g[e] & 0xffff0000u);
        o[e] = (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
      }
    }
    *reinterpret_cast<u32x4*>(out + rowi * ld + j) = o;
  }
}

// out[n][j] = in[j][n] for in of shape [rows, cols].
__global__ void transpose_kernel(const uint16_t* __restrict__ in, int rows, int cols,
                                 uint16_t* __restrict__ out) {
  __shared__ uint16_t tile[32][33];
  const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 256 threads: 32 x 8
  for (int y = ty; y < 32; y += 8) {
    const int r = r0 + y, c = c0 + tx;
    tile[y][tx] = (r < rows && c < cols) ? in[(int64_t)r * cols + c] : (uint16_t)0;
  }
  __syncthreads();
  for (int y = ty; y < 32; y += 8) {
    const int c = c0 + y, r = r0 + tx;
    if (c < cols && r < rows) out[(int64_t)c * rows + r] = tile[tx][y];
  }
}

// wcat[m][d + n] = sum_j wcat[m][j] * woT[n][j] for m < M = n_tiles*128, n < N = H*dh:
// the folded F_h[:, k] of every head h (n = h*dh + e), next to W' in the same row.
__global__ void __launch_bounds__(kThreads)
fold_kernel(uint16_t* __restrict__ wcat, const uint16_t* __restrict__ woT, int N, int d,
            int64_t ld) {
  __shared__ __attribute__((aligned(16))) uint16_t As[2][kBM * kLdsRow];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][kCols * kLdsRow];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int m0 = blockIdx.x * kBM, n0 = blockIdx.y * kCols;
  const uint16_t* a_base = wcat + (int64_t)m0 * ld;
  const uint16_t* b_base = woT + (int64_t)n0 * d;
  const int n_valid = N - n0;
  f32x16 acc[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) acc[b] = f32x16{};
  const int nch = (d + kKC - 1) / kKC;
  Stage<kKC> sa, sb;
  stage_load<kKC>(sa, a_base, ld, kBM, 0, d);
  stage_load<kKC>(sb, b_base, d, n_valid, 0, d);
  stage_store<kKC>(sa, As[0]);
  stage_store<kKC>(sb, Bs[0]);
  __syncthreads();
  for (int q = 0; q < nch; ++q) {
    const int buf = q & 1;
    if (q + 1 < nch) {
      stage_load<kKC>(sa, a_base, ld, kBM, (q + 1) * kKC, d);
      stage_load<kKC>(sb, b_base, d, n_valid, (q + 1) * kKC, d);
    }
    mfma_stage<kKC>(As[buf], Bs[buf], acc, wave, lane);
    if (q + 1 < nch) {
      stage_store<kKC>(sa, As[buf ^ 1]);
      stage_store<kKC>(sb, Bs[buf ^ 1]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const int n = n0 + b * 32 + (lane & 31);
    if (n >= N) continue;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int m = m0 + wave * 32 + acc_row(i, lane);
      wcat[(int64_t)m * ld + d + n] = f32_to_bf16(acc[b][i]);
    }
  }
}

// fp32 fold: F[h][gu][k][e] = sum_j W_o[j][h*dh + e] * gamma[j] * W_gu[k][j]
__global__ void fold_f32_kernel(const float* __restrict__ w_o, const float* __restrict__ gamma,
                                const float* __restrict__ w_gate, const float* __restrict__ w_up,
                                int d, int I, int H, int dh, float* __restrict__ fold) {
  const int64_t total = (int64_t)H * 2 * I * dh;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int e = (int)(idx % dh);
    const int k = (int)((idx / dh) % I);
    const int gu = (int)((idx / ((int64_t)dh * I)) % 2);
    const int h = (int)(idx / ((int64_t)dh * I * 2));
    const float* w = (gu == 0 ? w_gate : w_up) + (int64_t)k * d;
    float s = 0.0f;
    for (int j = 0; j < d; ++j) s = fmaf(w_o[(int64_t)j * H * dh + h * dh + e] * gamma[j], w[j], s);
    fold[idx] = s;
  }
}

// nd[k] = sum_j w_down[j][k]^2 in two passes: part[c][k] sums the rows of chunk c in row
// order, then the chunks are added in order.  A thread of the first pass takes 8 adjacent
// columns of its chunk, one 16-byte load per row where the rows allow it (VEC), so each
// load carries 8 columns and a thread's rows are in flight together.
template <typename T, bool VEC>
__global__ void __launch_bounds__(256)
down_norm_part_kernel(const T* __restrict__ w_down, int d, int I, int chunk_rows,
                      float* __restrict__ part) {
  const int k0 = 8 * (blockIdx.x * 256 + threadIdx.x);
  const int c = blockIdx.y;
  if (k0 >= I) return;
  const int j1 = min(d, (c + 1) * chunk_rows);
  float s[8] = {};
  if constexpr (VEC) {  // I % 8 == 0 and 16-byte aligned rows
#pragma unroll 4
    for (int j = c * chunk_rows; j < j1; ++j) {
      const T* row = w_down + (int64_t)j * I + k0;
      if constexpr (sizeof(T) == 2) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(row);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float lo = __uint_as_float(v[e] << 16), hi = __uint_as_float(v[e] & 0xffff0000u);
          s[2 * e] = fmaf(lo, lo, s[2 * e]);
          s[2 * e + 1] = fmaf(hi, hi, s[2 * e + 1]);
        }
      } else {
        const float4 a = *reinterpret_cast<const float4*>(row);
        const float4 b = *reinterpret_cast<const float4*>(row + 4);
        const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) s[e] = fmaf(v[e], v[e], s[e]);
      }
    }
  } else {
    for (int j = c * chunk_rows; j < j1; ++j)
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (k0 + e < I) {
          const float v = load_f32(w_down, (int64_t)j * I + k0 + e);
          s[e] = fmaf(v, v, s[e]);
        }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e)
    if (k0 + e < I) part[(int64_t)c * I + k0 + e] = s[e];
}

__global__ void __launch_bounds__(64)
down_norm_sum_kernel(const float* __restrict__ part, int chunks, int I, int I_pad,
                     float* __restrict__ nd) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= I_pad) return;
  double t = 0.0;
  if (k < I) {
#pragma unroll 8
    for (int c = 0; c < chunks; ++c) t += (double)part[(int64_t)c * I + k];
  }
  nd[k] = (float)t;
}

// ------------------------------------------------------------------ per-token scalars
// rinv[t] = 1 / sqrt(mean_j x[t][j]^2 + eps); one wavefront per token.
template <typename T>
__global__ void __launch_bounds__(256)
rms_kernel(const T* __restrict__ x, int64_t T_tokens, int d, float eps, float* __restrict__ rinv) {
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= T_tokens) return;  // whole wavefronts exit together
  const T* row = x + t * d;
  float s = 0.0f;
  if constexpr (sizeof(T) == 2) {
    // d % 16 == 0: 16-byte loads of 8 bf16
    for (int j = lane * 8; j < d; j += 64 * 8) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(row + j);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float lo = __uint_as_float(v[e] << 16), hi = __uint_as_float(v[e] & 0xffff0000u);
        s = fmaf(lo, lo, s);
        s = fmaf(hi, hi, s);
      }
    }
  } else {
    for (int j = lane; j < d; j += 64) {
      const float v = load_f32(row, j);
      s = fmaf(v, v, s);
    }
  }
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  if (lane == 0) rinv[t] = 1.0f / sqrtf(s / (float)d + eps);
}

// ------------------------------------------------------------------ token tiling (bf16)
// The MFMA operand layout gives lane l token row l % 32, so a wavefront reading its
// fragments straight from row-major [T][d] rows touches 32 rows per load, which the
// vector memory path serves at a quarter of its rate for contiguous loads.  Each slice of
// tokens is therefore first rewritten so that every fragment is one contiguous 1 KB run:
//   xt[rb][q][s][h][r][e] = [x | attn][32*rb + r][q*KC + h*KC/2 + 8*s + e]
// for 32-row block rb, stage q of KC columns, k-step s < KC/16, half h, row r < 32 and
// element e < 8 (rows past the last token are zero).  The head entries of token t are
// multiplied by p_t = pow2_floor(1/r_t), which is exact in bf16, so the per-head
// contractions come out as p_t (a_h . F) and the damage coefficients c1/p_t, c2/p_t that
// multiply them lie within a factor 2 of silu'(g) u and silu(g) (fp16 range, whatever
// the token scale).  One thread moves one 16-byte chunk; consecutive threads read
// consecutive chunks of a row.
__device__ __forceinline__ float pow2_floor(float v) {  // 2^floor(log2 v), v normal and > 0
  return __uint_as_float(__float_as_uint(v) & 0x7f800000u);
}

__device__ __forceinline__ float pow2_fraction(float v) {  // v / pow2_floor(v), in [1, 2)
  return __uint_as_float((__float_as_uint(v) & 0x007fffffu) | 0x3f800000u);
}

__device__ __forceinline__ uint32_t scale_bf16_pair(uint32_t w, float f) {
  // Both halves times a power of two; exact while the results stay normal.
  const float lo = __uint_as_float(w << 16) * f;
  const float hi = __uint_as_float(w & 0xffff0000u) * f;
  return (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xffff0000u);
}

template <int KC>
__global__ void __launch_bounds__(256)
tile_tokens_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ attn,
                   const float* __restrict__ rinv, int T, int d, int HD, int nq, int64_t n_chunks,
                   uint16_t* __restrict__ xt) {
  constexpr int kRowChunks = KC / 8;
  constexpr int kUnitChunks = 32 * kRowChunks;
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= n_chunks) return;
  const int64_t u = g / kUnitChunks;  // (row block, stage)
  const int w = (int)(g % kUnitChunks);
  const int r = w / kRowChunks, c = w % kRowChunks;
  const int64_t rb = u / nq;
  const int q = (int)(u % nq);
  const int64_t t = 32 * rb + r;
  const int k0 = q * KC + 8 * c;
  u32x4 v = {0u, 0u, 0u, 0u};
  if (t < T) {
    if (k0 < d) {
      v = *reinterpret_cast<const u32x4*>(x + t * d + k0);
    } else {
      v = *reinterpret_cast<const u32x4*>(attn + t * HD + (k0 - d));
      const float f = pow2_floor(rinv[t]);
#pragma unroll
      for (int j = 0; j < 4; ++j) v[j] = scale_bf16_pair(v[j], f);
    }
  }
  const int h = c / (KC / 16), s = c % (KC / 16);
  *reinterpret_cast<u32x4*>(xt + u * (32 * KC) + ((s * 2 + h) * 32 + r) * 8) = v;
}

// ------------------------------------------------------------------ fused affinity (bf16)
struct AffinityArgs {
  const uint16_t* xt;     // token rows [x | attn] in the tiled layout of tile_tokens_kernel
  const uint16_t* wcat;   // [n_tiles*128][Kt], Kt = d + H*dh
  const float* rinv;      // [T]
  const float* rinv_next; // [T] 1/r' of the residual entering the next layer, or NULL
  const float* nd;        // [I_pad]
  float* partial;         // [splits][G+1][I_pad]: G up rows, then the down statistic
  int T, d, H, G, dh, n_tiles, splits, I_pad, Kt, nrb;  // nrb: 32-row blocks in xt
};

// A stage of a block's weight tile: COLS columns x KC contraction elements spread over
// NT threads (KC*COLS/(8*NT) 16-byte segments each), staged through registers into LDS rows
// of KC + 8 bf16 (the 16 bytes of padding spread consecutive rows over the banks).
template <int KC, int COLS, int NT>
struct WeightStage {
  static constexpr int kSegs = KC / 8;                  // per column
  static constexpr int kPerThread = COLS * kSegs / NT;  // per thread
  static_assert(kPerThread >= 1 && COLS * kSegs % NT == 0, "stage does not split evenly");
  u32x4 v[kPerThread];
};

// Operand loads go through buffer resources: a scalar descriptor (base, byte size), a
// per-lane 32-bit byte offset fixed for a whole tile, and a wave-uniform byte offset per
// stage, so a stage spends no vector instructions on addresses (the first step from 64-bit
// per-lane addresses to 32-bit offsets measured 4% on the fused kernel, this one 1% more).
// A load past the descriptor's size returns zeros instead of touching memory.
// 0x00020000: the descriptor word that selects 32-bit raw access on gfx9-class GPUs.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}

__device__ __forceinline__ u32x4 buffer_load16(__amdgpu_buffer_rsrc_t r, uint32_t lane_off,
                                               uint32_t wave_off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)lane_off,
                                                                         (int)wave_off, 0));
}

// Per-thread byte offsets of a weight stage inside its tile (rows of ld elements).
template <int KC, int COLS, int NT>
struct WeightOffsets {
  uint32_t v[WeightStage<KC, COLS, NT>::kPerThread];
  __device__ explicit WeightOffsets(int ld) {
    constexpr int kSegs = WeightStage<KC, COLS, NT>::kSegs;
#pragma unroll
    for (int j = 0; j < WeightStage<KC, COLS, NT>::kPerThread; ++j) {
      const uint32_t i = threadIdx.x + NT * j;
      v[j] = 2u * ((i / kSegs) * (uint32_t)ld + 8u * (i % kSegs));
    }
  }
};

// Contraction columns k0 .. k0+KC-1 of the tile described by `tile`.
template <int KC, int COLS, int NT>
__device__ inline void load_weights(WeightStage<KC, COLS, NT>& w, __amdgpu_buffer_rsrc_t tile,
                                    const WeightOffsets<KC, COLS, NT>& off, int k0) {
#pragma unroll
  for (int j = 0; j < WeightStage<KC, COLS, NT>::kPerThread; ++j)
    w.v[j] = buffer_load16(tile, off.v[j], 2u * (uint32_t)k0);
}

template <int KC, int COLS, int NT>
__device__ inline void store_weights(const WeightStage<KC, COLS, NT>& w, uint16_t* lds) {
  constexpr int kSegs = WeightStage<KC, COLS, NT>::kSegs;
#pragma unroll
  for (int j = 0; j < WeightStage<KC, COLS, NT>::kPerThread; ++j) {
    const int i = threadIdx.x + NT * j;
    *reinterpret_cast<u32x4*>(lds + (i / kSegs) * (KC + 8) + 8 * (i % kSegs)) = w.v[j];
  }
}

// Contraction order inside a stage of KC columns.  Lane l of a wavefront serves token row
// (or weight column) l % 32 and the half h = l / 32 of the stage; its k-step s covers stage
// columns h*KC/2 + 8s .. +7.  Any assignment of contraction indices to (half, k-step)
// yields the same sums as long as both operands follow it; this one gives every lane one
// contiguous run of KC bytes of each of its token rows per stage, loaded straight into
// registers.
template <int KC, int RB>
struct TokenRows {
  u32x4 v[RB][KC / 16];
};

// lane_off[rb]: byte offset of this lane's part of row block rb's unit of stage 0;
// stage q adds q units of 32 x KC elements.
template <int KC, int RB>
__device__ inline void load_token_rows(TokenRows<KC, RB>& f, __amdgpu_buffer_rsrc_t xt,
                                       const uint32_t (&lane_off)[RB], int q) {
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int s = 0; s < KC / 16; ++s)
      f.v[rb][s] = buffer_load16(xt, lane_off[rb] + 1024u * s, (uint32_t)q * (64u * KC));
}

// MFMA work of one stage: the wave's RB token row blocks against the gate and up
// fragments of its NB neuron blocks; each LDS fragment feeds RB MFMAs.  Fragments are
// read kAhead k-steps ahead of their MFMAs (three register buffers, measured 1% faster
// than two at KC = 64), so the LDS latency hides behind the MFMAs in between.  ZERO starts
// the accumulators from zero (first stage of a contraction) instead of adding to them.
template <int KC, int RB, int NB, bool ZERO>
__device__ __forceinline__ void stage_mfma(const uint16_t* B, const TokenRows<KC, RB>& a,
                                           f32x16 (&acc)[RB][NB][2], const int (&gate_off)[NB],
                                           const int (&up_off)[NB]) {
  constexpr int kSteps = KC / 16;
  constexpr int kAhead = kSteps < 3 ? kSteps : 3;
  bf16x8 frag[kAhead][NB][2];
  auto read = [&](int buf, int s) __attribute__((always_inline)) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      frag[buf][nb][0] = *reinterpret_cast<const bf16x8*>(B + gate_off[nb] + 8 * s);
      frag[buf][nb][1] = *reinterpret_cast<const bf16x8*>(B + up_off[nb] + 8 * s);
    }
  };
#pragma unroll
  for (int s = 0; s < kAhead; ++s) read(s, s);
#pragma unroll
  for (int s = 0; s < kSteps; ++s) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const bf16x8 av = __builtin_bit_cast(bf16x8, a.v[rb][s]);
        const bool z = ZERO && s == 0;
#pragma unroll
        for (int gu = 0; gu < 2; ++gu)
          acc[rb][nb][gu] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              av, frag[s % kAhead][nb][gu], z ? f32x16{} : acc[rb][nb][gu], 0, 0, 0);
      }
    if (s + kAhead < kSteps) read(s % kAhead, s + kAhead);
  }
  // Keep that order through scheduling: the reads of the first kAhead k-steps, then each
  // k-step's MFMAs followed by the reads of the k-step kAhead later.
  constexpr int kFrags = 2 * NB, kMfma = 2 * NB * RB;
  __builtin_amdgcn_sched_group_barrier(0x100, kAhead * kFrags, 0);
#pragma unroll
  for (int s = 0; s < kSteps; ++s) {
    __builtin_amdgcn_sched_group_barrier(0x008, kMfma, 0);
    if (s + kAhead < kSteps) __builtin_amdgcn_sched_group_barrier(0x100, kFrags, 0);
  }
}

// Weight stages of KC = 64 or 32 copied into LDS by the buffer unit (buffer_load ... lds),
// no registers and no LDS store instructions: each instruction fills 1 KB of the 128-row
// stage, KC / 32 instructions per thread of the 512.  The rows (KC elements) are
// unpadded; row R keeps its 16-byte chunk c at position c ^ sw(R), with
// sw(R) = (R / (128 / KC)) mod (KC / 8), so the 16 lanes of a fragment read (16
// consecutive rows, one chunk) hit all 64 banks once.
template <int KC>
struct DmaWeights {
  static constexpr int kChunks = KC / 8;        // 16-byte chunks per row
  static constexpr int kRowsPerCopy = 512 / KC;  // rows per 1 KB instruction
  static constexpr int kCopies = KC / 32;        // instructions per thread
  __device__ static int swizzle(int row) { return (row / (128 / KC)) % kChunks; }
  uint32_t voff[kCopies];  // byte offset in the tile of this lane's chunk, per instruction
  __device__ DmaWeights(int Kt, int wave, int lane) {
#pragma unroll
    for (int j = 0; j < kCopies; ++j) {
      const int row = kRowsPerCopy * (kCopies * wave + j) + lane / kChunks;
      const int c = (lane % kChunks) ^ swizzle(row);
      voff[j] = 2u * ((uint32_t)row * (uint32_t)Kt + 8u * c);
    }
  }
  // Contraction columns k0 .. k0+KC-1 of the tile into dst (128 x KC elements).
  __device__ __forceinline__ void copy(__amdgpu_buffer_rsrc_t tile, uint16_t* dst, int wave,
                                       int k0) const {
#pragma unroll
    for (int j = 0; j < kCopies; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          tile, (__attribute__((address_space(3))) void*)(dst + (kCopies * wave + j) * 512), 16,
          (int)voff[j], 2 * k0, 0, 0);
  }
};

// stage_mfma over such a swizzled stage.  rowoff: element offset of the lane's gate row
// per neuron block (the up row is 64 rows further); choff[s]: element offset of k-step
// s's chunk within the row.
template <int KC, int RB, int NB, bool ZERO>
__device__ __forceinline__ void stage_mfma_swizzled(const uint16_t* B, const TokenRows<KC, RB>& a,
                                                    f32x16 (&acc)[RB][NB][2], const int (&rowoff)[NB],
                                                    const int (&choff)[KC / 16]) {
  constexpr int kSteps = KC / 16;
  constexpr int kAhead = kSteps < 3 ? kSteps : 3;
  bf16x8 frag[kAhead][NB][2];
  auto read = [&](int buf, int s) __attribute__((always_inline)) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      frag[buf][nb][0] = *reinterpret_cast<const bf16x8*>(B + rowoff[nb] + choff[s]);
      frag[buf][nb][1] = *reinterpret_cast<const bf16x8*>(B + rowoff[nb] + kBN * KC + choff[s]);
    }
  };
#pragma unroll
  for (int s = 0; s < kAhead; ++s) read(s, s);
#pragma unroll
  for (int s = 0; s < kSteps; ++s) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const bf16x8 av = __builtin_bit_cast(bf16x8, a.v[rb][s]);
        const bool z = ZERO && s == 0;
#pragma unroll
        for (int gu = 0; gu < 2; ++gu)
          acc[rb][nb][gu] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              av, frag[s % kAhead][nb][gu], z ? f32x16{} : acc[rb][nb][gu], 0, 0, 0);
      }
    if (s + kAhead < kSteps) read(s % kAhead, s + kAhead);
  }
  constexpr int kFrags = 2 * NB, kMfma = 2 * NB * RB;
  __builtin_amdgcn_sched_group_barrier(0x100, kAhead * kFrags, 0);
#pragma unroll
  for (int s = 0; s < kSteps; ++s) {
    __builtin_amdgcn_sched_group_barrier(0x008, kMfma, 0);
    if (s + kAhead < kSteps) __builtin_amdgcn_sched_group_barrier(0x100, kFrags, 0);
  }
}

// Per-lane coefficients c1/p_t and c2/p_t of the accumulator elements, either as fp32 or
// rounded to fp16 and packed as one 32-bit (c1, c2) pair (fp16 keeps 11 significant
// bits, and the scaled coefficients lie within a factor 2 of silu'(g) u and silu(g)).
template <int RB, int NB, bool PACK>
struct Coefs;

template <int RB, int NB>
struct Coefs<RB, NB, false> {
  float v1[RB][NB][16], v2[RB][NB][16];
  __device__ __forceinline__ void set(int rb, int nb, int i, float a, float b) {
    v1[rb][nb][i] = a;
    v2[rb][nb][i] = b;
  }
  __device__ __forceinline__ float c1(int rb, int nb, int i) const { return v1[rb][nb][i]; }
  __device__ __forceinline__ float c2(int rb, int nb, int i) const { return v2[rb][nb][i]; }
  // Delta = c1 G + c2 U of element i
  __device__ __forceinline__ float delta(int rb, int nb, int i, float g, float u) const {
    return v1[rb][nb][i] * g + v2[rb][nb][i] * u;
  }
};

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

template <int RB, int NB>
struct Coefs<RB, NB, true> {
  uint32_t v[RB][NB][16];  // c1 in the low half, c2 in the high half
  // a and b are first rounded to fp32 (the asm hides the products that made them), then to
  // fp16: otherwise the compiler may fuse some products with the conversion (one rounding)
  // and not others (two), and a token's coefficients would depend on its row slot.
  __device__ __forceinline__ void set(int rb, int nb, int i, float a, float b) {
    asm("" : "+v"(a), "+v"(b));
    half2_t c;
    c.x = (_Float16)a;
    c.y = (_Float16)b;
    v[rb][nb][i] = __builtin_bit_cast(uint32_t, c);
  }
  __device__ __forceinline__ float c1(int rb, int nb, int i) const {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)(v[rb][nb][i] & 0xffffu));
  }
  __device__ __forceinline__ float c2(int rb, int nb, int i) const {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)(v[rb][nb][i] >> 16));
  }
  // Delta = c1 G + c2 U as two mixed-precision fmas that read the fp16 halves in place
  // (three VALU operations per element with the square; measured 1% faster than
  // unpacking c2 first).  The packed word goes through a scalar before the cast.
  __device__ __forceinline__ float delta(int rb, int nb, int i, float g, float u) const {
    const uint32_t w = v[rb][nb][i];
    const half2_t c = __builtin_bit_cast(half2_t, w);
    return __builtin_fmaf((float)c.y, u, __builtin_fmaf((float)c.x, g, 0.0f));
  }
};

// Work item of block b.  Blocks are dealt to the 8 XCDs round-robin (block b runs on
// XCD b % 8), and each XCD has its own L2.  The (neuron group, token split) items are
// ordered in bands of SG splits, neuron group by neuron group inside a band, and each
// XCD takes one contiguous run of that order, so the blocks an XCD runs together share
// SG token tiles and a few weight tiles.  SG = 0 keeps the plain order.
template <int SG>
__device__ __forceinline__ void block_work(int b, int n_tg, int n_split, int& tg, int& split) {
  if (SG == 0) {
    tg = b / n_split;
    split = b % n_split;
    return;
  }
  const int n = n_tg * n_split;
  const int x = b % 8, slot = b / 8;
  const int j = x * (n / 8) + min(x, n % 8) + slot;
  const int g = j / (SG * n_tg), r = j % (SG * n_tg);
  const int gw = min(SG, n_split - SG * g);
  tg = r / gw;
  split = SG * g + r % gw;
}

// Block = (neuron group of 32*NB*WN neurons, token split) with WM x WN wavefronts.  Wave
// (wm, wn) owns RB 32-row blocks of tokens (rows 32*RB*wm ..) and NB 32-neuron blocks
// (neurons 32*NB*wn ..), each neuron block held as a gate and an up MFMA accumulator, so
// c1/c2 and both damage terms of a (token, neuron) pair sit in the same lane.  For every
// tile of 32*RB*WM tokens of its split the block runs one contraction over
// Kt = d + H*dh in stages of KC:
//   stages [0, d/KC)          acc = [x] . [W'_gate | W'_up]^T          -> c1, c2 in registers
//   each next dh/KC stages    acc = [a_h] . [Fg_h | Fu_h]^T            -> Delta^2 column sums
// The token fragments (one contiguous 1 KB load per k-step) are fetched two stages ahead
// into registers and go straight to the MFMAs.  The weight stage shared by the block goes
// through LDS: at KC = 64 and 32 copied there by the buffer unit two or three stages ahead
// into a ring of three or six swizzled buffers (DmaWeights), otherwise fetched into registers two
// stages ahead and stored into a padded double buffer one stage before use.  Each LDS
// fragment feeds RB MFMAs.  Rows past the last token get zero coefficients.  Column sums
// are kept per lane over its rows, folded across the two half-waves after the last query
// head of each KV group, and banked in LDS per (wave, group); the block writes the
// fixed-order sum over its WM row waves times ||w^d_k||^2 to its split's partial.
template <int KC, int WM, int WN, int RB, int NB, bool PACK, int SG, bool ADD, int RING>
__global__ void __launch_bounds__(64 * WM * WN, 2)  // two waves per SIMD
affinity_bf16_kernel(AffinityArgs p) {
  constexpr int NT = 64 * WM * WN;
  constexpr int kRows = 32 * RB * WM;     // tokens per block tile
  constexpr int kNeurons = 32 * NB * WN;  // neurons per block
  constexpr int kStageCols = 2 * kNeurons;
  static_assert(kNeurons % kBN == 0, "a block covers whole 64-neuron tiles");
  using WStage = WeightStage<KC, kStageCols, NT>;
  // KC = 64 or 32 with one 64-neuron group: weight stages copied straight into LDS (DmaWeights),
  // each stage's buffer a separate array, so the compiler can tell the reads of one stage
  // from the copy into another (one array indexed by the stage makes it wait for the copy
  // before every read).  Otherwise through registers into a padded double buffer.
  constexpr bool kDma = (KC == 64 || KC == 32) && kStageCols == 128 && NT == 512;
  // Copied stages rotate through RING buffers: with three, every stage ends at a barrier
  // (stage q+2 is copied during stage q); with six, every second one does (stage q+3
  // copied); with nine, every third (stage q+4 copied).
  static_assert(RING == 3 || ((RING == 6 || RING == 9) && kDma), "three, six or nine copy buffers");
  constexpr bool kPairs = RING >= 6;  // not every stage ends at a barrier
  constexpr int kLead = RING == 9 ? 4 : RING == 6 ? 3 : 2;  // stages a copy runs ahead
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][kDma ? 8 : kStageCols * (KC + 8)];
  __shared__ __attribute__((aligned(16))) uint16_t BsA[kDma ? kStageCols * KC : 8];
  __shared__ __attribute__((aligned(16))) uint16_t BsB[kDma ? kStageCols * KC : 8];
  __shared__ __attribute__((aligned(16))) uint16_t BsC[kDma ? kStageCols * KC : 8];
  __shared__ __attribute__((aligned(16))) uint16_t BsD[kPairs ? kStageCols * KC : 8];
  __shared__ __attribute__((aligned(16))) uint16_t BsE[kPairs ? kStageCols * KC : 8];
  __shared__ __attribute__((aligned(16))) uint16_t BsF[kPairs ? kStageCols * KC : 8];
  __shared__ __attribute__((aligned(16))) uint16_t BsG[RING == 9 ? kStageCols * KC : 8];
  __shared__ __attribute__((aligned(16))) uint16_t BsH[RING == 9 ? kStageCols * KC : 8];
  __shared__ __attribute__((aligned(16))) uint16_t BsI[RING == 9 ? kStageCols * KC : 8];
  __shared__ __attribute__((aligned(16))) float rv[kRows];  // 1/r of the tile's rows, 0 past T
  __shared__ __attribute__((aligned(16))) float rv2[kRows];  // 1/r' of the rows (down statistic)
  extern __shared__ float red[];  // [WM*WN][G+1][32*NB]
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wm = wave % WM, wn = wave / WM;
  int tg, split;  // neuron group and token split of this block
  block_work<SG>(blockIdx.x, (int)gridDim.x / p.splits, p.splits, tg, split);
  const int hpg = p.H / p.G;

  const int G1 = p.G + 1;  // banked rows: the G up groups, then the down statistic
  const bool down = p.rinv_next != nullptr;
  for (int i = threadIdx.x; i < WM * WN * G1 * 32 * NB; i += NT) red[i] = 0.0f;

  const int mtiles = (p.T + kRows - 1) / kRows;
  const int per = (mtiles + p.splits - 1) / p.splits;
  const int mt_begin = split * per;
  const int mt_end = min(mtiles, mt_begin + per);
  const int nq1 = p.d / KC;   // operating-point stages
  const int nqh = p.dh / KC;  // stages per head
  const int nq = nq1 + p.H * nqh;
  const uint16_t* w_tile = p.wcat + (int64_t)tg * kStageCols * p.Kt;
  // Byte sizes fit 32 bits: the tiled slice holds at most 2^30 elements, a weight tile
  // kStageCols x Kt with Kt <= 131,072.
  const __amdgpu_buffer_rsrc_t xt_rsrc = make_rsrc(p.xt, (uint32_t)p.nrb * 64u * (uint32_t)p.Kt);
  const __amdgpu_buffer_rsrc_t w_rsrc = make_rsrc(w_tile, 2u * kStageCols * (uint32_t)p.Kt);
  const WeightOffsets<KC, kStageCols, NT> w_off(p.Kt);
  // LDS offsets of this wave's gate and up fragments inside a weight stage: neuron n of
  // the block sits at stage row 128*(n/64) + n%64 (gate) and 64 rows further (up).
  int gate_off[NB], up_off[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int n0 = 32 * (NB * wn + nb);
    const int row = (n0 / kBN) * kCols + n0 % kBN + (lane & 31);
    gate_off[nb] = row * (KC + 8) + (lane >> 5) * (KC / 2);
    up_off[nb] = gate_off[nb] + kBN * (KC + 8);
  }
  // The same fragments in the swizzled stage: the lane's row, and the position of k-step
  // s's chunk (chunk (KC / 16) (lane / 32) + s, swizzled by the row; 32 nb and 64 are
  // multiples of 16, so the swizzle depends on lane % 32 only).
  int sw_row[NB], sw_chunk[KC / 16];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) sw_row[nb] = (32 * nb + (lane & 31)) * KC;
#pragma unroll
  for (int st = 0; st < KC / 16; ++st)
    sw_chunk[st] = 8 * (((KC / 16) * (lane >> 5) + st) ^ DmaWeights<KC>::swizzle(lane & 31));
  const DmaWeights<KC> dma(p.Kt, wave, lane);
  __syncthreads();

  for (int mt = mt_begin; mt < mt_end; ++mt) {
    const int m0 = mt * kRows;
    // Row blocks past the last one are clamped to it; their rows get zero coefficients.
    uint32_t lane_off[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
      lane_off[rb] = 2u * ((uint32_t)min(mt * RB * WM + RB * wm + rb, p.nrb - 1) *
                               (uint32_t)(32 * p.Kt) + 8u * lane);
    auto load_tokens_for = [&](TokenRows<KC, RB>& f, int q) __attribute__((always_inline)) {
      load_token_rows<KC, RB>(f, xt_rsrc, lane_off, q);
    };

    f32x16 acc[RB][NB][2];  // [row block][neuron block][gate, up]
    Coefs<RB, NB, PACK> cf;
    float colsum[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) colsum[nb] = 0.0f;
    int head_stage = 0;  // stages done of the current head
    int h = 0;
    TokenRows<KC, RB> t0, t1, t2;
    WStage w0, w1;
    load_tokens_for(t0, 0);
    if constexpr (!kDma) load_weights(w0, w_rsrc, w_off, 0);
    load_tokens_for(t1, min(1, nq - 1));
    if constexpr (kDma) {
      dma.copy(w_rsrc, BsA, wave, 0);
      dma.copy(w_rsrc, BsB, wave, min(1, nq - 1) * KC);
      if constexpr (kLead > 2) dma.copy(w_rsrc, BsC, wave, min(2, nq - 1) * KC);
      if constexpr (kLead > 3) dma.copy(w_rsrc, BsD, wave, min(3, nq - 1) * KC);
    } else {
      load_weights(w1, w_rsrc, w_off, min(1, nq - 1) * KC);
      store_weights(w0, Bs[0]);
    }
    for (int i = threadIdx.x; i < kRows; i += NT) {
      rv[i] = m0 + i < p.T ? p.rinv[m0 + i] : 0.0f;
      rv2[i] = down && m0 + i < p.T ? p.rinv_next[m0 + i] : 0.0f;
    }
    if constexpr (kDma) __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0): stage 0's copy landed
    __syncthreads();

    // Stage q: tokens in `cur`, stage q+1's weights in `wnext` (stored to LDS here unless
    // they are copied),
    // stage q+2 fetched into `tnew` / `wnew`.
    // In the copy mode with three buffers: bcur holds stage q's weights, stage q+1's are
    // in flight or landed, and stage q+2's are copied into bnxt, which stage q-1 read (free
    // since the last barrier).  With six, barriers end the even stages only, so during
    // stages 2p-1 and 2p every wave is within those two: stage q+3 is copied into the
    // buffer of stage q-3, which all waves left before the last barrier, and the barrier
    // after stage 2p waits for the copies of stages 2p+1 and 2p+2.  A head of two stages
    // then ends with no barrier after its epilogue, so one wave's epilogue can run beside
    // the other wave's next MFMAs.  Nine buffers do the same with windows of three stages
    // (barriers after stages 3m; stage q+4 copied into the buffer of stage q-5), for
    // heads of three stages.  `sync`: the stage ends at a barrier (with three buffers,
    // every stage does).
    auto stage = [&](int q, TokenRows<KC, RB>& cur, TokenRows<KC, RB>& tnew, WStage& wnext,
                     WStage& wnew, uint16_t* bcur, uint16_t* bnxt, bool sync) __attribute__((always_inline)) {
      const int buf = q & 1;
      // Unconditional (the last two stages re-fetch the last stage), so that the wait
      // counts before each use stay exact instead of falling back to a full drain.
      const int qn = min(q + 2, nq - 1);
      if constexpr (kDma) {
        dma.copy(w_rsrc, bnxt, wave, min(q + kLead, nq - 1) * KC);
        // Keep the copy ahead of the token loads: the wait at the end of the stage counts
        // on the loads issued after it.
        __builtin_amdgcn_sched_barrier(0);
      }
      load_tokens_for(tnew, qn);
      if constexpr (!kDma) load_weights(wnew, w_rsrc, w_off, qn * KC);
      const bool zero = q == 0 || (q >= nq1 && head_stage == 0);
      if constexpr (kDma) {
        if (zero)
          stage_mfma_swizzled<KC, RB, NB, true>(bcur, cur, acc, sw_row, sw_chunk);
        else
          stage_mfma_swizzled<KC, RB, NB, false>(bcur, cur, acc, sw_row, sw_chunk);
      } else {
        if (zero)
          stage_mfma<KC, RB, NB, true>(Bs[buf], cur, acc, gate_off, up_off);
        else
          stage_mfma<KC, RB, NB, false>(Bs[buf], cur, acc, gate_off, up_off);
      }
      if (q == nq1 - 1) {
        // Operating point: g, u -> c1 = silu'(g) u / r, c2 = silu(g) / r, stored divided
        // by p_t (the head entries were multiplied by it).  Lane l's element i is row
        // 8(i/4) + 4(l/32) + i%4 of its row block: four runs of four rows.
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float4 r4 = *reinterpret_cast<const float4*>(rv + 32 * (RB * wm + rb) + 8 * j + 4 * (lane >> 5));
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              const int i = 4 * j + k;
              const float ri = r4[k];
              const float rs = ri > 0.0f ? pow2_fraction(ri) : 0.0f;  // ri / p_t
#pragma unroll
              for (int nb = 0; nb < NB; ++nb) {
                const float g = acc[rb][nb][0][i] * ri;
                const float u = acc[rb][nb][1][i] * ri;
                const float sg = __builtin_amdgcn_rcpf(1.0f + __expf(-g));
                if (ADD) {
                  cf.set(rb, nb, i, rs, rs);
                } else {
                  // silu(g) = g sg, silu'(g) = sg + silu(g) (1 - sg)
                  const float sl = g * sg;
                  cf.set(rb, nb, i, (fmaf(-sl, sg, sl) + sg) * u * rs, sl * rs);
                }
              }
            }
          }
        if (down) {
          // Down-edge statistic: (alpha / r')^2 with alpha = silu(g) u, summed over rows.
          float ds[NB];
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) ds[nb] = 0.0f;
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const int row = 32 * (RB * wm + rb) + 8 * j + 4 * (lane >> 5);
              const float4 r4 = *reinterpret_cast<const float4*>(rv + row);
              const float4 n4 = *reinterpret_cast<const float4*>(rv2 + row);
#pragma unroll
              for (int k = 0; k < 4; ++k)
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                  const float g = acc[rb][nb][0][4 * j + k] * r4[k];
                  const float u = acc[rb][nb][1][4 * j + k] * r4[k];
                  const float a = g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u * n4[k];
                  ds[nb] = fmaf(a, a, ds[nb]);
                }
            }
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) {
            const float t = ds[nb] + __shfl_xor(ds[nb], 32, 64);
            if (lane < 32) red[(wave * G1 + p.G) * (32 * NB) + 32 * nb + lane] += t;
          }
        }
      } else if (q >= nq1 && ++head_stage == nqh) {
        // Head h done: Delta = c1 (a_h . Fg) + c2 (a_h . Fu); sum Delta^2 over the rows.
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
              if (ADD) {  // (p_h . w^g_k)^2 + (p_h . w^u_k)^2, both coefficients 1/r
                const float dg = cf.c1(rb, nb, i) * acc[rb][nb][0][i];
                const float du = cf.c2(rb, nb, i) * acc[rb][nb][1][i];
                colsum[nb] = fmaf(du, du, fmaf(dg, dg, colsum[nb]));
              } else {
                const float dl = cf.delta(rb, nb, i, acc[rb][nb][0][i], acc[rb][nb][1][i]);
                colsum[nb] = fmaf(dl, dl, colsum[nb]);
              }
            }
        head_stage = 0;
        if (h % hpg == hpg - 1) {
          // Last query head of its KV group: fold the two half-waves and bank the sums.
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) {
            const float t = colsum[nb] + __shfl_xor(colsum[nb], 32, 64);
            if (lane < 32) red[(wave * G1 + h / hpg) * (32 * NB) + 32 * nb + lane] += t;
            colsum[nb] = 0.0f;
          }
        }
        ++h;
      }
      if constexpr (kDma) {
        // The copies the next stages read (stage q+1's; with six buffers also stage q+2's)
        // have landed for this wave once at most the loads issued after the last of them
        // are outstanding.  That one was issued at the start of stage q-1, and after it
        // came stage q-1's token loads, then this stage's copy and token loads (vmcnt);
        // this wave's LDS reads are done (lgkmcnt 0); then the barrier.  __syncthreads()
        // would drain every load.
        constexpr int kLater = 2 * (RB * KC / 16) + DmaWeights<KC>::kCopies;
        static_assert(kLater < 16, "vmcnt field");
        if (!kPairs || sync || q == nq - 1) {
          __builtin_amdgcn_s_waitcnt(0x0070 | kLater);  // vmcnt(kLater) expcnt(7) lgkmcnt(0)
          __builtin_amdgcn_s_barrier();
        }
      } else {
        store_weights(wnext, Bs[buf ^ 1]);  // unused after the last stage
        __syncthreads();
      }
    };

    // Unrolled by six so the three token and two weight register sets, and the three or
    // six copy buffers, rotate in place.
    int q = 0;
    if constexpr (RING == 9) {
      // Barriers after the stages q = 0 mod 3: with the operating point a multiple of three
      // stages and three-stage heads, no head epilogue is followed by a barrier.
      for (; q + 8 < nq; q += 9) {
        stage(q, t0, t2, w1, w0, BsA, BsE, true);
        stage(q + 1, t1, t0, w0, w1, BsB, BsF, false);
        stage(q + 2, t2, t1, w1, w0, BsC, BsG, false);
        stage(q + 3, t0, t2, w0, w1, BsD, BsH, true);
        stage(q + 4, t1, t0, w1, w0, BsE, BsI, false);
        stage(q + 5, t2, t1, w0, w1, BsF, BsA, false);
        stage(q + 6, t0, t2, w1, w0, BsG, BsB, true);
        stage(q + 7, t1, t0, w0, w1, BsH, BsC, false);
        stage(q + 8, t2, t1, w1, w0, BsI, BsD, false);
      }
      if (q < nq) stage(q, t0, t2, w1, w0, BsA, BsE, true);
      if (q + 1 < nq) stage(q + 1, t1, t0, w0, w1, BsB, BsF, false);
      if (q + 2 < nq) stage(q + 2, t2, t1, w1, w0, BsC, BsG, false);
      if (q + 3 < nq) stage(q + 3, t0, t2, w0, w1, BsD, BsH, true);
      if (q + 4 < nq) stage(q + 4, t1, t0, w1, w0, BsE, BsI, false);
      if (q + 5 < nq) stage(q + 5, t2, t1, w0, w1, BsF, BsA, false);
      if (q + 6 < nq) stage(q + 6, t0, t2, w1, w0, BsG, BsB, true);
      if (q + 7 < nq) stage(q + 7, t1, t0, w0, w1, BsH, BsC, false);
    } else if constexpr (kPairs) {
      for (; q + 5 < nq; q += 6) {
        stage(q, t0, t2, w1, w0, BsA, BsD, true);
        stage(q + 1, t1, t0, w0, w1, BsB, BsE, false);
        stage(q + 2, t2, t1, w1, w0, BsC, BsF, true);
        stage(q + 3, t0, t2, w0, w1, BsD, BsA, false);
        stage(q + 4, t1, t0, w1, w0, BsE, BsB, true);
        stage(q + 5, t2, t1, w0, w1, BsF, BsC, false);
      }
      if (q < nq) stage(q, t0, t2, w1, w0, BsA, BsD, true);
      if (q + 1 < nq) stage(q + 1, t1, t0, w0, w1, BsB, BsE, false);
      if (q + 2 < nq) stage(q + 2, t2, t1, w1, w0, BsC, BsF, true);
      if (q + 3 < nq) stage(q + 3, t0, t2, w0, w1, BsD, BsA, false);
      if (q + 4 < nq) stage(q + 4, t1, t0, w1, w0, BsE, BsB, true);
    } else {
      for (; q + 5 < nq; q += 6) {
        stage(q, t0, t2, w1, w0, BsA, BsC, true);
        stage(q + 1, t1, t0, w0, w1, BsB, BsA, true);
        stage(q + 2, t2, t1, w1, w0, BsC, BsB, true);
        stage(q + 3, t0, t2, w0, w1, BsA, BsC, true);
        stage(q + 4, t1, t0, w1, w0, BsB, BsA, true);
        stage(q + 5, t2, t1, w0, w1, BsC, BsB, true);
      }
      if (q < nq) stage(q, t0, t2, w1, w0, BsA, BsC, true);
      if (q + 1 < nq) stage(q + 1, t1, t0, w0, w1, BsB, BsA, true);
      if (q + 2 < nq) stage(q + 2, t2, t1, w1, w0, BsC, BsB, true);
      if (q + 3 < nq) stage(q + 3, t0, t2, w0, w1, BsA, BsC, true);
      if (q + 4 < nq) stage(q + 4, t1, t0, w1, w0, BsB, BsA, true);
    }
  }

  // Sum the row waves in a fixed order and scale by ||w^d_k||^2.
  for (int i = threadIdx.x; i < G1 * kNeurons; i += NT) {
    const int g = i / kNeurons, nl = i % kNeurons;
    const int cw = nl / (32 * NB), k = nl % (32 * NB);
    float sum = 0.0f;
    for (int w = 0; w < WM; ++w) sum += red[((cw * WM + w) * G1 + g) * (32 * NB) + k];
    const int n = tg * kNeurons + nl;
    p.partial[((int64_t)split * G1 + g) * p.I_pad + n] = g < p.G && !ADD ? sum * p.nd[n] : sum;
  }
}

// Dynamic LDS of the fused kernel: the per-wave group sums.
template <int WM, int WN, int NB>
size_t affinity_dynamic_lds(int G) {
  return sizeof(float) * WM * WN * (G + 1) * 32 * NB;
}

// Whether a block of the kernel fits one CU's LDS, less `margin`, with `dynamic` bytes on
// top of its static arrays.  A block that fits no CU would never be scheduled and the
// launch would never finish, so launches check this first.  The static size is the
// larger of what the runtime reports and the sum of the copy buffers.
template <int KC, int WM, int WN, int RB, int NB, bool PACK, int SG, bool ADD, int RING>
bool affinity_lds_fits(size_t dynamic, size_t margin = 0) {
  static const size_t static_lds = [] {
    hipFuncAttributes a{};
    const hipError_t e = hipFuncGetAttributes(
        &a, (const void*)&affinity_bf16_kernel<KC, WM, WN, RB, NB, PACK, SG, ADD, RING>);
    const size_t buffers = sizeof(uint16_t) * RING * (2 * 32 * NB * WN) * KC;
    return e == hipSuccess ? std::max(a.sharedSizeBytes, buffers) : ~size_t(0) / 2;
  }();
  return static_lds + dynamic + margin <= kLdsPerCu;
}

// Compute units of the current device, cached per device (atomics: calls on different
// layers may run on several host threads at once).
int device_cus() {
  static std::atomic<int> cus[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cus[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cus[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

// Token splits of a launch.  A CU runs one block of the fused kernel at a time (its eight
// waves fill the register file), so blocks run in rounds of one per CU, and a block of a
// launch with S splits takes up to ceil(mtiles / S) token tiles: the launch lasts about
// ceil(groups * S / CUs) * ceil(mtiles / S) tile times.  From the smallest split count
// that reaches kTargetBlocks, up to four times it, take the first count that minimises
// that product.  (896 blocks of 32 tiles take four rounds of 256 CUs where 1,792 blocks
// of 16 take seven, 12.5% sooner; 768 blocks of up to 6 tiles take 18 units where 1,024
// of 4 take 16.)
int choose_splits(int groups, int mtiles) {
  const int cap = std::min(mtiles, kMaxSplits);
  const int lo = std::max(1, std::min((kTargetBlocks + groups - 1) / groups, cap));
  const int64_t cus = device_cus();
  int best = lo;
  int64_t best_cost = -1;
  for (int s = lo; s <= std::min(4 * lo, cap); ++s) {
    const int64_t rounds = ((int64_t)groups * s + cus - 1) / cus;
    const int64_t cost = rounds * ((mtiles + s - 1) / s);
    if (best_cost < 0 || cost < best_cost) {
      best = s;
      best_cost = cost;
    }
  }
  return best;
}

// Launches the fused kernel on one slice; returns the number of token splits used, or 0
// if a block does not fit the LDS.
template <int KC, int WM, int WN, int RB, int NB, bool PACK, int SG, bool ADD, int RING>
int launch_affinity(AffinityArgs p, hipStream_t s) {
  constexpr int kRows = 32 * RB * WM;
  constexpr int kNeurons = 32 * NB * WN;
  const int groups = p.n_tiles * kBN / kNeurons;
  const int mtiles = (p.T + kRows - 1) / kRows;
  p.splits = choose_splits(groups, mtiles);
  const size_t shm = affinity_dynamic_lds<WM, WN, NB>(p.G);
  if (!affinity_lds_fits<KC, WM, WN, RB, NB, PACK, SG, ADD, RING>(shm)) return 0;
  if (shm > 65536)  // beyond the default dynamic LDS limit (G close to 32)
    (void)hipFuncSetAttribute((const void*)&affinity_bf16_kernel<KC, WM, WN, RB, NB, PACK, SG, ADD, RING>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
  affinity_bf16_kernel<KC, WM, WN, RB, NB, PACK, SG, ADD, RING><<<groups * p.splits, 64 * WM * WN, shm, s>>>(p);
  return p.splits;
}

// The 64- and 32-deep kernels with six copy buffers where the block fits the LDS with 8 KB
// to spare (G up to 26 at KC = 64), else with three.  At KC = 32 with heads and operating
// point in multiples of three stages, nine buffers (72 KB, any G).
template <int KC, bool ADD>
int launch_affinity_copied(AffinityArgs p, hipStream_t s) {
  if constexpr (KC == 32) {
    if ((p.dh / KC) % 3 == 0 && (p.d / KC) % 3 == 0 &&
        affinity_lds_fits<KC, 8, 1, 1, 2, true, 4, ADD, 9>(affinity_dynamic_lds<8, 1, 2>(p.G), 8192))
      return launch_affinity<KC, 8, 1, 1, 2, true, 4, ADD, 9>(p, s);
  }
  if (affinity_lds_fits<KC, 8, 1, 1, 2, true, 4, ADD, 6>(affinity_dynamic_lds<8, 1, 2>(p.G), 8192))
    return launch_affinity<KC, 8, 1, 1, 2, true, 4, ADD, 6>(p, s);
  return launch_affinity<KC, 8, 1, 1, 2, true, 4, ADD, 3>(p, s);
}

// ------------------------------------------------------------------ fused affinity (fp32)
// One thread per (neuron, token lane); heads visited group by group.
struct AffinityF32Args {
  const float* x;      // [T][d]
  const float* attn;   // [T][H*dh]
  const float* wgu;    // [n_tiles*128][d] gamma-scaled gate | up rows per tile
  const float* fold;   // [H][2][I][dh]
  const float* rinv;
  const float* rinv_next;  // or NULL
  const float* nd;
  float* partial;      // [splits][G+1][I_pad]
  int T, d, H, G, dh, I, I_pad, splits;
  int add;             // ADD score instead of FO
};

__global__ void __launch_bounds__(256)
affinity_f32_kernel(AffinityF32Args p) {
  // blockDim = 256 = 4 token lanes x 64 neurons of one tile
  __shared__ float red[4][kMaxAffinityGroups + 1][kBN];
  const int kl = threadIdx.x & 63, tl = threadIdx.x >> 6;
  const int tile = blockIdx.x / p.splits, split = blockIdx.x % p.splits;
  const int k = tile * kBN + kl;
  const int HD = p.H * p.dh, hpg = p.H / p.G;
  const int per = (p.T + p.splits - 1) / p.splits;
  const int t0 = split * per, t1 = min(p.T, t0 + per);
  float acc[kMaxAffinityGroups + 1];
  for (int g = 0; g <= p.G; ++g) acc[g] = 0.0f;
  if (k < p.I) {
    const float* wg = p.wgu + (int64_t)tile * kCols * p.d + (int64_t)kl * p.d;
    const float* wu = wg + (int64_t)kBN * p.d;
    for (int t = t0 + tl; t < t1; t += 4) {
      const float* xr = p.x + (int64_t)t * p.d;
      const float ri = p.rinv[t];
      float g = 0.0f, u = 0.0f;
      for (int j = 0; j < p.d; ++j) {
        g = fmaf(wg[j], xr[j], g);
        u = fmaf(wu[j], xr[j], u);
      }
      g *= ri;
      u *= ri;
      const float sg = 1.0f / (1.0f + expf(-g));
      if (p.rinv_next) {
        const float a = g * sg * u * p.rinv_next[t];
        acc[p.G] = fmaf(a, a, acc[p.G]);
      }
      const float cc2 = p.add ? ri : g * sg * ri;
      const float cc1 = p.add ? ri : sg * (1.0f + g * (1.0f - sg)) * u * ri;
      for (int h = 0; h < p.H; ++h) {
        const float* ar = p.attn + (int64_t)t * HD + h * p.dh;
        const float* fg = p.fold + (((int64_t)h * 2 + 0) * p.I + k) * p.dh;
        const float* fu = p.fold + (((int64_t)h * 2 + 1) * p.I + k) * p.dh;
        float pg = 0.0f, pu = 0.0f;
        for (int e = 0; e < p.dh; ++e) {
          pg = fmaf(ar[e], fg[e], pg);
          pu = fmaf(ar[e], fu[e], pu);
        }
        if (p.add) {
          acc[h / hpg] = fmaf(cc1 * pg, cc1 * pg, fmaf(cc2 * pu, cc2 * pu, acc[h / hpg]));
        } else {
          const float dl = cc1 * pg + cc2 * pu;
          acc[h / hpg] = fmaf(dl, dl, acc[h / hpg]);
        }
      }
    }
  }
  for (int g = 0; g <= p.G; ++g) red[tl][g][kl] = acc[g];
  __syncthreads();
  for (int i = threadIdx.x; i < (p.G + 1) * kBN; i += 256) {
    const int g = i / kBN, kk = i % kBN;
    const float s = red[0][g][kk] + red[1][g][kk] + red[2][g][kk] + red[3][g][kk];
    const int n = tile * kBN + kk;
    p.partial[((int64_t)split * (p.G + 1) + g) * p.I_pad + n] = g < p.G && !p.add ? s * p.nd[n] : s;
  }
}

// A[g][k] += sum_s partial[s][g][k] for g < G (row g = blockIdx.y), and s_down[k] +=
// sum_s partial[s][G][k] when s_down is given, in fp64 and in a fixed order: eight split
// groups (splits r, r + 8, r + 16, ...) summed in parallel, then the groups in order.
constexpr int kReduceGroups = 8;
__global__ void __launch_bounds__(256)
reduce_splits_kernel(const float* __restrict__ partial, int splits, int G, int I, int I_pad,
                     float* __restrict__ A, float* __restrict__ s_down) {
  __shared__ double part[kReduceGroups][32];
  const int kk = threadIdx.x & 31, r = threadIdx.x >> 5;
  const int g = blockIdx.y;
  const int k = blockIdx.x * 32 + kk;
  double s = 0.0;
  if (k < I)
    for (int sp = r; sp < splits; sp += kReduceGroups)
      s += (double)partial[((int64_t)sp * (G + 1) + g) * I_pad + k];
  part[r][kk] = s;
  __syncthreads();
  if (r == 0 && k < I) {
    float* out = g < G ? A + (int64_t)g * I + k : s_down + k;
    double t = (double)*out;
    for (int q = 0; q < kReduceGroups; ++q) t += part[q][kk];
    *out = (float)t;
  }
}

inline unsigned grid_for(int64_t n, int threads) {
  const int64_t b = (n + threads - 1) / threads;
  return (unsigned)std::min<int64_t>(b, 1 << 20);
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

}  // namespace
}  // namespace dtp

using namespace dtp;

struct dtp_layer_s {
  dtp_layer_desc desc;
  int device = 0;
  int n_tiles = 0, I_pad = 0, Kt = 0;
  bool has_weights = false;
  void* w = nullptr;       // bf16 wcat [n_tiles*128][d + H*dh]; f32 W' [n_tiles*128][d]
  void* woT = nullptr;     // bf16 [H*dh][d]: W_o^T, operand of the fold
  float* fold32 = nullptr;   // f32 path: [H][2][I][dh]
  float* nd = nullptr;       // [I_pad]
  float* rinv = nullptr;     // [kSliceTokens]
  float* rinv_next = nullptr;  // [kSliceTokens], 1/r' for the down statistic
  float* partial = nullptr;  // [kMaxSplits][G][I_pad]
  uint16_t* xt = nullptr;    // bf16 path: one slice of tiled token rows
  int64_t tile_slice = 0;    // tokens per bf16 slice
  bool profiling = false;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> events;
};

namespace {

void layer_free(dtp_layer L) {
  void* bufs[] = {L->w, L->woT, L->fold32, L->nd, L->rinv, L->rinv_next, L->partial, L->xt};
  for (void* b : bufs)
    if (b) (void)hipFree(b);
  for (auto& e : L->events) {
    (void)hipEventDestroy(e.first);
    (void)hipEventDestroy(e.second);
  }
  delete L;
}

// n_d into L->nd, with the layer's split partials as the scratch of the row chunks (the
// affinity launches that use them are ordered after this on the stream).
template <typename T>
dtp_status down_norms(const T* w_down, dtp_layer L, hipStream_t s) {
  const dtp_layer_desc& d = L->desc;
  const int64_t cap = (int64_t)kMaxSplits * (d.n_kv_groups + 1) * L->I_pad;  // floats
  int chunk_rows = 32;
  while ((int64_t)((d.d_model + chunk_rows - 1) / chunk_rows) * d.n_neurons > cap) chunk_rows *= 2;
  const int chunks = (d.d_model + chunk_rows - 1) / chunk_rows;
  const dim3 grid((d.n_neurons + 8 * 256 - 1) / (8 * 256), chunks);
  if (d.n_neurons % 8 == 0 && aligned16(w_down))
    down_norm_part_kernel<T, true><<<grid, 256, 0, s>>>(w_down, d.d_model, d.n_neurons, chunk_rows,
                                                        L->partial);
  else
    down_norm_part_kernel<T, false><<<grid, 256, 0, s>>>(w_down, d.d_model, d.n_neurons, chunk_rows,
                                                         L->partial);
  DTP_HIP(hipGetLastError());
  down_norm_sum_kernel<<<(L->I_pad + 63) / 64, 64, 0, s>>>(L->partial, chunks, d.n_neurons, L->I_pad,
                                                           L->nd);
  DTP_HIP(hipGetLastError());
  return DTP_OK;
}

dtp_status check_device(dtp_layer L) {
  int dev = -1;
  DTP_HIP(hipGetDevice(&dev));
  DTP_CHECK(dev == L->device, DTP_ERR_INVALID_ARG,
            "layer was created on device %d but device %d is current", L->device, dev);
  return DTP_OK;
}

}  // namespace

namespace dtp {
namespace {

// Shared body of the two accumulate entry points; x_next / s_down are NULL for the up
// affinity alone.
dtp_status accumulate(dtp_layer L, const void* x, const void* attn, const void* x_next,
                      float eps_next, int64_t n_tokens, float* A, float* s_down, bool add,
                      void* stream) {
  DTP_CHECK(L != nullptr, DTP_ERR_INVALID_ARG, "layer is NULL");
  DTP_CHECK(n_tokens >= 0, DTP_ERR_INVALID_ARG, "n_tokens=%lld is negative", (long long)n_tokens);
  if (n_tokens == 0) return DTP_OK;
  DTP_CHECK(x && attn && A, DTP_ERR_INVALID_ARG, "x, attn or A is NULL");
  DTP_CHECK(aligned16(x) && aligned16(attn), DTP_ERR_INVALID_ARG,
            "x and attn must be 16-byte aligned");
  DTP_CHECK((x_next == nullptr) == (s_down == nullptr), DTP_ERR_INVALID_ARG,
            "x_next and s_down must be given together");
  DTP_CHECK(x_next == nullptr || aligned16(x_next), DTP_ERR_INVALID_ARG,
            "x_next must be 16-byte aligned");
  DTP_CHECK(std::isfinite(eps_next) && eps_next >= 0.0f, DTP_ERR_INVALID_ARG,
            "rms_eps_next=%g must be finite and >= 0", (double)eps_next);
  DTP_CHECK(L->has_weights, DTP_ERR_INVALID_ARG, "dtp_layer_set_weights was not called");
  dtp_status st = check_device(L);
  if (st != DTP_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  const dtp_layer_desc& d = L->desc;
  const int H = d.n_q_heads, dh = d.head_dim, HD = H * dh, G = d.n_kv_groups;
  const int I = d.n_neurons, dm = d.d_model;
  const size_t esz = d.dtype == DTP_BF16 ? 2 : 4;
  const size_t nt = (size_t)n_tokens;
  if ((st = check_dev_buffer(x, esz * nt * dm, "x")) != DTP_OK ||
      (st = check_dev_buffer(attn, esz * nt * HD, "attn")) != DTP_OK ||
      (st = check_dev_buffer(A, sizeof(float) * (size_t)G * I, "A")) != DTP_OK ||
      (st = check_dev_buffer(x_next, esz * nt * dm, "x_next", true)) != DTP_OK ||
      (st = check_dev_buffer(s_down, sizeof(float) * (size_t)I, "s_down", true)) != DTP_OK)
    return st;
  // Tokens per slice: the 1/r buffer size, and element offsets of a slice below 2^30.
  const int64_t width = std::max(dm, HD);
  int64_t slice = std::max<int64_t>(256, std::min<int64_t>(kSliceTokens, ((int64_t)1 << 30) / width) / 256 * 256);
  if (d.dtype == DTP_BF16) slice = std::min(slice, L->tile_slice);
  for (int64_t t0 = 0; t0 < n_tokens; t0 += slice) {
    const int T = (int)std::min<int64_t>(slice, n_tokens - t0);
    const char* xs = (const char*)x + esz * (size_t)t0 * dm;
    const char* as = (const char*)attn + esz * (size_t)t0 * HD;
    const char* xns = x_next ? (const char*)x_next + esz * (size_t)t0 * dm : nullptr;
    const unsigned rb = (unsigned)((T + 3) / 4);
    if (d.dtype == DTP_BF16) {
      rms_kernel<uint16_t><<<rb, 256, 0, s>>>((const uint16_t*)xs, T, dm, d.rms_eps, L->rinv);
      if (xns)
        rms_kernel<uint16_t><<<rb, 256, 0, s>>>((const uint16_t*)xns, T, dm, eps_next, L->rinv_next);
    } else {
      rms_kernel<float><<<rb, 256, 0, s>>>((const float*)xs, T, dm, d.rms_eps, L->rinv);
      if (xns)
        rms_kernel<float><<<rb, 256, 0, s>>>((const float*)xns, T, dm, eps_next, L->rinv_next);
    }
    DTP_HIP(hipGetLastError());
    const float* rinv_next = xns ? L->rinv_next : nullptr;
    // bf16: rewrite the slice's token rows into the fragment-contiguous layout.  Stages
    // are as deep as the operating point and the heads both divide.
    const int kc = dm % 64 == 0 && dh % 64 == 0 ? 64 : dm % 32 == 0 && dh % 32 == 0 ? 32 : 16;
    const int nrb = (T + 31) / 32;
    if (d.dtype == DTP_BF16) {
      const int64_t n_chunks = (int64_t)nrb * 32 * L->Kt / 8;
      const unsigned tgrid = (unsigned)((n_chunks + 255) / 256);
      if (kc == 64)
        tile_tokens_kernel<64><<<tgrid, 256, 0, s>>>((const uint16_t*)xs, (const uint16_t*)as, L->rinv, T,
                                                     dm, HD, L->Kt / kc, n_chunks, L->xt);
      else if (kc == 32)
        tile_tokens_kernel<32><<<tgrid, 256, 0, s>>>((const uint16_t*)xs, (const uint16_t*)as, L->rinv, T,
                                                     dm, HD, L->Kt / kc, n_chunks, L->xt);
      else
        tile_tokens_kernel<16><<<tgrid, 256, 0, s>>>((const uint16_t*)xs, (const uint16_t*)as, L->rinv, T,
                                                     dm, HD, L->Kt / kc, n_chunks, L->xt);
      DTP_HIP(hipGetLastError());
    }

    int splits;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (L->profiling) {
      DTP_HIP(hipEventCreate(&e0));
      DTP_HIP(hipEventCreate(&e1));
      DTP_HIP(hipEventRecord(e0, s));
    }
    if (d.dtype == DTP_BF16) {
      AffinityArgs p;
      p.xt = L->xt;
      p.wcat = (const uint16_t*)L->w;
      p.rinv = L->rinv;
      p.rinv_next = rinv_next;
      p.nd = L->nd;
      p.partial = L->partial;
      p.T = T;
      p.d = dm;
      p.H = H;
      p.G = G;
      p.dh = dh;
      p.n_tiles = L->n_tiles;
      p.I_pad = L->I_pad;
      p.Kt = L->Kt;
      p.nrb = nrb;
      p.splits = 0;
      // Eight wavefronts per block (one block per CU): 256 tokens x 64 neurons per tile;
      // four for 16-wide stages, whose weight stage has only 256 16-byte pieces.
      if (kc == 64)
        splits = add ? launch_affinity_copied<64, true>(p, s) : launch_affinity_copied<64, false>(p, s);
      else if (kc == 32)
        splits = add ? launch_affinity_copied<32, true>(p, s) : launch_affinity_copied<32, false>(p, s);
      else
        splits = add ? launch_affinity<16, 4, 1, 1, 2, true, 4, true, 3>(p, s)
                     : launch_affinity<16, 4, 1, 1, 2, true, 4, false, 3>(p, s);
      DTP_CHECK(splits > 0, DTP_ERR_UNSUPPORTED,
                "affinity kernel: %d groups need more LDS than a CU holds", G);
    } else {
      splits = (kTargetBlocksF32 + L->n_tiles - 1) / L->n_tiles;
      splits = std::max(1, std::min(splits, std::min(T, kMaxSplits)));
      AffinityF32Args p;
      p.x = (const float*)xs;
      p.attn = (const float*)as;
      p.wgu = (const float*)L->w;
      p.fold = L->fold32;
      p.rinv = L->rinv;
      p.rinv_next = rinv_next;
      p.nd = L->nd;
      p.partial = L->partial;
      p.T = T;
      p.d = dm;
      p.H = H;
      p.G = G;
      p.dh = dh;
      p.I = I;
      p.I_pad = L->I_pad;
      p.splits = splits;
      p.add = add ? 1 : 0;
      affinity_f32_kernel<<<L->n_tiles * splits, 256, 0, s>>>(p);
    }
    DTP_HIP(hipGetLastError());
    if (L->profiling) {
      DTP_HIP(hipEventRecord(e1, s));
      L->events.emplace_back(e0, e1);
    }
    reduce_splits_kernel<<<dim3((I + 31) / 32, s_down ? G + 1 : G), 256, 0, s>>>(
        L->partial, splits, G, I, L->I_pad, A, s_down);
    DTP_HIP(hipGetLastError());
  }
  return DTP_OK;
}

}  // namespace
}  // namespace dtp

extern "C" {

dtp_status dtp_layer_create(const dtp_layer_desc* desc, dtp_layer* out) {
  return guarded([&]() -> dtp_status {
    clear_error();
    DTP_CHECK(desc != nullptr && out != nullptr, DTP_ERR_INVALID_ARG, "desc or out is NULL");
    const dtp_layer_desc& d = *desc;
    DTP_CHECK(d.d_model > 0 && d.n_neurons > 0 && d.n_q_heads > 0 && d.n_kv_groups > 0 &&
                  d.head_dim > 0,
              DTP_ERR_INVALID_ARG, "every size must be positive (d=%d I=%d H=%d G=%d dh=%d)",
              d.d_model, d.n_neurons, d.n_q_heads, d.n_kv_groups, d.head_dim);
    DTP_CHECK(d.n_q_heads % d.n_kv_groups == 0, DTP_ERR_INVALID_ARG,
              "H=%d is not a multiple of G=%d", d.n_q_heads, d.n_kv_groups);
    DTP_CHECK(d.n_kv_groups <= kMaxAffinityGroups, DTP_ERR_UNSUPPORTED, "G=%d exceeds %d",
              d.n_kv_groups, kMaxAffinityGroups);
    DTP_CHECK(d.head_dim % 16 == 0, DTP_ERR_INVALID_ARG, "head_dim=%d is not a multiple of 16",
              d.head_dim);
    DTP_CHECK(d.d_model % 16 == 0, DTP_ERR_INVALID_ARG, "d_model=%d is not a multiple of 16",
              d.d_model);
    DTP_CHECK(d.d_model <= 65536 && d.n_neurons <= (1 << 20) &&
                  (int64_t)d.n_q_heads * d.head_dim <= 65536,
              DTP_ERR_UNSUPPORTED, "shape too large (d <= 65536, I <= 2^20, H*dh <= 65536)");
    DTP_CHECK(std::isfinite(d.rms_eps) && d.rms_eps >= 0.0f, DTP_ERR_INVALID_ARG,
              "rms_eps=%g must be finite and >= 0", (double)d.rms_eps);
    DTP_CHECK(d.dtype == DTP_BF16 || d.dtype == DTP_F32, DTP_ERR_UNSUPPORTED, "dtype %d",
              d.dtype);
    dtp_layer L = new (std::nothrow) dtp_layer_s();
    DTP_CHECK(L != nullptr, DTP_ERR_NO_MEMORY, "host allocation failed");
    L->desc = d;
    hipError_t e = hipGetDevice(&L->device);
    L->n_tiles = (d.n_neurons + 2 * kBN - 1) / (2 * kBN) * 2;  // even: a block may span two tiles
    L->I_pad = L->n_tiles * kBN;
    const int64_t HD = (int64_t)d.n_q_heads * d.head_dim;
    const size_t rows = (size_t)L->n_tiles * kCols;
    if (d.dtype == DTP_BF16) {
      L->Kt = d.d_model + (int)HD;
      // Element offsets inside the tiled slice stay below 2^30.
      L->tile_slice = std::max<int64_t>(256, std::min<int64_t>(kTileTokens, ((int64_t)1 << 30) / L->Kt) / 256 * 256);
      if (e == hipSuccess) e = hipMalloc(&L->w, 2 * rows * L->Kt);
      if (e == hipSuccess) e = hipMalloc(&L->woT, 2 * (size_t)HD * d.d_model);
      if (e == hipSuccess) e = hipMalloc(&L->xt, 2 * (size_t)L->tile_slice * L->Kt);
    } else {
      L->Kt = d.d_model;
      if (e == hipSuccess) e = hipMalloc(&L->w, 4 * rows * d.d_model);
      if (e == hipSuccess) e = hipMalloc(&L->fold32, 4 * (size_t)HD * 2 * d.n_neurons);
    }
    if (e == hipSuccess) e = hipMalloc(&L->nd, 4 * (size_t)L->I_pad);
    if (e == hipSuccess) e = hipMalloc(&L->rinv, 4 * (size_t)kSliceTokens);
    if (e == hipSuccess)
      e = hipMalloc(&L->partial, 4 * (size_t)kMaxSplits * (d.n_kv_groups + 1) * L->I_pad);
    if (e == hipSuccess) e = hipMalloc(&L->rinv_next, 4 * (size_t)kSliceTokens);
    if (e != hipSuccess) {
      layer_free(L);
      return fail(e == hipErrorOutOfMemory ? DTP_ERR_NO_MEMORY : DTP_ERR_HIP,
                  "layer allocation failed: %s", hipGetErrorString(e));
    }
    *out = L;
    return DTP_OK;
  });
}

dtp_status dtp_layer_destroy(dtp_layer layer) {
  return guarded([&]() -> dtp_status {
    clear_error();
    if (layer) layer_free(layer);
    return DTP_OK;
  });
}

dtp_status dtp_layer_set_weights(dtp_layer L, const void* w_o, const void* gamma,
                                 const void* w_gate, const void* w_up, const void* w_down,
                                 void* stream) {
  return guarded([&]() -> dtp_status {
    clear_error();
    DTP_CHECK(L != nullptr, DTP_ERR_INVALID_ARG, "layer is NULL");
    DTP_CHECK(w_o && gamma && w_gate && w_up && w_down, DTP_ERR_INVALID_ARG,
              "a weight pointer is NULL");
    dtp_status st = check_device(L);
    if (st != DTP_OK) return st;
    hipStream_t s = (hipStream_t)stream;
    const dtp_layer_desc& d = L->desc;
    const int H = d.n_q_heads, dh = d.head_dim, HD = H * dh, I = d.n_neurons, dm = d.d_model;
    const int64_t n = (int64_t)L->n_tiles * kCols * dm;
    {
      const size_t esz = d.dtype == DTP_BF16 ? 2 : 4;
      const void* ptrs[5] = {w_o, gamma, w_gate, w_up, w_down};
      const size_t elems[5] = {(size_t)dm * HD, (size_t)dm, (size_t)I * dm, (size_t)I * dm,
                               (size_t)dm * I};
      const char* names[5] = {"w_o", "gamma", "w_gate", "w_up", "w_down"};
      for (int i = 0; i < 5; ++i)
        if ((st = check_dev_buffer(ptrs[i], esz * elems[i], names[i])) != DTP_OK) return st;
    }
    if (d.dtype == DTP_BF16) {
      if (aligned16(w_gate) && aligned16(w_up) && aligned16(gamma))
        prep_gate_up_bf16x8_kernel<<<grid_for(n / 8, 256), 256, 0, s>>>(
            (const uint16_t*)w_gate, (const uint16_t*)w_up, (const uint16_t*)gamma, I, dm,
            L->n_tiles, L->Kt, (uint16_t*)L->w);
      else
        prep_gate_up_kernel<uint16_t><<<grid_for(n, 256), 256, 0, s>>>(
            (const uint16_t*)w_gate, (const uint16_t*)w_up, (const uint16_t*)gamma, I, dm,
            L->n_tiles, L->Kt, (uint16_t*)L->w);
      DTP_HIP(hipGetLastError());
      dim3 tg((HD + 31) / 32, (dm + 31) / 32);
      transpose_kernel<<<tg, 256, 0, s>>>((const uint16_t*)w_o, dm, HD, (uint16_t*)L->woT);
      DTP_HIP(hipGetLastError());
      dim3 fg(L->n_tiles * kCols / kBM, (HD + kCols - 1) / kCols);
      fold_kernel<<<fg, kThreads, 0, s>>>((uint16_t*)L->w, (const uint16_t*)L->woT, HD, dm, L->Kt);
      DTP_HIP(hipGetLastError());
      st = down_norms((const uint16_t*)w_down, L, s);
      if (st != DTP_OK) return st;
    } else {
      prep_gate_up_kernel<float><<<grid_for(n, 256), 256, 0, s>>>(
          (const float*)w_gate, (const float*)w_up, (const float*)gamma, I, dm, L->n_tiles, dm,
          (float*)L->w);
      DTP_HIP(hipGetLastError());
      const int64_t nf = (int64_t)H * 2 * I * dh;
      fold_f32_kernel<<<grid_for(nf, 256), 256, 0, s>>>((const float*)w_o, (const float*)gamma,
                                                         (const float*)w_gate, (const float*)w_up,
                                                         dm, I, H, dh, L->fold32);
      DTP_HIP(hipGetLastError());
      st = down_norms((const float*)w_down, L, s);
      if (st != DTP_OK) return st;
    }
    L->has_weights = true;
    return DTP_OK;
  });
}

dtp_status dtp_affinity_accumulate(dtp_layer L, const void* x, const void* attn, int64_t n_tokens,
                                   float* A, void* stream) {
  return guarded([&]() -> dtp_status {
    clear_error();
    return dtp::accumulate(L, x, attn, nullptr, 0.0f, n_tokens, A, nullptr, false, stream);
  });
}

dtp_status dtp_affinity_accumulate_add(dtp_layer L, const void* x, const void* attn,
                                       int64_t n_tokens, float* A, void* stream) {
  return guarded([&]() -> dtp_status {
    clear_error();
    return dtp::accumulate(L, x, attn, nullptr, 0.0f, n_tokens, A, nullptr, true, stream);
  });
}

dtp_status dtp_affinity_accumulate_down(dtp_layer L, const void* x, const void* attn,
                                        const void* x_next, float rms_eps_next, int64_t n_tokens,
                                        float* A, float* s_down, void* stream) {
  return guarded([&]() -> dtp_status {
    clear_error();
    DTP_CHECK(x_next && s_down, DTP_ERR_INVALID_ARG, "x_next or s_down is NULL");
    return dtp::accumulate(L, x, attn, x_next, rms_eps_next, n_tokens, A, s_down, false, stream);
  });
}

dtp_status dtp_layer_profile(dtp_layer L, int32_t enable) {
  return guarded([&]() -> dtp_status {
    clear_error();
    DTP_CHECK(L != nullptr, DTP_ERR_INVALID_ARG, "layer is NULL");
    L->profiling = enable != 0;
    return DTP_OK;
  });
}

dtp_status dtp_layer_profile_read(dtp_layer L, double* total_ms, int64_t* launches) {
  return guarded([&]() -> dtp_status {
    clear_error();
    DTP_CHECK(L != nullptr && total_ms && launches, DTP_ERR_INVALID_ARG, "NULL argument");
    double sum = 0.0;
    for (auto& e : L->events) {
      DTP_HIP(hipEventSynchronize(e.second));
      float ms = 0.0f;
      DTP_HIP(hipEventElapsedTime(&ms, e.first, e.second));
      sum += ms;
    }
    *total_ms = sum;
    *launches = (int64_t)L->events.size();
    for (auto& e : L->events) {
      (void)hipEventDestroy(e.first);
      (void)hipEventDestroy(e.second);
    }
    L->events.clear();
    return DTP_OK;
  });
}

}  // extern "C"
