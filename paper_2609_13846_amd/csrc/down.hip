// Down-edge affinity on MI355X (gfx950): Section 3 of the paper, "Affinity scores", down
// edge.  Neuron k of layer i writes alpha_k w^d_k into the residual stream; through the
// attention pre-norm of layer i+1 (gain gamma', rms r') it reaches the q/k/v projections of
// KV group g as (alpha_k / r') b_gk with b_gk = W^{qkv}_g (gamma' * w^d_k), so
//   S_down[k, g] = sum_t alpha_k^2 / r'^2 * ||b_gk||^2      (raw token sum).
// The token statistic s[k] = sum_t alpha_k^2 / r'^2 comes out of the affinity kernel's
// operating point (dtp_affinity_accumulate_down).  This file holds the weight-only factor
// B[g, k] = ||b_gk||^2 and the product of the two.
//
// W^{qkv}_g stacks the q rows of the group's query heads (consecutive heads share a group),
// then its k rows and its v rows, from the q_proj / k_proj / v_proj weight layouts.
//
// Kernels:
//   scale_transpose_down_kernel  gamma' * W_down transposed to [I][d] bf16, once per call
//   down_weight_bf16_kernel  one block per (128 neurons, 128 rows of W^{qkv}_g, group):
//                            MFMA over d, then per-column sums of squares of the 128 rows
//   down_weight_f32_kernel   the same with plain FMAs, one thread per (group, neuron)
//   down_rows_reduce_kernel  B[g, k] = fixed-order fp64 sum over the row chunks
//   down_combine_kernel      S_down[k, g] = s[k] B[g, k]
#include <cmath>
#include <mutex>

#include "dtp_internal.h"
#include "tile_mfma.h"

namespace dtp {
namespace {

constexpr int kDKC = 32;              // contraction depth per LDS stage
constexpr int kDRow = kDKC + 8;       // bf16 per LDS row (16 bytes of padding)
constexpr int kDRows = 128;           // rows of W^{qkv}_g per block (4 waves x 32)
constexpr int kDCols = 128;           // neurons per block

// Row rho of W^{qkv}_g inside the three projection matrices (each row d long).
template <typename T>
__device__ inline const T* qkv_row(const T* w_q, const T* w_k, const T* w_v, int g, int rho,
                                   int hpg, int dh, int d) {
  if (rho < hpg * dh) return w_q + ((int64_t)g * hpg * dh + rho) * d;
  rho -= hpg * dh;
  if (rho < dh) return w_k + ((int64_t)g * dh + rho) * d;
  return w_v + ((int64_t)g * dh + rho - dh) * d;
}

// tw[k][j] = bf16(w_down[j][k] * gamma'[j]): W_down scaled and transposed once per call, so
// that the weight kernel reads each neuron's column contiguous along the contraction
// instead of scaling and transposing it again for every group and row chunk.  64 x 64
// tiles through LDS, reads along k and writes along j.
__global__ void __launch_bounds__(256)
scale_transpose_down_kernel(const uint16_t* __restrict__ w_down, const uint16_t* __restrict__ gamma,
                            int d, int I, uint16_t* __restrict__ tw) {
  __shared__ uint16_t tile[64][64 + 2];
  const int k0 = blockIdx.x * 64, j0 = blockIdx.y * 64;
  for (int idx = threadIdx.x; idx < 64 * 64; idx += 256) {
    const int r = idx / 64, c = idx % 64;
    const int j = j0 + r, k = k0 + c;
    tile[r][c] = j < d && k < I
                     ? f32_to_bf16(bf16_to_f32(w_down[(int64_t)j * I + k]) * bf16_to_f32(gamma[j]))
                     : (uint16_t)0;
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < 64 * 64; idx += 256) {
    const int r = idx / 64, c = idx % 64;
    const int k = k0 + r, j = j0 + c;
    if (k < I && j < d) tw[(int64_t)k * d + j] = tile[c][r];
  }
}

// partial[g][chunk][k] = sum over the chunk's rows rho of (W^{qkv}_g[rho] . (gamma' * w^d_k))^2.
// TW: the B operand comes from scale_transpose_down_kernel's tw; otherwise each stage
// scales and transposes its slice of W_down itself (the allocation-free path, which has no
// room for tw).  Both fill the LDS tile with the same values, so B is the same to the bit.
template <bool TW>
__global__ void __launch_bounds__(kTileThreads)
down_weight_bf16_kernel(const uint16_t* __restrict__ w_q, const uint16_t* __restrict__ w_k,
                        const uint16_t* __restrict__ w_v, const uint16_t* __restrict__ gamma,
                        const uint16_t* __restrict__ w_down, const uint16_t* __restrict__ tw,
                        int d, int I, int hpg, int dh, float* __restrict__ partial) {
  __shared__ __attribute__((aligned(16))) uint16_t As[2][kDRows * kDRow];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][kDCols * kDRow];
  __shared__ float red[4][kDCols];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int k0 = blockIdx.x * kDCols, chunk = blockIdx.y, g = blockIdx.z;
  const int n_chunks = gridDim.y;
  const int R = (hpg + 2) * dh;
  f32x16 acc[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) acc[b] = f32x16{};
  // A stage's operands in registers: A, 128 rows x 32 columns of W^{qkv}_g, and B, 128
  // neurons x 32 columns of gamma' * W_down, 16 bytes per thread and pass (2 passes each).
  // Stage kc+32 is fetched into registers during stage kc's MFMAs and stored into the
  // other LDS buffer after them.
  u32x4 av[2], bv[2];
  float bg[2];
  auto fetch = [&](int kc) __attribute__((always_inline)) {
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
      const int row = threadIdx.x / 4 + 64 * pass, seg = threadIdx.x % 4;
      const int rho = chunk * kDRows + row, j = kc + 8 * seg;
      av[pass] = u32x4{0u, 0u, 0u, 0u};
      if (rho < R && j < d)
        av[pass] = *reinterpret_cast<const u32x4*>(qkv_row(w_q, w_k, w_v, g, rho, hpg, dh, d) + j);
    }
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
      bv[pass] = u32x4{0u, 0u, 0u, 0u};
      if constexpr (TW) {
        const int row = threadIdx.x / 4 + 64 * pass, seg = threadIdx.x % 4;
        const int k = k0 + row, j = kc + 8 * seg;
        if (k < I && j < d) bv[pass] = *reinterpret_cast<const u32x4*>(tw + (int64_t)k * d + j);
      } else {
        const int idx = threadIdx.x + kTileThreads * pass;
        const int jj = idx / 16, kseg = idx % 16;
        const int j = kc + jj, k = k0 + 8 * kseg;
        // I % 8 == 0: the 8 neurons are all valid or all past I
        if (j < d && k < I) bv[pass] = *reinterpret_cast<const u32x4*>(w_down + (int64_t)j * I + k);
        bg[pass] = j < d ? bf16_to_f32(gamma[j]) : 0.0f;
      }
    }
  };
  auto store = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
      const int row = threadIdx.x / 4 + 64 * pass, seg = threadIdx.x % 4;
      *reinterpret_cast<u32x4*>(As[buf] + row * kDRow + 8 * seg) = av[pass];
    }
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
      if constexpr (TW) {
        const int row = threadIdx.x / 4 + 64 * pass, seg = threadIdx.x % 4;
        *reinterpret_cast<u32x4*>(Bs[buf] + row * kDRow + 8 * seg) = bv[pass];
      } else {  // scaled by gamma'[j] and stored transposed, [k][j]
        const int idx = threadIdx.x + kTileThreads * pass;
        const int jj = idx / 16, kseg = idx % 16;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint16_t w = (uint16_t)(bv[pass][e / 2] >> (16 * (e % 2)));
          Bs[buf][(8 * kseg + e) * kDRow + jj] = f32_to_bf16(bf16_to_f32(w) * bg[pass]);
        }
      }
    }
  };
  fetch(0);
  store(0);
  __syncthreads();
  for (int kc = 0, buf = 0; kc < d; kc += kDKC, buf ^= 1) {
    const bool more = kc + kDKC < d;
    if (more) fetch(kc + kDKC);
    mfma_stage<kDKC>(As[buf], Bs[buf], acc, wave, lane);
    if (more) store(buf ^ 1);
    __syncthreads();
  }
  // Sum of squares over the wave's 32 rows, per column; rows past R are zero.
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    float c = 0.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i) c = fmaf(acc[b][i], acc[b][i], c);
    c += __shfl_xor(c, 32, 64);
    if (lane < 32) red[wave][b * 32 + lane] = c;
  }
  __syncthreads();
  for (int c = threadIdx.x; c < kDCols; c += kTileThreads) {
    const int k = k0 + c;
    if (k < I)
      partial[((int64_t)g * n_chunks + chunk) * I + k] = red[0][c] + red[1][c] + red[2][c] + red[3][c];
  }
}

// B[g][k] directly, fp32 FMAs: one thread per (group, neuron).
__global__ void __launch_bounds__(256)
down_weight_f32_kernel(const float* __restrict__ w_q, const float* __restrict__ w_k,
                       const float* __restrict__ w_v, const float* __restrict__ gamma,
                       const float* __restrict__ w_down, int d, int I, int G, int hpg, int dh,
                       float* __restrict__ B) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)G * I) return;
  const int g = (int)(idx / I), k = (int)(idx % I);
  const int R = (hpg + 2) * dh;
  double acc = 0.0;
  for (int rho = 0; rho < R; ++rho) {
    const float* row = qkv_row(w_q, w_k, w_v, g, rho, hpg, dh, d);
    float b = 0.0f;
    for (int j = 0; j < d; ++j) b = fmaf(row[j], gamma[j] * w_down[(int64_t)j * I + k], b);
    acc += (double)b * b;
  }
  B[idx] = (float)acc;
}

__global__ void down_rows_reduce_kernel(const float* __restrict__ partial, int G, int n_chunks,
                                        int I, float* __restrict__ B) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)G * I) return;
  const int g = (int)(idx / I), k = (int)(idx % I);
  double s = 0.0;
  for (int c = 0; c < n_chunks; ++c) s += (double)partial[((int64_t)g * n_chunks + c) * I + k];
  B[idx] = (float)s;
}

__global__ void down_combine_kernel(const float* __restrict__ s, const float* __restrict__ B,
                                    int I, int G, float* __restrict__ A_down) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)I * G) return;
  const int k = (int)(idx / G), g = (int)(idx % G);
  A_down[idx] = s[k] * B[(int64_t)g * I + k];
}

unsigned blocks_for(int64_t n, int threads) { return (unsigned)((n + threads - 1) / threads); }

// Scratch of dtp_down_weights_noalloc: the per-chunk partial sums, in device memory the
// library never allocates.  Each device the library runs on holds its own copy until the
// process ends.  In host code `scratch` names a host-side stand-in, not a device address:
// the kernels only ever receive the address hipGetSymbolAddress returns for the current
// device (noalloc_scratch below).  Every slot a call reads is written earlier in the same
// call, so nothing needs clearing between calls.
constexpr size_t kNoAllocScratchFloats = size_t(1) << 20;  // 4 MiB
constexpr int kNoAllocMaxDevices = 64;
static __device__ __align__(256) float scratch[kNoAllocScratchFloats];

std::mutex g_scratch_mu;
float* g_scratch_dev[kNoAllocMaxDevices] = {};

// The current device's copy of `scratch`, looked up once per device on first use.
dtp_status noalloc_scratch(float** out) {
  int dev = -1;
  DTP_HIP(hipGetDevice(&dev));
  DTP_CHECK(dev >= 0 && dev < kNoAllocMaxDevices, DTP_ERR_UNSUPPORTED,
            "device %d: the allocation-free scratch is kept for devices 0..%d", dev,
            kNoAllocMaxDevices - 1);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_dev[dev] == nullptr) {
    void* p = nullptr;
    DTP_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    DTP_CHECK(p != nullptr, DTP_ERR_HIP, "no device address for the scratch on device %d", dev);
    g_scratch_dev[dev] = (float*)p;
  }
  *out = g_scratch_dev[dev];
  return DTP_OK;
}

// Shared body of dtp_down_weights and dtp_down_weights_noalloc.  The scratch of the row-chunk
// sums comes from the stream-ordered allocator, or with `use_static` from the current
// device's copy of `scratch` (the call is refused when it would not fit).
dtp_status down_weights(int32_t d_model, int32_t n_neurons, int32_t n_q_heads, int32_t n_kv_groups,
                        int32_t head_dim, dtp_dtype dtype, const void* w_q, const void* w_k,
                        const void* w_v, const void* gamma_next, const void* w_down, float* B,
                        bool use_static, void* stream) {
  DTP_CHECK(d_model > 0 && n_neurons > 0 && n_q_heads > 0 && n_kv_groups > 0 && head_dim > 0,
            DTP_ERR_INVALID_ARG, "every size must be positive (d=%d I=%d H=%d G=%d dh=%d)",
            d_model, n_neurons, n_q_heads, n_kv_groups, head_dim);
  DTP_CHECK(n_q_heads % n_kv_groups == 0, DTP_ERR_INVALID_ARG, "H=%d is not a multiple of G=%d",
            n_q_heads, n_kv_groups);
  DTP_CHECK(d_model <= 65536 && n_neurons <= (1 << 20) && (int64_t)n_q_heads * head_dim <= 65536,
            DTP_ERR_UNSUPPORTED, "shape too large (d <= 65536, I <= 2^20, H*dh <= 65536)");
  DTP_CHECK(dtype == DTP_BF16 || dtype == DTP_F32, DTP_ERR_UNSUPPORTED, "dtype %d", dtype);
  const int hpg = n_q_heads / n_kv_groups;
  const int64_t GI = (int64_t)n_kv_groups * n_neurons;
  const int R = (hpg + 2) * head_dim;
  const int n_chunks = (R + kDRows - 1) / kDRows;
  if (use_static && dtype == DTP_BF16)
    DTP_CHECK((size_t)GI * n_chunks <= kNoAllocScratchFloats, DTP_ERR_UNSUPPORTED,
              "G * I * ceil((H/G + 2) * dh / 128) = %lld partial sums exceed the %zu floats of "
              "the allocation-free scratch (use dtp_down_weights)",
              (long long)(GI * n_chunks), kNoAllocScratchFloats);
  DTP_CHECK(w_q && w_k && w_v && gamma_next && w_down && B, DTP_ERR_INVALID_ARG,
            "a weight pointer or B is NULL");
  auto al16 = [](const void* p) { return ((uintptr_t)p & 15u) == 0; };
  DTP_CHECK(al16(w_q) && al16(w_k) && al16(w_v) && al16(w_down), DTP_ERR_INVALID_ARG,
            "w_q, w_k, w_v and w_down must be 16-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  {
    const size_t esz = dtype == DTP_BF16 ? 2 : 4, dm = (size_t)d_model;
    const size_t gd = (size_t)n_kv_groups * head_dim;
    dtp_status st;
    if ((st = check_dev_buffer(w_q, esz * n_q_heads * head_dim * dm, "w_q")) != DTP_OK ||
        (st = check_dev_buffer(w_k, esz * gd * dm, "w_k")) != DTP_OK ||
        (st = check_dev_buffer(w_v, esz * gd * dm, "w_v")) != DTP_OK ||
        (st = check_dev_buffer(gamma_next, esz * dm, "gamma_next")) != DTP_OK ||
        (st = check_dev_buffer(w_down, esz * dm * n_neurons, "w_down")) != DTP_OK ||
        (st = check_dev_buffer(B, sizeof(float) * (size_t)GI, "B")) != DTP_OK)
      return st;
  }
  if (dtype == DTP_F32) {
    DTP_CHECK(d_model % 4 == 0, DTP_ERR_INVALID_ARG, "d_model=%d is not a multiple of 4", d_model);
    down_weight_f32_kernel<<<blocks_for(GI, 256), 256, 0, s>>>(
        (const float*)w_q, (const float*)w_k, (const float*)w_v, (const float*)gamma_next,
        (const float*)w_down, d_model, n_neurons, n_kv_groups, hpg, head_dim, B);
    DTP_HIP(hipGetLastError());
    return DTP_OK;
  }
  DTP_CHECK(d_model % 8 == 0, DTP_ERR_INVALID_ARG, "d_model=%d is not a multiple of 8", d_model);
  DTP_CHECK(n_neurons % 8 == 0, DTP_ERR_INVALID_ARG, "n_neurons=%d is not a multiple of 8",
            n_neurons);
  float* partial = nullptr;
  uint16_t* tw = nullptr;
  if (use_static) {
    dtp_status st = noalloc_scratch(&partial);
    if (st != DTP_OK) return st;
  } else {
    DTP_HIP(hipMallocAsync((void**)&partial, sizeof(float) * (size_t)GI * n_chunks, s));
    const hipError_t ea = hipMallocAsync((void**)&tw, sizeof(uint16_t) * (size_t)n_neurons * d_model, s);
    if (ea != hipSuccess) {
      (void)hipFreeAsync(partial, s);
      DTP_HIP(ea);
    }
  }
  dim3 grid((n_neurons + kDCols - 1) / kDCols, n_chunks, n_kv_groups);
  hipError_t e = hipSuccess;
  if (tw) {
    const dim3 tg((n_neurons + 63) / 64, (d_model + 63) / 64);
    scale_transpose_down_kernel<<<tg, 256, 0, s>>>((const uint16_t*)w_down,
                                                   (const uint16_t*)gamma_next, d_model, n_neurons, tw);
    e = hipGetLastError();
    if (e == hipSuccess)
      down_weight_bf16_kernel<true><<<grid, kTileThreads, 0, s>>>(
          (const uint16_t*)w_q, (const uint16_t*)w_k, (const uint16_t*)w_v,
          (const uint16_t*)gamma_next, (const uint16_t*)w_down, tw, d_model, n_neurons, hpg,
          head_dim, partial);
  } else {
    down_weight_bf16_kernel<false><<<grid, kTileThreads, 0, s>>>(
        (const uint16_t*)w_q, (const uint16_t*)w_k, (const uint16_t*)w_v,
        (const uint16_t*)gamma_next, (const uint16_t*)w_down, nullptr, d_model, n_neurons, hpg,
        head_dim, partial);
  }
  if (e == hipSuccess) e = hipGetLastError();
  if (e == hipSuccess) {
    down_rows_reduce_kernel<<<blocks_for(GI, 256), 256, 0, s>>>(partial, n_kv_groups, n_chunks,
                                                                n_neurons, B);
    e = hipGetLastError();
  }
  const hipError_t ef = use_static ? hipSuccess : hipFreeAsync(partial, s);
  const hipError_t et = tw ? hipFreeAsync(tw, s) : hipSuccess;
  DTP_HIP(e);
  DTP_HIP(ef);
  DTP_HIP(et);
  return DTP_OK;
}

}  // namespace
}  // namespace dtp

using namespace dtp;

extern "C" {

dtp_status dtp_down_weights(int32_t d_model, int32_t n_neurons, int32_t n_q_heads,
                            int32_t n_kv_groups, int32_t head_dim, dtp_dtype dtype,
                            const void* w_q, const void* w_k, const void* w_v,
                            const void* gamma_next, const void* w_down, float* B, void* stream) {
  return guarded([&]() -> dtp_status {
    clear_error();
    return down_weights(d_model, n_neurons, n_q_heads, n_kv_groups, head_dim, dtype, w_q, w_k, w_v,
                        gamma_next, w_down, B, false, stream);
  });
}

dtp_status dtp_down_weights_noalloc(int32_t d_model, int32_t n_neurons, int32_t n_q_heads,
                                    int32_t n_kv_groups, int32_t head_dim, dtp_dtype dtype,
                                    const void* w_q, const void* w_k, const void* w_v,
                                    const void* gamma_next, const void* w_down, float* B,
                                    void* stream) {
  return guarded([&]() -> dtp_status {
    clear_error();
    return down_weights(d_model, n_neurons, n_q_heads, n_kv_groups, head_dim, dtype, w_q, w_k, w_v,
                        gamma_next, w_down, B, true, stream);
  });
}

dtp_status dtp_down_affinity(int32_t n_neurons, int32_t n_kv_groups, const float* s_down,
                             const float* B, float* A_down, void* stream) {
  return guarded([&]() -> dtp_status {
    clear_error();
    DTP_CHECK(n_neurons > 0 && n_kv_groups > 0, DTP_ERR_INVALID_ARG, "I=%d and G=%d must be positive",
              n_neurons, n_kv_groups);
    DTP_CHECK(s_down && B && A_down, DTP_ERR_INVALID_ARG, "s_down, B or A_down is NULL");
    hipStream_t s = (hipStream_t)stream;
    const int64_t n = (int64_t)n_neurons * n_kv_groups;
    dtp_status st;
    if ((st = check_dev_buffer(s_down, sizeof(float) * (size_t)n_neurons, "s_down")) != DTP_OK ||
        (st = check_dev_buffer(B, sizeof(float) * (size_t)n, "B")) != DTP_OK ||
        (st = check_dev_buffer(A_down, sizeof(float) * (size_t)n, "A_down")) != DTP_OK)
      return st;
    down_combine_kernel<<<blocks_for(n, 256), 256, 0, s>>>(s_down, B, n_neurons, n_kv_groups, A_down);
    DTP_HIP(hipGetLastError());
    return DTP_OK;
  });
}

}  // extern "C"
