// bf16 MFMA tile helpers shared by the HIP kernels of libdtp.so (gfx950).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace dtp {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

constexpr int kTileThreads = 256;  // threads of the blocks that use the tile helpers

__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

__device__ inline uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;  // NaN stays NaN
  u += 0x7fffu + ((u >> 16) & 1u);                      // round to nearest even
  return (uint16_t)(u >> 16);
}

// ------------------------------------------------------------------ tile staging (bf16)
// A stage is 128 rows x KC contraction columns; each of the 256 threads moves KC/16
// segments of 16 bytes (8 bf16) from global memory into registers, then into LDS.
template <int KC>
struct Stage {
  u32x4 v[KC / 16];
};

template <int KC>
__device__ inline void stage_load(Stage<KC>& s, const uint16_t* __restrict__ base, int64_t ld,
                                  int rows_valid, int k0, int k_valid) {
  constexpr int kSegs = KC / 8;              // 16-byte segments per row
  constexpr int kRowsPerPass = kTileThreads / kSegs;
  const int t = threadIdx.x;
  const int k = k0 + (t % kSegs) * 8;
#pragma unroll
  for (int j = 0; j < KC / 16; ++j) {
    const int row = t / kSegs + kRowsPerPass * j;
    if (row < rows_valid && k < k_valid)
      s.v[j] = *reinterpret_cast<const u32x4*>(base + (int64_t)row * ld + k);
    else
      s.v[j] = u32x4{0u, 0u, 0u, 0u};
  }
}

template <int KC>
__device__ inline void stage_store(const Stage<KC>& s, uint16_t* lds) {
  constexpr int kSegs = KC / 8;
  constexpr int kRowsPerPass = kTileThreads / kSegs;
  const int t = threadIdx.x;
#pragma unroll
  for (int j = 0; j < KC / 16; ++j) {
    const int row = t / kSegs + kRowsPerPass * j;
    *reinterpret_cast<u32x4*>(lds + row * (KC + 8) + (t % kSegs) * 8) = s.v[j];
  }
}

// One stage of MFMA work: the wave's 32 rows of A against the 128 columns of B, with LDS
// rows of KC + 8 bf16 (the 16 bytes of padding spread consecutive rows over the banks).
// v_mfma_f32_32x32x16_bf16: lane l feeds row (l % 32) of A / column (l % 32) of B with the
// 8 contraction elements starting at 8 * (l / 32).
template <int KC>
__device__ inline void mfma_stage(const uint16_t* As, const uint16_t* Bs, f32x16 (&acc)[4],
                                  int wave, int lane) {
  constexpr int kRow = KC + 8;
  const int r = lane & 31;
  const int kh = (lane >> 5) * 8;
#pragma unroll
  for (int ks = 0; ks < KC; ks += 16) {
    const bf16x8 a = *reinterpret_cast<const bf16x8*>(As + (wave * 32 + r) * kRow + ks + kh);
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const bf16x8 bb = *reinterpret_cast<const bf16x8*>(Bs + (b * 32 + r) * kRow + ks + kh);
      acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bb, acc[b], 0, 0, 0);
    }
  }
}

// Row (within the wave's 32) held by accumulator element i of lane l.
__device__ inline int acc_row(int i, int lane) { return 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3); }

}  // namespace dtp
