// Applying a layout to a decoder layer's weights (Section 3, "The layout as a free
// variable").  Let group_order[p] be the original KV group placed at new position p and
// neuron_order[p] the original neuron at new position p, where each list runs through
// device 0's members in increasing original index, then device 1's, and so on.  With
// hpg = H/G query heads per group, the permuted weights are
//   w_q     row block p      (hpg*dh rows)  <- row block group_order[p]
//   w_k,w_v row block p      (dh rows)      <- row block group_order[p]
//   w_o     column block p   (hpg*dh cols)  <- column block group_order[p]
//   w_gate, w_up  row p      <- row neuron_order[p]
//   w_down  column p         <- column neuron_order[p]
// so device l's shard is one contiguous range of groups and of neurons.  Gains and
// per-head norm weights do not move.
//
// Kernels (pure data movement, bit-exact):
//   permute_rows_kernel  out row r = in row of block order[r / block] (16-byte vectors)
//   permute_cols_kernel  out[:, c] = in[:, column of block order[c / block]]
#include <algorithm>
#include <vector>

#include "dtp_internal.h"

namespace dtp {
namespace {

typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;

// rows x (row_bytes / 16) vectors; row r of `out` is row order[r / block]*block + r % block.
__global__ void __launch_bounds__(256)
permute_rows_kernel(const u32x4* __restrict__ in, u32x4* __restrict__ out, int64_t rows,
                    int64_t vecs_per_row, int block, const int32_t* __restrict__ order) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * vecs_per_row) return;
  const int64_t r = i / vecs_per_row, v = i % vecs_per_row;
  const int64_t src = (int64_t)order[r / block] * block + r % block;
  out[r * vecs_per_row + v] = in[src * vecs_per_row + v];
}

template <typename T>
__global__ void __launch_bounds__(256)
permute_cols_kernel(const T* __restrict__ in, T* __restrict__ out, int64_t rows, int64_t cols,
                    int block, const int32_t* __restrict__ order) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * cols) return;
  const int64_t r = i / cols, c = i % cols;
  out[i] = in[r * cols + (int64_t)order[c / block] * block + c % block];
}

unsigned grid1(int64_t n) { return (unsigned)((n + 255) / 256); }

// group_order / neuron_order: new position -> original index.
void orders(int G, int I, int L, const int32_t* h, const int32_t* nu, int32_t* go, int32_t* no) {
  int p = 0;
  for (int l = 0; l < L; ++l)
    for (int g = 0; g < G; ++g)
      if (h[g] == l) go[p++] = g;
  p = 0;
  for (int l = 0; l < L; ++l)
    for (int k = 0; k < I; ++k)
      if (nu[k] == l) no[p++] = k;
}

dtp_status check_assignment(const int32_t* a, int n, int L, const char* what) {
  std::vector<int> cnt(L, 0);
  for (int i = 0; i < n; ++i) {
    DTP_CHECK(a[i] >= 0 && a[i] < L, DTP_ERR_INVALID_ARG, "%s[%d] = %d is not a device in [0, %d)",
              what, i, a[i], L);
    ++cnt[a[i]];
  }
  for (int l = 0; l < L; ++l)
    DTP_CHECK(cnt[l] == n / L, DTP_ERR_INVALID_ARG, "%s is not balanced (device %d holds %d)",
              what, l, cnt[l]);
  return DTP_OK;
}

}  // namespace
}  // namespace dtp

using namespace dtp;

extern "C" {

dtp_status dtp_layout_orders(int32_t G, int32_t I, int32_t L, const int32_t* h, const int32_t* nu,
                             int32_t* group_order, int32_t* neuron_order) {
  return guarded([&]() -> dtp_status {
    clear_error();
    DTP_CHECK(G > 0 && I > 0 && L > 0 && G % L == 0 && I % L == 0, DTP_ERR_INVALID_ARG,
              "G=%d and I=%d must be positive multiples of L=%d", G, I, L);
    DTP_CHECK(h && nu && group_order && neuron_order, DTP_ERR_INVALID_ARG, "a pointer is NULL");
    dtp_status st = check_assignment(h, G, L, "h");
    if (st != DTP_OK) return st;
    if ((st = check_assignment(nu, I, L, "nu")) != DTP_OK) return st;
    orders(G, I, L, h, nu, group_order, neuron_order);
    return DTP_OK;
  });
}

dtp_status dtp_apply_layout(const dtp_layer_desc* desc, int32_t L, const int32_t* h,
                            const int32_t* nu, const void* const* src, void* const* dst,
                            void* stream) {
  return guarded([&]() -> dtp_status {
    clear_error();
    DTP_CHECK(desc && h && nu && src && dst, DTP_ERR_INVALID_ARG, "a pointer is NULL");
    const dtp_layer_desc& d = *desc;
    const int G = d.n_kv_groups, H = d.n_q_heads, dh = d.head_dim, I = d.n_neurons, dm = d.d_model;
    DTP_CHECK(dm > 0 && I > 0 && H > 0 && G > 0 && dh > 0 && H % G == 0, DTP_ERR_INVALID_ARG,
              "invalid layer shape (d=%d I=%d H=%d G=%d dh=%d)", dm, I, H, G, dh);
    DTP_CHECK(L > 0 && G % L == 0 && I % L == 0, DTP_ERR_INVALID_ARG,
              "G=%d and I=%d must be multiples of L=%d", G, I, L);
    DTP_CHECK(d.dtype == DTP_BF16 || d.dtype == DTP_F32, DTP_ERR_UNSUPPORTED, "dtype %d", d.dtype);
    const int esz = d.dtype == DTP_BF16 ? 2 : 4;
    DTP_CHECK(((int64_t)dm * esz) % 16 == 0, DTP_ERR_INVALID_ARG,
              "rows of d=%d elements must be a multiple of 16 bytes", dm);
    for (int i = 0; i < 7; ++i) {
      DTP_CHECK(src[i] && dst[i], DTP_ERR_INVALID_ARG, "weight %d is NULL", i);
      DTP_CHECK(((uintptr_t)src[i] & 15u) == 0 && ((uintptr_t)dst[i] & 15u) == 0,
                DTP_ERR_INVALID_ARG, "weight %d is not 16-byte aligned", i);
      DTP_CHECK(src[i] != dst[i], DTP_ERR_INVALID_ARG, "weight %d: in-place permutation", i);
    }
    dtp_status st = check_assignment(h, G, L, "h");
    if (st != DTP_OK) return st;
    if ((st = check_assignment(nu, I, L, "nu")) != DTP_OK) return st;
    {
      const size_t hd = (size_t)H * dh, gd = (size_t)G * dh;
      const size_t elems[7] = {hd * dm, gd * dm, gd * dm, (size_t)dm * hd, (size_t)I * dm,
                               (size_t)I * dm, (size_t)dm * I};
      const char* src_names[7] = {"src w_q", "src w_k", "src w_v", "src w_o", "src w_gate",
                                  "src w_up", "src w_down"};
      const char* dst_names[7] = {"dst w_q", "dst w_k", "dst w_v", "dst w_o", "dst w_gate",
                                  "dst w_up", "dst w_down"};
      for (int i = 0; i < 7; ++i) {
        if ((st = check_dev_buffer(src[i], esz * elems[i], src_names[i])) != DTP_OK) return st;
        if ((st = check_dev_buffer(dst[i], esz * elems[i], dst_names[i])) != DTP_OK) return st;
      }
    }
    std::vector<int32_t> ord(G + I);
    orders(G, I, L, h, nu, ord.data(), ord.data() + G);
    hipStream_t s = (hipStream_t)stream;
    int32_t* dord = nullptr;
    DTP_HIP(hipMallocAsync((void**)&dord, sizeof(int32_t) * (G + I), s));
    hipError_t e = hipMemcpyAsync(dord, ord.data(), sizeof(int32_t) * (G + I), hipMemcpyHostToDevice, s);
    const int32_t* go = dord;
    const int32_t* no = dord + G;
    const int hpg = H / G;
    const int64_t vr = (int64_t)dm * esz / 16;  // 16-byte vectors per row of d elements
    auto rows = [&](int i, int64_t n_rows, int block, const int32_t* ord_dev) {
      if (e != hipSuccess) return;
      permute_rows_kernel<<<grid1(n_rows * vr), 256, 0, s>>>((const u32x4*)src[i], (u32x4*)dst[i],
                                                             n_rows, vr, block, ord_dev);
      e = hipGetLastError();
    };
    auto cols = [&](int i, int64_t n_cols, int block, const int32_t* ord_dev) {
      if (e != hipSuccess) return;
      if (esz == 2)
        permute_cols_kernel<uint16_t><<<grid1((int64_t)dm * n_cols), 256, 0, s>>>(
            (const uint16_t*)src[i], (uint16_t*)dst[i], dm, n_cols, block, ord_dev);
      else
        permute_cols_kernel<float><<<grid1((int64_t)dm * n_cols), 256, 0, s>>>(
            (const float*)src[i], (float*)dst[i], dm, n_cols, block, ord_dev);
      e = hipGetLastError();
    };
    rows(0, (int64_t)H * dh, hpg * dh, go);  // w_q: a group's query heads are one block
    rows(1, (int64_t)G * dh, dh, go);        // w_k
    rows(2, (int64_t)G * dh, dh, go);        // w_v
    cols(3, (int64_t)H * dh, hpg * dh, go);  // w_o columns, like the q rows
    rows(4, I, 1, no);                       // w_gate
    rows(5, I, 1, no);                       // w_up
    cols(6, I, 1, no);                       // w_down columns
    const hipError_t ef = hipFreeAsync(dord, s);
    DTP_HIP(e);
    DTP_HIP(ef);
    // The order upload reads `ord`, which dies on return.
    DTP_HIP(hipStreamSynchronize(s));
    return DTP_OK;
  });
}

}  // extern "C"
