// Head step on the GPU (Section 3, "Optimiser"): score every labelled balanced partition
// of a layer's KV groups given the neighbouring neuron assignments.
//
// The objective is linear in h_i once nu_{i-1} and nu_i are fixed, so
//   score(h) = sum_g C[g, h(g)],
//   C[g, l]  = sum_{k: nu_i(k)=l} Q_up_i[g, k] + sum_{k: nu_{i-1}(k)=l} Q_down_{i-1}[k, g].
// All quantities are int64 fixed-point codes, so sums are exact in any order.
//
// Kernels (all over N layers at once):
//   head_gain_kernel      one block per (layer, group): C[g, :] in per-device LDS bins
//   partition_score_kernel one wavefront per (layer, partition): lane g adds C[g, h(g)]
//   best_partition_kernel one block per layer: best score, lowest rank on ties
#include "dtp_internal.h"

namespace dtp {

namespace {

constexpr int kGainThreads = 256;

__device__ inline int64_t wave_sum_i64(int64_t v) {
  for (int off = 32; off > 0; off >>= 1) {
    const int lo = __shfl_xor((int)(uint32_t)(uint64_t)v, off, 64);
    const int hi = __shfl_xor((int)(uint32_t)((uint64_t)v >> 32), off, 64);
    v += (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint64_t)(uint32_t)lo);
  }
  return v;
}

// At most kMaxGainDevices devices: a balanced layout over L devices has at least L!
// labelled partitions (G is a multiple of L), and 11! is beyond what the scoring accepts.
constexpr int kMaxGainDevices = 10;
static_assert(39916800 > kMaxPartitions, "11 devices would need more than 10 device sums");

// C[g, :] of one (layer, group) in one pass over the neurons: each lane keeps one register
// sum per device (DEV >= L of them, selects rather than a branch on the device index, so
// a thread's loads of successive neurons are in flight together), then each sum is added
// across the wavefront and one lane per wavefront adds it to the block's LDS bin.
// Integer sums: exact in any order.  A device index outside [0, L) adds to no sum.
template <int DEV>
__global__ void __launch_bounds__(kGainThreads)
head_gain_kernel(const int64_t* __restrict__ Q_up, const int32_t* __restrict__ nu,
                 const int64_t* __restrict__ Q_down, const int32_t* __restrict__ nu_down,
                 int G, int I, int L, int64_t* __restrict__ C) {
  __shared__ unsigned long long bins[DEV];
  const int layer = blockIdx.x / G;
  const int g = blockIdx.x % G;
  if (threadIdx.x < DEV) bins[threadIdx.x] = 0ull;
  __syncthreads();
  const int64_t* qu = Q_up + ((size_t)layer * G + g) * I;
  const int32_t* nl = nu + (size_t)layer * I;
  const bool down = Q_down != nullptr && layer > 0;
  const int64_t* qd = down ? Q_down + (size_t)(layer - 1) * I * G : nullptr;
  const int32_t* nd = down ? nu_down + (size_t)(layer - 1) * I : nullptr;
  int64_t sum[DEV] = {};
  auto add = [&](int l, int64_t v) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < DEV; ++j) sum[j] += l == j ? v : 0;
  };
#pragma unroll 4
  for (int k = threadIdx.x; k < I; k += kGainThreads) add(nl[k], qu[k]);
  if (down) {
#pragma unroll 4
    for (int k = threadIdx.x; k < I; k += kGainThreads) add(nd[k], qd[(size_t)k * G + g]);
  }
#pragma unroll
  for (int j = 0; j < DEV; ++j) {
    const int64_t t = wave_sum_i64(sum[j]);
    if ((threadIdx.x & 63) == 0) atomicAdd(&bins[j], (unsigned long long)t);
  }
  __syncthreads();
  for (int l = threadIdx.x; l < L; l += kGainThreads)
    C[((size_t)layer * G + g) * L + l] = (int64_t)bins[l];
}

// One wavefront per (layer, partition); lanes index KV groups (G <= 64).
__global__ void __launch_bounds__(256)
partition_score_kernel(const uint8_t* __restrict__ table, const int64_t* __restrict__ C,
                       int N, int G, int L, int64_t P, int64_t* __restrict__ scores) {
  const int64_t wid = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  if (wid >= (int64_t)N * P) return;  // whole wavefronts exit together
  const int layer = (int)(wid / P);
  const int64_t p = wid % P;
  int64_t v = 0;
  if (lane < G) {
    const int dev = table[p * G + lane];
    v = C[((size_t)layer * G + lane) * L + dev];
  }
  v = wave_sum_i64(v);
  if (lane == 0) scores[(size_t)layer * P + p] = v;
}

__device__ inline bool better(int64_t s, int64_t r, int64_t bs, int64_t br, int minimise) {
  if (s != bs) return minimise ? (s < bs) : (s > bs);
  return r < br;
}

__global__ void __launch_bounds__(256)
best_partition_kernel(const int64_t* __restrict__ scores, int64_t P, int minimise,
                      int64_t* __restrict__ best) {
  __shared__ int64_t ss[256];
  __shared__ int64_t sr[256];
  const int layer = blockIdx.x;
  const int64_t* sc = scores + (size_t)layer * P;
  int64_t bs = 0, br = -1;
  for (int64_t p = threadIdx.x; p < P; p += blockDim.x) {
    if (br < 0 || better(sc[p], p, bs, br, minimise)) {
      bs = sc[p];
      br = p;
    }
  }
  ss[threadIdx.x] = bs;
  sr[threadIdx.x] = br;
  __syncthreads();
  for (int step = 128; step > 0; step >>= 1) {
    if (threadIdx.x < step) {
      const int o = threadIdx.x + step;
      if (sr[o] >= 0 && (sr[threadIdx.x] < 0 ||
                         better(ss[o], sr[o], ss[threadIdx.x], sr[threadIdx.x], minimise))) {
        ss[threadIdx.x] = ss[o];
        sr[threadIdx.x] = sr[o];
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) best[layer] = sr[0];
}

}  // namespace

dtp_status score_workspace_create(ScoreWorkspace* ws, int N, int G, int I, int L, hipStream_t s) {
  ws->stream = s;
  ws->N = N;
  ws->G = G;
  ws->I = I;
  ws->L = L;
  ws->P = count_partitions(G, L);
  DTP_CHECK(ws->P > 0 && ws->P <= kMaxPartitions, DTP_ERR_UNSUPPORTED,
            "%lld partitions of %d groups over %d devices exceed the limit of %lld",
            (long long)ws->P, G, L, (long long)kMaxPartitions);
  ws->host_table = enumerate_partitions(G, L);
  const std::vector<uint8_t>& table = ws->host_table;
  // One allocation: [C | scores | best | table], each part 256-byte aligned.
  auto up = [](size_t b) { return (b + 255) & ~size_t(255); };
  const size_t c_bytes = up(sizeof(int64_t) * (size_t)N * G * L);
  const size_t s_bytes = up(sizeof(int64_t) * (size_t)N * ws->P);
  const size_t b_bytes = up(sizeof(int64_t) * (size_t)N);
  char* base = nullptr;
  DTP_HIP(stream_alloc((void**)&base, c_bytes + s_bytes + b_bytes + table.size(), s));
  ws->C = (int64_t*)base;
  ws->scores = (int64_t*)(base + c_bytes);
  ws->best = (int64_t*)(base + c_bytes + s_bytes);
  ws->table = (uint8_t*)(base + c_bytes + s_bytes + b_bytes);
  DTP_HIP(hipMemcpyAsync(ws->table, table.data(), table.size(), hipMemcpyHostToDevice, s));
  return DTP_OK;
}

// The host table must outlive its upload: callers synchronise the stream before this.
void score_workspace_destroy(ScoreWorkspace* ws) {
  if (ws->C) (void)stream_free(ws->C, ws->stream);
  *ws = ScoreWorkspace();
}

dtp_status launch_partition_scores(const ScoreWorkspace& ws, const int64_t* Q_up,
                                   const int32_t* nu, const int64_t* Q_down,
                                   const int32_t* nu_down, int minimise, hipStream_t stream) {
  DTP_CHECK(ws.L <= kMaxGainDevices && ws.G <= kMaxGroups, DTP_ERR_UNSUPPORTED,
            "partition scoring supports G <= %d and L <= %d", kMaxGroups, kMaxGainDevices);
  const unsigned gain_blocks = (unsigned)(ws.N * ws.G);
  if (ws.L <= 2)
    head_gain_kernel<2><<<gain_blocks, kGainThreads, 0, stream>>>(Q_up, nu, Q_down, nu_down, ws.G,
                                                                  ws.I, ws.L, ws.C);
  else if (ws.L <= 4)
    head_gain_kernel<4><<<gain_blocks, kGainThreads, 0, stream>>>(Q_up, nu, Q_down, nu_down, ws.G,
                                                                  ws.I, ws.L, ws.C);
  else
    head_gain_kernel<kMaxGainDevices><<<gain_blocks, kGainThreads, 0, stream>>>(
        Q_up, nu, Q_down, nu_down, ws.G, ws.I, ws.L, ws.C);
  DTP_HIP(hipGetLastError());
  const int64_t waves = (int64_t)ws.N * ws.P;
  const int64_t blocks = (waves + 3) / 4;
  partition_score_kernel<<<(unsigned)blocks, 256, 0, stream>>>(ws.table, ws.C, ws.N, ws.G,
                                                               ws.L, ws.P, ws.scores);
  DTP_HIP(hipGetLastError());
  best_partition_kernel<<<ws.N, 256, 0, stream>>>(ws.scores, ws.P, minimise, ws.best);
  DTP_HIP(hipGetLastError());
  return DTP_OK;
}

}  // namespace dtp
