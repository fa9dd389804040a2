// C ABI of the layout side of libdtp.so: status strings, error reporting, validation,
// the encoder, partition enumeration, the neuron step and the coordinate-ascent driver
// (Section 3, "Objective" and "Optimiser").  The affinity entry points live in
// affinity.hip.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <thread>

#include "dtp_internal.h"

namespace dtp {

namespace {
thread_local char g_last_error[1024] = "";
}

dtp_status fail(dtp_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return s;
}

void clear_error() { g_last_error[0] = '\0'; }

dtp_status check_dev_buffer(const void* p, size_t bytes, const char* what, bool optional) {
  if (p == nullptr) {
    DTP_CHECK(optional, DTP_ERR_INVALID_ARG, "%s is NULL", what);
    return DTP_OK;
  }
  int dev = -1;
  DTP_HIP(hipGetDevice(&dev));
  hipPointerAttribute_t a{};
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();  // keep the failed query out of later launch checks
    return fail(DTP_ERR_INVALID_ARG, "%s (%p) is not device memory", what, p);
  }
  DTP_CHECK(a.type == hipMemoryTypeDevice || a.type == hipMemoryTypeManaged, DTP_ERR_INVALID_ARG,
            "%s (%p) is not device memory (HIP memory type %d)", what, p, (int)a.type);
  DTP_CHECK(a.device == dev, DTP_ERR_INVALID_ARG, "%s (%p) is memory of device %d, not of the current device %d",
            what, p, a.device, dev);
  hipDeviceptr_t base = nullptr;
  size_t size = 0;
  if (hipMemGetAddressRange(&base, &size, const_cast<void*>(p)) != hipSuccess) {
    (void)hipGetLastError();
    return fail(DTP_ERR_INVALID_ARG, "%s (%p): no device allocation contains it", what, p);
  }
  const size_t off = (size_t)((const char*)p - (const char*)base);
  DTP_CHECK(off <= size && bytes <= size - off, DTP_ERR_INVALID_ARG,
            "%s (%p) has %zu bytes left in its allocation, the call reads or writes %zu", what, p,
            off <= size ? size - off : (size_t)0, bytes);
  return DTP_OK;
}

namespace {

// M[k][l] = sum_{g: h(g)=l} Q_up[g][k] + sum_{g: h_next(g)=l} Q_down[k][g], negated when
// minimising (the solver maximises).
void neuron_gain(int G, int I, int L, const int64_t* Q_up, const int32_t* h,
                 const int64_t* Q_down, const int32_t* h_next, bool minimise,
                 std::vector<int64_t>* M) {
  M->assign((size_t)I * L, 0);
  for (int g = 0; g < G; ++g) {
    const int l = h[g];
    const int64_t* q = Q_up + (size_t)g * I;
    for (int k = 0; k < I; ++k) (*M)[(size_t)k * L + l] += q[k];
  }
  if (Q_down) {
    for (int k = 0; k < I; ++k) {
      const int64_t* q = Q_down + (size_t)k * G;
      for (int g = 0; g < G; ++g) (*M)[(size_t)k * L + h_next[g]] += q[g];
    }
  }
  if (minimise)
    for (auto& v : *M) v = -v;
}

dtp_status check_balanced(const int32_t* h, int G, int L, const char* what) {
  int count[kMaxGroups] = {0};
  for (int g = 0; g < G; ++g) {
    DTP_CHECK(h[g] >= 0 && h[g] < L, DTP_ERR_INVALID_ARG, "%s[%d] = %d is not a device in [0, %d)",
              what, g, h[g], L);
    ++count[h[g]];
  }
  for (int l = 0; l < L; ++l)
    DTP_CHECK(count[l] == G / L, DTP_ERR_INVALID_ARG,
              "%s is not balanced: device %d holds %d groups, expected %d", what, l, count[l],
              G / L);
  return DTP_OK;
}

dtp_status check_layout_sizes(int G, int I, int L, int max_devices) {
  DTP_CHECK(G > 0 && I > 0 && L > 0, DTP_ERR_INVALID_ARG, "G=%d, I=%d, L=%d must be positive", G,
            I, L);
  DTP_CHECK(G % L == 0, DTP_ERR_INVALID_ARG, "G=%d is not a multiple of L=%d", G, L);
  DTP_CHECK(I % L == 0, DTP_ERR_INVALID_ARG, "I=%d is not a multiple of L=%d", I, L);
  DTP_CHECK(G <= kMaxGroups, DTP_ERR_UNSUPPORTED, "G=%d exceeds %d", G, kMaxGroups);
  DTP_CHECK(L <= max_devices, DTP_ERR_UNSUPPORTED, "L=%d exceeds %d", L, max_devices);
  DTP_CHECK(I <= (1 << 24), DTP_ERR_UNSUPPORTED, "I=%d exceeds 2^24", I);
  return DTP_OK;
}

int64_t objective_int(int N, int G, int I, const int64_t* Qu, const int64_t* Qd, bool has_down,
                      const int32_t* h, const int32_t* nu) {
  int64_t J = 0;
  for (int i = 0; i < N; ++i) {
    const int64_t* q = Qu + (size_t)i * G * I;
    const int32_t* hi = h + (size_t)i * G;
    const int32_t* ni = nu + (size_t)i * I;
    for (int g = 0; g < G; ++g)
      for (int k = 0; k < I; ++k)
        if (hi[g] == ni[k]) J += q[(size_t)g * I + k];
    if (has_down && i + 1 < N) {
      const int64_t* qd = Qd + (size_t)i * I * G;
      const int32_t* hn = h + (size_t)(i + 1) * G;
      for (int k = 0; k < I; ++k)
        for (int g = 0; g < G; ++g)
          if (ni[k] == hn[g]) J += qd[(size_t)k * G + g];
    }
  }
  return J;
}

// SplitMix64 output n from state `seed` (Steele, Lea and Flood, OOPSLA 2014).
uint64_t splitmix64(uint64_t seed, uint64_t n) {
  uint64_t z = seed + (n + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Fisher-Yates from the last position down; position j swaps with floor(r (j+1) / 2^64).
void shuffle(int32_t* a, int n, uint64_t seed, uint64_t* counter) {
  for (int j = n - 1; j > 0; --j) {
    const uint64_t r = splitmix64(seed, (*counter)++);
    const int i = (int)(((unsigned __int128)r * (uint64_t)(j + 1)) >> 64);
    std::swap(a[j], a[i]);
  }
}

// Stream-ordered scratch released on the stream it was allocated on.
struct DevBuf {
  void* p = nullptr;
  hipStream_t s = nullptr;
  explicit DevBuf(hipStream_t stream) : s(stream) {}
  ~DevBuf() {
    if (p) (void)stream_free(p, s);
  }
};

// Pinned host blocks for the device <-> host copies of the coordinate ascent.  A copy
// between device memory and pageable host memory goes through the runtime's staging
// buffer and costs several times the kernels around it (the codes of one 8 x 3072 layer,
// 196 KB, took longer than every kernel of the ascent together); from pinned memory it is
// one transfer.  Blocks come from a process-wide free list and go back to it when the call
// returns; they are never released, so the list holds at most one block per call that ran
// concurrently (each as large as the largest such call needed).
class PinnedPool {
 public:
  struct Block {
    void* p = nullptr;
    size_t bytes = 0;
  };
  Block take(size_t bytes) {
    {
      std::lock_guard<std::mutex> lock(mu_);
      for (size_t i = 0; i < free_.size(); ++i)
        if (free_[i].bytes >= bytes) {
          const Block b = free_[i];
          free_.erase(free_.begin() + (std::ptrdiff_t)i);
          return b;
        }
    }
    Block b;
    b.bytes = std::max(bytes, (size_t)64 << 10);
    if (hipHostMalloc(&b.p, b.bytes, hipHostMallocPortable) != hipSuccess) b = Block();
    return b;
  }
  void give(const Block& b) {
    if (b.p == nullptr) return;
    std::lock_guard<std::mutex> lock(mu_);
    free_.push_back(b);
  }

 private:
  std::mutex mu_;
  std::vector<Block> free_;
};

PinnedPool& pinned_pool() {
  static PinnedPool* pool = new PinnedPool;  // lives until the process ends
  return *pool;
}

// A pinned block for one call, or (if pinned memory cannot be had) pageable memory.
struct HostStaging {
  PinnedPool::Block pinned;
  std::vector<char> pageable;
  char* base = nullptr;
  explicit HostStaging(size_t bytes) : pinned(pinned_pool().take(bytes)) {
    if (pinned.p) {
      base = (char*)pinned.p;
    } else {
      pageable.resize(bytes);
      base = pageable.data();
    }
  }
  ~HostStaging() { pinned_pool().give(pinned); }
};

}  // namespace

hipError_t stream_alloc(void** p, size_t bytes, hipStream_t s) {
  static std::mutex mu;
  static bool retained[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < 64) {
    std::lock_guard<std::mutex> lock(mu);
    if (!retained[dev]) {
      hipMemPool_t pool;
      if (hipDeviceGetDefaultMemPool(&pool, dev) == hipSuccess) {
        uint64_t keep = UINT64_MAX;
        (void)hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep);
      }
      retained[dev] = true;
    }
  }
  return hipMallocAsync(p, bytes, s);
}

hipError_t stream_free(void* p, hipStream_t s) { return hipFreeAsync(p, s); }
}  // namespace dtp

using namespace dtp;

extern "C" {

const char* dtp_status_string(dtp_status s) {
  switch (s) {
    case DTP_OK: return "DTP_OK";
    case DTP_ERR_INVALID_ARG: return "DTP_ERR_INVALID_ARG";
    case DTP_ERR_UNSUPPORTED: return "DTP_ERR_UNSUPPORTED";
    case DTP_ERR_DEGENERATE: return "DTP_ERR_DEGENERATE";
    case DTP_ERR_NO_MEMORY: return "DTP_ERR_NO_MEMORY";
    case DTP_ERR_HIP: return "DTP_ERR_HIP";
  }
  return "DTP_ERR_UNKNOWN";
}

const char* dtp_last_error(void) { return g_last_error; }

int64_t dtp_partition_count(int32_t G, int32_t L) { return count_partitions(G, L); }

dtp_status dtp_partition_unrank(int32_t G, int32_t L, int64_t rank, int32_t* h) {
  return guarded([&]() -> dtp_status {
    clear_error();
    DTP_CHECK(h != nullptr, DTP_ERR_INVALID_ARG, "h is NULL");
    const int64_t P = count_partitions(G, L);
    DTP_CHECK(P > 0, DTP_ERR_INVALID_ARG, "no balanced partitions for G=%d, L=%d", G, L);
    DTP_CHECK(rank >= 0 && rank < P, DTP_ERR_INVALID_ARG, "rank %lld outside [0, %lld)",
              (long long)rank, (long long)P);
    unrank_partition(G, L, rank, h);
    return DTP_OK;
  });
}

dtp_status dtp_encode_affinity(const float* A, int64_t n, int64_t* Q) {
  return guarded([&]() -> dtp_status {
    clear_error();
    DTP_CHECK(A != nullptr && Q != nullptr, DTP_ERR_INVALID_ARG, "A or Q is NULL");
    DTP_CHECK(n >= 1 && n <= (int64_t(1) << 20), DTP_ERR_INVALID_ARG,
              "n=%lld outside [1, 2^20]", (long long)n);
    return encode_unit_mass(A, n, Q);
  });
}

dtp_status dtp_encode_affinity_device(const float* A, int64_t n, int64_t* Q, void* stream) {
  return guarded([&]() -> dtp_status {
    clear_error();
    DTP_CHECK(A != nullptr && Q != nullptr, DTP_ERR_INVALID_ARG, "A or Q is NULL");
    DTP_CHECK(n >= 1 && n <= (int64_t(1) << 30), DTP_ERR_INVALID_ARG,
              "n=%lld outside [1, 2^30]", (long long)n);
    dtp_status st0;
    if ((st0 = check_dev_buffer(A, sizeof(float) * (size_t)n, "A")) != DTP_OK ||
        (st0 = check_dev_buffer(Q, sizeof(int64_t) * (size_t)n, "Q")) != DTP_OK)
      return st0;
    hipStream_t s = (hipStream_t)stream;
    DevBuf stats_dev(s);
    DTP_HIP(stream_alloc(&stats_dev.p, sizeof(EncodeStats), s));
    dtp_status st = launch_encode_unit_mass(A, 1, nullptr, 0, n, Q, nullptr,
                                            (EncodeStats*)stats_dev.p, s);
    if (st != DTP_OK) return st;
    EncodeStats stats;
    DTP_HIP(hipMemcpyAsync(&stats, stats_dev.p, sizeof(EncodeStats), hipMemcpyDeviceToHost, s));
    DTP_HIP(hipStreamSynchronize(s));
    return check_encode_stats(stats, "matrix", 0);
  });
}

dtp_status dtp_balanced_assign(int32_t G, int32_t I, int32_t L, const int64_t* Q_up,
                               const int32_t* h, const int64_t* Q_down, const int32_t* h_next,
                               int32_t minimise, int32_t* nu, int64_t* value) {
  return guarded([&]() -> dtp_status {
    clear_error();
    dtp_status st = check_layout_sizes(G, I, L, kMaxAssignDevices);
    if (st != DTP_OK) return st;
    DTP_CHECK(Q_up && h && nu && value, DTP_ERR_INVALID_ARG, "a required pointer is NULL");
    DTP_CHECK((Q_down == nullptr) == (h_next == nullptr), DTP_ERR_INVALID_ARG,
              "Q_down and h_next must both be given or both be NULL");
    if ((st = check_balanced(h, G, L, "h")) != DTP_OK) return st;
    if (h_next && (st = check_balanced(h_next, G, L, "h_next")) != DTP_OK) return st;
    std::vector<int64_t> M;
    neuron_gain(G, I, L, Q_up, h, Q_down, h_next, minimise != 0, &M);
    int64_t v = 0;
    balanced_assign_exact(I, L, M.data(), nu, &v);
    *value = minimise ? -v : v;
    return DTP_OK;
  });
}

dtp_status dtp_balanced_assign_dual_ascent(int32_t G, int32_t I, int32_t L, const int64_t* Q_up,
                                           const int32_t* h, const int64_t* Q_down,
                                           const int32_t* h_next, int32_t minimise, int32_t* nu,
                                           int64_t* value) {
  return guarded([&]() -> dtp_status {
    clear_error();
    dtp_status st = check_layout_sizes(G, I, L, kMaxAssignDevices);
    if (st != DTP_OK) return st;
    DTP_CHECK(Q_up && h && nu && value, DTP_ERR_INVALID_ARG, "a required pointer is NULL");
    DTP_CHECK((Q_down == nullptr) == (h_next == nullptr), DTP_ERR_INVALID_ARG,
              "Q_down and h_next must both be given or both be NULL");
    if ((st = check_balanced(h, G, L, "h")) != DTP_OK) return st;
    if (h_next && (st = check_balanced(h_next, G, L, "h_next")) != DTP_OK) return st;
    std::vector<int64_t> M;
    neuron_gain(G, I, L, Q_up, h, Q_down, h_next, minimise != 0, &M);
    int64_t v = 0;
    balanced_assign_dual_ascent(I, L, M.data(), kDualAscentIterations, kDualAscentDecay, nu, &v);
    *value = minimise ? -v : v;
    return DTP_OK;
  });
}

dtp_status dtp_partition_scores(int32_t G, int32_t I, int32_t L, const int64_t* Q_up,
                                const int32_t* nu, const int64_t* Q_down_prev,
                                const int32_t* nu_prev, int32_t minimise, int64_t* scores,
                                int64_t* best_rank, void* stream) {
  return guarded([&]() -> dtp_status {
    clear_error();
    dtp_status st = check_layout_sizes(G, I, L, 64);
    if (st != DTP_OK) return st;
    DTP_CHECK(Q_up && nu && scores && best_rank, DTP_ERR_INVALID_ARG, "a required pointer is NULL");
    DTP_CHECK((Q_down_prev == nullptr) == (nu_prev == nullptr), DTP_ERR_INVALID_ARG,
              "Q_down_prev and nu_prev must both be given or both be NULL");
    const int64_t P = count_partitions(G, L);
    DTP_CHECK(P > 0 && P <= kMaxPartitions, DTP_ERR_UNSUPPORTED,
              "%lld partitions exceed the limit of %lld", (long long)P, (long long)kMaxPartitions);
    if ((st = check_dev_buffer(Q_up, sizeof(int64_t) * (size_t)G * I, "Q_up")) != DTP_OK ||
        (st = check_dev_buffer(nu, sizeof(int32_t) * (size_t)I, "nu")) != DTP_OK ||
        (st = check_dev_buffer(Q_down_prev, sizeof(int64_t) * (size_t)I * G, "Q_down_prev", true)) != DTP_OK ||
        (st = check_dev_buffer(nu_prev, sizeof(int32_t) * (size_t)I, "nu_prev", true)) != DTP_OK ||
        (st = check_dev_buffer(scores, sizeof(int64_t) * (size_t)P, "scores")) != DTP_OK)
      return st;
    hipStream_t s = (hipStream_t)stream;
    // A two-layer view: layer 0 is empty padding so that layer 1 reads Q_down_prev / nu_prev
    // as its incoming down edge.  Without a down edge one layer suffices.
    const bool down = Q_down_prev != nullptr;
    ScoreWorkspace ws;
    st = score_workspace_create(&ws, down ? 2 : 1, G, I, L, s);
    if (st != DTP_OK) {
      score_workspace_destroy(&ws);
      return st;
    }
    DevBuf qbuf(s), nbuf(s);
    const int64_t* qu = Q_up;
    const int32_t* nl = nu;
    if (down) {
      // layer 0 gets zero codes; layer 1 is the real layer
      const size_t qbytes = sizeof(int64_t) * (size_t)G * I;
      const size_t nbytes = sizeof(int32_t) * (size_t)I;
      hipError_t e = stream_alloc(&qbuf.p, 2 * qbytes, s);
      if (e == hipSuccess) e = stream_alloc(&nbuf.p, 2 * nbytes, s);
      if (e == hipSuccess) e = hipMemsetAsync(qbuf.p, 0, qbytes, s);
      if (e == hipSuccess)
        e = hipMemcpyAsync((char*)qbuf.p + qbytes, Q_up, qbytes, hipMemcpyDeviceToDevice, s);
      if (e == hipSuccess) e = hipMemcpyAsync(nbuf.p, nu_prev, nbytes, hipMemcpyDeviceToDevice, s);
      if (e == hipSuccess)
        e = hipMemcpyAsync((char*)nbuf.p + nbytes, nu, nbytes, hipMemcpyDeviceToDevice, s);
      if (e != hipSuccess) {
        score_workspace_destroy(&ws);
        return fail(DTP_ERR_HIP, "staging the two-layer view failed: %s", hipGetErrorString(e));
      }
      qu = (const int64_t*)qbuf.p;
      nl = (const int32_t*)nbuf.p;
    }
    st = launch_partition_scores(ws, qu, nl, Q_down_prev, nl, minimise, s);
    if (st == DTP_OK) {
      const int layer = down ? 1 : 0;
      hipError_t e = hipMemcpyAsync(scores, ws.scores + (size_t)layer * P, sizeof(int64_t) * P,
                                    hipMemcpyDeviceToDevice, s);
      if (e == hipSuccess)
        e = hipMemcpyAsync(best_rank, ws.best + layer, sizeof(int64_t), hipMemcpyDeviceToHost, s);
      if (e == hipSuccess) e = hipStreamSynchronize(s);
      if (e != hipSuccess) st = fail(DTP_ERR_HIP, "partition scoring failed: %s", hipGetErrorString(e));
    }
    score_workspace_destroy(&ws);
    return st;
  });
}

dtp_status dtp_coordinate_ascent(int32_t N, int32_t G, int32_t I, int32_t L, const float* A_up,
                                 const float* A_down, const dtp_ca_options* options, int32_t* h,
                                 int32_t* nu, double* J, int64_t* J_fixed, int32_t* sweeps,
                                 void* stream) {
  return guarded([&]() -> dtp_status {
    clear_error();
    DTP_CHECK(N >= 1, DTP_ERR_INVALID_ARG, "N=%d must be >= 1", N);
    dtp_status st = check_layout_sizes(G, I, L, kMaxAssignDevices);
    if (st != DTP_OK) return st;
    DTP_CHECK(A_up && h && nu && J && J_fixed && sweeps, DTP_ERR_INVALID_ARG,
              "a required pointer is NULL");
    DTP_CHECK(A_down == nullptr || N >= 2, DTP_ERR_INVALID_ARG, "A_down needs N >= 2");
    dtp_ca_options opt = {64, 0, 0, 0, nullptr, 0};
    if (options) opt = *options;
    DTP_CHECK(opt.max_sweeps >= 1, DTP_ERR_INVALID_ARG, "max_sweeps=%d must be >= 1",
              opt.max_sweeps);
    const int64_t P = count_partitions(G, L);
    DTP_CHECK(P > 0 && P <= kMaxPartitions, DTP_ERR_UNSUPPORTED, "too many partitions (%lld)",
              (long long)P);
    const bool has_down = A_down != nullptr;
    const size_t nup = (size_t)N * G * I, ndown = has_down ? (size_t)(N - 1) * I * G : 0;
    if ((st = check_dev_buffer(A_up, sizeof(float) * nup, "A_up")) != DTP_OK ||
        (st = check_dev_buffer(A_down, sizeof(float) * ndown, "A_down", true)) != DTP_OK)
      return st;
    hipStream_t s = (hipStream_t)stream;

    // Unit-mass codes of every matrix, computed on the device where the head step reads
    // them; the host copy feeds the neuron step and J.  Layout of the scratch block:
    // [encode stats | Q_up | Q_down | nu].
    const int nmat = N + (has_down ? N - 1 : 0);
    const size_t st_bytes = sizeof(EncodeStats) * nmat;
    const size_t qu_bytes = sizeof(int64_t) * nup, qd_bytes = sizeof(int64_t) * ndown;
    DevBuf block(s);
    DTP_HIP(stream_alloc(&block.p, st_bytes + qu_bytes + qd_bytes + sizeof(int32_t) * (size_t)N * I, s));
    EncodeStats* st_dev = (EncodeStats*)block.p;
    int64_t* qu_dev = (int64_t*)((char*)block.p + st_bytes);
    int64_t* qd_dev = has_down ? qu_dev + nup : nullptr;
    int32_t* nu_dev = (int32_t*)((char*)qu_dev + qu_bytes + qd_bytes);
    st = launch_encode_unit_mass(A_up, N, A_down, has_down ? N - 1 : 0, (int64_t)G * I, qu_dev,
                                 qd_dev, st_dev, s);
    if (st != DTP_OK) return st;
    // Host mirror of [encode stats | Q_up | Q_down], then the staging of the uploaded nu and
    // of the best ranks, in pinned memory: one copy brings the stats and codes back.
    const size_t nu_bytes = sizeof(int32_t) * (size_t)N * I;
    const size_t best_off = (st_bytes + qu_bytes + qd_bytes + nu_bytes + 7) / 8 * 8;
    HostStaging host(best_off + sizeof(int64_t) * (size_t)N);
    const EncodeStats* stats = (const EncodeStats*)host.base;
    const int64_t* Qu = (const int64_t*)(host.base + st_bytes);
    const int64_t* Qd = has_down ? Qu + nup : nullptr;
    int32_t* nu_host = (int32_t*)(host.base + st_bytes + qu_bytes + qd_bytes);
    const int64_t* best = (const int64_t*)(host.base + best_off);
    DTP_HIP(hipMemcpyAsync(host.base, block.p, st_bytes + qu_bytes + qd_bytes, hipMemcpyDeviceToHost, s));
    // The partition table is enumerated and queued while the stream encodes.  Every return
    // below synchronises the stream before the guard releases the table's host copy.
    ScoreWorkspace ws;
    st = score_workspace_create(&ws, N, G, I, L, s);
    struct WsGuard {
      ScoreWorkspace* w;
      hipStream_t s;
      ~WsGuard() {
        (void)hipStreamSynchronize(s);
        score_workspace_destroy(w);
      }
    } guard{&ws, s};
    if (st != DTP_OK) return st;
    DTP_HIP(hipStreamSynchronize(s));
    for (int m = 0; m < nmat; ++m) {
      st = m < N ? check_encode_stats(stats[m], "up affinity of layer", m)
                 : check_encode_stats(stats[m], "down affinity of layer", m - N);
      if (st != DTP_OK) return st;
    }
    const std::vector<uint8_t>& table = ws.host_table;

    // Contiguous start.
    std::vector<int32_t> hs((size_t)N * G), nus((size_t)N * I);
    for (int i = 0; i < N; ++i) {
      for (int g = 0; g < G; ++g) hs[(size_t)i * G + g] = g / (G / L);
      for (int k = 0; k < I; ++k) nus[(size_t)i * I + k] = k / (I / L);
    }
    auto moves = [&](int i) { return opt.layer_mask == nullptr || opt.layer_mask[i] != 0; };
    const bool minimise = opt.minimise != 0;
    int64_t J_prev = 0;
    int sweep = 0;
    while (sweep < opt.max_sweeps) {
      ++sweep;
      if (!opt.freeze_neurons) {
        // Neuron block: layers are independent given the heads; solve them in parallel.
        const unsigned hw = std::max(1u, std::thread::hardware_concurrency());
        const int nthreads = (int)std::min<unsigned>(hw, (unsigned)N);
        auto work = [&](int t) {
          std::vector<int64_t> M;
          for (int i = t; i < N; i += nthreads) {
            if (!moves(i)) continue;
            const bool dn = has_down && i + 1 < N;
            neuron_gain(G, I, L, Qu + (size_t)i * G * I, hs.data() + (size_t)i * G,
                        dn ? Qd + (size_t)i * I * G : nullptr,
                        dn ? hs.data() + (size_t)(i + 1) * G : nullptr, minimise, &M);
            if (opt.dual_ascent_neurons)
              balanced_assign_dual_ascent(I, L, M.data(), kDualAscentIterations, kDualAscentDecay,
                                          nus.data() + (size_t)i * I, nullptr);
            else
              balanced_assign_exact(I, L, M.data(), nus.data() + (size_t)i * I, nullptr);
          }
        };
        if (nthreads == 1) {
          work(0);
        } else {
          std::vector<std::thread> pool;
          for (int t = 0; t < nthreads; ++t) pool.emplace_back(work, t);
          for (auto& th : pool) th.join();
        }
      }
      if (!opt.freeze_heads) {
        // staged: the previous sweep's upload from nu_host ended at its synchronisation
        std::memcpy(nu_host, nus.data(), nu_bytes);
        DTP_HIP(hipMemcpyAsync(nu_dev, nu_host, nu_bytes, hipMemcpyHostToDevice, s));
        st = launch_partition_scores(ws, qu_dev, nu_dev, qd_dev, nu_dev, minimise ? 1 : 0, s);
        if (st != DTP_OK) return st;
        DTP_HIP(hipMemcpyAsync((void*)best, ws.best, sizeof(int64_t) * N, hipMemcpyDeviceToHost, s));
        DTP_HIP(hipStreamSynchronize(s));
        for (int i = 0; i < N; ++i) {
          if (!moves(i)) continue;
          DTP_CHECK(best[i] >= 0 && best[i] < P, DTP_ERR_HIP, "partition scoring returned rank %lld",
                    (long long)best[i]);
          for (int g = 0; g < G; ++g) hs[(size_t)i * G + g] = table[(size_t)best[i] * G + g];
        }
      }
      const int64_t Jc = objective_int(N, G, I, Qu, Qd, has_down, hs.data(), nus.data());
      const bool improved = sweep == 1 || (minimise ? Jc < J_prev : Jc > J_prev);
      J_prev = Jc;
      if (!improved) break;
    }
    // The uploads read host memory that is released on return.
    DTP_HIP(hipStreamSynchronize(s));
    std::memcpy(h, hs.data(), sizeof(int32_t) * hs.size());
    std::memcpy(nu, nus.data(), sizeof(int32_t) * nus.size());
    *J_fixed = J_prev;
    *J = (double)J_prev / (double)(int64_t(1) << kFracBits);
    *sweeps = sweep;
    return DTP_OK;
  });
}

dtp_status dtp_random_layout(int32_t N, int32_t G, int32_t I, int32_t L, uint64_t seed,
                             int32_t* h, int32_t* nu) {
  return guarded([&]() -> dtp_status {
    clear_error();
    DTP_CHECK(N >= 1, DTP_ERR_INVALID_ARG, "N=%d must be >= 1", N);
    dtp_status st = check_layout_sizes(G, I, L, kMaxGroups);
    if (st != DTP_OK) return st;
    DTP_CHECK(h && nu, DTP_ERR_INVALID_ARG, "h or nu is NULL");
    uint64_t counter = 0;
    for (int i = 0; i < N; ++i) {
      int32_t* hi = h + (size_t)i * G;
      int32_t* ni = nu + (size_t)i * I;
      for (int g = 0; g < G; ++g) hi[g] = g / (G / L);
      shuffle(hi, G, seed, &counter);
      for (int k = 0; k < I; ++k) ni[k] = k / (I / L);
      shuffle(ni, I, seed, &counter);
    }
    return DTP_OK;
  });
}

dtp_status dtp_layout_objective(int32_t N, int32_t G, int32_t I, int32_t L, const int64_t* Q_up,
                                const int64_t* Q_down, const int32_t* h, const int32_t* nu,
                                int64_t* J_fixed) {
  return guarded([&]() -> dtp_status {
    clear_error();
    DTP_CHECK(N >= 1, DTP_ERR_INVALID_ARG, "N=%d must be >= 1", N);
    dtp_status st = check_layout_sizes(G, I, L, kMaxGroups);
    if (st != DTP_OK) return st;
    DTP_CHECK(Q_up && h && nu && J_fixed, DTP_ERR_INVALID_ARG, "a required pointer is NULL");
    DTP_CHECK(Q_down == nullptr || N >= 2, DTP_ERR_INVALID_ARG, "Q_down needs N >= 2");
    for (int i = 0; i < N; ++i) {
      if ((st = check_balanced(h + (size_t)i * G, G, L, "h")) != DTP_OK) return st;
      std::vector<int32_t> cnt(L, 0);
      for (int k = 0; k < I; ++k) {
        const int32_t l = nu[(size_t)i * I + k];
        DTP_CHECK(l >= 0 && l < L, DTP_ERR_INVALID_ARG, "nu[%d][%d] = %d is not a device", i, k, l);
        ++cnt[l];
      }
      for (int l = 0; l < L; ++l)
        DTP_CHECK(cnt[l] == I / L, DTP_ERR_INVALID_ARG, "nu[%d] is not balanced", i);
    }
    *J_fixed = objective_int(N, G, I, Q_up, Q_down, Q_down != nullptr, h, nu);
    return DTP_OK;
  });
}

dtp_status dtp_layer_optimum(int32_t G, int32_t I, int32_t L, const int64_t* Q_up, int32_t* h,
                             int32_t* nu, int64_t* J_fixed) {
  return guarded([&]() -> dtp_status {
    clear_error();
    dtp_status st = check_layout_sizes(G, I, L, kMaxAssignDevices);
    if (st != DTP_OK) return st;
    DTP_CHECK(Q_up && h && nu && J_fixed, DTP_ERR_INVALID_ARG, "a required pointer is NULL");
    const int64_t P = count_partitions(G, L);
    DTP_CHECK(P > 0 && P <= kMaxPartitions, DTP_ERR_UNSUPPORTED, "too many partitions (%lld)",
              (long long)P);
    // One representative per partition up to device relabelling: labels first appear in
    // the order 0, 1, ..., L-1.
    const std::vector<uint8_t> table = enumerate_partitions(G, L);
    std::vector<int64_t> reps;
    for (int64_t r = 0; r < P; ++r) {
      const uint8_t* hp = table.data() + (size_t)r * G;
      int next = 0;
      bool ok = true;
      for (int g = 0; g < G && ok; ++g) {
        if (hp[g] > next) ok = false;
        else if (hp[g] == next) ++next;
      }
      if (ok) reps.push_back(r);
    }
    std::vector<int64_t> value(reps.size());
    std::vector<std::vector<int32_t>> nus(reps.size(), std::vector<int32_t>(I));
    auto solve = [&](size_t j) {
      int32_t hh[kMaxGroups];
      for (int g = 0; g < G; ++g) hh[g] = table[(size_t)reps[j] * G + g];
      std::vector<int64_t> M;
      neuron_gain(G, I, L, Q_up, hh, nullptr, nullptr, false, &M);
      balanced_assign_exact(I, L, M.data(), nus[j].data(), &value[j]);
    };
    const unsigned hw = std::max(1u, std::min(16u, std::thread::hardware_concurrency()));
    std::vector<std::thread> pool;
    for (unsigned t = 0; t < hw; ++t)
      pool.emplace_back([&, t] {
        for (size_t j = t; j < reps.size(); j += hw) solve(j);
      });
    for (auto& th : pool) th.join();
    size_t best = 0;  // first partition (lexicographic) attaining the maximum
    for (size_t j = 1; j < reps.size(); ++j)
      if (value[j] > value[best]) best = j;
    for (int g = 0; g < G; ++g) h[g] = table[(size_t)reps[best] * G + g];
    std::copy(nus[best].begin(), nus[best].end(), nu);
    *J_fixed = value[best];
    return DTP_OK;
  });
}

}  // extern "C"
