// Internal declarations shared by the translation units of libdtp.so.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <exception>
#include <new>
#include <string>
#include <vector>

#include "dtp.h"

namespace dtp {

// Records a thread-local message for dtp_last_error() and returns `s`.
dtp_status fail(dtp_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

// A caller's device buffer: `p` must be memory of the current HIP device whose allocation
// holds at least `bytes` from `p` on.  A host pointer, another device's memory or a short
// allocation would make a kernel read or write outside what the caller owns, so every
// entry point checks its device arguments this way before enqueueing work.  NULL is
// accepted when `optional` (the argument is then unused).
dtp_status check_dev_buffer(const void* p, size_t bytes, const char* what, bool optional = false);

// Runs an entry point's body and turns any C++ exception (a host allocation, a thread the
// neuron step could not start) into a status, so that nothing unwinds through the C ABI.
template <typename F>
dtp_status guarded(F&& body) noexcept {
  try {
    return body();
  } catch (const std::bad_alloc&) {
    return fail(DTP_ERR_NO_MEMORY, "host memory allocation failed");
  } catch (const std::exception& e) {
    return fail(DTP_ERR_NO_MEMORY, "host resource failure: %s", e.what());
  } catch (...) {
    return fail(DTP_ERR_NO_MEMORY, "unexpected host failure");
  }
}

#define DTP_HIP(call)                                                                 \
  do {                                                                                \
    hipError_t e_ = (call);                                                           \
    if (e_ != hipSuccess)                                                             \
      return ::dtp::fail(DTP_ERR_HIP, "%s failed: %s (%s:%d)", #call,                 \
                         hipGetErrorString(e_), __FILE__, __LINE__);                  \
  } while (0)

#define DTP_CHECK(cond, status, ...)                                                  \
  do {                                                                                \
    if (!(cond)) return ::dtp::fail((status), __VA_ARGS__);                           \
  } while (0)

constexpr int kMaxGroups = 64;        // partition scoring: one lane per KV group
constexpr int kMaxAffinityGroups = 32;  // affinity kernel: per-group sums kept in LDS
constexpr int kMaxAssignDevices = 8;  // exact assignment: Hall checks over 2^L subsets
constexpr int64_t kMaxPartitions = int64_t(1) << 24;
constexpr int kFracBits = 48;
constexpr int kMantBits = 40;

// ---- stream-ordered scratch (abi.cpp): hipMallocAsync / hipFreeAsync from the device's
// default pool, which is told once per device to keep freed memory, so per-call scratch
// costs neither a device-wide synchronisation nor a trip to the driver.
hipError_t stream_alloc(void** p, size_t bytes, hipStream_t s);
hipError_t stream_free(void* p, hipStream_t s);

// ---- unit-mass fixed point (encode.cpp)
dtp_status encode_unit_mass(const float* A, int64_t n, int64_t* Q);

// ---- the same codes on the GPU (encode_device.hip), for n_up + n_down matrices of n
// entries: matrix m < n_up reads A_up + m n and writes Q_up + m n, the others A_down and
// Q_down.  Enqueues on `s`; stats (device, one per matrix) says, once the stream has run,
// whether each matrix was encodable (check_encode_stats on a host copy); the codes of a
// matrix that was not are left unwritten.
struct EncodeStats {
  unsigned long long maxbits;  // fp32 bits of the largest entry
  unsigned long long badidx;   // smallest index of a negative or non-finite entry, or ~0
  unsigned long long s_lo, s_hi;  // sum of the q codes, 128-bit
};
dtp_status launch_encode_unit_mass(const float* A_up, int n_up, const float* A_down, int n_down,
                                   int64_t n, int64_t* Q_up, int64_t* Q_down, EncodeStats* stats,
                                   hipStream_t s);
dtp_status check_encode_stats(const EncodeStats& st, const char* what, int index);

// ---- labelled balanced partitions (partitions.cpp)
int64_t count_partitions(int G, int L);               // -1 if invalid or > 2^62
std::vector<uint8_t> enumerate_partitions(int G, int L);  // [P][G], lexicographic
bool unrank_partition(int G, int L, int64_t rank, int32_t* h);

// ---- exact balanced assignment (assign.cpp).  M is [I][L] row-major.
// Returns the lexicographically smallest assignment maximising sum_k M[k][nu[k]].
void balanced_assign_exact(int I, int L, const int64_t* M, int32_t* nu, int64_t* value);
// The paper's approximate solver (dual ascent on device offsets, capacity fix-up, pairwise
// swaps); balanced, never above the optimum, exact when L = 2.
void balanced_assign_dual_ascent(int I, int L, const int64_t* M, int iterations, double decay,
                                 int32_t* nu, int64_t* value);
constexpr int kDualAscentIterations = 300;
constexpr double kDualAscentDecay = 0.98;

// ---- GPU partition scoring (scores.hip)
struct ScoreWorkspace {
  int N = 0, G = 0, I = 0, L = 0;
  int64_t P = 0;
  hipStream_t stream = nullptr;    // the allocation and its release are ordered on it
  std::vector<uint8_t> host_table;  // source of the table upload, kept until release
  uint8_t* table = nullptr;   // dev [P][G]
  int64_t* C = nullptr;       // dev [N][G][L]
  int64_t* scores = nullptr;  // dev [N][P]
  int64_t* best = nullptr;    // dev [N]
};
dtp_status score_workspace_create(ScoreWorkspace* ws, int N, int G, int I, int L, hipStream_t s);
void score_workspace_destroy(ScoreWorkspace* ws);
// Q_up dev [N][G][I]; nu dev [N][I]; Q_down dev [N-1][I][G] or null (layer i uses
// Q_down[i-1] with nu[i-1]).  Enqueues C, scores and best on `stream`.
dtp_status launch_partition_scores(const ScoreWorkspace& ws, const int64_t* Q_up,
                                   const int32_t* nu, const int64_t* Q_down,
                                   const int32_t* nu_down, int minimise, hipStream_t stream);

}  // namespace dtp
