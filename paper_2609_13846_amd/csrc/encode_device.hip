// Unit-mass fixed-point codes of affinity matrices on the GPU (Section 3, "Objective":
// each matrix is normalised to unit mass before co-located entries are summed).
//
// The same integers as the host encoder: with E = floor(log2 max A),
//   q_i = floor(A_i * 2^(40 - E))        exact in fp64, q_i < 2^41
//   S   = sum_i q_i                      exact, 128-bit
//   Q_i = floor(q_i * 2^48 / S)          fp64 estimate, then exact 128-bit correction
// The maximum, the first bad index and S are integer reductions (atomic max / min / add on
// 64-bit words, the add carrying into a second word), so the result does not depend on
// the order in which blocks finish.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "dtp_internal.h"

namespace dtp {
namespace {

constexpr int kEncThreads = 256;
constexpr unsigned long long kNoBad = ~0ull;

__device__ __forceinline__ const float* matrix_in(const float* A_up, const float* A_down, int nup,
                                                  int64_t n, int m) {
  return m < nup ? A_up + (int64_t)m * n : A_down + (int64_t)(m - nup) * n;
}

__device__ __forceinline__ int64_t* matrix_out(int64_t* Q_up, int64_t* Q_down, int nup, int64_t n,
                                               int m) {
  return m < nup ? Q_up + (int64_t)m * n : Q_down + (int64_t)(m - nup) * n;
}

__device__ __forceinline__ unsigned long long shfl_xor_u64(unsigned long long v, int off) {
  const unsigned lo = __shfl_xor((unsigned)(v & 0xffffffffull), off, 64);
  const unsigned hi = __shfl_xor((unsigned)(v >> 32), off, 64);
  return ((unsigned long long)hi << 32) | lo;
}

__global__ void encode_init_kernel(EncodeStats* st, int count) {
  const int m = blockIdx.x * blockDim.x + threadIdx.x;
  if (m < count) {
    st[m].maxbits = 0;
    st[m].badidx = kNoBad;
    st[m].s_lo = 0;
    st[m].s_hi = 0;
  }
}

// Per matrix (blockIdx.y): the largest entry (as fp32 bits, which order like the values for
// entries >= 0) and the smallest index of a negative or non-finite entry.
__global__ void __launch_bounds__(kEncThreads)
encode_stats_kernel(const float* __restrict__ A_up, const float* __restrict__ A_down, int nup,
                    int64_t n, EncodeStats* st) {
  const int m = blockIdx.y;
  const float* A = matrix_in(A_up, A_down, nup, n, m);
  unsigned long long mx = 0, bad = kNoBad;
  for (int64_t i = (int64_t)blockIdx.x * kEncThreads + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * kEncThreads) {
    const float a = A[i];
    if (!(a >= 0.0f) || !isfinite(a))  // NaN fails the comparison
      bad = min(bad, (unsigned long long)i);
    else
      mx = max(mx, (unsigned long long)(__float_as_uint(a) & 0x7fffffffu));  // -0 counts as 0
  }
  for (int off = 32; off > 0; off >>= 1) {
    mx = max(mx, shfl_xor_u64(mx, off));
    bad = min(bad, shfl_xor_u64(bad, off));
  }
  if ((threadIdx.x & 63) == 0) {
    if (mx) atomicMax(&st[m].maxbits, mx);
    if (bad != kNoBad) atomicMin(&st[m].badidx, bad);
  }
}

__device__ __forceinline__ bool encodable(const EncodeStats& s) {
  return s.badidx == kNoBad && s.maxbits != 0;
}

// q_i into Q, and S = sum q_i: per-wave sums (at most 65 x 64 codes below 2^41, so under
// 2^54 at the grid sizes of blocks_for) added to the
// low word of S, a wrap of the low word adding one to the high word.
__global__ void __launch_bounds__(kEncThreads)
encode_q_kernel(const float* __restrict__ A_up, const float* __restrict__ A_down, int nup,
                int64_t n, EncodeStats* st, int64_t* Q_up, int64_t* Q_down) {
  const int m = blockIdx.y;
  if (!encodable(st[m])) return;
  const float* A = matrix_in(A_up, A_down, nup, n, m);
  int64_t* Q = matrix_out(Q_up, Q_down, nup, n, m);
  int e = 0;
  (void)frexp((double)__uint_as_float((unsigned)st[m].maxbits), &e);  // max = f 2^e, f in [0.5, 1)
  const double p2 = ldexp(1.0, kMantBits - (e - 1));
  unsigned long long sum = 0;
  for (int64_t i = (int64_t)blockIdx.x * kEncThreads + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * kEncThreads) {
    const unsigned long long q = (unsigned long long)(int64_t)((double)A[i] * p2);  // floor, >= 0
    Q[i] = (int64_t)q;
    sum += q;
  }
  for (int off = 32; off > 0; off >>= 1) sum += shfl_xor_u64(sum, off);
  if ((threadIdx.x & 63) == 0 && sum) {
    const unsigned long long old = atomicAdd(&st[m].s_lo, sum);
    if (old + sum < old) atomicAdd(&st[m].s_hi, 1ull);
  }
}

struct U128 {
  unsigned long long lo, hi;
};

__device__ __forceinline__ bool less_eq(U128 a, U128 b) {
  return a.hi < b.hi || (a.hi == b.hi && a.lo <= b.lo);
}

__device__ __forceinline__ U128 add(U128 a, U128 b) {
  U128 r;
  r.lo = a.lo + b.lo;
  r.hi = a.hi + b.hi + (r.lo < a.lo ? 1ull : 0ull);
  return r;
}

__device__ __forceinline__ U128 sub(U128 a, U128 b) {  // a >= b
  U128 r;
  r.lo = a.lo - b.lo;
  r.hi = a.hi - b.hi - (a.lo < b.lo ? 1ull : 0ull);
  return r;
}

// Q_i = floor(q_i 2^48 / S): c from fp64, then c * S <= q_i 2^48 < (c + 1) * S enforced.
__global__ void __launch_bounds__(kEncThreads)
encode_div_kernel(int nup, int64_t n, const EncodeStats* st, int64_t* Q_up, int64_t* Q_down) {
  const int m = blockIdx.y;
  if (!encodable(st[m])) return;
  int64_t* Q = matrix_out(Q_up, Q_down, nup, n, m);
  const U128 S = {st[m].s_lo, st[m].s_hi};  // S < 2^72: n <= 2^30 entries below 2^41 each
  const double scale = ldexp(1.0, kFracBits) / ((double)S.hi * 18446744073709551616.0 + (double)S.lo);
  for (int64_t i = (int64_t)blockIdx.x * kEncThreads + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * kEncThreads) {
    const unsigned long long q = (unsigned long long)Q[i];
    const U128 num = {q << kFracBits, q >> (64 - kFracBits)};
    unsigned long long c = (unsigned long long)((double)q * scale);
    U128 prod = {c * S.lo, __umul64hi(c, S.lo) + c * S.hi};  // c <= 2^48, so c S < 2^120
    while (!less_eq(prod, num)) {
      --c;
      prod = sub(prod, S);
    }
    for (U128 next = add(prod, S); less_eq(next, num); next = add(prod, S)) {
      ++c;
      prod = next;
    }
    Q[i] = (int64_t)c;
  }
}

unsigned blocks_for(int64_t n) {
  // About 4 entries per thread (a layer's G x I matrix then spreads over tens of CUs
  // instead of a few, whose threads would wait on their loads one after another), and at
  // most 65535 blocks: a thread then sums at most 2^30 / (65535 * 256) + 1 = 65 codes
  // below 2^41 each.
  const int64_t b = (n + kEncThreads * 4 - 1) / (kEncThreads * 4);
  return (unsigned)std::max<int64_t>(1, std::min<int64_t>(b, 65535));
}

}  // namespace

dtp_status launch_encode_unit_mass(const float* A_up, int n_up, const float* A_down, int n_down,
                                   int64_t n, int64_t* Q_up, int64_t* Q_down, EncodeStats* stats,
                                   hipStream_t s) {
  const int count = n_up + n_down;
  DTP_CHECK(n >= 1 && n <= (int64_t(1) << 30), DTP_ERR_UNSUPPORTED,
            "matrix of %lld entries (1 to 2^30 supported)", (long long)n);
  DTP_CHECK(count >= 1 && count <= 65535, DTP_ERR_UNSUPPORTED, "%d matrices (1 to 65535)", count);
  encode_init_kernel<<<(count + 255) / 256, 256, 0, s>>>(stats, count);
  const dim3 grid(blocks_for(n), (unsigned)count);
  encode_stats_kernel<<<grid, kEncThreads, 0, s>>>(A_up, A_down, n_up, n, stats);
  encode_q_kernel<<<grid, kEncThreads, 0, s>>>(A_up, A_down, n_up, n, stats, Q_up, Q_down);
  encode_div_kernel<<<grid, kEncThreads, 0, s>>>(n_up, n, stats, Q_up, Q_down);
  DTP_HIP(hipGetLastError());
  return DTP_OK;
}

dtp_status check_encode_stats(const EncodeStats& st, const char* what, int index) {
  if (st.badidx != kNoBad)
    return fail(DTP_ERR_DEGENERATE, "%s %d: affinity entry %llu is negative or not finite", what,
                index, st.badidx);
  if (st.maxbits == 0) return fail(DTP_ERR_DEGENERATE, "%s %d: affinity matrix is all zero", what, index);
  return DTP_OK;
}

}  // namespace dtp
