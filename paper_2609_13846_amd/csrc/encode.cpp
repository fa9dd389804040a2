// Unit-mass normalisation of an affinity matrix as exact fixed point.
//
// The paper normalises every affinity matrix to unit mass before summing co-located
// entries into the objective J (Section 3, "Objective").  To make J, the head-partition
// scores and the neuron gains independent of summation order, the library carries the
// normalised matrix as integers:
//   E   = floor(log2 max A)
//   q_i = floor(A_i * 2^(40 - E))        exact: A_i is an fp32 value, q_i < 2^41
//   Q_i = floor(q_i * 2^48 / sum_j q_j)  128-bit intermediate
// so sum_i Q_i lies in (2^48 - n, 2^48] and J = (sum of co-located Q) / 2^48.
#include <cmath>
#include <cstring>

#include "dtp_internal.h"

namespace dtp {

dtp_status encode_unit_mass(const float* A, int64_t n, int64_t* Q) {
  float amax = 0.0f;
  for (int64_t i = 0; i < n; ++i) {
    const float a = A[i];
    if (!std::isfinite(a) || a < 0.0f)
      return fail(DTP_ERR_DEGENERATE, "affinity entry %lld is %g (must be finite and >= 0)",
                  (long long)i, (double)a);
    if (a > amax) amax = a;
  }
  if (!(amax > 0.0f)) return fail(DTP_ERR_DEGENERATE, "affinity matrix is all zero");
  int e = 0;
  std::frexp(amax, &e);  // amax = m * 2^e, m in [0.5, 1)
  const int E = e - 1;   // amax in [2^E, 2^(E+1))
  // Scaling an fp32 value by a power of two is exact in fp64 (the product is below 2^41,
  // and one that underflows truncates to 0 either way); truncation is floor for x >= 0.
  const double p2 = std::ldexp(1.0, kMantBits - E);
  unsigned __int128 S = 0;
  for (int64_t i = 0; i < n; ++i) {
    Q[i] = (int64_t)((double)A[i] * p2);  // temporarily q_i
    S += (unsigned __int128)(uint64_t)Q[i];
  }
  // floor(q * 2^48 / S): a double estimate (within a few units), then an exact integer
  // correction.
  const double scale = std::ldexp(1.0, kFracBits) / (double)S;
  for (int64_t i = 0; i < n; ++i) {
    const unsigned __int128 num = (unsigned __int128)(uint64_t)Q[i] << kFracBits;
    uint64_t c = (uint64_t)((double)Q[i] * scale);
    while ((unsigned __int128)c * S > num) --c;
    while ((unsigned __int128)(c + 1) * S <= num) ++c;
    Q[i] = (int64_t)c;
  }
  return DTP_OK;
}

}  // namespace dtp
