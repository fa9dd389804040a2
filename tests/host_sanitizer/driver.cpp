// Checks of the library's host code under AddressSanitizer and UndefinedBehaviorSanitizer.
// tests/test_host_sanitizer.py builds this file with the host sources of libdtp.so (g++,
// no GPU) and runs it.  The GPU launchers that the host sources call are stubbed out
// below.  Every host entry point runs on seeded random and tie-heavy inputs, small
// instances are checked against brute force, and the argument errors the ABI must reject
// are exercised.  A failed check prints its case and exits non-zero; a memory error or
// undefined behaviour aborts through the sanitizers.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <limits>
#include <vector>

#include "dtp.h"
#include "dtp_internal.h"

namespace dtp {
// The GPU side of the coordinate ascent and of the device encoder, absent here.
dtp_status launch_encode_unit_mass(const float*, int, const float*, int, int64_t, int64_t*,
                                   int64_t*, EncodeStats*, hipStream_t) {
  return fail(DTP_ERR_UNSUPPORTED, "no GPU in the host-only build");
}
dtp_status check_encode_stats(const EncodeStats&, const char*, int) {
  return fail(DTP_ERR_UNSUPPORTED, "no GPU in the host-only build");
}
dtp_status score_workspace_create(ScoreWorkspace*, int, int, int, int, hipStream_t) {
  return fail(DTP_ERR_UNSUPPORTED, "no GPU in the host-only build");
}
void score_workspace_destroy(ScoreWorkspace* ws) { *ws = ScoreWorkspace(); }
dtp_status launch_partition_scores(const ScoreWorkspace&, const int64_t*, const int32_t*,
                                   const int64_t*, const int32_t*, int, hipStream_t) {
  return fail(DTP_ERR_UNSUPPORTED, "no GPU in the host-only build");
}
}  // namespace dtp

namespace {

int g_checks = 0;

#define CHECK(cond, ...)                                                 \
  do {                                                                   \
    ++g_checks;                                                          \
    if (!(cond)) {                                                       \
      std::fprintf(stderr, "FAILED %s:%d: %s: ", __FILE__, __LINE__, #cond); \
      std::fprintf(stderr, __VA_ARGS__);                                 \
      std::fprintf(stderr, "\n");                                        \
      std::exit(1);                                                      \
    }                                                                    \
  } while (0)

// SplitMix64 (Steele, Lea and Flood, 2014): the seeded source of every input here.
struct Rng {
  uint64_t s;
  uint64_t next() {
    uint64_t z = (s += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
  }
  int below(int n) { return (int)(next() % (uint64_t)n); }
  double unit() { return (double)(next() >> 11) * 0x1.0p-53; }
};

bool balanced(const int32_t* a, int n, int L) {
  std::vector<int> c(L, 0);
  for (int i = 0; i < n; ++i) {
    if (a[i] < 0 || a[i] >= L) return false;
    ++c[a[i]];
  }
  for (int l = 0; l < L; ++l)
    if (c[l] != n / L) return false;
  return true;
}

// A uniformly shuffled balanced assignment of n items to L devices.
std::vector<int32_t> random_balanced(Rng& r, int n, int L) {
  std::vector<int32_t> a(n);
  for (int i = 0; i < n; ++i) a[i] = i / (n / L);
  for (int i = n - 1; i > 0; --i) std::swap(a[i], a[r.below(i + 1)]);
  return a;
}

// Calls fn on every balanced assignment of n items to L devices, in lexicographic order.
template <typename F>
void each_balanced(int n, int L, F fn) {
  std::vector<int32_t> a(n);
  std::vector<int> left(L, n / L);
  auto rec = [&](auto&& self, int i) -> void {
    if (i == n) {
      fn(a);
      return;
    }
    for (int l = 0; l < L; ++l)
      if (left[l] > 0) {
        --left[l];
        a[i] = l;
        self(self, i + 1);
        ++left[l];
      }
  };
  rec(rec, 0);
}

int64_t multinomial(int G, int L) {  // G! / ((G/L)!)^L, small G
  int64_t r = 1;
  int used = 0;
  for (int l = 0; l < L; ++l)
    for (int j = 1; j <= G / L; ++j) {
      ++used;
      r = r * used / j;  // exact: r is C(used, j) times an earlier product at each step
    }
  return r;
}

// ---------------------------------------------------------------- partitions
void check_partitions() {
  for (int G = 1; G <= 12; ++G)
    for (int L = 1; L <= G; ++L) {
      const int64_t P = dtp_partition_count(G, L);
      if (G % L) {
        CHECK(P == -1, "G=%d L=%d count %lld", G, L, (long long)P);
        continue;
      }
      CHECK(P == multinomial(G, L), "G=%d L=%d count %lld", G, L, (long long)P);
      std::vector<int32_t> h(G), prev(G);
      const int64_t n = std::min<int64_t>(P, 20000);
      for (int64_t r = 0; r < n; ++r) {
        CHECK(dtp_partition_unrank(G, L, r, h.data()) == DTP_OK, "unrank G=%d L=%d r=%lld", G, L,
              (long long)r);
        CHECK(balanced(h.data(), G, L), "unbalanced G=%d L=%d r=%lld", G, L, (long long)r);
        if (r == 0)
          for (int g = 0; g < G; ++g) CHECK(h[g] == g / (G / L), "rank 0 not contiguous G=%d L=%d", G, L);
        else
          CHECK(std::lexicographical_compare(prev.begin(), prev.end(), h.begin(), h.end()),
                "ranks out of order G=%d L=%d r=%lld", G, L, (long long)r);
        prev = h;
      }
      CHECK(dtp_partition_unrank(G, L, P, h.data()) != DTP_OK, "rank P accepted G=%d L=%d", G, L);
      CHECK(dtp_partition_unrank(G, L, -1, h.data()) != DTP_OK, "rank -1 accepted");
      CHECK(dtp_partition_unrank(G, L, 0, nullptr) != DTP_OK, "null h accepted");
    }
  CHECK(dtp_partition_count(8, 0) == -1, "L=0");
  CHECK(dtp_partition_count(65, 5) == -1, "G=65");
}

// ---------------------------------------------------------------- encoding
void check_encode(Rng& r) {
  for (int trial = 0; trial < 300; ++trial) {
    const int n = 1 + r.below(trial < 100 ? 64 : 4096);
    std::vector<float> A(n);
    const int kind = trial % 5;
    for (int i = 0; i < n; ++i) {
      double v = r.unit();
      if (kind == 1) v = std::ldexp(v, r.below(60) - 30);          // wide exponent spread
      if (kind == 2 && r.below(3)) v = 0.0;                          // mostly zeros
      if (kind == 3) v = r.below(2) ? 1e-40 * r.unit() : v * 1e-38;  // subnormals
      if (kind == 4) v = std::ldexp(v, 100);                         // near the fp32 top
      A[i] = (float)v;
    }
    A[r.below(n)] = kind == 3 ? 1e-38f : 1.0f;  // at least one nonzero entry
    std::vector<int64_t> Q(n);
    CHECK(dtp_encode_affinity(A.data(), n, Q.data()) == DTP_OK, "trial %d n=%d", trial, n);
    int64_t sum = 0;
    for (int i = 0; i < n; ++i) {
      CHECK(Q[i] >= 0, "negative code trial %d", trial);
      sum += Q[i];
    }
    const int64_t one = (int64_t)1 << 48;
    CHECK(sum <= one && sum > one - n, "trial %d: sum of codes %lld", trial, (long long)sum);
    for (int t = 0; t < 64; ++t) {
      const int i = r.below(n), j = r.below(n);
      if (A[i] <= A[j]) CHECK(Q[i] <= Q[j], "not monotone trial %d", trial);
    }
    if (kind == 0) {  // a power of two leaves the codes unchanged
      std::vector<float> B(A);
      for (float& v : B) v = std::ldexp(v, 7);
      std::vector<int64_t> QB(n);
      CHECK(dtp_encode_affinity(B.data(), n, QB.data()) == DTP_OK, "scaled trial %d", trial);
      CHECK(QB == Q, "power-of-two scaling changed the codes, trial %d", trial);
    }
  }
  std::vector<float> A(16, 0.0f);
  std::vector<int64_t> Q(16);
  CHECK(dtp_encode_affinity(A.data(), 16, Q.data()) == DTP_ERR_DEGENERATE, "all zero");
  const float bad[3] = {-1.0f, std::numeric_limits<float>::quiet_NaN(),
                        std::numeric_limits<float>::infinity()};
  for (float b : bad) {
    std::fill(A.begin(), A.end(), 1.0f);
    A[5] = b;
    CHECK(dtp_encode_affinity(A.data(), 16, Q.data()) == DTP_ERR_DEGENERATE, "bad entry %g", (double)b);
  }
  CHECK(dtp_encode_affinity(A.data(), 0, Q.data()) == DTP_ERR_INVALID_ARG, "n=0");
  // larger than the documented limit: refused before anything is read
  CHECK(dtp_encode_affinity(A.data(), (1 << 20) + 1, Q.data()) == DTP_ERR_INVALID_ARG, "n > 2^20");
  CHECK(dtp_encode_affinity(nullptr, 16, Q.data()) == DTP_ERR_INVALID_ARG, "null A");
  CHECK(dtp_encode_affinity(A.data(), 16, nullptr) == DTP_ERR_INVALID_ARG, "null Q");
}

// ---------------------------------------------------------------- neuron step
struct AssignCase {
  int G, I, L;
  bool minimise;
  std::vector<int64_t> Qu, Qd;  // [G, I] and [I, G] (empty: no down edge)
  std::vector<int32_t> h, hn;
};

int64_t gain(const AssignCase& c, int k, int l) {
  int64_t m = 0;
  for (int g = 0; g < c.G; ++g) {
    if (c.h[g] == l) m += c.Qu[(size_t)g * c.I + k];
    if (!c.Qd.empty() && c.hn[g] == l) m += c.Qd[(size_t)k * c.G + g];
  }
  return m;
}

AssignCase random_case(Rng& r, int G, int I, int L, bool ties) {
  AssignCase c{G, I, L, r.below(4) == 0, {}, {}, {}, {}};
  const bool down = r.below(2) == 0;
  auto code = [&]() { return ties ? (int64_t)r.below(4) : (int64_t)(r.next() >> 24); };
  c.Qu.resize((size_t)G * I);
  for (auto& v : c.Qu) v = code();
  c.h = random_balanced(r, G, L);
  if (down) {
    c.Qd.resize((size_t)I * G);
    for (auto& v : c.Qd) v = code();
    c.hn = random_balanced(r, G, L);
  }
  return c;
}

void check_assign(Rng& r) {
  const int Ls[] = {1, 2, 3, 4, 8};
  for (int trial = 0; trial < 600; ++trial) {
    const int L = Ls[r.below(5)];
    const int G = L * (1 + r.below(L <= 4 ? 4 : 2));
    const bool small = trial % 2 == 0;
    const int I = small ? L * (1 + r.below(std::max(1, 10 / L))) : L * (1 + r.below(64 / L + 8));
    const bool ties = trial % 3 == 0;
    const AssignCase c = random_case(r, G, I, L, ties);
    const int64_t* qd = c.Qd.empty() ? nullptr : c.Qd.data();
    const int32_t* hn = c.Qd.empty() ? nullptr : c.hn.data();
    std::vector<int32_t> nu(I, -1), nu2(I, -1);
    int64_t value = 0, value2 = 0;
    CHECK(dtp_balanced_assign(G, I, L, c.Qu.data(), c.h.data(), qd, hn, c.minimise, nu.data(), &value) == DTP_OK,
          "trial %d G=%d I=%d L=%d", trial, G, I, L);
    CHECK(balanced(nu.data(), I, L), "trial %d: unbalanced", trial);
    int64_t v = 0;
    for (int k = 0; k < I; ++k) v += gain(c, k, nu[k]);
    CHECK(v == value, "trial %d: value %lld, recomputed %lld", trial, (long long)value, (long long)v);
    if (I <= 10) {  // brute force: the optimum, and the lexicographically smallest optimiser
      int64_t best = c.minimise ? std::numeric_limits<int64_t>::max() : std::numeric_limits<int64_t>::min();
      std::vector<int32_t> arg;
      each_balanced(I, L, [&](const std::vector<int32_t>& a) {
        int64_t s = 0;
        for (int k = 0; k < I; ++k) s += gain(c, k, a[k]);
        if (c.minimise ? s < best : s > best) {
          best = s;
          arg = a;
        }
      });
      CHECK(best == value, "trial %d: optimum %lld, library %lld (G=%d I=%d L=%d min=%d)", trial,
            (long long)best, (long long)value, G, I, L, (int)c.minimise);
      CHECK(arg == nu, "trial %d: not the lexicographically smallest optimiser", trial);
    }
    CHECK(dtp_balanced_assign_dual_ascent(G, I, L, c.Qu.data(), c.h.data(), qd, hn, c.minimise, nu2.data(),
                                          &value2) == DTP_OK,
          "dual ascent trial %d", trial);
    CHECK(balanced(nu2.data(), I, L), "dual ascent trial %d: unbalanced", trial);
    int64_t v2 = 0;
    for (int k = 0; k < I; ++k) v2 += gain(c, k, nu2[k]);
    CHECK(v2 == value2, "dual ascent trial %d: value", trial);
    CHECK(c.minimise ? value2 >= value : value2 <= value, "dual ascent beats the optimum, trial %d", trial);
    if (L == 2) CHECK(value2 == value, "dual ascent trial %d: L = 2 not optimal", trial);
  }
  // argument errors
  std::vector<int64_t> Q(8 * 16, 1);
  std::vector<int32_t> h = {0, 0, 0, 0, 1, 1, 1, 1}, bad = {0, 0, 0, 1, 1, 1, 1, 1}, nu(16);
  int64_t value = 0;
  CHECK(dtp_balanced_assign(8, 16, 2, Q.data(), bad.data(), nullptr, nullptr, 0, nu.data(), &value) ==
            DTP_ERR_INVALID_ARG, "unbalanced h");
  CHECK(dtp_balanced_assign(8, 15, 2, Q.data(), h.data(), nullptr, nullptr, 0, nu.data(), &value) ==
            DTP_ERR_INVALID_ARG, "I %% L");
  CHECK(dtp_balanced_assign(8, 16, 3, Q.data(), h.data(), nullptr, nullptr, 0, nu.data(), &value) ==
            DTP_ERR_INVALID_ARG, "G %% L");
  CHECK(dtp_balanced_assign(8, 16, 0, Q.data(), h.data(), nullptr, nullptr, 0, nu.data(), &value) ==
            DTP_ERR_INVALID_ARG, "L = 0");
  CHECK(dtp_balanced_assign(8, 16, 2, nullptr, h.data(), nullptr, nullptr, 0, nu.data(), &value) ==
            DTP_ERR_INVALID_ARG, "null Q");
  CHECK(dtp_balanced_assign(8, 16, 2, Q.data(), h.data(), Q.data(), nullptr, 0, nu.data(), &value) ==
            DTP_ERR_INVALID_ARG, "Q_down without h_next");
  CHECK(dtp_balanced_assign(8, 16, 2, Q.data(), h.data(), nullptr, nullptr, 0, nullptr, &value) ==
            DTP_ERR_INVALID_ARG, "null nu");
  CHECK(dtp_balanced_assign_dual_ascent(8, 16, 2, Q.data(), bad.data(), nullptr, nullptr, 0, nu.data(),
                                        &value) == DTP_ERR_INVALID_ARG, "dual ascent, unbalanced h");
}

// ---------------------------------------------------------------- layouts and J
void check_layouts(Rng& r) {
  for (int trial = 0; trial < 60; ++trial) {
    const int N = 1 + r.below(4), L = 1 << r.below(3), G = L * (1 + r.below(3)), I = L * (1 + r.below(12));
    const uint64_t seed = r.next();
    std::vector<int32_t> h((size_t)N * G), nu((size_t)N * I), h2(h.size()), nu2(nu.size());
    CHECK(dtp_random_layout(N, G, I, L, seed, h.data(), nu.data()) == DTP_OK, "random layout %d", trial);
    CHECK(dtp_random_layout(N, G, I, L, seed, h2.data(), nu2.data()) == DTP_OK, "random layout %d", trial);
    CHECK(h == h2 && nu == nu2, "random layout %d not reproducible", trial);
    for (int i = 0; i < N; ++i) {
      CHECK(balanced(h.data() + (size_t)i * G, G, L), "random h %d", trial);
      CHECK(balanced(nu.data() + (size_t)i * I, I, L), "random nu %d", trial);
    }
    // J of the layout against the co-located sum written out
    std::vector<int64_t> Qu((size_t)N * G * I), Qd((size_t)(N - 1) * I * G);
    for (auto& v : Qu) v = (int64_t)(r.next() >> 20);
    for (auto& v : Qd) v = (int64_t)(r.next() >> 20);
    const bool down = N > 1 && r.below(2);
    int64_t J = -1;
    CHECK(dtp_layout_objective(N, G, I, L, Qu.data(), down ? Qd.data() : nullptr, h.data(), nu.data(), &J) ==
              DTP_OK, "objective %d", trial);
    int64_t ref = 0;
    for (int i = 0; i < N; ++i)
      for (int g = 0; g < G; ++g)
        for (int k = 0; k < I; ++k) {
          if (h[(size_t)i * G + g] == nu[(size_t)i * I + k]) ref += Qu[((size_t)i * G + g) * I + k];
          if (down && i + 1 < N && nu[(size_t)i * I + k] == h[(size_t)(i + 1) * G + g])
            ref += Qd[((size_t)i * I + k) * G + g];
        }
    CHECK(J == ref, "objective %d: %lld against %lld", trial, (long long)J, (long long)ref);
    if (L > 1) {  // an unbalanced layout is refused
      std::vector<int32_t> hb(h);
      hb[0] = (hb[0] + 1) % L;
      CHECK(dtp_layout_objective(N, G, I, L, Qu.data(), nullptr, hb.data(), nu.data(), &J) == DTP_ERR_INVALID_ARG,
            "unbalanced layout accepted, trial %d", trial);
    }
  }
  // the exact per-layer optimum against brute force over every layout of small layers
  for (int trial = 0; trial < 40; ++trial) {
    const int L = 2 + r.below(2), G = L * (1 + r.below(2)), I = L * (1 + r.below(8 / L));
    std::vector<int64_t> Q((size_t)G * I);
    for (auto& v : Q) v = trial % 2 ? (int64_t)r.below(3) : (int64_t)(r.next() >> 20);
    std::vector<int32_t> h(G), nu(I);
    int64_t J = -1;
    CHECK(dtp_layer_optimum(G, I, L, Q.data(), h.data(), nu.data(), &J) == DTP_OK, "optimum %d", trial);
    int64_t best = std::numeric_limits<int64_t>::min();
    each_balanced(G, L, [&](const std::vector<int32_t>& hh) {
      each_balanced(I, L, [&](const std::vector<int32_t>& nn) {
        int64_t s = 0;
        for (int g = 0; g < G; ++g)
          for (int k = 0; k < I; ++k)
            if (hh[g] == nn[k]) s += Q[(size_t)g * I + k];
        best = std::max(best, s);
      });
    });
    CHECK(J == best, "optimum %d: %lld against brute force %lld (G=%d I=%d L=%d)", trial, (long long)J,
          (long long)best, G, I, L);
    int64_t s = 0;
    for (int g = 0; g < G; ++g)
      for (int k = 0; k < I; ++k)
        if (h[g] == nu[k]) s += Q[(size_t)g * I + k];
    CHECK(s == J && balanced(h.data(), G, L) && balanced(nu.data(), I, L), "optimum %d: layout", trial);
    int seen = 0;  // device labels first appear in the order 0, 1, ..., L - 1
    for (int g = 0; g < G; ++g) {
      CHECK(h[g] <= seen, "optimum %d: labels out of order", trial);
      if (h[g] == seen) ++seen;
    }
  }
  std::vector<int32_t> h(8), nu(8);
  CHECK(dtp_random_layout(1, 8, 8, 3, 1, h.data(), nu.data()) == DTP_ERR_INVALID_ARG, "G %% L");
  CHECK(dtp_random_layout(0, 8, 8, 2, 1, h.data(), nu.data()) == DTP_ERR_INVALID_ARG, "N = 0");
}

// ---------------------------------------------------------------- the rest of the ABI
void check_misc() {
  const dtp_status all[] = {DTP_OK, DTP_ERR_INVALID_ARG, DTP_ERR_UNSUPPORTED, DTP_ERR_DEGENERATE,
                            DTP_ERR_NO_MEMORY, DTP_ERR_HIP};
  for (dtp_status s : all) CHECK(dtp_status_string(s) != nullptr, "status string %d", (int)s);
  CHECK(dtp_status_string((dtp_status)12345) != nullptr, "unknown status string");
  std::vector<int32_t> h(8);
  (void)dtp_partition_unrank(8, 3, 0, h.data());  // fails: leaves a message behind
  CHECK(dtp_last_error() != nullptr, "last error");
  // Entry points with device arguments refuse bad sizes before any GPU call.
  int64_t best = 0;
  CHECK(dtp_partition_scores(8, 16, 3, nullptr, nullptr, nullptr, nullptr, 0, nullptr, &best, nullptr) !=
            DTP_OK, "partition scores, G %% L");
}

}  // namespace

int main() {
  Rng r{2609'13846ull};
  check_partitions();
  check_encode(r);
  check_assign(r);
  check_layouts(r);
  check_misc();
  std::printf("host checks passed: %d\n", g_checks);
  return 0;
}
