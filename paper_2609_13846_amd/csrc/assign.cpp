// Exact balanced neuron assignment (Section 3, "Optimiser", neuron step).
//
// Given the gain M[k][l] of putting neuron k on device l, find nu maximising
// sum_k M[k][nu[k]] with exactly I/L neurons per device: a linear assignment with I/L
// replicated slots per device.  The paper solves it approximately (dual ascent, a
// capacity fix-up, pairwise swaps); this solver is exact.
//
// 1. Optimum.  With two devices, a selection by M[k][0] - M[k][1] is exact and gives the
//    canonical optimum of step 2 directly (canonical_two_devices).  Otherwise neurons
//    are inserted one at a time, each along a best augmenting path of
//    the current optimal partial assignment (the successive-shortest-path method of the
//    assignment problem, one row at a time).  Because there are only L devices, a path is
//    a walk over devices: the new neuron enters device a0, then for every hop a -> b the
//    neuron of a with the largest M[j][b] - M[j][a] moves to b, and the walk ends at a
//    device with a free slot.  Best moves per device pair come from lazy max-heaps, and
//    the longest walk is Bellman-Ford over the L devices (no gaining cycle exists while
//    the partial assignment is optimal).
// 2. Canonical optimum.  Device prices lambda are longest-path distances in the exchange
//    graph of the optimum; every optimal assignment uses only "tight" pairs
//    (k, l) with M[k][l] - lambda_l = max_l' (M[k][l'] - lambda_l') (complementary
//    slackness), and every balanced assignment on tight pairs is optimal.  The answer is
//    the lexicographically smallest of them: neurons in index order take the smallest
//    tight device that leaves a feasible completion, feasibility being Hall's condition
//    over device subsets, evaluated by a subset-sum over tight-set masks.
#include <algorithm>
#include <functional>
#include <queue>
#include <utility>
#include <vector>

#include "dtp_internal.h"

namespace dtp {

namespace {

using Entry = std::pair<int64_t, int32_t>;  // (gain of moving j from a to b, j)

struct PairHeaps {
  int L;
  std::vector<std::priority_queue<Entry>> heap;  // [a * L + b]
  explicit PairHeaps(int L_) : L(L_), heap((size_t)L_ * L_) {}

  void add(const int64_t* M, int j, int a) {
    const int64_t* m = M + (size_t)j * L;
    for (int b = 0; b < L; ++b)
      if (b != a) heap[(size_t)a * L + b].push(Entry(m[b] - m[a], j));
  }
  // Best (gain, neuron) currently on device a for a move to b; false if a is empty.
  bool top(int a, int b, const std::vector<int32_t>& nu, Entry* out) {
    auto& h = heap[(size_t)a * L + b];
    while (!h.empty() && nu[h.top().second] != a) h.pop();
    if (h.empty()) return false;
    *out = h.top();
    return true;
  }
};

void optimal_by_insertion(int I, int L, const int64_t* M, std::vector<int32_t>& nu) {
  const int cap = I / L;
  std::vector<int> count(L, 0);
  PairHeaps heaps(L);
  std::vector<int64_t> dist(L);
  std::vector<int> pred(L);
  std::vector<Entry> edge((size_t)L * L);
  std::vector<char> has_edge((size_t)L * L);
  for (int k = 0; k < I; ++k) {
    for (int a = 0; a < L; ++a)
      for (int b = 0; b < L; ++b) {
        const size_t e = (size_t)a * L + b;
        has_edge[e] = (a != b) && heaps.top(a, b, nu, &edge[e]);
      }
    const int64_t* mk = M + (size_t)k * L;
    for (int a = 0; a < L; ++a) {
      dist[a] = mk[a];
      pred[a] = -1;
    }
    for (int round = 0; round + 1 < L; ++round) {
      bool changed = false;
      for (int a = 0; a < L; ++a)
        for (int b = 0; b < L; ++b) {
          const size_t e = (size_t)a * L + b;
          if (!has_edge[e]) continue;
          const int64_t cand = dist[a] + edge[e].first;
          if (cand > dist[b]) {
            dist[b] = cand;
            pred[b] = a;
            changed = true;
          }
        }
      if (!changed) break;
    }
    int end = -1;
    for (int b = 0; b < L; ++b)
      if (count[b] < cap && (end < 0 || dist[b] > dist[end])) end = b;
    // Collect the moves along the walk before touching the heaps.
    std::vector<std::pair<int32_t, int>> moves;
    int b = end;
    while (pred[b] >= 0) {
      const int a = pred[b];
      moves.emplace_back(edge[(size_t)a * L + b].second, b);
      b = a;
    }
    const int entry = b;
    for (const auto& mv : moves) {
      nu[mv.first] = mv.second;
      heaps.add(M, mv.first, mv.second);
    }
    nu[k] = entry;
    heaps.add(M, k, entry);
    ++count[end];
  }
}

void canonicalise(int I, int L, const int64_t* M, std::vector<int32_t>& nu) {
  // Exchange graph of the optimum and prices by longest paths from a zero source.
  std::vector<int64_t> w((size_t)L * L, 0);
  std::vector<char> has((size_t)L * L, 0);
  for (int j = 0; j < I; ++j) {
    const int a = nu[j];
    const int64_t* m = M + (size_t)j * L;
    for (int b = 0; b < L; ++b) {
      if (b == a) continue;
      const size_t e = (size_t)a * L + b;
      const int64_t gain = m[b] - m[a];
      if (!has[e] || gain > w[e]) {
        w[e] = gain;
        has[e] = 1;
      }
    }
  }
  std::vector<int64_t> lam(L, 0);
  for (int round = 0; round < L; ++round)
    for (int a = 0; a < L; ++a)
      for (int b = 0; b < L; ++b) {
        const size_t e = (size_t)a * L + b;
        if (has[e] && lam[a] + w[e] > lam[b]) lam[b] = lam[a] + w[e];
      }
  // Tight-set mask of every neuron.
  const int nmask = 1 << L;
  std::vector<uint32_t> mask(I);
  std::vector<int64_t> cnt(nmask, 0);
  for (int k = 0; k < I; ++k) {
    const int64_t* m = M + (size_t)k * L;
    int64_t best = m[0] - lam[0];
    for (int l = 1; l < L; ++l) best = std::max(best, m[l] - lam[l]);
    uint32_t mk = 0;
    for (int l = 0; l < L; ++l)
      if (m[l] - lam[l] == best) mk |= 1u << l;
    mask[k] = mk;
    ++cnt[mk];
  }
  std::vector<int64_t> cap(L, I / L), need(nmask);
  auto feasible = [&]() {
    // need[S] = number of remaining neurons whose tight set lies inside S
    for (int s = 0; s < nmask; ++s) need[s] = cnt[s];
    for (int l = 0; l < L; ++l)
      for (int s = 0; s < nmask; ++s)
        if (s >> l & 1) need[s] += need[s ^ (1 << l)];
    for (int s = 1; s < nmask; ++s) {
      int64_t have = 0;
      for (int l = 0; l < L; ++l)
        if (s >> l & 1) have += cap[l];
      if (need[s] > have) return false;
    }
    return true;
  };
  for (int k = 0; k < I; ++k) {
    --cnt[mask[k]];
    if ((mask[k] & (mask[k] - 1)) == 0) {  // one tight device: the invariant keeps it feasible
      const int l = __builtin_ctz(mask[k]);
      --cap[l];
      nu[k] = l;
      continue;
    }
    for (int l = 0; l < L; ++l) {
      if (!(mask[k] >> l & 1) || cap[l] == 0) continue;
      --cap[l];
      if (feasible()) {
        nu[k] = l;
        break;
      }
      ++cap[l];
    }
  }
}

// Two devices, optimum and canonical form in one pass.  An assignment is optimal exactly
// when device 0 holds I/2 neurons of largest d_k = M[k][0] - M[k][1] (exchanging any pair
// across the cut cannot gain), so the optima differ only in which neurons with d_k = t,
// the I/2-th largest value, fill device 0's last places; the lexicographically smallest
// gives those places to the lowest indices.
void canonical_two_devices(int I, const int64_t* M, std::vector<int32_t>& nu) {
  std::vector<int64_t> d(I);
  for (int k = 0; k < I; ++k) d[k] = M[2 * (size_t)k] - M[2 * (size_t)k + 1];
  std::vector<int64_t> sorted(d);
  std::nth_element(sorted.begin(), sorted.begin() + (I / 2 - 1), sorted.end(), std::greater<int64_t>());
  const int64_t t = sorted[I / 2 - 1];
  int above = 0;
  for (int k = 0; k < I; ++k) above += d[k] > t;
  int ties_to_0 = I / 2 - above;  // >= 1: fewer than I/2 values exceed t, at least I/2 reach it
  for (int k = 0; k < I; ++k) {
    if (d[k] > t) {
      nu[k] = 0;
    } else if (d[k] == t && ties_to_0 > 0) {
      nu[k] = 0;
      --ties_to_0;
    } else {
      nu[k] = 1;
    }
  }
}

}  // namespace

void balanced_assign_exact(int I, int L, const int64_t* M, int32_t* nu_out, int64_t* value) {
  std::vector<int32_t> nu(I, -1);
  if (L == 1) {
    std::fill(nu.begin(), nu.end(), 0);
  } else {
    if (L == 2) {
      canonical_two_devices(I, M, nu);
    } else {
      optimal_by_insertion(I, L, M, nu);
      canonicalise(I, L, M, nu);
    }
  }
  int64_t v = 0;
  for (int k = 0; k < I; ++k) {
    nu_out[k] = nu[k];
    v += M[(size_t)k * L + nu[k]];
  }
  if (value) *value = v;
}

// ------------------------------------------------------------------ the paper's heuristic
// The approximate solver the paper uses for the same problem (Section 3, "Optimiser", and
// the appendix's 300 iterations with step decay 0.98), kept to measure its distance from
// the optimum:
// 1. Dual ascent on device offsets lambda (starting at 0, first step (max M - min M) / I):
//    every neuron takes argmax_l (M[k][l] - lambda_l), lowest l on ties, and each device's
//    offset rises by step * (load_l - I/L); the step is multiplied by the decay.
// 2. Fix-up: from the assignment the final offsets induce, move one neuron at a time from
//    an overloaded device to an underloaded one, the move losing the least gain first
//    (smallest neuron, then smallest device, on ties).
// 3. Pairwise swaps: scan device pairs (a, b), a < b; exchange the neuron of a gaining most
//    by moving to b with the neuron of b gaining most by moving to a (smallest indices on
//    ties) when the two gains sum to more than zero; repeat until a scan exchanges nothing.
// The offsets are doubles: M's entries are exact in fp64 below 2^53.  Each update is a
// product and then a sum in separate statements, so no fused multiply-add changes it.
void balanced_assign_dual_ascent(int I, int L, const int64_t* M, int iterations, double decay,
                                 int32_t* nu_out, int64_t* value) {
  const int cap = I / L;
  std::vector<double> lam(L, 0.0);
  int64_t lo = M[0], hi = M[0];
  for (int64_t i = 0; i < (int64_t)I * L; ++i) {
    lo = std::min(lo, M[i]);
    hi = std::max(hi, M[i]);
  }
  double step = ((double)hi - (double)lo) / (double)I;
  std::vector<int32_t> nu(I);
  std::vector<int> load(L);
  auto induce = [&]() {
    std::fill(load.begin(), load.end(), 0);
    for (int k = 0; k < I; ++k) {
      int best = 0;
      double bv = (double)M[(size_t)k * L] - lam[0];
      for (int l = 1; l < L; ++l) {
        const double v = (double)M[(size_t)k * L + l] - lam[l];
        if (v > bv) {
          bv = v;
          best = l;
        }
      }
      nu[k] = best;
      ++load[best];
    }
  };
  for (int it = 0; it < iterations; ++it) {
    induce();
    for (int l = 0; l < L; ++l) {
      const double inc = step * (double)(load[l] - cap);
      lam[l] = lam[l] + inc;
    }
    step = step * decay;
  }
  induce();
  // fix-up
  for (;;) {
    bool over = false;
    for (int l = 0; l < L; ++l) over = over || load[l] > cap;
    if (!over) break;
    int64_t best_loss = 0;
    int bk = -1, bb = -1;
    for (int k = 0; k < I; ++k) {
      const int a = nu[k];
      if (load[a] <= cap) continue;
      for (int b = 0; b < L; ++b) {
        if (load[b] >= cap) continue;
        const int64_t loss = M[(size_t)k * L + a] - M[(size_t)k * L + b];
        if (bk < 0 || loss < best_loss) {
          best_loss = loss;
          bk = k;
          bb = b;
        }
      }
    }
    --load[nu[bk]];
    ++load[bb];
    nu[bk] = bb;
  }
  // pairwise swaps
  for (bool changed = true; changed;) {
    changed = false;
    for (int a = 0; a < L; ++a)
      for (int b = a + 1; b < L; ++b) {
        int ka = -1, kb = -1;
        int64_t ga = 0, gb = 0;
        for (int k = 0; k < I; ++k) {
          if (nu[k] == a) {
            const int64_t g = M[(size_t)k * L + b] - M[(size_t)k * L + a];
            if (ka < 0 || g > ga) {
              ga = g;
              ka = k;
            }
          } else if (nu[k] == b) {
            const int64_t g = M[(size_t)k * L + a] - M[(size_t)k * L + b];
            if (kb < 0 || g > gb) {
              gb = g;
              kb = k;
            }
          }
        }
        if (ka >= 0 && kb >= 0 && ga + gb > 0) {
          nu[ka] = b;
          nu[kb] = a;
          changed = true;
        }
      }
  }
  int64_t v = 0;
  for (int k = 0; k < I; ++k) {
    nu_out[k] = nu[k];
    v += M[(size_t)k * L + nu[k]];
  }
  if (value) *value = v;
}

}  // namespace dtp
