// Labelled balanced partitions of G KV groups over L devices (Section 3, "Optimiser":
// the head step scores all G!/((G/L)!)^L of them, 2520 for G = 8, L = 4).
// A partition is h in {0..L-1}^G with G/L groups per device; ranks follow the
// lexicographic order of (h(0), h(1), ..., h(G-1)), so rank 0 is the contiguous layout.
#include "dtp_internal.h"

namespace dtp {

namespace {

// Number of ways to fill the remaining positions given per-device remaining counts.
unsigned __int128 completions(const int* rem, int L, bool* overflow) {
  unsigned __int128 total = 1;
  int left = 0;
  for (int l = 0; l < L; ++l) {
    // multiply by C(left + rem[l], rem[l]) step by step (exact at every step)
    for (int j = 1; j <= rem[l]; ++j) {
      total = total * (unsigned __int128)(left + j) / (unsigned __int128)j;
      if (total > ((unsigned __int128)1 << 62)) {
        *overflow = true;
        return 0;
      }
    }
    left += rem[l];
  }
  return total;
}

void enumerate_rec(int g, int G, int L, int* rem, uint8_t* cur, std::vector<uint8_t>* out) {
  if (g == G) {
    out->insert(out->end(), cur, cur + G);
    return;
  }
  for (int l = 0; l < L; ++l) {
    if (rem[l] == 0) continue;
    --rem[l];
    cur[g] = (uint8_t)l;
    enumerate_rec(g + 1, G, L, rem, cur, out);
    ++rem[l];
  }
}

}  // namespace

int64_t count_partitions(int G, int L) {
  if (L < 1 || G < 1 || G > kMaxGroups || G % L) return -1;
  int rem[kMaxGroups];
  for (int l = 0; l < L; ++l) rem[l] = G / L;
  bool overflow = false;
  const unsigned __int128 c = completions(rem, L, &overflow);
  return overflow ? -1 : (int64_t)c;
}

std::vector<uint8_t> enumerate_partitions(int G, int L) {
  std::vector<uint8_t> out;
  const int64_t P = count_partitions(G, L);
  if (P < 0) return out;
  out.reserve((size_t)P * G);
  int rem[kMaxGroups];
  uint8_t cur[kMaxGroups];
  for (int l = 0; l < L; ++l) rem[l] = G / L;
  enumerate_rec(0, G, L, rem, cur, &out);
  return out;
}

bool unrank_partition(int G, int L, int64_t rank, int32_t* h) {
  const int64_t P = count_partitions(G, L);
  if (P < 0 || rank < 0 || rank >= P) return false;
  int rem[kMaxGroups];
  for (int l = 0; l < L; ++l) rem[l] = G / L;
  unsigned __int128 r = (unsigned __int128)rank;
  for (int g = 0; g < G; ++g) {
    for (int l = 0; l < L; ++l) {
      if (rem[l] == 0) continue;
      --rem[l];
      bool of = false;
      const unsigned __int128 c = completions(rem, L, &of);
      if (r < c) {
        h[g] = l;
        break;
      }
      r -= c;
      ++rem[l];
    }
  }
  return true;
}

}  // namespace dtp
