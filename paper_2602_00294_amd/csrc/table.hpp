// Host-side feature table: the constant index matrix M_p of every degree and
// the per-feature weights (Sec. 2.4, "Efficient Computation": both are
// constant and precomputed once per (d, P)).
//
// Order: degree-major; inside degree p the tuples i1 <= ... <= ip (0-based) in
// lexicographic order; feature 0 is the degree-0 empty product (App. A1).
// Weight of tuple m of degree p: d^(-p/4) / sqrt(prod over distinct indices of
// (count)!), which is sqrt(alpha_p * C_p[m]) with alpha_p = 1/(p! d^(p/2)) and
// C_p[m] = p!/prod(count!) (Sec. 2.1, Sec. 2.3).
#pragma once

#include <cmath>
#include <cstdint>
#include <cstring>
#include <vector>

namespace sata {

constexpr int kMaxP = 8;      // degrees 0..7: seven index bytes plus a degree byte
constexpr int kMaxDim = 255;  // indices are stored in one byte

// Binomial coefficient C(n, k); returns -1 when the result exceeds int64.
inline int64_t binom(int64_t n, int64_t k) {
  if (k < 0 || n < 0 || k > n) return 0;
  if (k > n - k) k = n - k;
  __int128 r = 1;
  for (int64_t i = 1; i <= k; ++i) {
    r = r * (n - k + i) / i;  // exact: r * (n-k+i) is divisible by i at every step
    if (r > (__int128)INT64_MAX) return -1;
  }
  return (int64_t)r;
}

inline int64_t feature_count(int d, int P) {
  if (d < 1 || P < 1) return -1;
  return binom((int64_t)d + P - 1, P - 1);
}

// Packed form of one feature: byte j (j < 7) holds index i_{j+1}, byte 7 the degree.
inline uint64_t pack_feature(int p, const int* idx) {
  uint64_t v = (uint64_t)p << 56;
  for (int j = 0; j < p; ++j) v |= (uint64_t)(idx[j] & 0xff) << (8 * j);
  return v;
}

inline int packed_degree(uint64_t v) { return (int)(v >> 56); }
inline int packed_index(uint64_t v, int j) { return (int)((v >> (8 * j)) & 0xff); }

// Visits the features of degree p in lexicographic order of non-decreasing tuples.
template <typename F>
inline void for_each_tuple(int d, int p, F&& visit) {
  int idx[kMaxP] = {0};
  while (true) {
    visit(idx);
    int j = p - 1;
    while (j >= 0 && idx[j] == d - 1) --j;
    if (j < 0) return;
    const int nv = idx[j] + 1;
    for (int t = j; t < p; ++t) idx[t] = nv;  // smallest non-decreasing successor
  }
}

inline double feature_weight(int d, int p, const int* idx) {
  double denom = 1.0;
  int run = 1;
  for (int j = 1; j <= p; ++j) {
    if (j < p && idx[j] == idx[j - 1]) {
      ++run;
    } else {
      for (int c = 2; c <= run; ++c) denom *= c;
      run = 1;
    }
  }
  return std::pow((double)d, -0.25 * p) / std::sqrt(denom);
}

struct FeatureTable {
  int d = 0, P = 0;
  int64_t D = 0;
  std::vector<uint64_t> packed;  // [D]
  std::vector<float> weight;     // [D]
};

inline FeatureTable build_table(int d, int P) {
  FeatureTable t;
  t.d = d;
  t.P = P;
  t.D = feature_count(d, P);
  t.packed.reserve((size_t)t.D);
  t.weight.reserve((size_t)t.D);
  for (int p = 0; p < P; ++p) {
    if (p == 0) {
      t.packed.push_back(pack_feature(0, nullptr));
      t.weight.push_back(1.0f);
      continue;
    }
    for_each_tuple(d, p, [&](const int* idx) {
      t.packed.push_back(pack_feature(p, idx));
      t.weight.push_back((float)feature_weight(d, p, idx));
    });
  }
  return t;
}

// Generation program of the matrix-core prefill that computes features from
// their monomials, two 32-bit words per feature (followed by `pad` entries
// for slices that run past the last feature):
//   word 0: bits 0-9: byte offset 4 i_p of the feature's last index in a
//           float32 row of coordinates (degree 0 and padding: 4 d, a column
//           that holds 1); bits 10-17 and 18-25: the first two of the other
//           indices (d where the feature has fewer); bit 30: it has more than
//           two other indices (the rest are read from the packed entry);
//           bit 31: the product of the other indices must be formed anew, at
//           every multiple of `block` features and wherever the degree or an
//           index other than the last changes;
//   word 1: the feature weight (0 for padding).
// Features run through their last index in order (for_each_tuple), so the
// product of the others is shared by runs of up to d consecutive features.
inline std::vector<uint32_t> build_gen_program(const FeatureTable& t, int pad, int block) {
  std::vector<uint32_t> g(2 * ((size_t)t.D + pad));
  const uint32_t d = (uint32_t)t.d;
  uint64_t prev_key = ~(uint64_t)0;
  for (int64_t f = 0; f < t.D + pad; ++f) {
    uint32_t off = 4u * d, a0 = d, a1 = d, more = 0, w = 0;
    uint64_t key = ~(uint64_t)0 - 1;  // padding: one key for all
    if (f < t.D) {
      const uint64_t e = t.packed[(size_t)f];
      const int p = packed_degree(e);
      if (p > 0) off = 4u * (uint32_t)packed_index(e, p - 1);
      if (p > 1) a0 = (uint32_t)packed_index(e, 0);
      if (p > 2) a1 = (uint32_t)packed_index(e, 1);
      more = p > 3 ? 1u : 0u;
      key = p > 0 ? e & ~((uint64_t)0xff << (8 * (p - 1))) : e;
      std::memcpy(&w, &t.weight[(size_t)f], sizeof(w));
    }
    const bool fresh = f % block == 0 || key != prev_key;
    prev_key = key;
    g[2 * (size_t)f] = off | (a0 << 10) | (a1 << 18) | (more << 30) | (fresh ? 0x80000000u : 0u);
    g[2 * (size_t)f + 1] = w;
  }
  return g;
}

}  // namespace sata
