// Stochastic-length training batches (Sec. 3.3, "train sparsely, infer
// densely"; App. "Extrapolation details"): host-side batch construction that
// feeds the ragged training path.
//
//  1. Length sampling: s ~ Beta(alpha, beta) with beta from the expectation
//     constraint (Eq. beta), L_raw = L_min + s (L_max - L_min) (Eq.
//     beta-scale), rounded to the nearest multiple of 8.
//  2. Global length allocation: each request keeps min(L_train, its history
//     length); if the batch total exceeds the token budget B * L_avg, the
//     longest requests are cut to a common cap (the largest multiple of 8
//     that fits the budget), the shorter ones keep their sampled length.
//  3. Element selection: the temporal suffix (the most recent L rows).
//  4. Compaction: the kept rows are packed without padding into the flat
//     history layout, segmented by offsets (the index-based ragged layout).
//
// Random numbers: SplitMix64 (Steele, Lea and Flood, 2014) over a counter per
// (seed, request), uniform doubles from its top 53 bits; normal variates by
// Box-Muller; Gamma variates by Marsaglia and Tsang (2000), with the
// shape < 1 case from Gamma(a + 1) U^(1/a) taken in log space (at a = 0.02 the
// power underflows); Beta = G_a / (G_a + G_b) formed from the logs.
#include <cmath>
#include <cstdint>
#include <vector>
#include <algorithm>

#include "../../include/stca.h"

namespace {

struct Stream {
  uint64_t state;
  explicit Stream(uint64_t seed, uint64_t id) : state(seed ^ (0x9E3779B97F4A7C15ull * (id + 1))) {}
  uint64_t next() {
    uint64_t z = (state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  // uniform in (0, 1)
  double uniform() { return (static_cast<double>(next() >> 11) + 0.5) * (1.0 / 9007199254740992.0); }
  double normal() {
    const double u1 = uniform(), u2 = uniform();
    return std::sqrt(-2.0 * std::log(u1)) * std::cos(6.283185307179586 * u2);
  }
  // log of a Gamma(shape, 1) variate
  double log_gamma_variate(double a) {
    if (a < 1.0) return log_gamma_variate(a + 1.0) + std::log(uniform()) / a;
    const double d = a - 1.0 / 3.0, c = 1.0 / std::sqrt(9.0 * d);
    for (;;) {
      double x, v;
      do {
        x = normal();
        v = 1.0 + c * x;
      } while (v <= 0.0);
      v = v * v * v;
      const double u = uniform();
      if (std::log(u) < 0.5 * x * x + d - d * v + d * std::log(v)) return std::log(d * v);
    }
  }
  double beta(double a, double b) {
    const double la = log_gamma_variate(a), lb = log_gamma_variate(b);
    // G_a / (G_a + G_b) = 1 / (1 + exp(lb - la))
    const double t = lb - la;
    return t > 0 ? std::exp(-t) / (1.0 + std::exp(-t)) : 1.0 / (1.0 + std::exp(t));
  }
};

int32_t round8(double x) { return static_cast<int32_t>(std::floor(x / 8.0 + 0.5)) * 8; }

bool valid_lengths(int32_t l_min, int32_t l_avg, int32_t l_max) {
  return l_min >= 0 && l_min < l_avg && l_avg < l_max;
}

}  // namespace

extern "C" {

double stca_sl_beta(double alpha, int32_t l_min, int32_t l_avg, int32_t l_max) {
  if (!(alpha > 0) || !valid_lengths(l_min, l_avg, l_max)) return NAN;
  return alpha * static_cast<double>(l_max - l_avg) / static_cast<double>(l_avg - l_min);
}

stca_status_t stca_sl_sample(uint64_t seed, int32_t n, double alpha, int32_t l_min, int32_t l_avg, int32_t l_max,
                             double* l_raw, int32_t* l_train) {
  const double b = stca_sl_beta(alpha, l_min, l_avg, l_max);
  if (n < 0 || !(b > 0) || (n > 0 && !l_train)) return STCA_ERR_INVALID_ARG;
  const int32_t lo = std::max<int32_t>(8, round8(l_min)), hi = round8(l_max) > l_max ? round8(l_max) - 8
                                                                                         : round8(l_max);
  for (int32_t r = 0; r < n; ++r) {
    Stream s(seed, static_cast<uint64_t>(r));
    const double raw = l_min + s.beta(alpha, b) * (l_max - l_min);
    if (l_raw) l_raw[r] = raw;
    l_train[r] = std::min(hi, std::max(lo, round8(raw)));
  }
  return STCA_OK;
}

stca_status_t stca_sl_allocate(int32_t n, const int32_t* l_full, const int32_t* l_train, int64_t budget,
                               int32_t* l_keep) {
  if (n < 0 || budget < 0 || (n > 0 && (!l_full || !l_train || !l_keep))) return STCA_ERR_INVALID_ARG;
  int64_t total = 0;
  int32_t longest = 0;
  for (int32_t r = 0; r < n; ++r) {
    if (l_full[r] < 0 || l_train[r] < 0) return STCA_ERR_INVALID_ARG;
    l_keep[r] = std::min(l_full[r], l_train[r]);
    total += l_keep[r];
    longest = std::max(longest, l_keep[r]);
  }
  if (total <= budget) return STCA_OK;
  // the largest cap (multiple of 8, at least 8) with sum(min(keep, cap)) <= budget
  auto sum_at = [&](int64_t cap) {
    int64_t t = 0;
    for (int32_t r = 0; r < n; ++r) t += std::min<int64_t>(l_keep[r], cap);
    return t;
  };
  int64_t lo = 8, hi = (static_cast<int64_t>(longest) + 7) / 8 * 8;
  if (sum_at(lo) > budget) {
    hi = lo;  // even the smallest cap is over: keep 8 rows of each (every request keeps some history)
  } else {
    while (hi - lo > 8) {
      const int64_t mid = (lo + hi) / 16 * 8;
      if (sum_at(mid) <= budget) lo = mid;
      else hi = mid;
    }
    hi = sum_at(hi) <= budget ? hi : lo;
  }
  for (int32_t r = 0; r < n; ++r) l_keep[r] = static_cast<int32_t>(std::min<int64_t>(l_keep[r], hi));
  return STCA_OK;
}

stca_status_t stca_sl_pack(int32_t n, const int32_t* full_off, const int32_t* l_keep, int32_t* hist_off,
                           int32_t* src_rows) {
  if (n < 0 || !full_off || !hist_off || (n > 0 && !l_keep)) return STCA_ERR_INVALID_ARG;
  int64_t k = 0;
  hist_off[0] = 0;
  for (int32_t r = 0; r < n; ++r) {
    const int32_t f0 = full_off[r], f1 = full_off[r + 1];
    if (f1 < f0 || l_keep[r] < 0 || l_keep[r] > f1 - f0) return STCA_ERR_INVALID_ARG;
    if (k + l_keep[r] > INT32_MAX) return STCA_ERR_INVALID_ARG;
    // the temporal suffix: the most recent l_keep rows, oldest first
    if (src_rows)
      for (int32_t i = 0; i < l_keep[r]; ++i) src_rows[k + i] = f1 - l_keep[r] + i;
    k += l_keep[r];
    hist_off[r + 1] = static_cast<int32_t>(k);
  }
  return STCA_OK;
}

}  // extern "C"
