// Host-side helpers shared by the C-ABI translation units: workspace
// bump allocation, argument checks, the attention split size and optional
// per-launch event recording.
#pragma once

#include <cstdint>
#include <cstring>
#include <algorithm>
#include <functional>
#include <vector>

#include "common.h"
#include "internal.h"

namespace stca {
namespace api {

constexpr size_t kAlign = 256;

struct Bump {
  size_t off = 0;
  size_t take(size_t bytes) {
    size_t o = off;
    off = round_up(static_cast<int64_t>(off + bytes), kAlign);
    return o;
  }
};

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// 1 = bf16 MFMA path, 0 = generic, <0 = status
inline int path_of(const stca_dims_t* d) {
  if (!d) return STCA_ERR_INVALID_ARG;
  if (d->d_model <= 0 || d->n_heads <= 0 || d->n_layers <= 0 || d->ffn_hidden <= 0 ||
      d->d_model % d->n_heads != 0 || (d->dtype != STCA_F32 && d->dtype != STCA_BF16))
    return STCA_ERR_INVALID_ARG;
  if (d->kv_form < STCA_KV_AUTO || d->kv_form > STCA_KV_MATERIALIZE || d->attn_form < STCA_ATTN_AUTO ||
      d->attn_form > STCA_ATTN_REORDERED || d->bwd_form < STCA_BWD_AUTO || d->bwd_form > STCA_BWD_REORDERED ||
      d->chunk_blocks < 0)
    return STCA_ERR_INVALID_ARG;
  const int dh = d->d_model / d->n_heads;
  if (d->ffn_hidden % 32 != 0) return STCA_ERR_UNSUPPORTED;
  if (d->dtype == STCA_BF16 && dh == 32 && (d->d_model == 64 || d->d_model == 128 || d->d_model == 256) &&
      d->ffn_hidden % 256 == 0)
    return 1;
  if (dh == 8 || dh == 16 || dh == 32 || dh == 64) return 0;
  return STCA_ERR_UNSUPPORTED;
}

inline stca_status_t check_batch(const stca_batch_t* b) {
  if (!b || b->n_requests < 1 || b->n_hist < 0 || b->n_tgt < 0 || b->n_hist >= (int64_t(1) << 31) ||
      b->n_tgt >= (int64_t(1) << 31) || !b->hist_off || !b->tgt_off)
    return STCA_ERR_INVALID_ARG;
  if ((b->hist_off_host == nullptr) != (b->tgt_off_host == nullptr)) return STCA_ERR_INVALID_ARG;
  if (b->hist_off_host) {
    const int32_t *h = b->hist_off_host, *t = b->tgt_off_host;
    if (h[0] != 0 || t[0] != 0 || h[b->n_requests] != b->n_hist || t[b->n_requests] != b->n_tgt)
      return STCA_ERR_INVALID_ARG;
    for (int r = 0; r < b->n_requests; ++r) {
      if (h[r + 1] < h[r] || t[r + 1] < t[r]) return STCA_ERR_INVALID_ARG;
      if (t[r + 1] > t[r] && h[r + 1] == h[r]) return STCA_ERR_INVALID_ARG;
    }
  }
  return STCA_OK;
}

inline int device_cus() {
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cache[dev] = n;
  }
  return cache[dev];
}

// Chunk length (in 32-row blocks) of the split over history rows: aim at about
// `per_cu` attention units per CU (four for the standard form; one for the
// reordered form, whose units stream X with little work per block and whose
// merge cost grows with the chunk count), over `rows` history rows (the
// whole batch by default).  A positive `forced` (the caller's
// stca_dims_t.chunk_blocks) replaces the choice.
inline int chunk_blocks_for(const stca_batch_t* b, int n_cu, int per_cu, int forced, int64_t rows = -1) {
  if (forced >= 1) return forced;
  const int64_t nb = ceil_div(rows >= 0 ? rows : b->n_hist, kBlockTokens);
  int64_t c = ceil_div(nb, per_cu * static_cast<int64_t>(n_cu));
  if (c < 8) c = 8;
  if (c > (1 << 20)) c = 1 << 20;
  return static_cast<int>(c);
}

// Chunk length of the standard form's units: with host offsets, the one of
// one, two, four or eight units per CU whose estimated makespan is least
// (fewer units on ties).  The estimate cuts the requests the standard form serves
// (targets in [m_lo, m_hi]) as the device scheduler does and deals their
// units (those of up to 32 and of more targets run in separate launches, so
// their makespans add) in descending size,
// round-robin over the CUs in alternating directions as the device
// scheduler does, and charges each unit one block of fixed cost (its query
// load, partial stores and merge).  Equal histories then run one unit per
// CU when the chunks divide evenly (headline batch 1.45 -> 1.41 ms per step),
// while ragged ones take many (the ragged batch: eight per CU, 2.06 ms per
// step; four 2.13, two 2.68).
inline int chunk_blocks_auto(const stca_batch_t* b, int n_cu, int forced, int m_lo = 1, int m_hi = 1 << 30) {
  if (forced >= 1 || !b->hist_off_host || !b->tgt_off_host || n_cu < 1) return chunk_blocks_for(b, n_cu, 4, forced);
  int best = 0;
  int64_t best_span = -1;
  std::vector<int64_t> jobs[2], load, cnt;
  for (int per_cu = 1; per_cu <= 8; per_cu *= 2) {
    const int c = chunk_blocks_for(b, n_cu, per_cu, 0);
    jobs[0].clear();
    jobs[1].clear();
    for (int r = 0; r < b->n_requests; ++r) {
      const int64_t m = b->tgt_off_host[r + 1] - b->tgt_off_host[r];
      if (m < m_lo || m > m_hi || m < 1) continue;
      const int64_t h0 = b->hist_off_host[r], h1 = b->hist_off_host[r + 1];
      if (h1 <= h0) continue;
      // the device scheduler's cut: ceil(nbr / c) chunks (at most
      // kMaxChunks) of equal length, the last one shorter
      const int64_t nbr = ceil_div(h1, kBlockTokens) - h0 / kBlockTokens;
      int64_t nch = std::min<int64_t>(kMaxChunks, std::max<int64_t>(1, ceil_div(nbr, c)));
      const int64_t cb = ceil_div(nbr, nch);
      nch = ceil_div(nbr, cb);
      const int64_t groups = m <= 64 ? 1 : ceil_div(m, 64);
      for (int64_t g = 0; g < groups; ++g)
        for (int64_t k = 0; k < nch; ++k) jobs[m > 32].push_back(std::min<int64_t>(cb, nbr - k * cb) + 1);
    }
    if (jobs[0].size() + jobs[1].size() > (1u << 18)) return chunk_blocks_for(b, n_cu, 4, 0);  // bound the host work
    int64_t span = 0;
    for (auto& j : jobs) {
      if (j.empty()) continue;
      // descending order: counted when the sizes are small (a request of more
      // than kMaxChunks chunks has chunks longer than c)
      const int64_t top = *std::max_element(j.begin(), j.end());
      if (top <= (1 << 16)) {
        cnt.assign(top + 1, 0);
        for (const int64_t x : j) ++cnt[x];
        size_t i = 0;
        for (int64_t x = top; x >= 0; --x)
          for (int64_t k = 0; k < cnt[x]; ++k) j[i++] = x;
      } else {
        std::sort(j.begin(), j.end(), std::greater<int64_t>());
      }
      load.assign(n_cu, 0);
      for (size_t i = 0; i < j.size(); ++i) {
        const size_t round = i / n_cu, pos = i % n_cu;
        load[round % 2 ? n_cu - 1 - pos : pos] += j[i];
      }
      span += *std::max_element(load.begin(), load.end());
    }
    if (best_span < 0 || span < best_span) {
      best_span = span;
      best = c;
    }
  }
  return best;
}

inline int64_t max_units_for(const stca_batch_t* b, int chunk_blocks, int group, int m_lo = 1,
                             int m_hi = 1 << 30) {
  if (b->hist_off_host)
    return host_count_units(b->hist_off_host, b->tgt_off_host, b->n_requests, chunk_blocks, group, m_lo, m_hi);
  return (ceil_div(b->n_tgt, group) + b->n_requests) * kMaxChunks;
}

template <typename T>
inline T* at(void* base, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(base) + off);
}
template <typename T>
inline const T* at(const void* base, size_t off) {
  return reinterpret_cast<const T*>(static_cast<const char*>(base) + off);
}

// Optional per-launch event recording for measurement: ev[0] is recorded
// before the first launch and ev[k+1] right after launch k.
struct Rec {
  hipEvent_t* ev = nullptr;
  int n = 0, k = 0;
  const char** labels = nullptr;
  hipStream_t st = nullptr;
  hipError_t start() {
    if (!ev) return hipSuccess;
    if (k >= n) return hipErrorInvalidValue;
    return hipEventRecord(ev[k++], st);
  }
  hipError_t mark(const char* name) {
    if (!ev) return hipSuccess;
    if (k >= n) return hipErrorInvalidValue;
    if (labels) labels[k - 1] = name;
    return hipEventRecord(ev[k++], st);
  }
};

#define HIPCHK(x)                             \
  do {                                        \
    if ((x) != hipSuccess) return STCA_ERR_HIP; \
  } while (0)

}  // namespace api
}  // namespace stca
