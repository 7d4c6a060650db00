// Varlen scheduler: device offsets -> attention work units.
//
// The ragged batch is packed without padding and segmented by per-request
// offsets (App. A.4, index-based ragged target attention).  Each request's
// history rows are covered by whole 32-row blocks of the packed history
// ([floor(h0/32), ceil(h1/32))); the blocks are cut into at most kMaxChunks
// chunks of about `chunk_blocks` blocks, and the request's targets into groups
// of `group` (at most kWideGroup).  One unit = (target group, chunk).  Units of groups with at
// most 32 targets are listed first, the wider ones after them, so kernels
// specialised on the group width each get one contiguous range.  With
// deal = G > 0, each range holds its units in descending order of history
// blocks (32 size buckets, any order inside a bucket), every complete round
// of G units after the first in reverse order: a persistent kernel of G
// workgroups that deals units round-robin (unit w, w + G, ...) then pairs
// large units with small ones.  Every
// target's chunk count is recorded so the combine step knows how many partial
// results to merge.
//
// One workgroup of 1024 threads; each thread owns a contiguous run of requests.
// Invalid segments produce no units and set the workspace status, so no later
// kernel reads outside the buffers whatever the offsets hold.  Only requests
// with m_lo..m_hi targets get units (a batch can be split between two forms
// of the attention, each with its own schedule); every request is validated.
#include "common.h"
#include "internal.h"

namespace stca {

namespace {

constexpr int kSchedThreads = 1024;

struct ReqPlan {
  int32_t h0, h1, t0, t1, nch, cb, ng, bl;
  bool ok;
};

__device__ ReqPlan plan_request(const int32_t* hoff, const int32_t* toff, int r, int64_t n_hist,
                                int64_t n_tgt, int chunk_blocks, int group, int m_lo, int m_hi) {
  ReqPlan p{};
  p.h0 = hoff[r];
  p.h1 = hoff[r + 1];
  p.t0 = toff[r];
  p.t1 = toff[r + 1];
  p.ok = p.h0 >= 0 && p.h0 <= p.h1 && p.h1 <= n_hist && p.t0 >= 0 && p.t0 <= p.t1 && p.t1 <= n_tgt &&
         (p.t1 == p.t0 || p.h1 > p.h0);
  p.nch = 0;
  p.ng = 0;
  if (!p.ok || p.t1 == p.t0 || p.t1 - p.t0 < m_lo || p.t1 - p.t0 > m_hi) return p;
  p.bl = p.h0 / kBlockTokens;
  const int32_t bh = static_cast<int32_t>(ceil_div(p.h1, kBlockTokens));
  const int32_t nb = bh - p.bl;
  int32_t nch = static_cast<int32_t>(ceil_div(nb, chunk_blocks));
  nch = nch < 1 ? 1 : (nch > kMaxChunks ? kMaxChunks : nch);
  p.cb = static_cast<int32_t>(ceil_div(nb, nch));
  p.nch = static_cast<int32_t>(ceil_div(nb, p.cb));  // no empty chunk
  p.ng = static_cast<int32_t>(ceil_div(p.t1 - p.t0, group));
  return p;
}

__device__ __forceinline__ int group_size(const ReqPlan& p, int g, int group) {
  return min(group, p.t1 - (p.t0 + g * group));
}

// Exclusive prefix sum over the workgroup: an inclusive scan inside each
// wave by shuffles, then one scan of the 16 wave totals by the first wave.
// scan[kSchedThreads - 1] holds the total afterwards.
__device__ int64_t block_scan(int64_t* scan, int64_t mine) {
  constexpr int kWaves = kSchedThreads / 64;
  __shared__ int64_t wsum[kWaves];
  const int tid = threadIdx.x, lane = tid % 64, w = tid / 64;
  int64_t v = mine;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int64_t t = __shfl_up(v, off, 64);
    if (lane >= off) v += t;
  }
  if (lane == 63) wsum[w] = v;
  __syncthreads();
  if (w == 0) {
    int64_t x = lane < kWaves ? wsum[lane] : 0;
#pragma unroll
    for (int off = 1; off < kWaves; off <<= 1) {
      const int64_t t = __shfl_up(x, off, 64);
      if (lane >= off) x += t;
    }
    if (lane < kWaves) wsum[lane] = x;  // inclusive prefix of the wave totals
  }
  __syncthreads();
  const int64_t excl = (w > 0 ? wsum[w - 1] : 0) + v - mine;
  if (tid == kSchedThreads - 1) scan[tid] = wsum[kWaves - 1];
  __syncthreads();
  return excl;
}

// Size buckets of the by-size order: bucket of a unit of `size` blocks.
constexpr int kSizeBuckets = 32;
__device__ __forceinline__ int size_bucket(int size, int chunk_blocks) {
  return min(kSizeBuckets - 1, static_cast<int>((int64_t)size * kSizeBuckets / (chunk_blocks + 1)));
}

__global__ __launch_bounds__(kSchedThreads) void sched_kernel(const int32_t* __restrict__ hoff,
                                                              const int32_t* __restrict__ toff, int R,
                                                              int64_t n_hist, int64_t n_tgt,
                                                              int chunk_blocks, int group, int m_lo, int m_hi,
                                                              int by_size, unsigned deal,
                                                              Unit* __restrict__ units,
                                                              int64_t max_units,
                                                              int32_t* __restrict__ tchunks,
                                                              WsHeader* __restrict__ hdr) {
  __shared__ int64_t scan[kSchedThreads];
  __shared__ int bad;
  __shared__ unsigned cursor[2][kSizeBuckets];  // by_size: units, then next rank, per (class, bucket)
  const int tid = threadIdx.x;
  if (tid == 0) bad = (hoff[0] != 0 || toff[0] != 0 || hoff[R] != n_hist || toff[R] != n_tgt) ? 1 : 0;
  if (tid < 2 * kSizeBuckets) cursor[tid / kSizeBuckets][tid % kSizeBuckets] = 0;
  for (int64_t t = tid; t < n_tgt; t += kSchedThreads) tchunks[t] = 0;
  __syncthreads();

  const int per = static_cast<int>(ceil_div(R, kSchedThreads));
  const int rb = tid * per;
  const int re = min(R, rb + per);
  int64_t narrow = 0, wide = 0;
  bool any_bad = false;
  for (int r = rb; r < re; ++r) {
    ReqPlan p = plan_request(hoff, toff, r, n_hist, n_tgt, chunk_blocks, group, m_lo, m_hi);
    any_bad |= !p.ok;
    const int32_t bh = static_cast<int32_t>(ceil_div(p.h1, kBlockTokens));
    for (int g = 0; g < p.ng; ++g) {
      const int cls = group_size(p, g, group) > 32 ? 1 : 0;
      (cls ? wide : narrow) += p.nch;
      if (by_size)  // units per (class, size bucket)
        for (int c = 0; c < p.nch; ++c) {
          const int b0 = p.bl + c * p.cb;
          atomicAdd(&cursor[cls][size_bucket(min(b0 + p.cb, bh) - b0, chunk_blocks)], 1u);
        }
    }
  }
  if (any_bad) atomicOr(&bad, 1);
  int64_t un = block_scan(scan, narrow);
  const int64_t total_narrow = scan[kSchedThreads - 1];
  __syncthreads();
  int64_t uw = total_narrow + block_scan(scan, wide);
  const int64_t total = total_narrow + scan[kSchedThreads - 1];
  if (by_size) {
    // each bucket's rank range within its class, from the largest bucket down
    if (tid < 2) {
      unsigned pos = 0u;
      for (int k = kSizeBuckets - 1; k >= 0; --k) {
        const unsigned n = cursor[tid][k];
        cursor[tid][k] = pos;
        pos += n;
      }
    }
    __syncthreads();
  }
  for (int r = rb; r < re; ++r) {
    ReqPlan p = plan_request(hoff, toff, r, n_hist, n_tgt, chunk_blocks, group, m_lo, m_hi);
    if (p.nch == 0) continue;
    const int32_t bh = static_cast<int32_t>(ceil_div(p.h1, kBlockTokens));
    for (int g = 0; g < p.ng; ++g) {
      const int cls = group_size(p, g, group) > 32 ? 1 : 0;
      int64_t& ur = cls ? uw : un;
      for (int c = 0; c < p.nch; ++c, ++ur) {
        const int b0 = p.bl + c * p.cb;
        int64_t u = ur;
        if (by_size) {
          // rank k in the class's descending order; complete rounds of
          // `deal` units are dealt in alternating directions, so that a
          // workgroup taking a large unit in one round takes a small one in
          // the next
          const unsigned k = atomicAdd(&cursor[cls][size_bucket(min(b0 + p.cb, bh) - b0, chunk_blocks)], 1u);
          const unsigned nc = static_cast<unsigned>(cls ? total - total_narrow : total_narrow);
          const unsigned j = k / deal, i = k - j * deal;
          const bool back = (j & 1) && (j + 1) * deal <= nc;
          u = (cls ? total_narrow : 0) + static_cast<int64_t>(j) * deal + (back ? deal - 1 - i : i);
        }
        if (u >= max_units) continue;
        Unit un_;
        un_.r = r;
        un_.t0 = p.t0 + g * group;
        un_.nt = group_size(p, g, group);
        un_.c = c;
        un_.b0 = p.bl + c * p.cb;
        un_.b1 = min(un_.b0 + p.cb, bh);
        un_.l0 = p.h0;
        un_.l1 = p.h1;
        units[u] = un_;
      }
    }
    for (int t = p.t0; t < p.t1; ++t) tchunks[t] = p.nch;
  }
  if (tid == 0) {
    hdr->n_units = static_cast<int32_t>(total < max_units ? total : max_units);
    hdr->n_narrow = static_cast<int32_t>(total_narrow < max_units ? total_narrow : max_units);
    hdr->status = (bad || total > max_units) ? STCA_ERR_INVALID_ARG : STCA_OK;
    hdr->range = 0;  // set by later kernels of the call that find an fp16 overflow
  }
}

}  // namespace

hipError_t launch_sched(const int32_t* hoff, const int32_t* toff, int R, int64_t n_hist, int64_t n_tgt,
                        int chunk_blocks, int group, Unit* units, int64_t max_units, int32_t* tchunks,
                        WsHeader* hdr, hipStream_t st, int m_lo, int m_hi, int deal) {
  if (group < 1 || group > kWideGroup || deal < 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(sched_kernel, dim3(1), dim3(kSchedThreads), 0, st, hoff, toff, R, n_hist, n_tgt,
                     chunk_blocks, group, m_lo, m_hi, deal > 0 ? 1 : 0, static_cast<unsigned>(deal > 0 ? deal : 1),
                     units, max_units, tchunks, hdr);
  return hipGetLastError();
}

// Host mirror of plan_request for exact unit counts when host offsets exist.
int64_t host_count_units(const int32_t* hoff, const int32_t* toff, int R, int chunk_blocks, int group, int m_lo,
                         int m_hi) {
  int64_t n = 0;
  for (int r = 0; r < R; ++r) {
    const int64_t h0 = hoff[r], h1 = hoff[r + 1], t0 = toff[r], t1 = toff[r + 1];
    if (t1 == t0 || t1 - t0 < m_lo || t1 - t0 > m_hi) continue;
    const int64_t nb = ceil_div(h1, kBlockTokens) - h0 / kBlockTokens;
    int64_t nch = ceil_div(nb, chunk_blocks);
    nch = nch < 1 ? 1 : (nch > kMaxChunks ? kMaxChunks : nch);
    const int64_t cb = ceil_div(nb, nch);
    n += ceil_div(nb, cb) * ceil_div(t1 - t0, group);
  }
  return n;
}

}  // namespace stca
