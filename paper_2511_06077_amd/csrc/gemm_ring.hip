// Streaming MFMA GEMM for the backward's products over history rows, the
// largest of the training step: the projection weight gradients
// [dW_K | dW_V] = X^T [dK | dV] (K = every history row of the batch, split
// over K) and the history gradient dX = [dK | dV] [W_K | W_V]^T (M = every
// history row).  Both stream one large bf16 operand ([dK | dV], about 1 KB
// per history row and layer pair) past a small one that stays in L2, so they
// are bound by how many bytes each CU keeps in flight rather than by the
// matrix cores.
//
// One workgroup of eight waves per CU (two per SIMD, each with a 64 x 64
// share of the output tile), persistent over its work items (output
// tile x K range).  Operand tiles go from global memory straight into an LDS
// ring of NS stages with gfx950's direct loads (16 bytes per lane, no
// register staging); NS - 1 stages are in flight while one is multiplied, and
// a wave's loads for the next work item start while it finishes the current
// one.  The output tile spans the whole of the small output extent (256 or
// 128 x 256), so the streamed operand is read from HBM exactly once.  At the
// 256-request, 2048-row training window this takes [dW_K | dW_V] from 0.81 to
// 0.67 ms and dX from 0.72 to 0.64 ms against the register-staged kernel of
// gemm.hip; one wave per SIMD (four waves with 64 x 128 shares), four per
// SIMD (32 x 64 shares) and 32-deep stages (six in the ring) were all slower.
//
// LDS forms (16-byte units, no padding, so that the direct loads, which write
// 1 KB runs, can fill them; conflict-free for the 16-byte and transposing
// reads that feed v_mfma_f32_32x32x16_bf16):
//   k contiguous in the source: one row per output row, BK k; unit u of row
//     r sits at position u ^ ((r / G) % (BK / 8)), G = 128 / BK, so that the
//     16 rows a 16-lane read phase touches cover all 64 banks;
//   rows contiguous in the source: one run of R rows per k; unit c of k row
//     k sits at position c ^ 4 (k % 4), so that the four k rows one
//     transposing read gathers (same 32 rows) fall on disjoint bank quarters.
// The direct loads place lane i's 16 bytes at a fixed LDS offset, so each
// lane fetches the source unit that the permutation puts there; vectors
// outside the operands (row or k tails) are fetched from a zero vector.
#include <algorithm>

#include "common.h"
#include "internal.h"
#include "ring.h"

namespace stca {

namespace {

constexpr int kRingWaves = 8;
constexpr int kRingThreads = 64 * kRingWaves;
constexpr int kRingLds = 144 * 1024;
constexpr int kXcds = 8;

// the source of every vector outside the operands
__device__ const uint4 kZero16[1] = {};

__device__ __forceinline__ f32x16 mfma_bf(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// s_waitcnt: at most N vector memory operations of this wave outstanding,
// LDS operations drained (gfx9 encoding: vmcnt bits 3:0 and 15:14)
template <int N>
__device__ __forceinline__ void wait_vm_n() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
}

// Geometry of one operand tile of R rows (output rows or columns) x BK k.
template <bool KC, int R, int BK>
struct Tile {
  static constexpr int kBytes = R * BK * 2;
  static constexpr int kChunks = kBytes / 1024;  // 1 KB runs of the direct loads
  static constexpr int kUpr = BK / 8;            // k units per row (k contiguous)
  static constexpr int kGrp = 16 / kUpr;         // rows per bank-permutation step
  static_assert(kChunks % kRingWaves == 0, "each wave loads whole runs");

  // byte offset of the unit holding (row r, k 8 u .. 8 u + 7) [k contiguous]
  __device__ static int kc_off(int r, int u) { return r * (BK * 2) + 16 * (u ^ ((r / kGrp) % kUpr)); }
  // byte offset of (k row k, rows 8 c .. 8 c + 7) [rows contiguous]
  __device__ static int rc_off(int k, int c) { return k * (2 * R) + 16 * (c ^ (4 * (k % 4))); }

  // This wave's share of the direct loads of the tile rows row0.., k k0..
  // (valid below nrows and kend) into lds.
  __device__ static void load(const bf16_bits* __restrict__ src, int64_t ld, int row0, int nrows, int k0, int kend,
                              const unsigned char* lds, int wave, int lane) {
#pragma unroll
    for (int i = 0; i < kChunks / kRingWaves; ++i) {
      const int q = wave + kRingWaves * i;
      const int o = 1024 * q + 16 * lane;
      int r, kk;
      if (KC) {
        r = o / (BK * 2);
        kk = 8 * (((o / 16) % kUpr) ^ ((r / kGrp) % kUpr));
      } else {
        kk = o / (2 * R);
        r = 8 * (((o / 16) % (R / 8)) ^ (4 * (kk % 4)));
      }
      const bool ok = row0 + r < nrows && k0 + kk < kend;
      const bf16_bits* g = KC ? src + (int64_t)(row0 + r) * ld + k0 + kk : src + (int64_t)(k0 + kk) * ld + row0 + r;
      dma16(ok ? static_cast<const void*>(g) : static_cast<const void*>(kZero16), lds + 1024 * q);
    }
  }

  // MFMA operand of rows m0 .. m0 + 31 for k-step ks: lane l holds row
  // m0 + l % 32, k = 16 ks + 8 (l / 32) + e.  Rows contiguous: two
  // transposing reads of four k each; in a 16-lane group lane j addresses k
  // row j / 4 and rows 4 (j % 4) .. + 3 and receives its own row's four k.
  __device__ static bf16x8 op(const unsigned char* lds, int m0, int ks, int lane) {
    if (KC) return *reinterpret_cast<const bf16x8*>(lds + kc_off(m0 + lane % 32, 2 * ks + lane / 32));
    const int j = lane % 16;
    const int m = m0 + 16 * ((lane / 16) % 2) + 4 * (j % 4);
    const int k = 16 * ks + 8 * (lane / 32) + j / 4;
    const tr16x4 lo = lds_read_tr16(lds + rc_off(k, m / 8) + 2 * (m % 8));
    const tr16x4 hi = lds_read_tr16(lds + rc_off(k + 4, m / 8) + 2 * (m % 8));
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  }
};

struct RingProblem {
  int M, N, K;
  const bf16_bits* A;
  int64_t lda;
  const bf16_bits* B;
  int64_t ldb;
  float* C;
  int64_t ldc;
  float alpha;
  int accumulate, k_chunk, tiles_m, tiles_n, splits, n_work;
  float* part;  // per-split partial tiles, or null (no split)
  // unit mode (units non-null): work item u covers rows
  // [max(32 b0, l0), min(32 b1, l1)) of unit u (of hdr->n_units), all N and
  // all K, with B advanced by b_stride per request
  const Unit* units;
  const WsHeader* hdr;
  int64_t b_stride;
};

// Work item in flight: output rows (from m0, below mend, BM per tile), K
// range, and progress (ks over tiles x kpt k-steps).
struct Cursor {
  int round, ks, nks, kpt, m0, mend, n0, kb, ke, split;
  int64_t bofs;
  bool done;
};

template <int BM, int BN, int BK>
__device__ __forceinline__ void set_item(const RingProblem& P, Cursor& c) {
  // Workgroups are dealt to the XCDs round robin: in each round, XCD x takes
  // a contiguous range of work items (those of one K range share an operand).
  const int G = gridDim.x, b = blockIdx.x;
  c.ks = 0;
  if (P.units) {
    const int n = P.hdr->n_units;
    for (;;) {  // the next unit with rows (units are never empty; the check keeps the loop safe)
      const int id = c.round * G + (b % kXcds) * (G / kXcds) + b / kXcds;
      if (id >= n) {
        c.done = true;
        return;
      }
      const Unit u = P.units[id];
      c.m0 = max(u.b0 * kBlockTokens, u.l0);
      c.mend = min(u.b1 * kBlockTokens, u.l1);
      c.n0 = 0;
      c.kb = 0;
      c.ke = P.K;
      c.split = 0;
      c.bofs = (int64_t)u.r * P.b_stride;
      c.kpt = (P.K + BK - 1) / BK;
      c.nks = c.mend > c.m0 ? c.kpt * ((c.mend - c.m0 + BM - 1) / BM) : 0;
      if (c.nks > 0) return;
      ++c.round;
    }
  }
  const int id = c.round * G + (b % kXcds) * (G / kXcds) + b / kXcds;
  if (id >= P.n_work) {
    c.done = true;
    return;
  }
  const int tiles = P.tiles_m * P.tiles_n;
  c.split = id / tiles;
  const int t = id % tiles;
  c.m0 = (t / P.tiles_n) * BM;
  c.mend = P.M;
  c.n0 = (t % P.tiles_n) * BN;
  c.kb = c.split * P.k_chunk;
  c.ke = min(P.K, c.kb + P.k_chunk);
  c.bofs = 0;
  c.nks = c.kpt = (c.ke - c.kb + BK - 1) / BK;
}

template <int BM, int BN, int BK>
__device__ __forceinline__ void advance(const RingProblem& P, Cursor& c) {
  if (++c.ks == c.nks) {
    ++c.round;
    set_item<BM, BN, BK>(P, c);
  }
}

// wait until at most `later` stages (of PER loads each) are still in flight
template <int PER, int NS>
__device__ __forceinline__ void wait_stages(int later) {
  static_assert(NS <= 6, "up to four later stages");
  if (NS > 5 && later >= 4) return wait_vm_n<(NS > 5 ? 4 * PER : 0)>();
  if (NS > 4 && later >= 3) return wait_vm_n<(NS > 4 ? 3 * PER : 0)>();
  if (NS > 3 && later >= 2) return wait_vm_n<(NS > 3 ? 2 * PER : 0)>();
  if (later >= 1) return wait_vm_n<PER>();
  wait_vm_n<0>();
}

// Store alpha * acc for a wave's TM x TN result tiles at rows m0..,
// columns n0.. and clear them; CHECK: bounds per element.
// Result lane layout: column n = lane % 32, rows 8 (v / 4) + 4 hi + v % 4.
template <int TM, int TN, bool CHECK>
__device__ __forceinline__ void put_tile(f32x16 (&acc)[TM][TN], float* __restrict__ out, int64_t ldo, int m0, int n0,
                                         int M, int N, float alpha, int lane) {
  const int hi = lane / 32;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = n0 + 32 * j + lane % 32;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int m = m0 + 32 * i + 8 * (v / 4) + 4 * hi + (v % 4);
        if (!CHECK || (m < M && n < N)) out[(int64_t)m * ldo + n] = alpha * acc[i][j][v];
      }
      acc[i][j] = f32x16{};
    }
}

template <bool A_KC, bool B_KC, int BM, int BN, int BK, int NS>
__global__ __launch_bounds__(kRingThreads, 2) void ring_gemm_kernel(RingProblem P) {
  using TA = Tile<A_KC, BM, BK>;
  using TB = Tile<B_KC, BN, BK>;
  constexpr int SB = TA::kBytes + TB::kBytes;
  constexpr int PER = (TA::kChunks + TB::kChunks) / kRingWaves;  // loads per wave per stage
  constexpr int WM = BM / 64;  // waves along M, each with a 64 x 64 share: 2 x 2 tiles of 32 x 32
  constexpr int TM = 2, TN = 2;
  static_assert(WM * (BN / 64) == kRingWaves, "one 64 x 64 share per wave");
  static_assert(NS * SB <= kRingLds, "LDS ring size");
  __shared__ __attribute__((aligned(1024))) unsigned char ring[NS * SB];

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
  const int lane = threadIdx.x % 64;
  const int wm = (wave % WM) * 64, wn = (wave / WM) * 64;

  Cursor ci{0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, false};
  set_item<BM, BN, BK>(P, ci);
  if (ci.done) return;
  Cursor cc = ci;

  auto issue = [&](int slot) {
    const unsigned char* s = ring + slot * SB;
    const int k0 = ci.kb + (ci.ks % ci.kpt) * BK;
    TA::load(P.A, P.lda, ci.m0 + (ci.ks / ci.kpt) * BM, ci.mend, k0, ci.ke, s, wave, lane);
    TB::load(P.B + ci.bofs, P.ldb, ci.n0, P.N, k0, ci.ke, s + TA::kBytes, wave, lane);
    advance<BM, BN, BK>(P, ci);
  };

  int issued = 0;
#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    if (!ci.done) {
      issue(s);
      ++issued;
    }

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x16{};

  for (int step = 0; !cc.done; ++step) {
    wait_stages<PER, NS>(issued - step - 1);
    ring_barrier();
    if (!ci.done) {
      issue(issued % NS);
      ++issued;
    }
    const unsigned char* as = ring + (step % NS) * SB;
    const unsigned char* bs = as + TA::kBytes;
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 a[TM], b[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) a[i] = TA::op(as, wm + 32 * i, ks, lane);
#pragma unroll
      for (int j = 0; j < TN; ++j) b[j] = TB::op(bs, wn + 32 * j, ks, lane);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma_bf(a[i], b[j], acc[i][j]);
    }
    if ((cc.ks + 1) % cc.kpt == 0) {
      const int mt = cc.m0 + (cc.ks / cc.kpt) * BM;
      const int m0 = mt + wm, n0 = cc.n0 + wn;
      const bool full = mt + BM <= cc.mend && cc.n0 + BN <= P.N;
      if (P.part) {
        float* out = P.part + (int64_t)cc.split * P.M * P.N;
        if (full) put_tile<TM, TN, false>(acc, out, P.N, m0, n0, P.M, P.N, 1.f, lane);
        else put_tile<TM, TN, true>(acc, out, P.N, m0, n0, P.M, P.N, 1.f, lane);
      } else {
        if (full) put_tile<TM, TN, false>(acc, P.C, P.ldc, m0, n0, cc.mend, P.N, P.alpha, lane);
        else put_tile<TM, TN, true>(acc, P.C, P.ldc, m0, n0, cc.mend, P.N, P.alpha, lane);
      }
    }
    advance<BM, BN, BK>(P, cc);
  }
}

__global__ void ring_split_sum_kernel(const float* __restrict__ part, int splits, int M, int N,
                                      float* __restrict__ C, int64_t ldc, float alpha, int accumulate) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)M * N) return;
  float s = 0.f;
  for (int k = 0; k < splits; ++k) s += part[(int64_t)k * M * N + i];
  float* c = C + (i / N) * ldc + i % N;
  *c = accumulate ? *c + alpha * s : alpha * s;
}

constexpr int kBK = 64, kNS = 3;

bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Output tile: the whole of the smaller output extent where it fits (256 x
// 128 when M <= N, else 128 x 256), so that the long operand is read once.
bool wide_m(int M, int N) { return M <= N; }

// Splits over K of a product with fewer output tiles than twice the CUs: about
// two work items per CU, each K range at least 1024 deep.
int64_t ring_splits(int M, int N, int K, int n_cu) {
  const bool wm = wide_m(M, N);
  const int64_t tiles = ceil_div(M, wm ? 256 : 128) * ceil_div(N, wm ? 128 : 256);
  if (tiles >= 2 * n_cu || K < 2048) return 1;
  return std::max<int64_t>(1, std::min<int64_t>(ceil_div(2 * n_cu, tiles), K / 1024));
}

template <typename Launch>
void by_form(bool a_kc, bool b_kc, bool wm, Launch launch) {
  auto pick = [&](auto f) {
    if (wm) launch(f, std::integral_constant<bool, true>{});
    else launch(f, std::integral_constant<bool, false>{});
  };
  if (a_kc && b_kc) pick(std::integral_constant<int, 3>{});
  else if (a_kc) pick(std::integral_constant<int, 2>{});
  else if (b_kc) pick(std::integral_constant<int, 1>{});
  else pick(std::integral_constant<int, 0>{});
}

}  // namespace

int64_t gemm_ring_part_floats(int M, int N, int K, int n_cu) {
  const int64_t s = ring_splits(M, N, K, n_cu);
  return s > 1 ? s * M * N : 0;
}

hipError_t gemm_ring(int M, int N, int K, const bf16_bits* A, int64_t lda, int transA, const bf16_bits* B,
                     int64_t ldb, int transB, float* C, int64_t ldc, float alpha, int accumulate, float* part,
                     int64_t part_floats, int n_cu, hipStream_t st) {
  if (M == 0 || N == 0) return hipSuccess;
  if (K == 0)
    return gemm_mfma(M, N, K, A, lda, transA, B, ldb, transB, C, ldc, alpha, accumulate, nullptr, 0, st);
  const bool a_kc = !transA, b_kc = transB != 0;
  if ((a_kc ? K : M) % 8 || (b_kc ? K : N) % 8 || lda % 8 || ldb % 8 || !al16(A) || !al16(B) || n_cu < 1)
    return hipErrorInvalidValue;
  const bool wm = wide_m(M, N);
  const int bm = wm ? 256 : 128, bn = wm ? 128 : 256;
  int splits = 1;
  if (part) {
    splits = static_cast<int>(ring_splits(M, N, K, n_cu));
    while (splits > 1 && (int64_t)splits * M * N > part_floats) --splits;
  }
  const int k_chunk = static_cast<int>(round_up(ceil_div(K, splits), kBK));
  splits = static_cast<int>(ceil_div(K, k_chunk));
  // the kernel stores its tiles (adding to C is left to the split sum)
  if (accumulate && splits == 1)
    return gemm_mfma(M, N, K, A, lda, transA, B, ldb, transB, C, ldc, alpha, accumulate, nullptr, 0, st);
  const int64_t tm = ceil_div(M, bm), tn = ceil_div(N, bn);
  const int64_t work = tm * tn * splits;
  if (work > 0x7fffffff) return hipErrorInvalidValue;
  RingProblem P{M, N, K, A, lda, B, ldb, C, ldc, alpha, accumulate, k_chunk, static_cast<int>(tm),
                static_cast<int>(tn), splits, static_cast<int>(work), splits > 1 ? part : nullptr, nullptr, nullptr,
                0};
  // one workgroup per CU (the ring takes most of the LDS), a multiple of
  // the XCD count
  const int64_t grid = round_up(std::min<int64_t>(work, n_cu), kXcds);
  by_form(a_kc, b_kc, wm, [&](auto f, auto w) {
    constexpr int F = decltype(f)::value;
    constexpr bool W = decltype(w)::value;
    hipLaunchKernelGGL((ring_gemm_kernel<(F & 2) != 0, (F & 1) != 0, W ? 256 : 128, W ? 128 : 256, kBK, kNS>),
                       dim3(static_cast<unsigned>(grid)), dim3(kRingThreads), 0, st, P);
  });
  if (P.part)
    hipLaunchKernelGGL(ring_split_sum_kernel, dim3(static_cast<unsigned>(ceil_div((int64_t)M * N, 256))), dim3(256),
                       0, st, P.part, P.splits, M, N, C, ldc, alpha, accumulate);
  return hipGetLastError();
}

hipError_t gemm_ring_units(int N, int K, const bf16_bits* A, int64_t lda, const bf16_bits* B, int64_t ldb,
                           int64_t b_stride, float* C, int64_t ldc, const Unit* units, const WsHeader* hdr,
                           int n_cu, hipStream_t st) {
  if (N == 0 || K == 0) return hipSuccess;
  if (K % 8 || N % 8 || lda % 8 || ldb % 8 || b_stride % 8 || !al16(A) || !al16(B) || n_cu < 1)
    return hipErrorInvalidValue;
  RingProblem P{0, N, K, A, lda, B, ldb, C, ldc, 1.f, 0, K, 1, static_cast<int>(ceil_div(N, 256)), 1, 0, nullptr,
                units, hdr, b_stride};
  if (N > 256) return hipErrorInvalidValue;  // one tile spans N
  hipLaunchKernelGGL((ring_gemm_kernel<true, false, 128, 256, kBK, kNS>), dim3(static_cast<unsigned>(round_up(n_cu, kXcds))),
                     dim3(kRingThreads), 0, st, P);
  return hipGetLastError();
}

}  // namespace stca
