// MFMA GEMM with bf16 operands and fp32 accumulation for the backward pass:
//   C[M,N] (fp32) = alpha * op(A) op(B)  (+ C when accumulating)
// Products: the per-layer K/V of the history ([K | V] = X [W_K | W_V], one
// product for both), the projection weight gradients ([dW_K | dW_V] =
// X^T [dK | dV], K = history rows, split over K), the history gradient
// (dX += [dK | dV] [W_K | W_V]^T) and the target-side products of the
// training window (weight gradients with K = targets).
//
// 128 x 128 output tile per workgroup of four waves (2 x 2), each wave 64 x 64
// as 2 x 2 v_mfma_f32_32x32x16_bf16 tiles.  64-deep k tiles go global ->
// registers (16-byte loads, the next tile's loads in flight while the current
// one is multiplied) -> LDS (one buffer, 37 KB, so four workgroups share a
// CU) -> MFMA operands.  An operand whose source has k contiguous is copied
// row by row into rows padded by 16 bytes and read back 16 bytes per lane.
// One whose source has the row index contiguous (X and dK | dV in
// [dW_K | dW_V], both operands of the target-side weight gradients) keeps
// that layout in LDS (one 256-byte row per k, 16-byte units permuted per
// k row) and is read back with gfx950's transposing LDS reads, which hand
// each lane four consecutive k of its own row.  Neither form meets LDS bank
// conflicts on writes or reads.  Tiles are handed to the eight XCDs in
// contiguous ranges, so the tiles that share a row block of A (and, split
// over K, every tile of one K range) run on one XCD and share its L2.  A
// split over K writes per-split partial tiles that a second kernel sums.
#include <algorithm>

#include "common.h"
#include "internal.h"
#include "ring.h"

namespace stca {

namespace {

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int LROW = BK + 8;  // padded LDS row, in bf16 elements (144 bytes)
constexpr int kXcds = 8;

typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f32x16 mfma_bf(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// One operand tile: 128 rows x 64 k = 1024 vectors of 8 bf16, four per thread
// (vector v = thread + 256 i).  kcontig: element (row, k) at src[row * ld + k],
// vector v = row v / 8, k 8 (v % 8) .. + 7; else at src[k * ld + row],
// vector v = k v / 16, rows 8 (v % 16) .. + 7 (16 threads read one 256-byte
// run of a k row).  Vectors are whole or absent: the caller guarantees that
// the contiguous extent (K, or the row count) is a multiple of 8 and chunk
// ends are multiples of BK.
template <bool kcontig>
__device__ __forceinline__ void load_tile(u16x8 (&r)[4], const bf16_bits* __restrict__ src, int64_t ld, int row0,
                                          int nrows, int k0, int kend) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int v = threadIdx.x + 256 * i;
    bool ok;
    int64_t off;
    if (kcontig) {
      const int row = v / (BK / 8), kk = (v % (BK / 8)) * 8;
      ok = row0 + row < nrows && k0 + kk < kend;
      off = (int64_t)(row0 + row) * ld + k0 + kk;
    } else {
      const int kk = v / (BM / 8), row = (v % (BM / 8)) * 8;
      ok = k0 + kk < kend && row0 + row < nrows;
      off = (int64_t)(k0 + kk) * ld + row0 + row;
    }
    r[i] = ok ? *reinterpret_cast<const u16x8*>(src + off) : u16x8{0, 0, 0, 0, 0, 0, 0, 0};
  }
}

// LDS offsets, in bf16 elements.  k contiguous: the 8-k unit u (k = 8u ..
// 8u + 7) of row m in padded rows of LROW (144 bytes: the 16 lanes of a
// 16-byte read phase, 16 consecutive rows, start 9 units apart mod 16 and
// cover all 64 banks).  Rows contiguous: k row k is 256 bytes (128 rows m,
// exactly the 64 banks) whose 16-byte units are permuted by 4 (k % 4), so
// that the four k rows a transposing read gathers (same 64-byte run of m)
// fall on four disjoint quarters of the banks.
__device__ __forceinline__ int lds_kc(int m, int u) { return m * LROW + 8 * u; }
__device__ __forceinline__ int lds_rc(int k, int m) { return k * BM + 8 * ((m / 8) ^ (4 * (k % 4))) + m % 8; }

template <bool kcontig>
__device__ __forceinline__ void store_tile(bf16_bits* __restrict__ lds, const u16x8 (&r)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int v = threadIdx.x + 256 * i;
    const int off = kcontig ? lds_kc(v / (BK / 8), v % (BK / 8)) : lds_rc(v / (BM / 8), (v % (BM / 8)) * 8);
    *reinterpret_cast<u16x8*>(lds + off) = r[i];
  }
}

// MFMA operand of 32 rows m0 .. m0 + 31 for k-step ks (k = 16 ks .. + 15):
// lane l holds row m0 + l % 32, k = 16 ks + 8 (l / 32) + e, e = 0..7.  Rows
// contiguous in LDS: two transposing reads, each giving four k; within a
// 16-lane group (16 rows m) lane j addresses k row j / 4 of the four and the
// four rows m 4 (j % 4) .. + 3, and receives its own row m's four k.
template <bool kcontig>
__device__ __forceinline__ bf16x8 read_op(const bf16_bits* __restrict__ lds, int m0, int ks, int lane) {
  if (kcontig) return *reinterpret_cast<const bf16x8*>(lds + lds_kc(m0 + lane % 32, 2 * ks + lane / 32));
  const int j = lane % 16;
  const int m = m0 + 16 * ((lane / 16) % 2) + 4 * (j % 4);
  const int k = 16 * ks + 8 * (lane / 32) + j / 4;
  const tr16x4 lo = lds_read_tr16(reinterpret_cast<const unsigned char*>(lds + lds_rc(k, m)));
  const tr16x4 hi = lds_read_tr16(reinterpret_cast<const unsigned char*>(lds + lds_rc(k + 4, m)));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// op(A) element (m, k): A[m * lda + k] if A_KC else A[k * lda + m].
// op(B) element (k, n): B[n * ldb + k] if B_KC else B[k * ldb + n].
// One work item (output tile, K split) of a product.
struct GemmProblem {
  int M, N, K;
  const bf16_bits* A;
  int64_t lda;
  const bf16_bits* B;
  int64_t ldb;
  float* C;
  int64_t ldc;
  float alpha;
  int accumulate, k_chunk, n_tiles_m, n_tiles_n, splits;
  int work_begin;  // first work item of this product in a grouped launch
  float* part;     // per-split partial tiles, or null (no split)
};

// workgroups are dealt to the XCDs round robin by their linear index: give
// each XCD a contiguous range of work items
__device__ __forceinline__ int xcd_work_id() {
  const int per = gridDim.x / kXcds;
  return (blockIdx.x % kXcds) * per + blockIdx.x / kXcds;
}

template <bool A_KC, bool B_KC>
__device__ __forceinline__ void gemm_work(const GemmProblem& P, int w_id, bf16_bits* __restrict__ As,
                                          bf16_bits* __restrict__ Bs) {
  const int M = P.M, N = P.N, K = P.K, k_chunk = P.k_chunk, n_tiles_m = P.n_tiles_m, n_tiles_n = P.n_tiles_n;
  const bf16_bits* __restrict__ A = P.A;
  const bf16_bits* __restrict__ B = P.B;
  const int64_t lda = P.lda, ldb = P.ldb, ldc = P.ldc;
  float* __restrict__ C = P.C;
  float* __restrict__ part = P.part;
  const float alpha = P.alpha;
  const int accumulate = P.accumulate;
  const int tiles = n_tiles_m * n_tiles_n;
  const int split = w_id / tiles, t = w_id % tiles;
  const int m0 = (t / n_tiles_n) * BM, n0 = (t % n_tiles_n) * BN;
  const int kb = split * k_chunk;
  const int ke = min(K, kb + k_chunk);

  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int wm = (wave / 2) * 64, wn = (wave % 2) * 64;
  const int r32 = lane % 32, hi = lane / 32;
  f32x16 acc[2][2] = {};
  u16x8 ra[4], rb[4];
  load_tile<A_KC>(ra, A, lda, m0, M, kb, ke);
  load_tile<B_KC>(rb, B, ldb, n0, N, kb, ke);
  store_tile<A_KC>(As, ra);
  store_tile<B_KC>(Bs, rb);
  __syncthreads();
  for (int k0 = kb; k0 < ke; k0 += BK) {
    const bool more = k0 + BK < ke;
    if (more) {
      load_tile<A_KC>(ra, A, lda, m0, M, k0 + BK, ke);
      load_tile<B_KC>(rb, B, ldb, n0, N, k0 + BK, ke);
    }
    const bf16_bits* as = As;
    const bf16_bits* bs = Bs;
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        a[i] = read_op<A_KC>(as, wm + 32 * i, ks, lane);
        b[i] = read_op<B_KC>(bs, wn + 32 * i, ks, lane);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = mfma_bf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
    if (more) {
      store_tile<A_KC>(As, ra);
      store_tile<B_KC>(Bs, rb);
    }
    __syncthreads();
  }
  // result lane layout: column n = lane % 32, rows 8 (v / 4) + 4 hi + v % 4
  float* out = part ? part + (int64_t)split * M * N : C;
  const int64_t ldo = part ? N : ldc;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int n = n0 + wn + 32 * j + r32;
      if (n >= N) continue;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int m = m0 + wm + 32 * i + 8 * (v / 4) + 4 * hi + (v % 4);
        if (m >= M) continue;
        float* c = out + (int64_t)m * ldo + n;
        if (part)
          *c = acc[i][j][v];
        else
          *c = accumulate ? *c + alpha * acc[i][j][v] : alpha * acc[i][j][v];
      }
    }
}

template <bool A_KC, bool B_KC>
__global__ __launch_bounds__(256) void mfma_gemm_kernel(GemmProblem P, int n_work) {
  __shared__ __attribute__((aligned(16))) bf16_bits As[BM * LROW];
  __shared__ __attribute__((aligned(16))) bf16_bits Bs[BN * LROW];
  const int w_id = xcd_work_id();
  if (w_id >= n_work) return;
  gemm_work<A_KC, B_KC>(P, w_id, As, Bs);
}

// Up to kMaxGroup products (same operand forms) in one launch, their work
// items numbered consecutively.
constexpr int kMaxGroup = 16;
struct GemmGroup {
  GemmProblem p[kMaxGroup];
  int n;
};

template <bool A_KC, bool B_KC>
__global__ __launch_bounds__(256) void mfma_gemm_group_kernel(GemmGroup G, int n_work) {
  __shared__ __attribute__((aligned(16))) bf16_bits As[BM * LROW];
  __shared__ __attribute__((aligned(16))) bf16_bits Bs[BN * LROW];
  const int w_id = xcd_work_id();
  if (w_id >= n_work) return;
  int q = 0;
#pragma unroll
  for (int i = 1; i < kMaxGroup; ++i)
    if (i < G.n && w_id >= G.p[i].work_begin) q = i;
  gemm_work<A_KC, B_KC>(G.p[q], w_id - G.p[q].work_begin, As, Bs);
}

__global__ void split_sum_kernel(const float* __restrict__ part, int splits, int M, int N, float* __restrict__ C,
                                 int64_t ldc, float alpha, int accumulate) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)M * N) return;
  float s = 0.f;
  for (int k = 0; k < splits; ++k) s += part[(int64_t)k * M * N + i];
  float* c = C + (i / N) * ldc + i % N;
  *c = accumulate ? *c + alpha * s : alpha * s;
}

// split_sum_kernel over every split product of a group, one thread per
// output element, the products' elements numbered consecutively
__global__ void split_sum_group_kernel(GemmGroup G) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (int q = 0; q < G.n; ++q) {
    const GemmProblem& P = G.p[q];
    if (!P.part) continue;
    const int64_t mn = (int64_t)P.M * P.N;
    if (i < mn) {
      float s = 0.f;
      for (int k = 0; k < P.splits; ++k) s += P.part[(int64_t)k * mn + i];
      float* c = P.C + (i / P.N) * P.ldc + i % P.N;
      *c = P.accumulate ? *c + P.alpha * s : P.alpha * s;
      return;
    }
    i -= mn;
  }
}

bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// dst[c * ldd + r] = src[r * lds + c] for r < R, c < C; dst columns r in
// [R, Rp) are zeroed.  64 x 64 tiles through LDS with 16-byte global reads
// and writes (eight consecutive columns in, eight consecutive rows out).
__global__ __launch_bounds__(256) void transpose_kernel(const bf16_bits* __restrict__ src, int64_t lds, int R, int C,
                                                        bf16_bits* __restrict__ dst, int64_t ldd, int Rp) {
  constexpr int TR = 64 + 2;  // padded LDS row (bf16): column reads spread over the banks
  __shared__ bf16_bits t[64 * TR];
  const int r0 = blockIdx.x * 64, c0 = blockIdx.y * 64;
  const bool vec_in = (C % 8) == 0 && (lds % 8) == 0;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int v = threadIdx.x + 256 * i;
    const int rr = v / 8, cc = (v % 8) * 8;
    const int r = r0 + rr, c = c0 + cc;
    u16x8 x = {0, 0, 0, 0, 0, 0, 0, 0};
    if (r < R) {
      if (vec_in && c + 8 <= C) {
        x = *reinterpret_cast<const u16x8*>(src + (int64_t)r * lds + c);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = c + e < C ? src[(int64_t)r * lds + c + e] : bf16_bits(0);
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) t[rr * TR + cc + e] = x[e];
  }
  __syncthreads();
  const bool vec_out = (ldd % 8) == 0 && (Rp % 8) == 0;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int v = threadIdx.x + 256 * i;
    const int cc = v / 8, rr = (v % 8) * 8;
    const int c = c0 + cc, r = r0 + rr;
    if (c >= C || r >= Rp) continue;
    u16x8 y;
#pragma unroll
    for (int e = 0; e < 8; ++e) y[e] = t[(rr + e) * TR + cc];
    if (vec_out && r + 8 <= Rp) {
      *reinterpret_cast<u16x8*>(dst + (int64_t)c * ldd + r) = y;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (r + e < Rp) dst[(int64_t)c * ldd + r + e] = y[e];
    }
  }
}

}  // namespace

hipError_t transpose_bf16(const bf16_bits* src, int64_t lds, int R, int C, bf16_bits* dst, int64_t ldd, int Rp,
                          hipStream_t st) {
  if (Rp == 0 || C == 0) return hipSuccess;
  hipLaunchKernelGGL(transpose_kernel, dim3(static_cast<unsigned>(ceil_div(Rp, 64)),
                                            static_cast<unsigned>(ceil_div(C, 64))),
                     dim3(256), 0, st, src, lds, R, C, dst, ldd, Rp);
  return hipGetLastError();
}

namespace {
// Splits over K of a product with few output tiles: enough partial tiles for
// about 2048 workgroups (two rounds of the four a CU holds, so one round's
// loads overlap the other's products: [dW_K | dW_V] at the training window
// 0.86 -> 0.82 ms against 1024), each split at least 512 deep (the target
// side's weight gradients over 4096 targets: 8 splits instead of 16 halve the
// partials the split sum reads, 0.54 -> 0.52 ms of target-side products per
// training step; 1024 deep starves the K/V-side products of workgroups).
int64_t k_splits(int M, int N, int K) {
  const int64_t tiles = ceil_div(M, BM) * ceil_div(N, BN);
  if (tiles >= 256 || K < 1024) return 1;
  return std::max<int64_t>(1, std::min<int64_t>(ceil_div(2048, tiles), K / 512));
}
}  // namespace

int64_t gemm_mfma_part_floats(int M, int N, int K) {
  const int64_t s = k_splits(M, N, K);
  return s > 1 ? s * M * N : 0;
}

namespace {
// Validate one product and plan its split over K (work items = tiles x splits).
hipError_t plan_problem(int M, int N, int K, const bf16_bits* A, int64_t lda, int transA, const bf16_bits* B,
                        int64_t ldb, int transB, float* C, int64_t ldc, float alpha, int accumulate, float* part,
                        int64_t part_floats, GemmProblem* P, int64_t* work) {
  const bool a_kc = !transA, b_kc = transB != 0;
  // whole 16-byte vectors: the contiguous extent of each operand is a
  // multiple of 8 elements and every row starts 16-byte aligned
  if ((a_kc ? K : M) % 8 || (b_kc ? K : N) % 8 || lda % 8 || ldb % 8 || !al16(A) || !al16(B))
    return hipErrorInvalidValue;
  const int tm = static_cast<int>(ceil_div(M, BM)), tn = static_cast<int>(ceil_div(N, BN));
  int splits = 1;
  if (part) {
    splits = static_cast<int>(k_splits(M, N, K));
    while (splits > 1 && (int64_t)splits * M * N > part_floats) --splits;
  }
  const int k_chunk = std::max(BK, static_cast<int>(round_up(ceil_div(K, splits), BK)));
  splits = static_cast<int>(ceil_div(K, k_chunk));
  *P = GemmProblem{M, N, K, A, lda, B, ldb, C, ldc, alpha, accumulate, k_chunk, tm, tn, splits, 0,
                   splits > 1 ? part : nullptr};
  *work = (int64_t)tm * tn * splits;
  return hipSuccess;
}

template <typename Launch>
hipError_t by_form(bool a_kc, bool b_kc, Launch launch) {
  if (a_kc && b_kc) launch(std::integral_constant<int, 3>{});
  else if (a_kc) launch(std::integral_constant<int, 2>{});
  else if (b_kc) launch(std::integral_constant<int, 1>{});
  else launch(std::integral_constant<int, 0>{});
  return hipSuccess;
}
}  // namespace

hipError_t gemm_mfma(int M, int N, int K, const bf16_bits* A, int64_t lda, int transA, const bf16_bits* B,
                     int64_t ldb, int transB, float* C, int64_t ldc, float alpha, int accumulate, float* part,
                     int64_t part_floats, hipStream_t st) {
  if (M == 0 || N == 0) return hipSuccess;
  GemmProblem P;
  int64_t work = 0;
  hipError_t e = plan_problem(M, N, K, A, lda, transA, B, ldb, transB, C, ldc, alpha, accumulate, part,
                              part_floats, &P, &work);
  if (e != hipSuccess) return e;
  const int64_t grid = round_up(work, kXcds);
  if (grid > 0x7fffffff) return hipErrorInvalidValue;
  by_form(!transA, transB != 0, [&](auto f) {
    constexpr int F = decltype(f)::value;
    hipLaunchKernelGGL((mfma_gemm_kernel<(F & 2) != 0, (F & 1) != 0>), dim3(static_cast<unsigned>(grid)), dim3(256),
                       0, st, P, static_cast<int>(work));
  });
  if (P.part)
    hipLaunchKernelGGL(split_sum_kernel, dim3(static_cast<unsigned>(ceil_div((int64_t)M * N, 256))), dim3(256), 0,
                       st, P.part, P.splits, M, N, C, ldc, alpha, accumulate);
  return hipGetLastError();
}

hipError_t gemm_mfma_group(const GemmSpec* specs, int n, float* part, int64_t part_floats, hipStream_t st) {
  if (n < 1 || n > kMaxGroup) return hipErrorInvalidValue;
  GemmGroup G{};
  int64_t total = 0, part_used = 0, sum_threads = 0;
  int form = -1;
  for (int i = 0; i < n; ++i) {
    const GemmSpec& g = specs[i];
    if (g.M == 0 || g.N == 0) return hipErrorInvalidValue;
    const int f = (!g.transA ? 2 : 0) | (g.transB != 0 ? 1 : 0);
    if (form >= 0 && f != form) return hipErrorInvalidValue;  // one operand form per launch
    form = f;
    int64_t work = 0;
    float* p = part ? part + part_used : nullptr;
    hipError_t e = plan_problem(g.M, g.N, g.K, g.A, g.lda, g.transA, g.B, g.ldb, g.transB, g.C, g.ldc, g.alpha,
                                g.accumulate, p, part ? part_floats - part_used : 0, &G.p[i], &work);
    if (e != hipSuccess) return e;
    G.p[i].work_begin = static_cast<int>(total);
    total += work;
    if (G.p[i].part) {
      part_used += (int64_t)G.p[i].splits * g.M * g.N;
      sum_threads += (int64_t)g.M * g.N;
    }
  }
  G.n = n;
  const int64_t grid = round_up(total, kXcds);
  if (grid > 0x7fffffff) return hipErrorInvalidValue;
  by_form(form & 2, form & 1, [&](auto f) {
    constexpr int F = decltype(f)::value;
    hipLaunchKernelGGL((mfma_gemm_group_kernel<(F & 2) != 0, (F & 1) != 0>), dim3(static_cast<unsigned>(grid)),
                       dim3(256), 0, st, G, static_cast<int>(total));
  });
  if (sum_threads > 0)
    hipLaunchKernelGGL(split_sum_group_kernel, dim3(static_cast<unsigned>(ceil_div(sum_threads, 256))), dim3(256), 0,
                       st, G);
  return hipGetLastError();
}

}  // namespace stca
