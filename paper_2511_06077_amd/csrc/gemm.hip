// General MFMA GEMM for the backward pass's history-side products:
//   C[M,N] (fp32) = alpha * op(A) op(B)  (+ C when accumulating)
// A and B are bf16 or fp32 (fp32 operands are rounded to bf16 as they are
// staged), either may be read transposed.  Products: the per-layer K/V of the
// history (X W_K, X W_V; bf16 inputs, exact up to fp32 accumulation), the
// history gradient (dX += dK W_K^T + dV W_V^T) and the projection weight
// gradients (dW_K = X^T dK, dW_V = X^T dV, split over the long K dimension).
//
// 128 x 128 output tile per workgroup of four waves (2 x 2), each wave 64 x 64
// as 2 x 2 v_mfma_f32_32x32x16_bf16 tiles; 32-deep k tiles staged in LDS with
// k contiguous per row (16-byte operand reads, rows padded against bank
// conflicts).
#include <algorithm>

#include "common.h"
#include "internal.h"

namespace stca {

namespace {

constexpr int BM = 128, BN = 128, BK = 32;
constexpr int LROW = BK + 8;  // padded LDS row (bf16)

__device__ __forceinline__ f32x16 mfma_bf(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

template <typename T>
__device__ __forceinline__ __bf16 as_bf16(T v);
template <>
__device__ __forceinline__ __bf16 as_bf16<bf16_bits>(bf16_bits v) {
  return __builtin_bit_cast(__bf16, v);
}
template <>
__device__ __forceinline__ __bf16 as_bf16<float>(float v) {
  return static_cast<__bf16>(v);  // round to nearest even
}

// Stage a [rows x BK] operand tile into LDS as rows with k contiguous.
// "row" is M for A and N for B.  kmajor: the source holds element (row, k) at
// src[k * ld + row] (k-major); otherwise at src[row * ld + k].
template <typename T>
__device__ __forceinline__ void stage(__bf16* __restrict__ lds, const T* __restrict__ src, int64_t ld, bool kmajor,
                                      int row0, int nrows, int k0, int nk) {
  // 128 rows x 32 k = 4096 elements, 256 threads: 16 elements each, as two
  // runs of 8 consecutive source elements
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int run = threadIdx.x + r * 256;  // 512 runs of 8
    if (!kmajor) {
      const int row = run / (BK / 8), kk = (run % (BK / 8)) * 8;
      __bf16 v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const bool ok = row0 + row < nrows && k0 + kk + e < nk;
        v[e] = ok ? as_bf16<T>(src[(int64_t)(row0 + row) * ld + k0 + kk + e]) : static_cast<__bf16>(0.f);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) lds[row * LROW + kk + e] = v[e];
    } else {
      const int kk = run / (BM / 8), row = (run % (BM / 8)) * 8;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const bool ok = row0 + row + e < nrows && k0 + kk < nk;
        lds[(row + e) * LROW + kk] =
            ok ? as_bf16<T>(src[(int64_t)(k0 + kk) * ld + row0 + row + e]) : static_cast<__bf16>(0.f);
      }
    }
  }
}

template <typename TA, typename TB>
__global__ __launch_bounds__(256) void mfma_gemm_kernel(int M, int N, int K, const TA* __restrict__ A, int64_t lda,
                                                        int transA, const TB* __restrict__ B, int64_t ldb,
                                                        int transB, float* __restrict__ C, int64_t ldc, float alpha,
                                                        int accumulate, int k_chunk) {
  __shared__ __attribute__((aligned(16))) __bf16 As[BM * LROW];
  __shared__ __attribute__((aligned(16))) __bf16 Bs[BN * LROW];
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int wm = (wave / 2) * 64, wn = (wave % 2) * 64;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int kb = blockIdx.z * k_chunk;
  const int ke = min(K, kb + k_chunk);
  f32x16 acc[2][2] = {};
  const int r32 = lane % 32, hi = lane / 32;
  for (int k0 = kb; k0 < ke; k0 += BK) {
    // A: op(A) element (m, k) is A[m][k] (not transposed) or A[k][m]
    stage<TA>(As, A, lda, transA != 0, m0, M, k0, ke);
    // B: op(B) element (k, n) is B[k][n] (not transposed: k-major as a
    // [n][k] tile) or B[n][k]
    stage<TB>(Bs, B, ldb, transB == 0, n0, N, k0, ke);
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        a[i] = *reinterpret_cast<const bf16x8*>(&As[(wm + 32 * i + r32) * LROW + ks * 16 + hi * 8]);
        b[i] = *reinterpret_cast<const bf16x8*>(&Bs[(wn + 32 * i + r32) * LROW + ks * 16 + hi * 8]);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) acc[i][jj] = mfma_bf(a[i], b[jj], acc[i][jj]);
    }
    __syncthreads();
  }
  // result lane layout: column n = lane % 32, rows 8 (v / 4) + 4 hi + v % 4
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      const int n = n0 + wn + 32 * jj + r32;
      if (n >= N) continue;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int m = m0 + wm + 32 * i + 8 * (v / 4) + 4 * hi + (v % 4);
        if (m >= M) continue;
        float* c = C + (int64_t)m * ldc + n;
        const float x = alpha * acc[i][jj][v];
        if (gridDim.z > 1)
          atomicAdd(c, x);
        else
          *c = accumulate ? *c + x : x;
      }
    }
}

__global__ void zero2d_kernel(float* __restrict__ C, int64_t ldc, int M, int N) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < (int64_t)M * N) C[(i / N) * ldc + i % N] = 0.f;
}

}  // namespace

hipError_t gemm_mfma(int a_bf16, int b_bf16, int M, int N, int K, const void* A, int64_t lda, int transA,
                     const void* B, int64_t ldb, int transB, float* C, int64_t ldc, float alpha, int accumulate,
                     hipStream_t st) {
  if (M == 0 || N == 0) return hipSuccess;
  const int64_t tiles = ceil_div(M, BM) * ceil_div(N, BN);
  int splits = 1;
  if (tiles < 256 && K >= 8192) splits = static_cast<int>(std::min<int64_t>(ceil_div(512, tiles), K / 4096));
  if (splits < 1) splits = 1;
  const int k_chunk = static_cast<int>(round_up(ceil_div(K, splits), BK));
  splits = static_cast<int>(ceil_div(K, k_chunk));
  if (splits > 1 && !accumulate)
    hipLaunchKernelGGL(zero2d_kernel, dim3(static_cast<unsigned>(ceil_div((int64_t)M * N, 256))), dim3(256), 0, st,
                       C, ldc, M, N);
  dim3 g(static_cast<unsigned>(ceil_div(N, BN)), static_cast<unsigned>(ceil_div(M, BM)), splits);
#define STCA_MG(TA, TB)                                                                                 \
  hipLaunchKernelGGL((mfma_gemm_kernel<TA, TB>), g, dim3(256), 0, st, M, N, K, (const TA*)A, lda, transA, \
                     (const TB*)B, ldb, transB, C, ldc, alpha, accumulate, k_chunk)
  if (a_bf16 && b_bf16) STCA_MG(bf16_bits, bf16_bits);
  else if (a_bf16) STCA_MG(bf16_bits, float);
  else if (b_bf16) STCA_MG(float, bf16_bits);
  else STCA_MG(float, float);
#undef STCA_MG
  return hipGetLastError();
}

}  // namespace stca
