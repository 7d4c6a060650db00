// Launchers shared between the C-ABI layer and the kernel files.
#pragma once

#include "common.h"

namespace stca {

// ---- scheduler (sched.hip)
// `group`: targets per unit (1..kWideGroup).  Only requests with m_lo..m_hi
// targets get units (and chunk counts); the others keep a zero chunk count.
// deal > 0: within each width class, units in descending order of their
// history blocks, complete rounds of `deal` units alternating in direction
// (for persistent kernels of `deal` workgroups that take units round-robin
// and place every partial by its chunk index); 0: request and chunk order.
hipError_t launch_sched(const int32_t* hoff, const int32_t* toff, int R, int64_t n_hist, int64_t n_tgt,
                        int chunk_blocks, int group, Unit* units, int64_t max_units, int32_t* tchunks,
                        WsHeader* hdr, hipStream_t st, int m_lo = 1, int m_hi = 1 << 30, int deal = 0);
int64_t host_count_units(const int32_t* hoff, const int32_t* toff, int R, int chunk_blocks, int group,
                         int m_lo = 1, int m_hi = 1 << 30);

// ---- generic fp32-arithmetic path (generic.hip)
enum GemmEpi { kEpiStore = 0, kEpiAddRes = 1, kEpiRelu = 2 };
// C[M,N] = epi(alpha * A[M,K] B[K,N]); A, B row-major with leading dims; C fp32.
// kEpiAddRes: C = R + alpha*AB.  kEpiRelu: C = max(AB, 0) and, if C2, C2 = AB.
// transA / transB read A as [K,M] / B as [N,K] (i.e. multiply by the transpose).
hipError_t gemm_generic(int a_bf16, int b_bf16, int M, int N, int K, const void* A, int64_t lda,
                        int transA, const void* B, int64_t ldb, int transB, float* C, int64_t ldc,
                        float alpha, GemmEpi epi, const float* R, int64_t ldr, float* C2,
                        int accumulate, hipStream_t st);
// MFMA GEMM, bf16 operands, fp32 accumulation and output:
// C = alpha op(A) op(B) (+ C when accumulating), operand conventions as in
// gemm_generic.  The contiguous extent of each operand (K for A untransposed
// and for B transposed, else M / N) and lda, ldb must be multiples of 8, A
// and B 16-byte aligned (hipErrorInvalidValue otherwise).  Long-K products
// with few output tiles split K when `part` holds splits * M * N floats
// (gemm_mfma_part_floats gives the most any split asks for).
int64_t gemm_mfma_part_floats(int M, int N, int K);
hipError_t gemm_mfma(int M, int N, int K, const bf16_bits* A, int64_t lda, int transA, const bf16_bits* B,
                     int64_t ldb, int transB, float* C, int64_t ldc, float alpha, int accumulate, float* part,
                     int64_t part_floats, hipStream_t st);
// Up to sixteen gemm_mfma products with the same operand forms (transA,
// transB) in one launch (and one launch summing their splits), so that small
// products fill the chip together; `part` is shared, the products' splits in
// order (the sum of their gemm_mfma_part_floats holds every split).
struct GemmSpec {
  int M, N, K;
  const bf16_bits* A;
  int64_t lda;
  int transA;
  const bf16_bits* B;
  int64_t ldb;
  int transB;
  float* C;
  int64_t ldc;
  float alpha;
  int accumulate;
};
hipError_t gemm_mfma_group(const GemmSpec* specs, int n, float* part, int64_t part_floats, hipStream_t st);
// The same product for the long history-row operands ([dW_K | dW_V] with K =
// history rows, dX with M = history rows): one persistent workgroup per CU
// (n_cu of them), operand tiles streamed into an LDS ring by direct loads.
// Same conventions and requirements as gemm_mfma (accumulating products
// without a split over K are left to gemm_mfma); splits over K need
// gemm_ring_part_floats floats in `part`.
int64_t gemm_ring_part_floats(int M, int N, int K, int n_cu);
hipError_t gemm_ring(int M, int N, int K, const bf16_bits* A, int64_t lda, int transA, const bf16_bits* B,
                     int64_t ldb, int transB, float* C, int64_t ldc, float alpha, int accumulate, float* part,
                     int64_t part_floats, int n_cu, hipStream_t st);
// The same kernel over the units of a schedule (hdr->n_units of them): unit
// u's rows [max(32 b0, l0), min(32 b1, l1)) of C ([rows][ldc] fp32, N <= 256
// columns) = A rows (bf16, k contiguous, lda) times B + r * b_stride (bf16
// [K][ldb], rows contiguous), r the unit's request.
hipError_t gemm_ring_units(int N, int K, const bf16_bits* A, int64_t lda, const bf16_bits* B, int64_t ldb,
                           int64_t b_stride, float* C, int64_t ldc, const Unit* units, const WsHeader* hdr,
                           int n_cu, hipStream_t st);
// dst[c][r] = src[r][c] (bf16; R x C source, row pitches lds / ldd); dst
// columns R..Rp-1 are zeroed.
hipError_t transpose_bf16(const bf16_bits* src, int64_t lds, int R, int C, bf16_bits* dst, int64_t ldd, int Rp,
                          hipStream_t st);
hipError_t attn_generic(int d_head, int n_heads, const Unit* units, int64_t max_units,
                        const WsHeader* hdr, const float* Q, const float* KV, int d,
                        float* part_acc, float* part_ml, int64_t n_tgt, hipStream_t st);
hipError_t merge_generic(int d_head, int n_heads, int64_t n_tgt, const int32_t* tchunks,
                         const float* part_acc, const float* part_ml, float* a, float* lse,
                         hipStream_t st);
hipError_t convert(int src_bf16, int dst_bf16, const void* src, void* dst, int64_t n, hipStream_t st);
hipError_t fill_f32(float* dst, float v, int64_t n, hipStream_t st);
// [W_K^0 | W_V^0 | W_K^1 | ...] ([d][n 2d] bf16) from the stacked W_K, W_V
// ([n][d][d] bf16, 16-byte aligned; d a multiple of 8).
hipError_t pack_wkv(const bf16_bits* wk, const bf16_bits* wv, int n, int d, bf16_bits* wkv, hipStream_t st);
// dW_K^i and dW_V^i ([n][d][d] fp32) from [dW_K^0 | dW_V^0 | ...] ([d][n 2d]).
hipError_t split_dwkv(const float* dwkv, int n, int d, float* dwk, float* dwv, hipStream_t st);
// generic backward pieces
// dKV ([N_hist] rows of 2d, row pitch ldkv elements; fp32 or bf16 when
// dkv_bf16) is written for every history row of a request with targets, and
// with bf16 also its transpose dKVT ([2d][ldt]) when dKVT is not null; rows of
// requests without targets are left untouched.
hipError_t attn_bwd_generic(int d_head, int n_heads, const Unit* units, int64_t max_units,
                            const WsHeader* hdr, const int32_t* toff, const float* Q, const float* KV, int d,
                            const float* a, const float* da, const float* lse, float* dq_part, void* dKV,
                            int64_t ldkv, int dkv_bf16, bf16_bits* dKVT, int64_t ldt, int64_t n_tgt,
                            hipStream_t st);
// Exact fp32 attention on the fp32 matrix cores (attn_mfma.hip) for d_h in
// {16, 32, 64}: the same outputs as attn_generic / attn_bwd_generic, which
// dispatch to them.
bool attn_mfma_supported(int d_head);
hipError_t attn_fwd_mfma(int d_head, int n_heads, const Unit* units, int64_t max_units, const WsHeader* hdr,
                         const float* Q, const float* KV, int d, float* part_acc, float* part_ml, int64_t n_tgt,
                         hipStream_t st);
hipError_t attn_bwd_mfma(int d_head, int n_heads, const Unit* units, int64_t max_units, const WsHeader* hdr,
                         const int32_t* toff, const float* Q, const float* KV, int d, const float* a, const float* da,
                         const float* lse, float* dq_part, void* dKV, int64_t ldkv, int dkv_bf16, bf16_bits* dKVT,
                         int64_t ldt, int64_t n_tgt, hipStream_t st);
// out (fp32) and out16 (bf16, rounded from the same fp32 value), either may
// be null: the scaled sum of each target's chunk partials
hipError_t reduce_chunks(int64_t n_tgt, int d, const int32_t* tchunks, const float* part, float* out,
                         bf16_bits* out16, float scale, hipStream_t st);
hipError_t relu_mask_mul(float* dh, const float* pre, int64_t n, hipStream_t st);
// Zero the history rows of requests without targets in dKV ([N_hist][ldkv]
// bf16, columns [0, cols)) and, when dKVT is given ([cols][ldt]), the
// matching entries of that transpose and its padding rows [n_hist, ldt).
hipError_t zero_untargeted(const int32_t* hoff, const int32_t* toff, int n_requests, int64_t n_hist,
                           bf16_bits* dKV, int64_t ldkv, int cols, bf16_bits* dKVT, int64_t ldt, hipStream_t st);

}  // namespace stca
