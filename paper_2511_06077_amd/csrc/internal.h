// Launchers shared between the C-ABI layer and the kernel files.
#pragma once

#include "common.h"

namespace stca {

// ---- scheduler (sched.hip)
hipError_t launch_sched(const int32_t* hoff, const int32_t* toff, int R, int64_t n_hist, int64_t n_tgt,
                        int chunk_blocks, Unit* units, int64_t max_units, int32_t* tchunks,
                        WsHeader* hdr, hipStream_t st);
int64_t host_count_units(const int32_t* hoff, const int32_t* toff, int R, int chunk_blocks);

// ---- generic fp32-arithmetic path (generic.hip)
enum GemmEpi { kEpiStore = 0, kEpiAddRes = 1, kEpiRelu = 2 };
// C[M,N] = epi(alpha * A[M,K] B[K,N]); A, B row-major with leading dims; C fp32.
// kEpiAddRes: C = R + alpha*AB.  kEpiRelu: C = max(AB, 0) and, if C2, C2 = AB.
// transA / transB read A as [K,M] / B as [N,K] (i.e. multiply by the transpose).
hipError_t gemm_generic(int a_bf16, int b_bf16, int M, int N, int K, const void* A, int64_t lda,
                        int transA, const void* B, int64_t ldb, int transB, float* C, int64_t ldc,
                        float alpha, GemmEpi epi, const float* R, int64_t ldr, float* C2,
                        int accumulate, hipStream_t st);
// MFMA GEMM with bf16 operands (fp32 operands rounded to bf16 when staged)
// and fp32 accumulation/output; same operand conventions as gemm_generic
// (kEpiStore only, optional accumulate).  For the backward's history-side
// products on bf16 inputs.
hipError_t gemm_mfma(int a_bf16, int b_bf16, int M, int N, int K, const void* A, int64_t lda, int transA,
                     const void* B, int64_t ldb, int transB, float* C, int64_t ldc, float alpha, int accumulate,
                     hipStream_t st);
hipError_t attn_generic(int d_head, int n_heads, const Unit* units, int64_t max_units,
                        const WsHeader* hdr, const float* Q, const float* KV, int d,
                        float* part_acc, float* part_ml, int64_t n_tgt, hipStream_t st);
hipError_t merge_generic(int d_head, int n_heads, int64_t n_tgt, const int32_t* tchunks,
                         const float* part_acc, const float* part_ml, float* a, float* lse,
                         hipStream_t st);
hipError_t convert(int src_bf16, int dst_bf16, const void* src, void* dst, int64_t n, hipStream_t st);
hipError_t fill_f32(float* dst, float v, int64_t n, hipStream_t st);
// generic backward pieces
hipError_t attn_bwd_generic(int d_head, int n_heads, const Unit* units, int64_t max_units,
                            const WsHeader* hdr, const float* Q, const float* KV, int d,
                            const float* a, const float* da, const float* lse, float* dq_part,
                            float* dKV, int64_t n_tgt, hipStream_t st);
hipError_t reduce_chunks(int64_t n_tgt, int d, const int32_t* tchunks, const float* part, float* out,
                         float scale, hipStream_t st);
hipError_t relu_mask_mul(float* dh, const float* pre, int64_t n, hipStream_t st);

}  // namespace stca
