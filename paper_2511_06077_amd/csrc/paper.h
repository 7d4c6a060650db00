// Launchers of the paper-exact layer stack's kernels (paper.hip).
#pragma once

#include "common.h"

namespace stca {

constexpr float kLnEps = 1e-5f;  // LayerNorm epsilon (scale 1, shift 0)

// Bytes of one layer's SwiGLU weights in per-chunk operand order.
size_t swiglu_packed_bytes(int D, int F);
// Repack W_u, W_v [n_layers][D][F] and W_o [n_layers][F][D] (bf16) into
// P [n_layers][swiglu_packed_bytes].
hipError_t swiglu_pack(const void* Wu, const void* Wv, const void* Wo, int n_layers, int D, int F, void* P,
                       hipStream_t st);
// out16 (bf16, required) and out32 (fp32, nullable) [n_rows][D] =
// LN(SwiGLUFFN(X)) with one layer's packed weights; D in {64, 128, 256},
// F % 32 == 0.
hipError_t swiglu_ln(int D, const void* X, int64_t n_rows, const void* Wp_layer, int F, void* out16, float* out32,
                     hipStream_t st);
// u = u * v * sigmoid(v), elementwise (fp32).
hipError_t swiglu_gate_f32(float* u, const float* v, int64_t n, hipStream_t st);
// out[r] = LN(y[r]) over d features (fp32; out may alias y).
hipError_t layer_norm_rows(const float* y, int64_t rows, int d, float* out, hipStream_t st);
// Scaled fp32 queries [n_tgt][D] -> the fused attention kernel's fp16 QN layout.
hipError_t qn_pack(const float* Q, void* QN, int64_t n_tgt, int D, hipStream_t st);

}  // namespace stca
