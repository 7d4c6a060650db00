// Kernels of the paper-exact layer stack (Sec. 3.1): the token-wise SwiGLU
// block of Eq. swigluffn followed by LayerNorm, on the history rows (the
// dominant cost: 6 r d^2 flop per row and layer) and the small target-side
// pieces (gate, row LayerNorm, query packing for the fused attention kernel).
//
// History transform X~ = LN(SwiGLUFFN(X)), bf16 in and out, one workgroup of
// eight waves (two per SIMD, so one wave's gate arithmetic overlaps the other's
// MFMAs) per 256 history rows, one wave per 32 rows:
//
//   U^T = W_u^T X^T, V^T = W_v^T X^T   (32 hidden columns at a time, MFMA
//                                       32x32x16 bf16, X^T held in registers)
//   G^T = U^T * V^T * sigmoid(V^T)     (registers, rounded to bf16)
//   Y^T += W_o^T G^T                   (all d rows accumulated in registers)
//   X~ = LN(Y) per row                 (the row's d values sit in one lane pair)
//
// The hidden activations never leave the registers: the result registers of
// U^T and V^T hold, for lane (row l%32, half hi), hidden columns
// 16kk + 4hi + {0..3, 8..11} (kk = 0, 1), which is a valid B operand of the
// down projection when W_o's rows are packed in that same order.  Weights are
// repacked once per call into per-chunk operand order (32 hidden columns:
// W_u^T fragments, W_v^T fragments, W_o^T fragments, contiguous) and each
// chunk is copied into LDS with direct global-to-LDS loads, double buffered,
// so the eight waves share one copy.
#include "common.h"
#include "paper.h"

namespace stca {

namespace {

__device__ __forceinline__ f32x16 mfma_bf16(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 zero8() {
  bf16x8 z;
#pragma unroll
  for (int i = 0; i < 8; ++i) z[i] = static_cast<__bf16>(0.f);
  return z;
}

// SiLU gate of Eq. swigluffn: u * v * sigmoid(v)
__device__ __forceinline__ float swiglu_gate(float u, float v) {
  return u * v * __builtin_amdgcn_rcpf(1.f + __expf(-v));
}

// hidden row of slot (kk, hi, i) of a packed W_o fragment: the order in which
// the up projection's result registers hold hidden columns
__device__ __forceinline__ int gate_row(int kk, int hi, int i) { return 16 * kk + 4 * hi + (i < 4 ? i : i + 4); }

__global__ void swiglu_pack_kernel(const bf16_bits* __restrict__ Wu, const bf16_bits* __restrict__ Wv,
                                   const bf16_bits* __restrict__ Wo, int D, int F, bf16_bits* __restrict__ P,
                                   int64_t groups_per_layer) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= groups_per_layer) return;
  const int layer = blockIdx.y;
  const int KS = D / 16;
  const int64_t per_chunk = (int64_t)(2 * KS + 2 * (D / 32)) * 64;
  const int c = static_cast<int>(g / per_chunk);
  int q = static_cast<int>(g % per_chunk);
  Wu += (int64_t)layer * D * F;
  Wv += (int64_t)layer * D * F;
  Wo += (int64_t)layer * F * D;
  bf16_bits* dst = P + ((int64_t)layer * groups_per_layer + g) * 8;
  const int l = q % 64, n = l % 32, hi = l / 32;
  if (q < 2 * KS * 64) {
    const bf16_bits* W = q < KS * 64 ? Wu : Wv;
    const int ks = (q / 64) % KS;
#pragma unroll
    for (int i = 0; i < 8; ++i) dst[i] = W[(int64_t)(16 * ks + 8 * hi + i) * F + 32 * c + n];
  } else {
    q -= 2 * KS * 64;
    const int nt = q / 128, kk = (q / 64) % 2;
#pragma unroll
    for (int i = 0; i < 8; ++i) dst[i] = Wo[(int64_t)(32 * c + gate_row(kk, hi, i)) * D + 32 * nt + n];
  }
}

constexpr int kSwWaves = 8;  // waves per workgroup (two per SIMD), 32 rows each

template <int D>
__global__ __launch_bounds__(kSwWaves * 64)
__attribute__((amdgpu_waves_per_eu(kSwWaves / 4, kSwWaves / 4))) void swiglu_ln_kernel(
    const bf16_bits* __restrict__ X, int64_t n_rows, const unsigned char* __restrict__ Wp, int F,
    bf16_bits* __restrict__ out16, float* __restrict__ out32) {
  constexpr int KS = D / 16;       // k-steps of the up projections
  constexpr int NT = D / 32;       // 32-row tiles of Y^T
  constexpr int UB = KS * 1024;    // bytes of one chunk's W_u^T (or W_v^T) fragments
  constexpr int CB = 2 * UB + NT * 2048;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];  // [2][CB]
  const int w = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int tcol = lane % 32, hi = lane / 32;
  const int64_t row = (int64_t)blockIdx.x * (32 * kSwWaves) + 32 * w + tcol;
  const bool live = row < n_rows;

  // X^T as B operands: lane (row, hi), k-step ks holds X[row][16ks + 8hi .. +7]
  bf16x8 xb[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
    xb[ks] = live ? *reinterpret_cast<const bf16x8*>(X + row * D + 16 * ks + 8 * hi) : zero8();
  f32x16 Y[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) Y[t] = f32x16{};

  const int nch = F / 32;
  auto dma = [&](int c, int buf) {
    const unsigned char* src = Wp + (size_t)c * CB + lane * 16;
    unsigned char* dst = smem + buf * CB;
    for (int i = w; i < CB / 1024; i += kSwWaves)
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(src + i * 1024),
                                       (void __attribute__((address_space(3)))*)(dst + i * 1024), 16, 0, 0);
  };
  dma(0, 0);
  for (int c = 0; c < nch; ++c) {
    const int cur = c & 1;
    // chunk c has landed (each wave waited for its own copies) and every wave
    // is done with chunk c - 1, whose buffer the next copy overwrites
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (c + 1 < nch) dma(c + 1, cur ^ 1);
    const bf16x8* Ua = reinterpret_cast<const bf16x8*>(smem + cur * CB) + lane;
    const bf16x8* Va = Ua + KS * 64;
    const bf16x8* Oa = Va + KS * 64;
    f32x16 u = {}, v = {};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      u = mfma_bf16(Ua[ks * 64], xb[ks], u);
      v = mfma_bf16(Va[ks * 64], xb[ks], v);
    }
    bf16x8 g[2];
#pragma unroll
    for (int i = 0; i < 16; ++i) g[i / 8][i % 8] = static_cast<__bf16>(swiglu_gate(u[i], v[i]));
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      Y[t] = mfma_bf16(Oa[(2 * t) * 64], g[0], Y[t]);
      Y[t] = mfma_bf16(Oa[(2 * t + 1) * 64], g[1], Y[t]);
    }
  }
  // LayerNorm of the row: lane (row, hi) holds Y[row][32t + 8(v/4) + 4hi + v%4]
  float s = 0.f;
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int v = 0; v < 16; ++v) s += Y[t][v];
  s += __shfl_xor(s, 32);
  const float mean = s * (1.f / D);
  float q = 0.f;
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const float e = Y[t][v] - mean;
      q += e * e;
    }
  q += __shfl_xor(q, 32);
  const float rstd = rsqrtf(q * (1.f / D) + kLnEps);
  if (!live) return;
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const int col = 32 * t + 8 * g4 + 4 * hi;
      float o[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) o[k] = (Y[t][4 * g4 + k] - mean) * rstd;
      uint2 pk;
      pk.x = (uint32_t)from_f32<bf16_bits>(o[0]) | ((uint32_t)from_f32<bf16_bits>(o[1]) << 16);
      pk.y = (uint32_t)from_f32<bf16_bits>(o[2]) | ((uint32_t)from_f32<bf16_bits>(o[3]) << 16);
      *reinterpret_cast<uint2*>(out16 + row * D + col) = pk;
      if (out32) *reinterpret_cast<float4*>(out32 + row * D + col) = make_float4(o[0], o[1], o[2], o[3]);
    }
}

template <int D>
constexpr size_t swiglu_chunk_bytes() {
  return (size_t)2 * (D / 16) * 1024 + (size_t)(D / 32) * 2048;
}

template <typename K>
hipError_t allow_lds(K kernel, size_t bytes) {
  static int set_for[64] = {0};  // per device: bytes granted so far
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < 64 && set_for[dev] >= static_cast<int>(bytes)) return hipSuccess;
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                          static_cast<int>(bytes));
  if (e == hipSuccess && dev >= 0 && dev < 64) set_for[dev] = static_cast<int>(bytes);
  return e;
}

// ------------------------------------------------------------ target side
__global__ void gate_kernel(float* __restrict__ u, const float* __restrict__ v, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) {
    const float vv = v[i];
    u[i] = u[i] * vv / (1.f + expf(-vv));
  }
}

// one wave per row; two passes over the row (mean, then centred squares)
__global__ __launch_bounds__(256) void ln_rows_kernel(const float* __restrict__ y, int64_t rows, int d,
                                                      float* __restrict__ out) {
  const int64_t r = (int64_t)blockIdx.x * 4 + threadIdx.x / 64;
  const int lane = threadIdx.x % 64;
  if (r >= rows) return;
  const float* p = y + r * d;
  float s = 0.f;
  for (int e = lane; e < d; e += 64) s += p[e];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o);
  const float mean = s / d;
  float q = 0.f;
  for (int e = lane; e < d; e += 64) {
    const float c = p[e] - mean;
    q += c * c;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) q += __shfl_xor(q, o);
  const float rstd = 1.f / sqrtf(q / d + kLnEps);
  for (int e = lane; e < d; e += 64) out[r * d + e] = (p[e] - mean) * rstd;
}

// fp32 queries (already scaled) -> the fused attention kernel's QN layout:
// per head, position 16s + 8hi + i holds dimension 16s + 4hi + (i<4 ? i : i+4), fp16
__global__ void qn_pack_kernel(const float* __restrict__ Q, _Float16* __restrict__ QN, int64_t n_groups) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= n_groups) return;
  const int64_t base = g * 8;  // first position of this group
  const int64_t head0 = base / 32 * 32;
  const int p = static_cast<int>(base % 32);
  const int s = p / 16, hi = (p / 8) % 2;
#pragma unroll
  for (int i = 0; i < 8; ++i) QN[base + i] = static_cast<_Float16>(Q[head0 + 16 * s + 4 * hi + (i < 4 ? i : i + 4)]);
}

}  // namespace

// ------------------------------------------------------------ launchers
size_t swiglu_packed_bytes(int D, int F) { return (size_t)(F / 32) * (2 * (D / 16) * 1024 + (D / 32) * 2048); }

hipError_t swiglu_pack(const void* Wu, const void* Wv, const void* Wo, int n_layers, int D, int F, void* P,
                       hipStream_t st) {
  if (D % 32 || F % 32) return hipErrorInvalidValue;
  const int64_t groups = (int64_t)(F / 32) * (2 * (D / 16) + 2 * (D / 32)) * 64;
  hipLaunchKernelGGL(swiglu_pack_kernel, dim3(static_cast<unsigned>(ceil_div(groups, 256)), n_layers), dim3(256), 0,
                     st, (const bf16_bits*)Wu, (const bf16_bits*)Wv, (const bf16_bits*)Wo, D, F, (bf16_bits*)P,
                     groups);
  return hipGetLastError();
}

hipError_t swiglu_ln(int D, const void* X, int64_t n_rows, const void* Wp_layer, int F, void* out16, float* out32,
                     hipStream_t st) {
  if (n_rows == 0) return hipSuccess;
  if (F % 32) return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(ceil_div(n_rows, 32 * kSwWaves)));
#define STCA_SWIGLU(DD)                                                                                      \
  {                                                                                                          \
    const size_t lds = 2 * swiglu_chunk_bytes<DD>();                                                         \
    hipError_t e = allow_lds(swiglu_ln_kernel<DD>, lds);                                                     \
    if (e != hipSuccess) return e;                                                                           \
    hipLaunchKernelGGL(swiglu_ln_kernel<DD>, grid, dim3(64 * kSwWaves), lds, st, (const bf16_bits*)X, n_rows, \
                       (const unsigned char*)Wp_layer, F, (bf16_bits*)out16, out32);                         \
  }
  switch (D) {
    case 64: STCA_SWIGLU(64); break;
    case 128: STCA_SWIGLU(128); break;
    case 256: STCA_SWIGLU(256); break;
    default: return hipErrorInvalidValue;
  }
#undef STCA_SWIGLU
  return hipGetLastError();
}

hipError_t swiglu_gate_f32(float* u, const float* v, int64_t n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(gate_kernel, dim3(static_cast<unsigned>(ceil_div(n, 256))), dim3(256), 0, st, u, v, n);
  return hipGetLastError();
}

hipError_t layer_norm_rows(const float* y, int64_t rows, int d, float* out, hipStream_t st) {
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(ln_rows_kernel, dim3(static_cast<unsigned>(ceil_div(rows, 4))), dim3(256), 0, st, y, rows, d,
                     out);
  return hipGetLastError();
}

hipError_t qn_pack(const float* Q, void* QN, int64_t n_tgt, int D, hipStream_t st) {
  const int64_t groups = n_tgt * D / 8;
  if (groups == 0) return hipSuccess;
  if (D % 32) return hipErrorInvalidValue;
  hipLaunchKernelGGL(qn_pack_kernel, dim3(static_cast<unsigned>(ceil_div(groups, 256))), dim3(256), 0, st, Q,
                     (_Float16*)QN, groups);
  return hipGetLastError();
}

}  // namespace stca
