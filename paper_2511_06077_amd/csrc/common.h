// Shared device/host definitions of the STCA HIP library (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/stca.h"

namespace stca {

typedef uint16_t bf16_bits;  // storage of a bfloat16 value
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlockTokens = 32;  // history rows per K/V block (one MFMA tile edge)
constexpr int kTargetGroup = 64;  // targets one attention unit holds (two 32-wide MFMA column groups)
constexpr int kWideGroup = 128;   // targets per unit of the materialised-K/V attention for m > 64
constexpr int kMaxChunks = 16;    // at most this many history chunks per request
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kF16Max = 65504.f;  // largest finite fp16 value

// One unit of attention work: targets [t0, t0+nt) of request r against the
// 32-row history blocks [b0, b1); rows outside [l0, l1) belong to neighbouring
// requests and are masked.  c is the chunk index of [b0, b1) within the request.
struct Unit {
  int32_t r, t0, nt, c, b0, b1, l0, l1;
};

// Header at the start of every workspace.
struct WsHeader {
  int32_t status;    // stca_status_t recorded by the device scheduler
  int32_t n_units;   // units the scheduler emitted
  int32_t n_narrow;  // units [0, n_narrow) have at most 32 targets, the rest more
  int32_t range;     // nonzero: an fp16 intermediate overflowed or a value was not finite
  int32_t pad[60];
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_bits x) {
  return __uint_as_float(static_cast<uint32_t>(x) << 16);
}
template <typename T>
__device__ __forceinline__ T from_f32(float x);
template <>
__device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <>
__device__ __forceinline__ bf16_bits from_f32<bf16_bits>(float x) {
  __bf16 b = static_cast<__bf16>(x);  // round to nearest even
  return __builtin_bit_cast(bf16_bits, b);
}

__host__ __device__ __forceinline__ int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
__host__ __device__ __forceinline__ int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }

}  // namespace stca
