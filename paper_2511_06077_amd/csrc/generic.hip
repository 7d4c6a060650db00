// Generic fp32-arithmetic kernels: any supported head width, fp32 or bf16
// storage.  They serve the fp32 storage type (whose tolerance bf16 MFMA
// arithmetic cannot meet) and the backward pass's small target-side GEMMs.
// LDS-tiled kernels; products with bf16 weights run on the bf16 matrix cores
// with the fp32 operand split into three bf16 terms (exact products), the
// others on the fp32 matrix cores; the bf16 hot path has its own kernels.
#include "common.h"
#include "internal.h"

#include <algorithm>

namespace stca {

namespace {

template <typename T>
__device__ __forceinline__ float ld(const T* p, int64_t i) {
  return to_f32(p[i]);
}

// ---------------------------------------------------------------- GEMM
// fp32 products (operands fp32 or bf16, widened exactly) on the fp32 MFMA,
// v_mfma_f32_32x32x2_f32: 64 x 64 output tile per workgroup of four waves,
// each wave a 32 x 32 quarter; 32-deep k tiles staged in LDS as [k][m] and
// [k][n], the next tile's global loads in flight during the current tile's
// MFMAs.
constexpr int GT = 64;  // output tile edge
constexpr int GK = 32;  // k step

template <typename TA, typename TB>
__global__ __launch_bounds__(256) void gemm_kernel(int M, int N, int K, const TA* __restrict__ A,
                                                   int64_t lda, int transA, const TB* __restrict__ B,
                                                   int64_t ldb, int transB, float* __restrict__ C,
                                                   int64_t ldc, float alpha, int epi,
                                                   const float* __restrict__ R, int64_t ldr,
                                                   float* __restrict__ C2, int accumulate, int k_chunk) {
  __shared__ float As[GK][GT + 1];
  __shared__ float Bs[GK][GT + 1];
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int wm = (wave / 2) * 32, wn = (wave % 2) * 32;
  const int r32 = lane % 32, hi = lane / 32;
  const int m0 = blockIdx.y * GT, n0 = blockIdx.x * GT;
  f32x16 acc = {};
  // split-K: workgroup z sums k in [z * k_chunk, (z + 1) * k_chunk) and adds
  // its partial into C atomically (C was cleared or holds what to add to)
  const int kb = blockIdx.z * k_chunk;
  const int ke = min(K, kb + k_chunk);
  constexpr int PER = GT * GK / 256;
  float ra[PER], rb[PER];
  // Consecutive threads walk each source's contiguous index, so global reads
  // coalesce.
  auto load = [&](int k0) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = threadIdx.x + 256 * i;
      const int mm = transA ? e % GT : e / GK, kk = transA ? e / GT : e % GK;
      const int gm = m0 + mm, gk = k0 + kk;
      ra[i] = (gm < M && gk < ke) ? (transA ? ld(A, (int64_t)gk * lda + gm) : ld(A, (int64_t)gm * lda + gk)) : 0.f;
      const int nn = transB ? e / GK : e % GT, kb2 = transB ? e % GK : e / GT;
      const int gn = n0 + nn, gk2 = k0 + kb2;
      rb[i] = (gn < N && gk2 < ke) ? (transB ? ld(B, (int64_t)gn * ldb + gk2) : ld(B, (int64_t)gk2 * ldb + gn))
                                   : 0.f;
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = threadIdx.x + 256 * i;
      const int mm = transA ? e % GT : e / GK, kk = transA ? e / GT : e % GK;
      As[kk][mm] = ra[i];
      const int nn = transB ? e / GK : e % GT, kb2 = transB ? e % GK : e / GT;
      Bs[kb2][nn] = rb[i];
    }
  };
  load(kb);
  store();
  __syncthreads();
  for (int k0 = kb; k0 < ke; k0 += GK) {
    const bool more = k0 + GK < ke;
    if (more) load(k0 + GK);
    // operand lane l holds A[m = l % 32][k = l / 32] and B[k = l / 32][n = l % 32]
#pragma unroll
    for (int kk = 0; kk < GK; kk += 2)
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(As[kk + hi][wm + r32], Bs[kk + hi][wn + r32], acc, 0, 0, 0);
    __syncthreads();
    if (more) {
      store();
      __syncthreads();
    }
  }
  // result lane layout: column n = lane % 32, rows 8 (v / 4) + 4 hi + v % 4
  const int gn = n0 + wn + r32;
  if (gn >= N) return;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int gm = m0 + wm + 8 * (v / 4) + 4 * hi + (v % 4);
    if (gm >= M) continue;
    float x = alpha * acc[v];
    float* c = C + (int64_t)gm * ldc + gn;
    if (gridDim.z > 1) {
      atomicAdd(c, x);
      continue;
    }
    if (epi == kEpiAddRes) x += R[(int64_t)gm * ldr + gn];
    if (epi == kEpiRelu) {
      if (C2) C2[(int64_t)gm * ldc + gn] = x;
      x = fmaxf(x, 0.f);
    }
    *c = accumulate ? *c + x : x;
  }
}

// fp32-accurate products with bf16 weights on the bf16 matrix cores:
// C = epi(alpha A B), A [M][K] fp32 (or bf16) row-major, B [K][N] bf16
// row-major.  Each fp32 value of A is split into three bf16 terms (the whole
// fp32 mantissa over fp32's exponent range); every product of two bf16
// values is exact in fp32 and the MFMA sums are fp32, so the result matches
// an fp32 product (a bf16 A is one term).  64 x 64 output tile per workgroup
// of four waves (each one 32 x 32 v_mfma_f32_32x32x16_bf16 tile), 32-deep k
// tiles double-buffered in LDS (A's terms as [m][k], B transposed to [n][k]).
typedef unsigned short u16x8g __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8g __attribute__((ext_vector_type(8)));
constexpr int SBK = 32;
constexpr int SROW = SBK + 8;  // padded LDS row (bf16 elements)

template <typename TA>
__global__ __launch_bounds__(256) void gemm_bf16w_kernel(int M, int N, int K, const TA* __restrict__ A, int64_t lda,
                                                         const bf16_bits* __restrict__ B, int64_t ldb,
                                                         float* __restrict__ C, int64_t ldc, float alpha, int epi,
                                                         const float* __restrict__ R, int64_t ldr,
                                                         float* __restrict__ C2, int accumulate) {
  constexpr int TERMS = sizeof(TA) == 4 ? 3 : 1;
  __shared__ __attribute__((aligned(16))) bf16_bits As[2][TERMS][GT * SROW];
  __shared__ __attribute__((aligned(16))) bf16_bits Bs[2][GT * SROW];
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int wm = (wave / 2) * 32, wn = (wave % 2) * 32;
  const int r32 = lane % 32, hi = lane / 32;
  const int m0 = blockIdx.y * GT, n0 = blockIdx.x * GT;
  // this thread's share of a k tile: A (64 x 32) and B (32 x 64)
  constexpr int AV = sizeof(TA) == 4 ? 2 : 1;  // 16-byte vectors of A per thread
  float4 ra[2];
  u16x8g ra16;
  u16x8g rb;
  auto load = [&](int k0) {
    if (sizeof(TA) == 4) {
#pragma unroll
      for (int i = 0; i < AV; ++i) {
        const int v = threadIdx.x + 256 * i;
        const int row = v / (SBK / 4), kk = (v % (SBK / 4)) * 4;
        const bool ok = m0 + row < M && k0 + kk < K;
        ra[i] = ok ? *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(A) + (int64_t)(m0 + row) * lda +
                                                      k0 + kk)
                   : make_float4(0.f, 0.f, 0.f, 0.f);
      }
    } else {
      const int row = threadIdx.x / (SBK / 8), kk = (threadIdx.x % (SBK / 8)) * 8;
      const bool ok = m0 + row < M && k0 + kk < K;
      ra16 = ok ? *reinterpret_cast<const u16x8g*>(reinterpret_cast<const bf16_bits*>(A) + (int64_t)(m0 + row) * lda +
                                                   k0 + kk)
                : u16x8g{0, 0, 0, 0, 0, 0, 0, 0};
    }
    const int kk = threadIdx.x / (GT / 8), nn = (threadIdx.x % (GT / 8)) * 8;
    const bool ok = k0 + kk < K && n0 + nn < N;
    rb = ok ? *reinterpret_cast<const u16x8g*>(B + (int64_t)(k0 + kk) * ldb + n0 + nn)
            : u16x8g{0, 0, 0, 0, 0, 0, 0, 0};
  };
  auto store = [&](int buf) {
    if (sizeof(TA) == 4) {
#pragma unroll
      for (int i = 0; i < AV; ++i) {
        const int v = threadIdx.x + 256 * i;
        const int row = v / (SBK / 4), kk = (v % (SBK / 4)) * 4;
        float x[4] = {ra[i].x, ra[i].y, ra[i].z, ra[i].w};
#pragma unroll
        for (int t = 0; t < TERMS; ++t) {
          uint2 pk;
          bf16_bits b[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            b[e] = from_f32<bf16_bits>(x[e]);
            x[e] -= to_f32(b[e]);
          }
          pk.x = (uint32_t)b[0] | ((uint32_t)b[1] << 16);
          pk.y = (uint32_t)b[2] | ((uint32_t)b[3] << 16);
          *reinterpret_cast<uint2*>(&As[buf][t][row * SROW + kk]) = pk;
        }
      }
    } else {
      const int row = threadIdx.x / (SBK / 8), kk = (threadIdx.x % (SBK / 8)) * 8;
      *reinterpret_cast<u16x8g*>(&As[buf][0][row * SROW + kk]) = ra16;
    }
    const int kk = threadIdx.x / (GT / 8), nn = (threadIdx.x % (GT / 8)) * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) Bs[buf][(nn + e) * SROW + kk] = rb[e];
  };
  f32x16 acc = {};
  load(0);
  store(0);
  __syncthreads();
  int buf = 0;
  for (int k0 = 0; k0 < K; k0 += SBK) {
    const bool more = k0 + SBK < K;
    if (more) load(k0 + SBK);
#pragma unroll
    for (int ks = 0; ks < SBK / 16; ++ks) {
      const bf16x8g b = *reinterpret_cast<const bf16x8g*>(&Bs[buf][(wn + r32) * SROW + ks * 16 + hi * 8]);
#pragma unroll
      for (int t = 0; t < TERMS; ++t) {
        const bf16x8g a = *reinterpret_cast<const bf16x8g*>(&As[buf][t][(wm + r32) * SROW + ks * 16 + hi * 8]);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
      }
    }
    if (more) store(buf ^ 1);  // that buffer was last read before the previous barrier
    __syncthreads();
    buf ^= 1;
  }
  // result lane layout: column n = lane % 32, rows 8 (v / 4) + 4 hi + v % 4
  const int gn = n0 + wn + r32;
  if (gn >= N) return;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int gm = m0 + wm + 8 * (v / 4) + 4 * hi + (v % 4);
    if (gm >= M) continue;
    float x = alpha * acc[v];
    float* c = C + (int64_t)gm * ldc + gn;
    if (epi == kEpiAddRes) x += R[(int64_t)gm * ldr + gn];
    if (epi == kEpiRelu) {
      if (C2) C2[(int64_t)gm * ldc + gn] = x;
      x = fmaxf(x, 0.f);
    }
    *c = accumulate ? *c + x : x;
  }
}

// ------------------------------------------------------------ attention
// Exact fp32 attention for the generic path and the backward pass.
//
// Lane layouts avoid reductions across lanes inside the token loops:
//  * target lanes: lane = (target t, stream st), 64 / TP streams for TP =
//    16, 32 or 64 target slots; each lane keeps its own target's state and
//    visits every (64 / TP)-th token of its wave's share of a 64-row K/V tile
//    staged in LDS (one row is read by many lanes at once, which LDS serves as
//    a broadcast; rows are padded to keep 16-byte reads conflict-free);
//  * token lanes: lane = history row; the targets' vectors are broadcast from
//    LDS.
// A workgroup (4 waves) handles one (unit, head).
constexpr int kTile = 64;

__device__ __forceinline__ int target_slots(int nt) { return nt <= 16 ? 16 : (nt <= 32 ? 32 : 64); }

template <int DH>
struct KvTile {
  float k[kTile][DH + 4];
  float v[kTile][DH + 4];
};

template <int DH>
__device__ __forceinline__ void stage_kv_tile(KvTile<DH>& T, const float* __restrict__ KV, int d, int j, int base,
                                              int lo, int hi) {
  for (int e = threadIdx.x; e < kTile * DH / 4; e += 256) {
    const int r = e / (DH / 4), c = (e % (DH / 4)) * 4;
    const int tok = base + r;
    const bool on = tok >= lo && tok < hi;
    const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
    *reinterpret_cast<float4*>(&T.k[r][c]) =
        on ? *reinterpret_cast<const float4*>(KV + (int64_t)tok * 2 * d + j * DH + c) : z;
    *reinterpret_cast<float4*>(&T.v[r][c]) =
        on ? *reinterpret_cast<const float4*>(KV + (int64_t)tok * 2 * d + d + j * DH + c) : z;
  }
}

template <int DH>
__device__ __forceinline__ float dot_row(const float (&x)[DH], const float* __restrict__ row) {
  float s = 0.f;
#pragma unroll
  for (int e = 0; e < DH; e += 4) {
    const float4 r = *reinterpret_cast<const float4*>(row + e);
    s = fmaf(x[e], r.x, s);
    s = fmaf(x[e + 1], r.y, s);
    s = fmaf(x[e + 2], r.z, s);
    s = fmaf(x[e + 3], r.w, s);
  }
  return s;
}

// acc = acc * f + p * row
template <int DH>
__device__ __forceinline__ void axpby_row(float (&acc)[DH], float f, float p, const float* __restrict__ row) {
#pragma unroll
  for (int e = 0; e < DH; e += 4) {
    const float4 r = *reinterpret_cast<const float4*>(row + e);
    acc[e] = fmaf(p, r.x, acc[e] * f);
    acc[e + 1] = fmaf(p, r.y, acc[e + 1] * f);
    acc[e + 2] = fmaf(p, r.z, acc[e + 2] * f);
    acc[e + 3] = fmaf(p, r.w, acc[e + 3] * f);
  }
}

// Online-softmax partial (acc, max, sum) per (chunk, target, head); Q holds
// the queries pre-scaled by log2(e)/sqrt(d_h), so scores are in log2 units.
template <int DH>
__global__ __launch_bounds__(256) void attn_generic_kernel(const Unit* __restrict__ units,
                                                           const WsHeader* __restrict__ hdr,
                                                           const float* __restrict__ Q,
                                                           const float* __restrict__ KV, int d,
                                                           float* __restrict__ part_acc,
                                                           float* __restrict__ part_ml, int64_t n_tgt,
                                                           int n_heads) {
  __shared__ __attribute__((aligned(16))) KvTile<DH> T;
  __shared__ float red[4][64][DH + 2];
  const int u = blockIdx.x;
  if (u >= hdr->n_units) return;
  const Unit un = units[u];
  const int j = blockIdx.y;
  const int lane = threadIdx.x % 64, w = threadIdx.x / 64;
  const int TP = target_slots(un.nt), S = 64 / TP;
  const int tt = lane % TP, st = lane / TP;
  const bool live = tt < un.nt;
  float q[DH], acc[DH];
#pragma unroll
  for (int e = 0; e < DH; ++e) {
    q[e] = live ? Q[(int64_t)(un.t0 + tt) * d + j * DH + e] : 0.f;
    acc[e] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  const int lo = max(un.b0 * kBlockTokens, un.l0), hi = min(un.b1 * kBlockTokens, un.l1);
  for (int base = lo; base < hi; base += kTile) {
    __syncthreads();
    stage_kv_tile<DH>(T, KV, d, j, base, lo, hi);
    __syncthreads();
    for (int r = w * 16 + st; r < w * 16 + 16; r += S) {
      if (base + r >= hi) break;
      const float sc = dot_row<DH>(q, T.k[r]);
      const float mn = fmaxf(m, sc);
      const float f = exp2f(m - mn);
      const float p = exp2f(sc - mn);
      l = l * f + p;
      axpby_row<DH>(acc, f, p, T.v[r]);
      m = mn;
    }
  }
  // merge the streams of each target (lanes tt + k TP), then the four waves
  for (int o = TP; o < 64; o <<= 1) {
    const float mo = __shfl_xor(m, o), lo_ = __shfl_xor(l, o);
    const float mn = fmaxf(m, mo);
    const float fa = m == -INFINITY ? 0.f : exp2f(m - mn), fb = mo == -INFINITY ? 0.f : exp2f(mo - mn);
    l = l * fa + lo_ * fb;
#pragma unroll
    for (int e = 0; e < DH; ++e) acc[e] = acc[e] * fa + __shfl_xor(acc[e], o) * fb;
    m = mn;
  }
  if (st == 0) {
    red[w][tt][0] = m;
    red[w][tt][1] = l;
#pragma unroll
    for (int e = 0; e < DH; ++e) red[w][tt][2 + e] = acc[e];
  }
  __syncthreads();
  for (int it = threadIdx.x; it < un.nt * (DH + 1); it += 256) {
    const int t = it / (DH + 1), e = it % (DH + 1);  // e == DH: (max, sum)
    float M = -INFINITY;
    for (int ww = 0; ww < 4; ++ww) M = fmaxf(M, red[ww][t][0]);
    float v = 0.f;
    for (int ww = 0; ww < 4; ++ww) {
      const float mw = red[ww][t][0];
      const float f = mw == -INFINITY ? 0.f : exp2f(mw - M);
      v += f * (e == DH ? red[ww][t][1] : red[ww][t][2 + e]);
    }
    const int64_t row = (int64_t)un.c * n_tgt + un.t0 + t;
    if (e == DH) {
      part_ml[(row * n_heads + j) * 2] = M;
      part_ml[(row * n_heads + j) * 2 + 1] = v;
    } else {
      part_acc[row * d + j * DH + e] = v;
    }
  }
}

// Merge the per-chunk partial results of every (target, head).
// One thread per (target, head, 4 consecutive dims): every chunk's (max, sum)
// and 16-byte slices of its accumulator, so a head's merge is d_h / 4 threads
// reading whole cache lines instead of one thread walking d_h floats.
__global__ void merge_generic_kernel(int dh, int n_heads, int64_t n_tgt, const int32_t* __restrict__ tchunks,
                                     const float* __restrict__ part_acc, const float* __restrict__ part_ml,
                                     float* __restrict__ a, float* __restrict__ lse) {
  const int q4 = dh / 4;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= n_tgt * n_heads * q4) return;
  const int64_t th = idx / q4;  // (target, head)
  const int e = static_cast<int>(idx % q4) * 4;
  const int64_t t = th / n_heads;
  const int j = static_cast<int>(th % n_heads);
  const int d = dh * n_heads;
  const int nch = tchunks[t];
  const float2* ml = reinterpret_cast<const float2*>(part_ml);
  float M = -INFINITY;
  for (int c = 0; c < nch; ++c) M = fmaxf(M, ml[((int64_t)c * n_tgt + t) * n_heads + j].x);
  float L = 0.f;
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int c = 0; c < nch; ++c) {
    const float2 m = ml[((int64_t)c * n_tgt + t) * n_heads + j];
    const float wc = exp2f(m.x - M);
    L += wc * m.y;
    const float4 x = *reinterpret_cast<const float4*>(part_acc + ((int64_t)c * n_tgt + t) * d + j * dh + e);
    v.x += wc * x.x, v.y += wc * x.y, v.z += wc * x.z, v.w += wc * x.w;
  }
  const float inv = 1.f / L;
  *reinterpret_cast<float4*>(a + t * d + j * dh + e) = make_float4(v.x * inv, v.y * inv, v.z * inv, v.w * inv);
  if (lse && e == 0) lse[t * n_heads + j] = (M + log2f(L)) * kLn2;
}

// ------------------------------------------------- attention backward
// With p = softmax weight, dp = dA . v, D = rowsum(dA * A):
//   de = p (dp - D);  dq = sum_rows de k / sqrt(d_h);  dk = sum_targets de q / sqrt(d_h);
//   dv = sum_targets p dA.
// dK/dV: token lanes; each history row's gradient is summed over every target
// of its request by one thread (the unit of the request's first target group
// does it, in batches of kTargetGroup targets), so it is written, not added.
// dq: target lanes.

template <typename T>
__device__ __forceinline__ void store_row(T* dst, const float* v, int n, float scale);
template <>
__device__ __forceinline__ void store_row<float>(float* dst, const float* v, int n, float scale) {
  for (int e = 0; e < n; e += 4)
    *reinterpret_cast<float4*>(dst + e) = make_float4(v[e] * scale, v[e + 1] * scale, v[e + 2] * scale,
                                                      v[e + 3] * scale);
}
template <>
__device__ __forceinline__ void store_row<bf16_bits>(bf16_bits* dst, const float* v, int n, float scale) {
  for (int e = 0; e < n; e += 4) {
    ushort4 o;
    o.x = from_f32<bf16_bits>(v[e] * scale);
    o.y = from_f32<bf16_bits>(v[e + 1] * scale);
    o.z = from_f32<bf16_bits>(v[e + 2] * scale);
    o.w = from_f32<bf16_bits>(v[e + 3] * scale);
    *reinterpret_cast<ushort4*>(dst + e) = o;
  }
}

template <int DH, typename OT>
__global__ __launch_bounds__(256) void attn_bwd_kv_kernel(
    const Unit* __restrict__ units, const WsHeader* __restrict__ hdr, const int32_t* __restrict__ toff,
    const float* __restrict__ Q, const float* __restrict__ KV, int d, const float* __restrict__ a,
    const float* __restrict__ da, const float* __restrict__ lse, OT* __restrict__ dKV, int64_t ldkv,
    bf16_bits* __restrict__ dKVT, int64_t ldt, int n_heads) {
  __shared__ __attribute__((aligned(16))) float qs[kTargetGroup][DH];
  __shared__ __attribute__((aligned(16))) float das[kTargetGroup][DH];
  __shared__ float cs[kTargetGroup][2];
  const int u = blockIdx.x;
  if (u >= hdr->n_units) return;
  const Unit un = units[u];
  const int T0 = toff[un.r], T1 = toff[un.r + 1];
  if (un.t0 != T0) return;  // not the request's first target group
  const int j = blockIdx.y;
  const int nbatch = static_cast<int>(ceil_div(T1 - T0, kTargetGroup));
  auto stage = [&](int tb) {
    const int nb = min(kTargetGroup, T1 - tb);
    for (int e = threadIdx.x; e < nb * DH; e += 256) {
      const int64_t t = tb + e / DH;
      qs[e / DH][e % DH] = Q[t * d + j * DH + e % DH];
      das[e / DH][e % DH] = da[t * d + j * DH + e % DH];
    }
    for (int tt = threadIdx.x; tt < nb; tt += 256) {
      const int64_t t = tb + tt;
      float D = 0.f;
      for (int e = 0; e < DH; ++e) D += da[t * d + j * DH + e] * a[t * d + j * DH + e];
      cs[tt][0] = lse[t * n_heads + j] * kLog2e;
      cs[tt][1] = D;
    }
  };
  if (nbatch == 1) stage(T0);
  __syncthreads();
  const int lo = max(un.b0 * kBlockTokens, un.l0), hi = min(un.b1 * kBlockTokens, un.l1);
  for (int base = lo; base < hi; base += 256) {
    const int tok = base + threadIdx.x;
    const bool on = tok < hi;
    float k[DH], v[DH], dk[DH], dv[DH];
#pragma unroll
    for (int e = 0; e < DH; e += 4) {
      const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
      const float4 kk = on ? *reinterpret_cast<const float4*>(KV + (int64_t)tok * 2 * d + j * DH + e) : z;
      const float4 vv = on ? *reinterpret_cast<const float4*>(KV + (int64_t)tok * 2 * d + d + j * DH + e) : z;
      k[e] = kk.x, k[e + 1] = kk.y, k[e + 2] = kk.z, k[e + 3] = kk.w;
      v[e] = vv.x, v[e + 1] = vv.y, v[e + 2] = vv.z, v[e + 3] = vv.w;
    }
#pragma unroll
    for (int e = 0; e < DH; ++e) dk[e] = dv[e] = 0.f;
    for (int bt = 0; bt < nbatch; ++bt) {
      const int tb = T0 + bt * kTargetGroup;
      if (nbatch > 1) {
        __syncthreads();
        stage(tb);
        __syncthreads();
      }
      const int nb = min(kTargetGroup, T1 - tb);
      for (int tt = 0; tt < nb; ++tt) {
        const float s = dot_row<DH>(k, qs[tt]);
        const float dp = dot_row<DH>(v, das[tt]);
        const float p = exp2f(s - cs[tt][0]);
        const float de = p * (dp - cs[tt][1]);
        axpby_row<DH>(dk, 1.f, de, qs[tt]);
        axpby_row<DH>(dv, 1.f, p, das[tt]);
      }
    }
    // Q holds log2(e)/sqrt(d_h) times the true query: dk of the true query
    // is de q / sqrt(d_h) = de * (stored q) * ln 2
    if (on) {
      store_row<OT>(dKV + (int64_t)tok * ldkv + j * DH, dk, DH, kLn2);
      store_row<OT>(dKV + (int64_t)tok * ldkv + d + j * DH, dv, DH, 1.f);
      if (dKVT) {  // transposed copy: consecutive lanes write consecutive rows
#pragma unroll
        for (int e = 0; e < DH; ++e) {
          dKVT[(int64_t)(j * DH + e) * ldt + tok] = from_f32<bf16_bits>(dk[e] * kLn2);
          dKVT[(int64_t)(d + j * DH + e) * ldt + tok] = from_f32<bf16_bits>(dv[e]);
        }
      }
    }
  }
}

template <int DH>
__global__ __launch_bounds__(256) void attn_bwd_q_kernel(
    const Unit* __restrict__ units, const WsHeader* __restrict__ hdr, const float* __restrict__ Q,
    const float* __restrict__ KV, int d, const float* __restrict__ a, const float* __restrict__ da,
    const float* __restrict__ lse, float* __restrict__ dq_part, int64_t n_tgt, int n_heads) {
  __shared__ __attribute__((aligned(16))) KvTile<DH> T;
  __shared__ float red[4][64][DH];
  const int u = blockIdx.x;
  if (u >= hdr->n_units) return;
  const Unit un = units[u];
  const int j = blockIdx.y;
  const int lane = threadIdx.x % 64, w = threadIdx.x / 64;
  const int TP = target_slots(un.nt), S = 64 / TP;
  const int tt = lane % TP, st = lane / TP;
  const bool live = tt < un.nt;
  const int64_t t = un.t0 + (live ? tt : 0);
  float q[DH], dat[DH], dq[DH];
  float D = 0.f;
#pragma unroll
  for (int e = 0; e < DH; ++e) {
    q[e] = live ? Q[t * d + j * DH + e] : 0.f;
    dat[e] = live ? da[t * d + j * DH + e] : 0.f;
    D += live ? dat[e] * a[t * d + j * DH + e] : 0.f;
    dq[e] = 0.f;
  }
  const float ls = live ? lse[t * n_heads + j] * kLog2e : 0.f;
  const int lo = max(un.b0 * kBlockTokens, un.l0), hi = min(un.b1 * kBlockTokens, un.l1);
  for (int base = lo; base < hi; base += kTile) {
    __syncthreads();
    stage_kv_tile<DH>(T, KV, d, j, base, lo, hi);
    __syncthreads();
    for (int r = w * 16 + st; r < w * 16 + 16; r += S) {
      if (base + r >= hi) break;
      const float sc = dot_row<DH>(q, T.k[r]);
      const float dp = dot_row<DH>(dat, T.v[r]);
      const float de = live ? exp2f(sc - ls) * (dp - D) : 0.f;
      axpby_row<DH>(dq, 1.f, de, T.k[r]);
    }
  }
  for (int o = TP; o < 64; o <<= 1)
#pragma unroll
    for (int e = 0; e < DH; ++e) dq[e] += __shfl_xor(dq[e], o);
  if (st == 0)
#pragma unroll
    for (int e = 0; e < DH; ++e) red[w][tt][e] = dq[e];
  __syncthreads();
  const float scale = 1.f / sqrtf((float)DH);
  for (int it = threadIdx.x; it < un.nt * DH; it += 256) {
    const int t2 = it / DH, e = it % DH;
    const float v = red[0][t2][e] + red[1][t2][e] + red[2][t2][e] + red[3][t2][e];
    dq_part[((int64_t)un.c * n_tgt + un.t0 + t2) * d + j * DH + e] = v * scale;
  }
}

__global__ void reduce_chunks_kernel(int64_t n_tgt, int d, const int32_t* __restrict__ tchunks,
                                     const float* __restrict__ part, float* __restrict__ out,
                                     bf16_bits* __restrict__ out16, float scale) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= n_tgt * d) return;
  const int64_t t = idx / d;
  float v = 0.f;
  for (int c = 0; c < tchunks[t]; ++c) v += part[(int64_t)c * n_tgt * d + idx];
  v *= scale;
  if (out) out[idx] = v;
  if (out16) out16[idx] = from_f32<bf16_bits>(v);
}

__global__ void relu_mask_kernel(float* __restrict__ dh, const float* __restrict__ pre, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n && !(pre[i] > 0.f)) dh[i] = 0.f;
}

// One workgroup per request (and one more for dKVT's padding columns); the
// row range is clamped to [0, n_hist), so malformed offsets write nothing
// outside the buffers (the scheduler reports them).
__global__ void zero_untargeted_kernel(const int32_t* __restrict__ hoff, const int32_t* __restrict__ toff,
                                       int n_requests, int64_t n_hist, bf16_bits* __restrict__ dKV, int64_t ldkv,
                                       int cols, bf16_bits* __restrict__ dKVT, int64_t ldt) {
  const int r = blockIdx.x;
  int64_t h0, h1;
  if (r < n_requests) {
    if (toff[r + 1] != toff[r]) return;
    h0 = max<int64_t>(0, hoff[r]);
    h1 = min<int64_t>(n_hist, hoff[r + 1]);
    const int64_t cnt = (h1 - h0) * cols;
    for (int64_t e = threadIdx.x; e < cnt; e += blockDim.x) dKV[(h0 + e / cols) * ldkv + e % cols] = 0;
  } else {
    h0 = n_hist;
    h1 = ldt;
  }
  if (h1 <= h0 || !dKVT) return;
  const int64_t w = h1 - h0, cnt = w * cols;
  for (int64_t e = threadIdx.x; e < cnt; e += blockDim.x) {
    const int64_t c = e / w, row = h0 + e % w;
    dKVT[c * ldt + row] = 0;
  }
}

// [W_K^0 | W_V^0 | W_K^1 | ...] ([d][n 2d] bf16) from the stacked W_K, W_V
// ([n][d][d]); one thread per 8 columns
__global__ void pack_wkv_kernel(const bf16_bits* __restrict__ wk, const bf16_bits* __restrict__ wv, int n, int d,
                                bf16_bits* __restrict__ wkv) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int per_row = n * 2 * d / 8;
  if (g >= (int64_t)d * per_row) return;
  const int r = static_cast<int>(g / per_row), c = static_cast<int>(g % per_row) * 8;
  const int i = c / (2 * d), cc = c % (2 * d);
  const bf16_bits* src = (cc < d ? wk : wv) + ((int64_t)i * d + r) * d + cc % d;
  *reinterpret_cast<uint4*>(wkv + (int64_t)r * n * 2 * d + c) = *reinterpret_cast<const uint4*>(src);
}

// dW_K^i, dW_V^i ([n][d][d] fp32) from [dW_K^0 | dW_V^0 | ...] ([d][n 2d]);
// one thread per 4 columns
__global__ void split_dwkv_kernel(const float* __restrict__ dwkv, int n, int d, float* __restrict__ dwk,
                                  float* __restrict__ dwv) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int per_row = n * 2 * d / 4;
  if (g >= (int64_t)d * per_row) return;
  const int r = static_cast<int>(g / per_row), c = static_cast<int>(g % per_row) * 4;
  const int i = c / (2 * d), cc = c % (2 * d);
  float* dst = (cc < d ? dwk : dwv) + ((int64_t)i * d + r) * d + cc % d;
  *reinterpret_cast<float4*>(dst) = *reinterpret_cast<const float4*>(dwkv + (int64_t)r * n * 2 * d + c);
}

template <typename S, typename D>
__global__ void convert_kernel(const S* __restrict__ src, D* __restrict__ dst, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = from_f32<D>(to_f32(src[i]));
}

__global__ void fill_kernel(float* __restrict__ dst, float v, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = v;
}

inline dim3 grid1(int64_t n, int b) { return dim3(static_cast<unsigned>(ceil_div(n, b))); }

}  // namespace

__global__ void fill2d_kernel(float* __restrict__ C, int64_t ldc, int M, int N) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < (int64_t)M * N) C[(i / N) * ldc + i % N] = 0.f;
}

hipError_t gemm_generic(int a_bf16, int b_bf16, int M, int N, int K, const void* A, int64_t lda,
                        int transA, const void* B, int64_t ldb, int transB, float* C, int64_t ldc,
                        float alpha, GemmEpi epi, const float* R, int64_t ldr, float* C2,
                        int accumulate, hipStream_t st) {
  if (M == 0 || N == 0) return hipSuccess;
  const int64_t tiles = ceil_div(N, GT) * ceil_div(M, GT);
  // long reductions (weight gradients over all rows) with few output tiles are
  // split over K so the whole chip works on them and each partial sum is short
  int splits = 1;
  if (epi == kEpiStore && tiles < 256 && K >= 1024) {
    splits = static_cast<int>(std::min<int64_t>(ceil_div(512, tiles), K / 512));
    if (splits < 1) splits = 1;
  }
  const int k_chunk = static_cast<int>(round_up(ceil_div(K, splits), GK));
  splits = static_cast<int>(ceil_div(K, k_chunk));
  // bf16 weights, untransposed operands, no split: the bf16 matrix cores with
  // A split into bf16 terms (whole 16-byte vectors: K, N and the leading
  // dimensions multiples of 8, 16-byte aligned operands)
  const auto al16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; };
  if (splits == 1 && b_bf16 && !transA && !transB && K % 8 == 0 && N % 8 == 0 && lda % 8 == 0 && ldb % 8 == 0 &&
      al16(A) && al16(B)) {
    dim3 g2(static_cast<unsigned>(ceil_div(N, GT)), static_cast<unsigned>(ceil_div(M, GT)));
    if (a_bf16)
      hipLaunchKernelGGL((gemm_bf16w_kernel<bf16_bits>), g2, dim3(256), 0, st, M, N, K, (const bf16_bits*)A, lda,
                         (const bf16_bits*)B, ldb, C, ldc, alpha, (int)epi, R, ldr, C2, accumulate);
    else
      hipLaunchKernelGGL((gemm_bf16w_kernel<float>), g2, dim3(256), 0, st, M, N, K, (const float*)A, lda,
                         (const bf16_bits*)B, ldb, C, ldc, alpha, (int)epi, R, ldr, C2, accumulate);
    return hipGetLastError();
  }
  if (splits > 1 && !accumulate)
    hipLaunchKernelGGL(fill2d_kernel, grid1((int64_t)M * N, 256), dim3(256), 0, st, C, ldc, M, N);
  dim3 g(static_cast<unsigned>(ceil_div(N, GT)), static_cast<unsigned>(ceil_div(M, GT)), splits);
#define STCA_GEMM(TA, TB)                                                                          \
  hipLaunchKernelGGL((gemm_kernel<TA, TB>), g, dim3(256), 0, st, M, N, K, (const TA*)A, lda, transA, \
                     (const TB*)B, ldb, transB, C, ldc, alpha, (int)epi, R, ldr, C2, accumulate, k_chunk)
  if (a_bf16 && b_bf16) STCA_GEMM(bf16_bits, bf16_bits);
  else if (a_bf16) STCA_GEMM(bf16_bits, float);
  else if (b_bf16) STCA_GEMM(float, bf16_bits);
  else STCA_GEMM(float, float);
#undef STCA_GEMM
  return hipGetLastError();
}

hipError_t attn_generic(int d_head, int n_heads, const Unit* units, int64_t max_units, const WsHeader* hdr,
                        const float* Q, const float* KV, int d, float* part_acc, float* part_ml,
                        int64_t n_tgt, hipStream_t st) {
  if (max_units == 0) return hipSuccess;
  if (attn_mfma_supported(d_head))
    return attn_fwd_mfma(d_head, n_heads, units, max_units, hdr, Q, KV, d, part_acc, part_ml, n_tgt, st);
  dim3 g(static_cast<unsigned>(max_units), n_heads);
#define STCA_ATT(DH)                                                                                    \
  hipLaunchKernelGGL(attn_generic_kernel<DH>, g, dim3(256), 0, st, units, hdr, Q, KV, d, part_acc, part_ml, \
                     n_tgt, n_heads)
  switch (d_head) {
    case 8: STCA_ATT(8); break;
    case 16: STCA_ATT(16); break;
    case 32: STCA_ATT(32); break;
    case 64: STCA_ATT(64); break;
    default: return hipErrorInvalidValue;
  }
#undef STCA_ATT
  return hipGetLastError();
}

hipError_t merge_generic(int d_head, int n_heads, int64_t n_tgt, const int32_t* tchunks, const float* part_acc,
                         const float* part_ml, float* a, float* lse, hipStream_t st) {
  if (n_tgt == 0) return hipSuccess;
  if (d_head % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(merge_generic_kernel, grid1(n_tgt * n_heads * (d_head / 4), 256), dim3(256), 0, st, d_head,
                     n_heads, n_tgt, tchunks, part_acc, part_ml, a, lse);
  return hipGetLastError();
}

hipError_t attn_bwd_generic(int d_head, int n_heads, const Unit* units, int64_t max_units,
                            const WsHeader* hdr, const int32_t* toff, const float* Q, const float* KV, int d,
                            const float* a, const float* da, const float* lse, float* dq_part, void* dKV,
                            int64_t ldkv, int dkv_bf16, bf16_bits* dKVT, int64_t ldt, int64_t n_tgt,
                            hipStream_t st) {
  if (max_units == 0) return hipSuccess;
  if (attn_mfma_supported(d_head))
    return attn_bwd_mfma(d_head, n_heads, units, max_units, hdr, toff, Q, KV, d, a, da, lse, dq_part, dKV, ldkv,
                         dkv_bf16, dKVT, ldt, n_tgt, st);
  dim3 g(static_cast<unsigned>(max_units), n_heads);
#define STCA_ATTB(DH)                                                                                      \
  if (dkv_bf16)                                                                                            \
    hipLaunchKernelGGL((attn_bwd_kv_kernel<DH, bf16_bits>), g, dim3(256), 0, st, units, hdr, toff, Q, KV, d, a, \
                       da, lse, static_cast<bf16_bits*>(dKV), ldkv, dKVT, ldt, n_heads);                    \
  else                                                                                                     \
    hipLaunchKernelGGL((attn_bwd_kv_kernel<DH, float>), g, dim3(256), 0, st, units, hdr, toff, Q, KV, d, a, da, \
                       lse, static_cast<float*>(dKV), ldkv, nullptr, 0, n_heads);                           \
  hipLaunchKernelGGL(attn_bwd_q_kernel<DH>, g, dim3(256), 0, st, units, hdr, Q, KV, d, a, da, lse, dq_part,  \
                     n_tgt, n_heads)
  switch (d_head) {
    case 8: STCA_ATTB(8); break;
    case 16: STCA_ATTB(16); break;
    case 32: STCA_ATTB(32); break;
    case 64: STCA_ATTB(64); break;
    default: return hipErrorInvalidValue;
  }
#undef STCA_ATTB
  return hipGetLastError();
}

hipError_t reduce_chunks(int64_t n_tgt, int d, const int32_t* tchunks, const float* part, float* out,
                         bf16_bits* out16, float scale, hipStream_t st) {
  if (n_tgt == 0) return hipSuccess;
  hipLaunchKernelGGL(reduce_chunks_kernel, grid1(n_tgt * d, 256), dim3(256), 0, st, n_tgt, d, tchunks, part,
                     out, out16, scale);
  return hipGetLastError();
}

hipError_t relu_mask_mul(float* dh, const float* pre, int64_t n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(relu_mask_kernel, grid1(n, 256), dim3(256), 0, st, dh, pre, n);
  return hipGetLastError();
}

hipError_t zero_untargeted(const int32_t* hoff, const int32_t* toff, int n_requests, int64_t n_hist,
                           bf16_bits* dKV, int64_t ldkv, int cols, bf16_bits* dKVT, int64_t ldt, hipStream_t st) {
  hipLaunchKernelGGL(zero_untargeted_kernel, dim3(static_cast<unsigned>(n_requests + 1)), dim3(256), 0, st, hoff,
                     toff, n_requests, n_hist, dKV, ldkv, cols, dKVT, ldt);
  return hipGetLastError();
}

hipError_t convert(int src_bf16, int dst_bf16, const void* src, void* dst, int64_t n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  dim3 g = grid1(n, 256);
  if (src_bf16 && dst_bf16)
    hipLaunchKernelGGL((convert_kernel<bf16_bits, bf16_bits>), g, dim3(256), 0, st, (const bf16_bits*)src,
                       (bf16_bits*)dst, n);
  else if (src_bf16)
    hipLaunchKernelGGL((convert_kernel<bf16_bits, float>), g, dim3(256), 0, st, (const bf16_bits*)src,
                       (float*)dst, n);
  else if (dst_bf16)
    hipLaunchKernelGGL((convert_kernel<float, bf16_bits>), g, dim3(256), 0, st, (const float*)src,
                       (bf16_bits*)dst, n);
  else
    hipLaunchKernelGGL((convert_kernel<float, float>), g, dim3(256), 0, st, (const float*)src, (float*)dst, n);
  return hipGetLastError();
}

hipError_t pack_wkv(const bf16_bits* wk, const bf16_bits* wv, int n, int d, bf16_bits* wkv, hipStream_t st) {
  if (d % 8) return hipErrorInvalidValue;
  const int64_t threads = (int64_t)d * n * 2 * d / 8;
  if (threads == 0) return hipSuccess;
  hipLaunchKernelGGL(pack_wkv_kernel, grid1(threads, 256), dim3(256), 0, st, wk, wv, n, d, wkv);
  return hipGetLastError();
}

hipError_t split_dwkv(const float* dwkv, int n, int d, float* dwk, float* dwv, hipStream_t st) {
  if (d % 4) return hipErrorInvalidValue;
  const int64_t threads = (int64_t)d * n * 2 * d / 4;
  if (threads == 0) return hipSuccess;
  hipLaunchKernelGGL(split_dwkv_kernel, grid1(threads, 256), dim3(256), 0, st, dwkv, n, d, dwk, dwv);
  return hipGetLastError();
}

hipError_t fill_f32(float* dst, float v, int64_t n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(fill_kernel, grid1(n, 256), dim3(256), 0, st, dst, v, n);
  return hipGetLastError();
}

}  // namespace stca
