// Exact fp32 attention (forward recomputation and backward) on the fp32 matrix
// cores, v_mfma_f32_16x16x4_f32, for head widths d_h in {16, 32, 64}.
//
// For this instruction lane l = 16 g + r (g = l / 16, r = l % 16) holds
//   A operand: A[i = r][k = g]    B operand: B[k = g][j = r]
//   result   : D[i = 4 g + v][j = r], v = 0..3
// and a product over K > 4 is a chain of k-steps.  Any bijection between
// (g, step) and the contracted index serves, as long as A and B use the same
// one; the kernels below pick, per product, the one that lets an operand come
// straight from the registers of an earlier result.
//
// Tiles are 16 history rows x 16 targets.  Scores are formed transposed,
// S^T = K Q^T (result lane r = target, v = row 4 g + v), so the per-target
// softmax statistics need only two lane exchanges (g), and P^T (and dE^T)
// feed products that contract over rows (O^T = V^T P^T, dQ^T = K^T dE^T) as
// their B operand directly.  Products that contract over targets (dV^T =
// dA^T P, dK^T = Q^T dE) take P and dE through a 16 x 16 transpose in LDS.
// Every other operand is loaded from global memory (L2) straight into the
// register layout it is used in, the next row tile's while the current one is
// multiplied; a wave works through its row tiles alone, so several waves per
// SIMD hide each other's latencies.
//
// Queries are stored pre-scaled by log2(e)/sqrt(d_h) (scores in log2 units);
// lse is natural-log.  With p = softmax weight, dp = dA . v, D = rowsum(dA*A):
//   de = p (dp - D);  dq = sum_rows de k / sqrt(d_h);
//   dk = sum_targets de q / sqrt(d_h) = sum_targets de (stored q) ln 2;
//   dv = sum_targets p dA.
#include "common.h"
#include "internal.h"

namespace stca {

namespace {

constexpr int kRows = 16;   // history rows per tile
constexpr int kWaves = 4;   // waves per workgroup; row tiles are dealt round robin

__device__ __forceinline__ f32x4 mma(float a, float b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// n consecutive floats (n % 4 == 0, 16-byte aligned) or zeros
template <int N>
__device__ __forceinline__ void load_run(float (&x)[N], const float* p, bool on) {
#pragma unroll
  for (int i = 0; i < N; i += 4) {
    const float4 v = on ? *reinterpret_cast<const float4*>(p + i) : make_float4(0.f, 0.f, 0.f, 0.f);
    x[i] = v.x, x[i + 1] = v.y, x[i + 2] = v.z, x[i + 3] = v.w;
  }
}

// Online-softmax partials per (chunk, target, head), as the SIMT kernel
// writes them: acc[c][t][d] unnormalised, (max in log2 units, sum).
// Targets go 16 at a time; for each, every wave runs through its row tiles,
// then the four waves' partials are merged.
template <int DH>
__global__ __launch_bounds__(64 * kWaves) void attn_fwd_mfma_kernel(const Unit* __restrict__ units,
                                                                    const WsHeader* __restrict__ hdr,
                                                                    const float* __restrict__ Q,
                                                                    const float* __restrict__ KV, int d,
                                                                    float* __restrict__ part_acc,
                                                                    float* __restrict__ part_ml, int64_t n_tgt,
                                                                    int n_heads) {
  constexpr int DT = DH / 16;  // 16-wide dimension tiles
  constexpr int KQ = DH / 4;   // k-steps over the head's dimensions
  __shared__ float red[kWaves][16][DH + 2];
  const int u = blockIdx.x;
  if (u >= hdr->n_units) return;
  const Unit un = units[u];
  const int j = blockIdx.y;
  const int w = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int r = lane % 16, g = lane / 16;
  const int lo = max(un.b0 * kBlockTokens, un.l0), hi = min(un.b1 * kBlockTokens, un.l1);
  const int nrt = (hi - lo + kRows - 1) / kRows;
  const float* Kh = KV + j * DH;
  const float* Vh = KV + d + j * DH;
  const int64_t ld = 2 * (int64_t)d;
  // the S^T operand (row r, dimensions g KQ ..) and the O^T operand (rows
  // 4 g + s, dimension 16 dt + r) of one row tile
  struct Tile {
    float k[KQ];
    float v[DT][4];
  };
  auto fetch = [&](int rt, Tile& T) {
    const int row0 = lo + rt * kRows;
    load_run<KQ>(T.k, Kh + (row0 + r) * ld + g * KQ, row0 + r < hi);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int row = row0 + 4 * g + ks;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) T.v[dt][ks] = row < hi ? Vh[row * ld + 16 * dt + r] : 0.f;
    }
  };
  for (int t0 = 0; t0 < un.nt; t0 += 16) {
    const int tq = t0 + r;
    float qb[KQ];
    load_run<KQ>(qb, Q + (int64_t)(un.t0 + tq) * d + j * DH + g * KQ, tq < un.nt);
    float m = -INFINITY, l = 0.f;
    f32x4 o[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    Tile cur, nxt;
    if (w < nrt) fetch(w, nxt);
    for (int rt = w; rt < nrt; rt += kWaves) {
      cur = nxt;
      if (rt + kWaves < nrt) fetch(rt + kWaves, nxt);
      const int row0 = lo + rt * kRows;
      // S^T: k-step s, lane group g <-> dimension g KQ + s (two chains)
      f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KQ; ks += 2) {
        s0 = mma(cur.k[ks], qb[ks], s0);
        s1 = mma(cur.k[ks + 1], qb[ks + 1], s1);
      }
      float sv[4], mx = -INFINITY;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        sv[v] = row0 + 4 * g + v < hi ? s0[v] + s1[v] : -INFINITY;
        mx = fmaxf(mx, sv[v]);
      }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mn = fmaxf(m, mx);
      const float f = m == -INFINITY ? 0.f : exp2f(m - mn);
      float p[4], ps = 0.f;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        p[v] = sv[v] == -INFINITY ? 0.f : exp2f(sv[v] - mn);
        ps += p[v];
      }
      ps += __shfl_xor(ps, 16);
      ps += __shfl_xor(ps, 32);
      l = l * f + ps;
      m = mn;
      // O^T += V^T P^T: k-step s, lane group g <-> row 4 g + s
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        f32x4 acc = o[dt] * f;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) acc = mma(cur.v[dt][ks], p[ks], acc);
        o[dt] = acc;
      }
    }
    // merge the four waves' partials of these 16 targets
    if (g == 0) {
      red[w][r][0] = m;
      red[w][r][1] = l;
    }
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int v = 0; v < 4; ++v) red[w][r][2 + 16 * dt + 4 * g + v] = o[dt][v];
    __syncthreads();
    const int ntile = min(16, un.nt - t0);
    for (int it = threadIdx.x; it < ntile * (DH + 1); it += 64 * kWaves) {
      const int t = it / (DH + 1), e = it % (DH + 1);  // e == DH: (max, sum)
      float M = -INFINITY;
      for (int ww = 0; ww < kWaves; ++ww) M = fmaxf(M, red[ww][t][0]);
      float val = 0.f;
      for (int ww = 0; ww < kWaves; ++ww) {
        const float mw = red[ww][t][0];
        const float fw = mw == -INFINITY ? 0.f : exp2f(mw - M);
        val += fw * (e == DH ? red[ww][t][1] : red[ww][t][2 + e]);
      }
      const int64_t row = (int64_t)un.c * n_tgt + un.t0 + t0 + t;
      if (e == DH) {
        part_ml[(row * n_heads + j) * 2] = M;
        part_ml[(row * n_heads + j) * 2 + 1] = val;
      } else {
        part_acc[row * d + j * DH + e] = val;
      }
    }
    __syncthreads();
  }
}

// four consecutive values (16-byte aligned fp32, 8-byte aligned bf16)
__device__ __forceinline__ void store4(float* p, const float (&x)[4]) {
  *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
}
__device__ __forceinline__ void store4(bf16_bits* p, const float (&x)[4]) {
  ushort4 o;
  o.x = from_f32<bf16_bits>(x[0]);
  o.y = from_f32<bf16_bits>(x[1]);
  o.z = from_f32<bf16_bits>(x[2]);
  o.w = from_f32<bf16_bits>(x[3]);
  *reinterpret_cast<ushort4*>(p) = o;
}
__device__ __forceinline__ void add4(float (&x)[4], const float* p) {
  const float4 v = *reinterpret_cast<const float4*>(p);
  x[0] += v.x, x[1] += v.y, x[2] += v.z, x[3] += v.w;
}
__device__ __forceinline__ void add4(float (&x)[4], const bf16_bits* p) {
  const ushort4 v = *reinterpret_cast<const ushort4*>(p);
  x[0] += to_f32(v.x), x[1] += to_f32(v.y), x[2] += to_f32(v.z), x[3] += to_f32(v.w);
}

// Backward of one (request chunk, head): dK/dV of the chunk's rows summed over
// every target of the request (the workgroup of the request's first target
// group does the whole request, 16 targets at a time; later batches add to
// what the first wrote), and the chunk's dq partial for each of those targets.
template <int DH, typename OT>
__global__ __launch_bounds__(64 * kWaves) void attn_bwd_mfma_kernel(
    const Unit* __restrict__ units, const WsHeader* __restrict__ hdr, const int32_t* __restrict__ toff,
    const float* __restrict__ Q, const float* __restrict__ KV, int d, const float* __restrict__ a,
    const float* __restrict__ da, const float* __restrict__ lse, OT* __restrict__ dKV, int64_t ldkv,
    bf16_bits* __restrict__ dKVT, int64_t ldt, float* __restrict__ dq_part, int64_t n_tgt, int n_heads) {
  constexpr int DT = DH / 16;
  constexpr int KQ = DH / 4;
  __shared__ float pT[kWaves][kRows][17], eT[kWaves][kRows][17];
  __shared__ float red[kWaves][16][DH];
  const int u = blockIdx.x;
  if (u >= hdr->n_units) return;
  const Unit un = units[u];
  const int T0 = toff[un.r], T1 = toff[un.r + 1];
  if (un.t0 != T0) return;  // not the request's first target group
  const int j = blockIdx.y;
  const int w = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int r = lane % 16, g = lane / 16;
  const int lo = max(un.b0 * kBlockTokens, un.l0), hi = min(un.b1 * kBlockTokens, un.l1);
  const int nrt = (hi - lo + kRows - 1) / kRows;
  const float* Kh = KV + j * DH;
  const float* Vh = KV + d + j * DH;
  const int64_t ld = 2 * (int64_t)d;
  // S^T / dP^T operands (row r, dimensions g KQ ..) and the dQ^T operand
  // (rows 4 g + s, dimension 16 dt + r) of one row tile
  struct Tile {
    float k[KQ], v[KQ];
    float kc[DT][4];
  };
  auto fetch = [&](int rt, Tile& T) {
    const int row0 = lo + rt * kRows;
    load_run<KQ>(T.k, Kh + (row0 + r) * ld + g * KQ, row0 + r < hi);
    load_run<KQ>(T.v, Vh + (row0 + r) * ld + g * KQ, row0 + r < hi);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int row = row0 + 4 * g + ks;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) T.kc[dt][ks] = row < hi ? Kh[row * ld + 16 * dt + r] : 0.f;
    }
  };
  for (int tb = T0; tb < T1; tb += 16) {
    const int nb = min(16, T1 - tb);
    const bool first = tb == T0;
    const bool live = r < nb;
    const int64_t t = tb + (live ? r : 0);
    // B operands of S^T and dP^T: target r, dimensions g KQ ..
    float qb[KQ], dab[KQ];
    load_run<KQ>(qb, Q + t * d + j * DH + g * KQ, live);
    load_run<KQ>(dab, da + t * d + j * DH + g * KQ, live);
    float Dt = 0.f;
    if (live)
      for (int e = 0; e < DH; ++e) Dt += da[t * d + j * DH + e] * a[t * d + j * DH + e];
    const float lt = live ? lse[t * n_heads + j] * kLog2e : INFINITY;
    // A operands of dV^T and dK^T: target 4 s + g, dimension 16 dt + r
    float qa[DT][4], daa[DT][4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int tt = 4 * ks + g;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        qa[dt][ks] = tt < nb ? Q[(int64_t)(tb + tt) * d + j * DH + 16 * dt + r] : 0.f;
        daa[dt][ks] = tt < nb ? da[(int64_t)(tb + tt) * d + j * DH + 16 * dt + r] : 0.f;
      }
    }
    f32x4 dq[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) dq[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    Tile cur, nxt;
    if (w < nrt) fetch(w, nxt);
    for (int rt = w; rt < nrt; rt += kWaves) {
      cur = nxt;
      if (rt + kWaves < nrt) fetch(rt + kWaves, nxt);
      const int row0 = lo + rt * kRows;
      // S^T and dP^T = V dA^T: k-step s, lane group g <-> dimension g KQ + s
      // (four independent chains: even and odd k-steps of each product)
      f32x4 s = {0.f, 0.f, 0.f, 0.f}, dp = {0.f, 0.f, 0.f, 0.f};
      f32x4 s1 = {0.f, 0.f, 0.f, 0.f}, dp1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KQ; ks += 2) {
        s = mma(cur.k[ks], qb[ks], s);
        dp = mma(cur.v[ks], dab[ks], dp);
        s1 = mma(cur.k[ks + 1], qb[ks + 1], s1);
        dp1 = mma(cur.v[ks + 1], dab[ks + 1], dp1);
      }
      s += s1;
      dp += dp1;
      float p[4], de[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        p[v] = row0 + 4 * g + v < hi ? exp2f(s[v] - lt) : 0.f;
        de[v] = p[v] * (dp[v] - Dt);
      }
      // dQ^T += K^T dE^T: k-step s, lane group g <-> row 4 g + s
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) dq[dt] = mma(cur.kc[dt][ks], de[ks], dq[dt]);
      // P and dE to row-major tiles for the products over targets
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        pT[w][4 * g + v][r] = p[v];
        eT[w][4 * g + v][r] = de[v];
      }
      wave_sync();
      // dV^T += dA^T P, dK^T += Q^T dE: k-step s, lane group g <-> target 4 s + g
      f32x4 dv[DT], dk[DT];
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        dv[dt] = dk[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          dv[dt] = mma(daa[dt][ks], pT[w][r][4 * ks + g], dv[dt]);
          dk[dt] = mma(qa[dt][ks], eT[w][r][4 * ks + g], dk[dt]);
        }
      }
      wave_sync();
      // dk[dt][v], dv[dt][v]: dimension 16 dt + 4 g + v of row row0 + r
      const int tok = row0 + r;
      if (tok < hi) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const int c = j * DH + 16 * dt + 4 * g;
          float kx[4], vx[4];
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            kx[v] = dk[dt][v] * kLn2;
            vx[v] = dv[dt][v];
          }
          OT* pk = dKV + (int64_t)tok * ldkv + c;
          OT* pv = dKV + (int64_t)tok * ldkv + d + c;
          if (!first) add4(kx, pk), add4(vx, pv);
          store4(pk, kx);
          store4(pv, vx);
          if (dKVT) {
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              dKVT[(int64_t)(c + v) * ldt + tok] = from_f32<bf16_bits>(kx[v]);
              dKVT[(int64_t)(d + c + v) * ldt + tok] = from_f32<bf16_bits>(vx[v]);
            }
          }
        }
      }
    }
    // dq of this batch's targets: sum the four waves' partials
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int v = 0; v < 4; ++v) red[w][r][16 * dt + 4 * g + v] = dq[dt][v];
    __syncthreads();
    const float scale = 1.f / sqrtf((float)DH);
    for (int it = threadIdx.x; it < nb * DH; it += 64 * kWaves) {
      const int tt = it / DH, e = it % DH;
      const float vsum = red[0][tt][e] + red[1][tt][e] + red[2][tt][e] + red[3][tt][e];
      dq_part[((int64_t)un.c * n_tgt + tb + tt) * d + j * DH + e] = vsum * scale;
    }
    __syncthreads();
  }
}

}  // namespace

bool attn_mfma_supported(int d_head) { return d_head == 16 || d_head == 32 || d_head == 64; }

hipError_t attn_fwd_mfma(int d_head, int n_heads, const Unit* units, int64_t max_units, const WsHeader* hdr,
                         const float* Q, const float* KV, int d, float* part_acc, float* part_ml, int64_t n_tgt,
                         hipStream_t st) {
  if (max_units == 0) return hipSuccess;
  dim3 grid(static_cast<unsigned>(max_units), n_heads);
#define STCA_AF(DH)                                                                                            \
  hipLaunchKernelGGL(attn_fwd_mfma_kernel<DH>, grid, dim3(64 * kWaves), 0, st, units, hdr, Q, KV, d, part_acc, \
                     part_ml, n_tgt, n_heads)
  switch (d_head) {
    case 16: STCA_AF(16); break;
    case 32: STCA_AF(32); break;
    case 64: STCA_AF(64); break;
    default: return hipErrorInvalidValue;
  }
#undef STCA_AF
  return hipGetLastError();
}

hipError_t attn_bwd_mfma(int d_head, int n_heads, const Unit* units, int64_t max_units, const WsHeader* hdr,
                         const int32_t* toff, const float* Q, const float* KV, int d, const float* a, const float* da,
                         const float* lse, float* dq_part, void* dKV, int64_t ldkv, int dkv_bf16, bf16_bits* dKVT,
                         int64_t ldt, int64_t n_tgt, hipStream_t st) {
  if (max_units == 0) return hipSuccess;
  dim3 grid(static_cast<unsigned>(max_units), n_heads);
#define STCA_AB(DH)                                                                                                \
  if (dkv_bf16)                                                                                                    \
    hipLaunchKernelGGL((attn_bwd_mfma_kernel<DH, bf16_bits>), grid, dim3(64 * kWaves), 0, st, units, hdr, toff, Q, \
                       KV, d, a, da, lse, static_cast<bf16_bits*>(dKV), ldkv, dKVT, ldt, dq_part, n_tgt,          \
                       n_heads);                                                                                   \
  else                                                                                                             \
    hipLaunchKernelGGL((attn_bwd_mfma_kernel<DH, float>), grid, dim3(64 * kWaves), 0, st, units, hdr, toff, Q, KV, \
                       d, a, da, lse, static_cast<float*>(dKV), ldkv, nullptr, 0, dq_part, n_tgt, n_heads)
  switch (d_head) {
    case 16: STCA_AB(16); break;
    case 32: STCA_AB(32); break;
    case 64: STCA_AB(64); break;
    default: return hipErrorInvalidValue;
  }
#undef STCA_AB
  return hipGetLastError();
}

}  // namespace stca
