// Target-side recomputation of the backward pass, one launch per layer: the
// merge of the attention partials into a (and its log-sum-exp), then
//   u = s + a W_O,  h = ReLU(u W_1),  s' = u + h W_2,  q' = s' W_Q^{next}
// (the layer output of Sec. 3.1 under the residual FFN stacking) for 32
// targets per workgroup, keeping every intermediate the backward needs in
// fp32.  These products decide the ReLU gates, so they are evaluated to fp32
// accuracy on the bf16 matrix cores: each fp32 activation is split into three
// bf16 terms (8 + 8 + 8 significant bits, the whole fp32 mantissa, over
// fp32's exponent range) and multiplied with the bf16 weights term by term;
// every product of two bf16 values is exact in fp32 and the sums are fp32.
//
// Each wave forms a 32 x 32 output tile (its 32 output columns for the
// workgroup's 32 targets) as acc = W^T act^T: A operand = packed weight tile
// (lane = output column), B operand = activations staged in LDS (lane =
// target), result lane = target, element v = output column 8 (v/4) + 4 hi +
// v%4.
#include "common.h"
#include "fast.h"

namespace stca {

namespace {

constexpr int DH = 32;

__device__ __forceinline__ f32x16 mma(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t pack2(float x, float y) {
  return (uint32_t)from_f32<bf16_bits>(x) | ((uint32_t)from_f32<bf16_bits>(y) << 16);
}

template <int D, int NC>
__global__ __launch_bounds__(64 * (D / 32)) void update_precise_kernel(UpdatePrecise A) {
  constexpr int NW = D / 32;
  constexpr int H = D / DH;
  constexpr int KS = D / 16;
  constexpr int AROW = D + 8;  // padded LDS row (bf16 elements)
  // three bf16 terms of the 32 current activation rows, and of D hidden
  // columns at a time
  __shared__ __attribute__((aligned(16))) bf16_bits act[3][32 * AROW];
  __shared__ __attribute__((aligned(16))) bf16_bits hid[3][32 * AROW];
  const int w = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int tcol = lane % 32, hi = lane / 32;
  const int64_t tb = (int64_t)blockIdx.x * 32;
  const int64_t t = tb + tcol;
  const bool tok = t < A.n_tgt;
  const int F = A.F;

  // stage 4 consecutive fp32 values (row r, columns c..c+3) as three bf16 terms
  auto put4 = [&](bf16_bits (*buf)[32 * AROW], int r, int c, float x0, float x1, float x2, float x3) {
    const float x[4] = {x0, x1, x2, x3};
    uint32_t pk[3][2];
#pragma unroll
    for (int e = 0; e < 4; e += 2) {
      float a0 = x[e], a1 = x[e + 1];
#pragma unroll
      for (int term = 0; term < 3; ++term) {
        const bf16_bits b0 = from_f32<bf16_bits>(a0), b1 = from_f32<bf16_bits>(a1);
        pk[term][e / 2] = (uint32_t)b0 | ((uint32_t)b1 << 16);
        a0 -= to_f32(b0);
        a1 -= to_f32(b1);
      }
    }
#pragma unroll
    for (int term = 0; term < 3; ++term)
      *reinterpret_cast<uint2*>(buf[term] + r * AROW + c) = make_uint2(pk[term][0], pk[term][1]);
  };
  // a wave's result tile (lane = target tcol, elements = columns col0 + 8 q + 4 hi + e)
  auto put_tile = [&](bf16_bits (*buf)[32 * AROW], int col0, const f32x16& v) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      put4(buf, tcol, col0 + 8 * q + 4 * hi, v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
  };
  auto store_tile = [&](float* dst, int64_t ld, int col0, const f32x16& v) {
    if (!tok) return;
    float* p = dst + t * ld + col0 + 4 * hi;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *reinterpret_cast<float4*>(p + 8 * q) = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
  };
  auto store_tile16 = [&](bf16_bits* dst, int64_t ld, int col0, const f32x16& v) {
    if (!tok || !dst) return;
    bf16_bits* p = dst + t * ld + col0 + 4 * hi;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *reinterpret_cast<uint2*>(p + 8 * q) =
          make_uint2(pack2(v[4 * q], v[4 * q + 1]), pack2(v[4 * q + 2], v[4 * q + 3]));
  };
  auto load_tile = [&](const float* src, int64_t ld, int col0) {
    f32x16 v = {};
    if (tok) {
      const float* p = src + t * ld + col0 + 4 * hi;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 x = *reinterpret_cast<const float4*>(p + 8 * q);
        v[4 * q] = x.x, v[4 * q + 1] = x.y, v[4 * q + 2] = x.z, v[4 * q + 3] = x.w;
      }
    }
    return v;
  };
  // acc += W^T act^T over KS k-steps with the packed weight tile's fragments
  // in registers (fetched from Wp, [KS][64] vectors, in one L2 round trip).
  // With NC (hidden chunks, F / D) known at compile time, each product's
  // fragments are fetched one product ahead into the other of two register
  // sets, so the weight stream overlaps the previous product; the chunk loop
  // is then fully unrolled.  NC = 0 (any other F) fetches right before.
  auto fetch = [&](bf16x8 (&r)[KS], const bf16x8* __restrict__ Wp) {
#pragma unroll
    for (int k = 0; k < KS; ++k) r[k] = Wp[k * 64 + lane];
  };
  auto gemm_r = [&](const bf16x8 (&wt)[KS], const bf16_bits (*src)[32 * AROW], f32x16 acc) {
#pragma unroll
    for (int k = 0; k < KS; ++k)
#pragma unroll
      for (int term = 0; term < 3; ++term)
        acc = mma(wt[k], *reinterpret_cast<const bf16x8*>(src[term] + tcol * AROW + 8 * hi + 16 * k), acc);
    return acc;
  };
  auto gemm = [&](const bf16x8* __restrict__ Wp, const bf16_bits (*src)[32 * AROW], f32x16 acc) {
    bf16x8 wt[KS];
    fetch(wt, Wp);
    return gemm_r(wt, src, acc);
  };
  constexpr bool PF = NC > 0;
  const bf16x8* WoP = static_cast<const bf16x8*>(A.WoP);
  const bf16x8* W1P = static_cast<const bf16x8*>(A.W1P);
  const bf16x8* W2P = static_cast<const bf16x8*>(A.W2P);
  const bf16x8* WqP = static_cast<const bf16x8*>(A.WqP);
  const float qscale = kLog2e * rsqrtf(static_cast<float>(DH));

  f32x16 s_next, q;
  if (A.mode == 0) {
    // s^(0) = x_t
    for (int c = threadIdx.x; c < 32 * D / 4; c += 64 * NW) {
      const int row = c / (D / 4), col = (c % (D / 4)) * 4;
      float x[4] = {0.f, 0.f, 0.f, 0.f};
      if (tb + row < A.n_tgt) {
        const uint2 v = *reinterpret_cast<const uint2*>(A.tgt + (tb + row) * D + col);
        x[0] = to_f32((bf16_bits)(v.x & 0xffff)), x[1] = to_f32((bf16_bits)(v.x >> 16));
        x[2] = to_f32((bf16_bits)(v.y & 0xffff)), x[3] = to_f32((bf16_bits)(v.y >> 16));
        *reinterpret_cast<float4*>(A.s_out + (tb + row) * D + col) = make_float4(x[0], x[1], x[2], x[3]);
        if (A.s16_out) *reinterpret_cast<uint2*>(A.s16_out + (tb + row) * D + col) = v;
      }
      put4(act, row, col, x[0], x[1], x[2], x[3]);
    }
    __syncthreads();
    q = gemm(WqP + ((int64_t)w * KS) * 64, act, f32x16{});
  } else {
    const int ql = A.layer + 1;
    const bool next_q = ql < A.n_layers;
    auto w1_tile = [&](int c) { return W1P + ((int64_t)A.layer * (F / 32) + c * NW + w) * KS * 64; };
    auto w2_tile = [&](int c) { return W2P + ((int64_t)(A.layer * NW + w) * (F / 16) + c * KS) * 64; };
    const bf16x8* wo_tile = WoP + ((int64_t)(A.layer * NW + w) * KS) * 64;
    const bf16x8* wq_tile = WqP + ((int64_t)(ql * NW + w) * KS) * 64;
    bf16x8 wa[KS], wb[KS];
    if (PF) fetch(wa, wo_tile);  // lands during the merge
    // merge the chunk partials: two threads per (target, head), 16 dims each
    {
      const int pair = threadIdx.x >> 1, half = threadIdx.x & 1;
      for (int pp = pair; pp < 32 * H; pp += 32 * NW) {
        const int row = pp / H, j = pp % H;
        const int64_t tt = tb + row;
        float av[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) av[i] = 0.f;
        if (tt < A.n_tgt) {
          // every chunk's (max, sum) requested at once, the accumulators four
          // chunks at a time (sums in chunk order)
          const int nch = A.tchunks[tt];
          float2 ml[kMaxChunks];
#pragma unroll
          for (int c = 0; c < kMaxChunks; ++c)
            ml[c] = c < nch ? A.part_ml[((int64_t)c * A.n_tgt + tt) * H + j] : make_float2(-INFINITY, 0.f);
          float M = ml[0].x;
#pragma unroll
          for (int c = 1; c < kMaxChunks; ++c) M = fmaxf(M, ml[c].x);
          float L = 0.f, wc[kMaxChunks];
#pragma unroll
          for (int c = 0; c < kMaxChunks; ++c) {
            wc[c] = c < nch ? exp2f(ml[c].x - M) : 0.f;
            L += wc[c] * ml[c].y;
          }
#pragma unroll
          for (int c0 = 0; c0 < kMaxChunks; c0 += 4) {
            if (c0 >= nch) break;
            float4 x[4][4];
#pragma unroll
            for (int cc = 0; cc < 4; ++cc) {
              const float4* pa = reinterpret_cast<const float4*>(
                  A.part_acc + ((int64_t)(c0 + cc) * A.n_tgt + tt) * D + j * DH + half * 16);
#pragma unroll
              for (int q = 0; q < 4; ++q) x[cc][q] = c0 + cc < nch ? pa[q] : make_float4(0.f, 0.f, 0.f, 0.f);
            }
#pragma unroll
            for (int cc = 0; cc < 4; ++cc) {
              const float w = wc[c0 + cc];
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                av[4 * q] += w * x[cc][q].x, av[4 * q + 1] += w * x[cc][q].y;
                av[4 * q + 2] += w * x[cc][q].z, av[4 * q + 3] += w * x[cc][q].w;
              }
            }
          }
          const float inv = 1.f / L;
#pragma unroll
          for (int i = 0; i < 16; ++i) av[i] *= inv;
          float4* sa = reinterpret_cast<float4*>(A.a_out + tt * D + j * DH + half * 16);
#pragma unroll
          for (int q = 0; q < 4; ++q) sa[q] = make_float4(av[4 * q], av[4 * q + 1], av[4 * q + 2], av[4 * q + 3]);
          if (A.a16_out) {
            uint2* s16 = reinterpret_cast<uint2*>(A.a16_out + tt * D + j * DH + half * 16);
#pragma unroll
            for (int q = 0; q < 4; ++q)
              s16[q] = make_uint2(pack2(av[4 * q], av[4 * q + 1]), pack2(av[4 * q + 2], av[4 * q + 3]));
          }
          if (half == 0) A.lse_out[tt * H + j] = (M + log2f(L)) * kLn2;
        }
#pragma unroll
        for (int q = 0; q < 4; ++q)
          put4(act, row, j * DH + half * 16 + 4 * q, av[4 * q], av[4 * q + 1], av[4 * q + 2], av[4 * q + 3]);
      }
    }
    __syncthreads();
    if (PF) fetch(wb, w1_tile(0));
    // u = s + a W_O
    f32x16 u = PF ? gemm_r(wa, act, load_tile(A.s_in, D, 32 * w)) : gemm(wo_tile, act, load_tile(A.s_in, D, 32 * w));
    store_tile(A.u_out, D, 32 * w, u);
    store_tile16(A.u16_out, D, 32 * w, u);
    __builtin_amdgcn_sched_barrier(0);
    if (PF) fetch(wa, w2_tile(0));
    __syncthreads();  // every wave is done reading a
    put_tile(act, 32 * w, u);
    __syncthreads();
    // s' = u + ReLU(u W_1) W_2, D hidden columns at a time
    s_next = u;
#pragma unroll
    for (int c = 0; c < (PF ? NC : F / D); ++c) {
      f32x16 h = PF ? gemm_r(wb, act, f32x16{}) : gemm(w1_tile(c), act, f32x16{});
#pragma unroll
      for (int v = 0; v < 16; ++v) h[v] = fmaxf(h[v], 0.f);
      store_tile(A.h_out, F, c * D + 32 * w, h);
      store_tile16(A.h16_out, F, c * D + 32 * w, h);
      __builtin_amdgcn_sched_barrier(0);
      if (PF) {
        if (c + 1 < NC)
          fetch(wb, w1_tile(c + 1));
        else if (next_q)
          fetch(wb, wq_tile);
      }
      put_tile(hid, 32 * w, h);
      __syncthreads();
      s_next = PF ? gemm_r(wa, hid, s_next) : gemm(w2_tile(c), hid, s_next);
      __builtin_amdgcn_sched_barrier(0);
      if (PF && c + 1 < NC) fetch(wa, w2_tile(c + 1));
      __syncthreads();  // hid is rewritten by the next chunk
    }
    store_tile(A.s_out, D, 32 * w, s_next);
    store_tile16(A.s16_out, D, 32 * w, s_next);
    if (!next_q) return;
    put_tile(act, 32 * w, s_next);  // act (u) was last read before the previous barrier
    __syncthreads();
    q = PF ? gemm_r(wb, act, f32x16{}) : gemm(wq_tile, act, f32x16{});
  }
  // next queries q' = s' W_Q^{next}, scaled into log2 units
#pragma unroll
  for (int v = 0; v < 16; ++v) q[v] *= qscale;
  store_tile(A.q_out, D, 32 * w, q);
}

// Reverse of the update: dH = (ds W_2^T) where h > 0, du = ds + dH W_1^T,
// da = du W_O^T, and first, when the next layer's query gradient is given,
// ds = du' + dq W_Q^T (the gradient of this layer's output state through the
// next layer's residual path and its queries).  Same tiling as the
// recomputation, one bf16 term per activation (these products only carry
// gradients).
template <int D, int NC>
__global__ __launch_bounds__(64 * (D / 32)) void update_grad_kernel(UpdateGrad A) {
  constexpr int NW = D / 32;
  constexpr int KS = D / 16;
  constexpr int AROW = D + 8;
  __shared__ __attribute__((aligned(16))) bf16_bits act[32 * AROW];
  __shared__ __attribute__((aligned(16))) bf16_bits hid[32 * AROW];
  const int w = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int tcol = lane % 32, hi = lane / 32;
  const int64_t tb = (int64_t)blockIdx.x * 32;
  const int64_t t = tb + tcol;
  const bool tok = t < A.n_tgt;
  const int F = A.F;
  const int KSF = F / 16;

  // weight fragments in registers, fetched one product ahead into the other
  // of two register sets when NC (F / D) is known at compile time, as in
  // the recomputation
  auto fetch = [&](bf16x8 (&r)[KS], const bf16x8* __restrict__ Wp) {
#pragma unroll
    for (int k = 0; k < KS; ++k) r[k] = Wp[k * 64 + lane];
  };
  auto gemm_r = [&](const bf16x8 (&wt)[KS], const bf16_bits* src, f32x16 acc) {
#pragma unroll
    for (int k = 0; k < KS; ++k)
      acc = mma(wt[k], *reinterpret_cast<const bf16x8*>(src + tcol * AROW + 8 * hi + 16 * k), acc);
    return acc;
  };
  auto gemm = [&](const bf16x8* __restrict__ Wp, const bf16_bits* src, f32x16 acc) {
    bf16x8 wt[KS];
    fetch(wt, Wp);
    return gemm_r(wt, src, acc);
  };
  constexpr bool PF = NC > 0;
  // a wave's tile (lane = target, elements = columns col0 + 8 q + 4 hi + e)
  auto put_tile = [&](bf16_bits* buf, int col0, const f32x16& v) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *reinterpret_cast<uint2*>(buf + tcol * AROW + col0 + 8 * q + 4 * hi) =
          make_uint2(pack2(v[4 * q], v[4 * q + 1]), pack2(v[4 * q + 2], v[4 * q + 3]));
  };
  auto store16 = [&](bf16_bits* dst, int64_t ld, int col0, const f32x16& v) {
    if (!tok) return;
    bf16_bits* p = dst + t * ld + col0 + 4 * hi;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *reinterpret_cast<uint2*>(p + 8 * q) =
          make_uint2(pack2(v[4 * q], v[4 * q + 1]), pack2(v[4 * q + 2], v[4 * q + 3]));
  };
  auto store32 = [&](float* dst, int64_t ld, int col0, const f32x16& v) {
    if (!tok) return;
    float* p = dst + t * ld + col0 + 4 * hi;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *reinterpret_cast<float4*>(p + 8 * q) = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
  };
  auto load32 = [&](const float* src, int64_t ld, int col0) {
    f32x16 v = {};
    if (tok) {
      const float* p = src + t * ld + col0 + 4 * hi;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 x = *reinterpret_cast<const float4*>(p + 8 * q);
        v[4 * q] = x.x, v[4 * q + 1] = x.y, v[4 * q + 2] = x.z, v[4 * q + 3] = x.w;
      }
    }
    return v;
  };
  const bf16x8* W2TP = static_cast<const bf16x8*>(A.W2TP);
  const bf16x8* W1TP = static_cast<const bf16x8*>(A.W1TP);
  const bf16x8* WoTP = static_cast<const bf16x8*>(A.WoTP);
  auto w2t_tile = [&](int c) { return W2TP + ((int64_t)A.layer * (F / 32) + c * NW + w) * KS * 64; };
  auto w1t_tile = [&](int c) { return W1TP + ((int64_t)(A.layer * NW + w) * KSF + c * KS) * 64; };
  const bf16x8* wot_tile = WoTP + ((int64_t)(A.layer * NW + w) * KS) * 64;
  bf16x8 wa[KS], wb[KS];  // wb: W_2^T of chunk c (then W_O^T), wa: W_Q^T, then W_1^T of chunk c
  if (PF && !A.ds_out) fetch(wb, w2t_tile(0));

  f32x16 du;
  if (A.dq16) {
    // ds = du' + dq W_Q^T: dq (bf16) into LDS, this wave's 32 columns of ds
    for (int c = threadIdx.x; c < 32 * D / 8; c += 64 * NW) {
      const int row = c / (D / 8), col = (c % (D / 8)) * 8;
      uint4 x = make_uint4(0, 0, 0, 0);
      if (tb + row < A.n_tgt) x = *reinterpret_cast<const uint4*>(A.dq16 + (tb + row) * D + col);
      *reinterpret_cast<uint4*>(act + row * AROW + col) = x;
    }
    __syncthreads();
    const bf16x8* WqTP = static_cast<const bf16x8*>(A.WqTP);
    const bf16x8* wqt_tile = WqTP + ((int64_t)(A.q_layer * NW + w) * KS) * 64;
    if (PF) {
      fetch(wa, wqt_tile);
      du = gemm_r(wa, act, f32x16{});
    } else {
      du = gemm(wqt_tile, act, f32x16{});
    }
    const f32x16 dprev = load32(A.du_in, D, 32 * w);
#pragma unroll
    for (int v = 0; v < 16; ++v) du[v] += dprev[v];
    if (A.ds_out) {
      store32(A.ds_out, D, 32 * w, du);
      return;
    }
    __syncthreads();  // every wave is done with dq
    put_tile(act, 32 * w, du);
    store16(A.ds16_out, D, 32 * w, du);
  } else {
    // ds (bf16) into LDS, and its bf16 copy
    for (int c = threadIdx.x; c < 32 * D / 4; c += 64 * NW) {
      const int row = c / (D / 4), col = (c % (D / 4)) * 4;
      float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
      if (tb + row < A.n_tgt) x = *reinterpret_cast<const float4*>(A.ds + (tb + row) * D + col);
      const uint2 v = make_uint2(pack2(x.x, x.y), pack2(x.z, x.w));
      *reinterpret_cast<uint2*>(act + row * AROW + col) = v;
      if (tb + row < A.n_tgt) *reinterpret_cast<uint2*>(A.ds16_out + (tb + row) * D + col) = v;
    }
    du = load32(A.ds, D, 32 * w);
  }
  __builtin_amdgcn_sched_barrier(0);
  if (PF) fetch(wa, w1t_tile(0));
  __syncthreads();
#pragma unroll
  for (int c = 0; c < (PF ? NC : F / D); ++c) {
    const int col = c * D + 32 * w;
    f32x16 dh = PF ? gemm_r(wb, act, f32x16{}) : gemm(w2t_tile(c), act, f32x16{});
    const f32x16 h = load32(A.h, F, col);
#pragma unroll
    for (int v = 0; v < 16; ++v) dh[v] = h[v] > 0.f ? dh[v] : 0.f;
    store16(A.dh16_out, F, col, dh);
    __builtin_amdgcn_sched_barrier(0);
    if (PF) fetch(wb, c + 1 < NC ? w2t_tile(c + 1) : wot_tile);
    put_tile(hid, 32 * w, dh);
    __syncthreads();
    du = PF ? gemm_r(wa, hid, du) : gemm(w1t_tile(c), hid, du);
    __builtin_amdgcn_sched_barrier(0);
    if (PF && c + 1 < NC) fetch(wa, w1t_tile(c + 1));
    __syncthreads();  // hid is rewritten by the next chunk
  }
  store32(A.du_out, D, 32 * w, du);
  store16(A.du16_out, D, 32 * w, du);
  put_tile(act, 32 * w, du);  // act (ds) was last read before the previous barrier
  __syncthreads();
  const f32x16 da = PF ? gemm_r(wb, act, f32x16{}) : gemm(wot_tile, act, f32x16{});
  store32(A.da_out, D, 32 * w, da);
}

}  // namespace

hipError_t fast_update_precise(int D, const UpdatePrecise& f, hipStream_t st) {
  if (f.n_tgt == 0) return hipSuccess;
  if (f.F % D != 0) return hipErrorInvalidValue;
  dim3 g(static_cast<unsigned>(ceil_div(f.n_tgt, 32)));
#define STCA_UPDP(DD)                                                                              \
  if (f.F == 4 * (DD))                                                                             \
    hipLaunchKernelGGL((update_precise_kernel<DD, 4>), g, dim3(64 * (DD / 32)), 0, st, f);         \
  else                                                                                             \
    hipLaunchKernelGGL((update_precise_kernel<DD, 0>), g, dim3(64 * (DD / 32)), 0, st, f)
  switch (D) {
    case 64: STCA_UPDP(64); break;
    case 128: STCA_UPDP(128); break;
    case 256: STCA_UPDP(256); break;
    default: return hipErrorInvalidValue;
  }
#undef STCA_UPDP
  return hipGetLastError();
}

hipError_t fast_update_grad(int D, const UpdateGrad& f, hipStream_t st) {
  if (f.n_tgt == 0) return hipSuccess;
  if (f.F % D != 0) return hipErrorInvalidValue;
  dim3 g(static_cast<unsigned>(ceil_div(f.n_tgt, 32)));
#define STCA_UPDG(DD)                                                                              \
  if (f.F == 4 * (DD))                                                                             \
    hipLaunchKernelGGL((update_grad_kernel<DD, 4>), g, dim3(64 * (DD / 32)), 0, st, f);            \
  else                                                                                             \
    hipLaunchKernelGGL((update_grad_kernel<DD, 0>), g, dim3(64 * (DD / 32)), 0, st, f)
  switch (D) {
    case 64: STCA_UPDG(64); break;
    case 128: STCA_UPDG(128); break;
    case 256: STCA_UPDG(256); break;
    default: return hipErrorInvalidValue;
  }
#undef STCA_UPDG
  return hipGetLastError();
}

}  // namespace stca
