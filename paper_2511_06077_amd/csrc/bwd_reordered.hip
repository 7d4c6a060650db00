// Attention backward in the reordered form (bf16 storage, d_h = 32, at most
// 128 / n_heads targets per request).
//
// The forward's reordering (Sec. 3.1, Eq. attn-optimized: the score of
// target t and head j is x_l . u_tj with u_tj = q_tj W_K^j^T, and the head
// output is (sum_l p_tl x_l) W_V^j) carries over to the gradients, so that
// neither K, V nor their gradients are formed.  With q scaled by
// log2(e)/sqrt(d_h) (scores in log2 units), per request, layer and head j
// and the softmax gradient de_tl = p_tl (dp_tl - D_t):
//   dp_tl = da_tj . v_l = x_l . h_tj,           h_tj = da_tj W_V^j^T
//   dX_l  = sum_j sum_t ln(2) de_tl u_tj + p_tl h_tj       (over every layer)
//   dW_K^j = ln(2) sum_t z_tj^T q_tj,  dW_V^j = sum_t y_tj^T da_tj
//   dq_tj = z_tj W_K^j / sqrt(d_h)
// with z_tj = sum_l de_tl x_l and y_tj = sum_l p_tl x_l.  The (target, head)
// pairs of a request are the rows of U and H (HM = 128 of them, index
// j' = head * M + t, M = 128 / n_heads, padded with zero rows).
//
//   rb_prep_kernel:  per request, U (fp16 for the scores; bf16 with H into
//                    the request's dX operand W_r), the softmax statistics
//                    (log2-unit lse, D) and bf16 copies of q and da.
//   rb_attn_kernel:  per unit (a history chunk of a request), history
//                    blocks of 32 rows streamed into an LDS ring by direct
//                    loads; eight waves, two per tile of 32 pairs: one forms
//                    S = X U^T (fp16) and P, and Y += P^T X; the other
//                    dP = X H^T (bf16) and, one block later, dE, the
//                    [ln(2) dE | P] words of this layer's columns of E and
//                    Z += dE^T X.  Z and Y (bf16, [head][target][D]) are
//                    written at the end of the request.
// The products that follow (dq, dW_K, dW_V from Z and Y; dX = E W_r after
// the last layer) are GEMMs.
#include <type_traits>

#include "common.h"
#include "fast.h"
#include "ring.h"

namespace stca {

namespace {

constexpr int DH = 32;
constexpr int HM = kRbPairs;  // (target, head) pairs per request, padded
constexpr int kRbStages = 5;  // X blocks in the LDS ring

__device__ __forceinline__ f32x16 mma(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mma(const f16x8& a, const f16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 pack_b(const f32x16& a, int off) {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = static_cast<__bf16>(a[off + i]);
  return r;
}

// bf16 bits -> fp16 (exact in fp16's normal range)
__device__ __forceinline__ f16x8 bf_to_f16(const bf16x8& x) {
  f16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = static_cast<_Float16>(static_cast<float>(x[i]));
  return r;
}

// v ~ hi + lo, both bf16
__device__ __forceinline__ void split_bf(float v, __bf16& hi, __bf16& lo) {
  hi = static_cast<__bf16>(v);
  lo = static_cast<__bf16>(v - static_cast<float>(hi));
}

// LDS position of 16-byte unit u of X-tile row r (D / 8 units per row): the
// permutation u ^ (4 (r % 4) + (r / 4) % 4) spreads both the 16 rows of a
// row read (same unit) and the 4 rows x 4 units of a transposing read over
// the banks.
__device__ __forceinline__ int xpos(int r, int u) { return u ^ (4 * (r % 4) + (r / 4) % 4); }

// The lane index, opaque to the compiler: addresses derived from it are
// formed where they are used instead of being kept live across a loop.
__device__ __forceinline__ int opaque_lane(int v) {
  asm volatile("" : "+v"(v));
  return v;
}

// the source of every direct load past the last history row
__device__ const uint4 kRbZero16[1] = {};

}  // namespace

namespace {

// ---- per request: U, H, statistics, bf16 q and da
template <int D>
__global__ __launch_bounds__(64 * (D / 32)) void rb_prep_kernel(RbPrep A) {
  constexpr int H = D / DH;
  constexpr int M = HM / H;   // target slots per head
  constexpr int MT = (M + 31) / 32;
  const int r = blockIdx.x;
  if (r >= A.n_requests) return;
  const int h = threadIdx.x / 64, lane = threadIdx.x % 64, l32 = lane % 32, hi = lane / 32;
  const int64_t t0 = A.tgt_off[r];
  const int m = static_cast<int>(A.tgt_off[r + 1] - t0);
  if (m == 0) return;
  const int cols = h * DH;
  _Float16* U16 = A.U16 + (int64_t)r * HM * D;
  bf16_bits* Wu = A.Wr + (((int64_t)r * A.n_layers + A.layer) * 2) * HM * D;
  bf16_bits* Wh = Wu + (int64_t)HM * D;
  for (int rt = 0; rt < MT; ++rt) {
    // A operands: row i = target slot 32 rt + l32, k = head dims 16 s + 8 hi + e
    // (fp32 q and da split into two bf16 terms); the same registers give the
    // pair statistic D = da . a and the bf16 copies of q and da
    const int t = 32 * rt + l32;
    const bool tok = t < m && t < M;
    bf16x8 qh[2], ql[2], dh[2], dl[2];
    float dsum = 0.f;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int64_t o = (t0 + (tok ? t : 0)) * D + cols + 16 * s + 8 * hi;
      float q[8], g[8], av[8];
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const float4 q4 = tok ? *reinterpret_cast<const float4*>(A.Q + o + 4 * half) : make_float4(0.f, 0.f, 0.f, 0.f);
        const float4 g4 = tok ? *reinterpret_cast<const float4*>(A.da + o + 4 * half) : make_float4(0.f, 0.f, 0.f, 0.f);
        const float4 a4 = tok ? *reinterpret_cast<const float4*>(A.a + o + 4 * half) : make_float4(0.f, 0.f, 0.f, 0.f);
        q[4 * half] = q4.x, q[4 * half + 1] = q4.y, q[4 * half + 2] = q4.z, q[4 * half + 3] = q4.w;
        g[4 * half] = g4.x, g[4 * half + 1] = g4.y, g[4 * half + 2] = g4.z, g[4 * half + 3] = g4.w;
        av[4 * half] = a4.x, av[4 * half + 1] = a4.y, av[4 * half + 2] = a4.z, av[4 * half + 3] = a4.w;
      }
      uint4 q16, g16;
      uint32_t* qw = reinterpret_cast<uint32_t*>(&q16);
      uint32_t* gw = reinterpret_cast<uint32_t*>(&g16);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        __bf16 a, b;
        split_bf(q[e], a, b);
        qh[s][e] = a, ql[s][e] = b;
        split_bf(g[e], a, b);
        dh[s][e] = a, dl[s][e] = b;
        dsum += g[e] * av[e];
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        qw[e] = (uint32_t)from_f32<bf16_bits>(q[2 * e]) | ((uint32_t)from_f32<bf16_bits>(q[2 * e + 1]) << 16);
        gw[e] = (uint32_t)from_f32<bf16_bits>(g[2 * e]) | ((uint32_t)from_f32<bf16_bits>(g[2 * e + 1]) << 16);
      }
      if (tok) {
        *reinterpret_cast<uint4*>(A.q16 + o) = q16;
        *reinterpret_cast<uint4*>(A.da16 + o) = g16;
      }
    }
    dsum += __shfl_xor(dsum, 32);  // the two lane halves hold 16 dims each
    if (t < M && hi == 0) {
      float* st = A.stats + ((int64_t)r * HM + h * M + t) * 2;
      st[0] = tok ? A.lse[(t0 + t) * H + h] * kLog2e : INFINITY;
      st[1] = tok ? dsum : 0.f;
    }
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) {
      const int dim = 32 * dt + l32;
      f32x16 u = {}, hv = {};
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const bf16x8 wk = *reinterpret_cast<const bf16x8*>(A.Wk + (int64_t)dim * D + cols + 16 * s + 8 * hi);
        const bf16x8 wv = *reinterpret_cast<const bf16x8*>(A.Wv + (int64_t)dim * D + cols + 16 * s + 8 * hi);
        u = mma(qh[s], wk, u);
        u = mma(ql[s], wk, u);
        hv = mma(dh[s], wv, hv);
        hv = mma(dl[s], wv, hv);
      }
      // lane = dim, element v = target slot 32 rt + 8 (v / 4) + 4 hi + v % 4
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int tt = 32 * rt + 8 * (v / 4) + 4 * hi + v % 4;
        if (tt < M) {
          const int64_t o = (int64_t)(h * M + tt) * D + dim;
          U16[o] = static_cast<_Float16>(u[v]);
          Wu[o] = from_f32<bf16_bits>(u[v]);
          Wh[o] = from_f32<bf16_bits>(hv[v]);
        }
      }
    }
  }
}

// ---- per request: S, dP, P, dE, E, Z, Y
template <int N>
__device__ __forceinline__ void wait_loads() {  // at most N vector memory operations outstanding
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
}
// at most `later` (0 .. L) blocks of PER loads each still in flight
template <int PER, int L>
__device__ __forceinline__ void wait_later(int later) {
  if constexpr (L > 0) {
    if (later >= L) return wait_loads<L * PER>();
    return wait_later<PER, L - 1>(later);
  } else {
    wait_loads<0>();
  }
}

// Eight waves, two per pair tile t (32 pairs each), in two roles that share
// the tile's SIMD: role 0 scores the block (S = X U^T on an fp16 copy of X),
// forms P, writes E's P columns and accumulates Y += P^T X; role 1 forms
// dP = X H^T and, one block later, when role 0's P of that block has come
// through LDS, dE = P (dP - D), E's dE columns and Z += dE^T X.  Each wave
// so holds one set of score operands (U or H rows) and one set of
// accumulators (Y or Z), which fit two waves per SIMD.  The ring keeps five
// blocks: the two in use (k for both roles, k - 1 for role 1's Z) and three
// in flight.
template <int D>
__global__ __launch_bounds__(512) void rb_attn_kernel(RbAttn A) {
  constexpr int KS = D / 16;       // k-steps of the score products
  constexpr int DT = D / 32;       // 32-column tiles of Z and Y
  constexpr int TB = 32 * D * 2;   // bytes of one X block in LDS
  constexpr int CH = TB / 1024;    // 1 KB direct-load runs per block
  static_assert(CH % 8 == 0, "whole runs per wave");
  constexpr int PER = CH / 8;      // direct loads per wave per block
  constexpr int STG = kRbStages;
  constexpr int AHEAD = STG - 2;   // blocks in flight beyond the two in use
  static_assert(AHEAD >= 1, "ring too short");
  __shared__ __attribute__((aligned(1024))) unsigned char ring[STG * TB];
  __shared__ __attribute__((aligned(1024))) unsigned char t16[2 * TB];  // fp16 copies of blocks k, k + 1
  __shared__ __attribute__((aligned(16))) float4 pex[2][4][4][64];      // P of block k per pair tile (role 0 -> 1)
  __shared__ __attribute__((aligned(16))) float4 dpx[4][4][64];         // role 1: dP of the previous block

  const Unit* __restrict__ units = static_cast<const Unit*>(A.units);
  const WsHeader* __restrict__ hdr = static_cast<const WsHeader*>(A.hdr);
  if (static_cast<int>(blockIdx.x) >= hdr->n_units) return;
  const Unit un = units[blockIdx.x];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
  const int tile_id = wave % 4, role = wave / 4;  // the pairs 32 tile_id ..
  const int lane = threadIdx.x % 64, l32 = lane % 32, hi = lane / 32;
  const int r = un.r;
  const int64_t t0 = un.t0;
  const int m = un.nt;
  const int jp = 32 * tile_id + l32;  // this lane's pair (result column)
  const bf16_bits* __restrict__ X = static_cast<const bf16_bits*>(A.X);
  constexpr int M = HM / (D / DH);

  float lse2 = A.stats[((int64_t)r * HM + jp) * 2];
  float dsum = A.stats[((int64_t)r * HM + jp) * 2 + 1];
  f32x16 acc[DT];  // role 0: Y, role 1: Z
#pragma unroll
  for (int i = 0; i < DT; ++i) acc[i] = f32x16{};

  // ring of X blocks b0 .. b1 - 1 (rows past the batch come from a zero vector)
  const int b0 = un.b0, nb = un.b1 - un.b0;
  auto issue = [&](int k) {
    const unsigned char* s = ring + (k % STG) * TB;
    const int64_t row0 = (int64_t)(b0 + k) * 32;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int q = wave + 8 * i;
      const int o = 1024 * q + 16 * lane;
      const int row = o / (2 * D), p = (o % (2 * D)) / 16;
      const int u = xpos(row, p);  // the permutation is an involution
      const int64_t g = row0 + row;
      dma16(g < A.n_hist ? static_cast<const void*>(X + g * D + 8 * u) : static_cast<const void*>(kRbZero16),
            s + 1024 * q);
    }
  };
  // fp16 copy of block k for the score products, same byte layout, made by
  // all 512 threads (two 16-byte units each at D = 256)
  auto convert = [&](int k) {
    const unsigned char* src = ring + (k % STG) * TB;
    unsigned char* dst = t16 + (k % 2) * TB;
#pragma unroll
    for (int i = 0; i < TB / (16 * 512); ++i) {
      const int off = 16 * (static_cast<int>(threadIdx.x) + 512 * i);
      *reinterpret_cast<f16x8*>(dst + off) = bf_to_f16(*reinterpret_cast<const bf16x8*>(src + off));
    }
  };
  const int64_t lde = A.lde;
  bf16_bits* __restrict__ ecol = A.E + (int64_t)A.layer * 2 * HM + jp + (role == 0 ? HM : 0);
  // acc[dt] += op^T X(block in `tile`): op = the 32 x 32 tile of P or dE in
  // result order (element p of k-step s is row 16 s + 4 hi + (p < 4 ? p : p + 4)),
  // X's columns by transposing reads of the same rows
  // With the permutation xpos, the byte address of row ra = 16 s + 4 hi +
  // j16 / 4 (rb = ra + 8), column col = 32 dt + 16 g16 + 4 (j16 % 4) is
  // (tb ^ 64 (dt % 4) [^ 32 for rb]) + 256 (dt / 4) + 16 s 2D [+ 8 2D for rb]
  // with one per-lane base tb; it is formed from an opaque lane index per
  // call, so no per-(s, dt) address is held across the loop.
  auto accumulate = [&](const unsigned char* tile, const bf16x8 (&op)[2]) {
    const int ln = opaque_lane(lane), jj = ln % 16, gg = (ln / 16) % 2, hh = ln / 32;
    const int a4 = jj / 4, c4 = 2 * gg + (jj % 4) / 2;
    const int tb = (4 * hh + a4) * (2 * D) + 16 * (c4 ^ hh) + 8 * ((jj % 4) & 1) + 64 * a4;
    // X^T operand of product i = s DT + dt
    auto operand = [&](int i) {
      const int s = i / DT, dt = i % DT;
      const int o = (tb ^ (64 * (dt % 4))) + 256 * (dt / 4) + 16 * s * (2 * D);
      const tr16x4 lo = lds_read_tr16(tile + o);
      const tr16x4 up = lds_read_tr16(tile + (o ^ 32) + 8 * (2 * D));
      return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, up, 0, 1, 2, 3, 4, 5, 6, 7));
    };
    // operands read two products ahead (scheduling barriers keep the
    // compiler from sinking the reads next to their use)
    constexpr int NA = 2;
    bf16x8 xb[NA];
#pragma unroll
    for (int i = 0; i < NA; ++i) xb[i] = operand(i);
#pragma unroll
    for (int i = 0; i < 2 * DT; ++i) {
      const bf16x8 x = xb[i % NA];
      if (i + NA < 2 * DT) xb[i % NA] = operand(i + NA);
      acc[i % DT] = mma(op[i / DT], x, acc[i % DT]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // byte address of row l32, 16-byte unit 2 ks + hi of a tile: sb ^ 32 ks
  auto score_base = [&]() {
    const int ln = opaque_lane(lane), r = ln % 32, h = ln / 32;
    return r * (2 * D) + ((16 * h) ^ (16 * (4 * (r % 4) + (r / 4) % 4)));
  };
  // E entries of block k (values in result order): this role's columns of
  // the rows inside the unit
  auto store_e = [&](int k, const f32x16& val, float scale) {
    const int64_t brow = (int64_t)(b0 + k) * 32;
    if (brow >= un.l0 && brow + 32 <= un.l1) {
      bf16_bits* __restrict__ eb = ecol + (brow + 4 * hi) * lde;
#pragma unroll
      for (int v = 0; v < 16; ++v) eb[(8 * (v / 4) + v % 4) * lde] = from_f32<bf16_bits>(scale * val[v]);
    } else {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t g = brow + 8 * (v / 4) + 4 * hi + v % 4;
        if (g >= un.l0 && g < un.l1) ecol[g * lde] = from_f32<bf16_bits>(scale * val[v]);
      }
    }
  };

  // One wave's walk over the blocks; both roles pass the same barriers.
  auto run = [&](auto role_tag) {
    constexpr int ROLE = decltype(role_tag)::value;
    // B operands of this role's score product: U (fp16) or H (bf16) rows
    typedef typename std::conditional<ROLE == 0, f16x8, bf16x8>::type OpT;
    OpT bop[KS];
    {
      const OpT* src = ROLE == 0
                           ? reinterpret_cast<const OpT*>(A.U16 + ((int64_t)r * HM + jp) * D)
                           : reinterpret_cast<const OpT*>(
                                 A.Wr + ((((int64_t)r * A.n_layers + A.layer) * 2 + 1) * HM + jp) * D);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) bop[ks] = src[2 * ks + hi];
    }
    // These loads land before the ring's first load is issued: the compiler
    // does not see the ring's loads, and would otherwise wait for these inside
    // the loop with counts that, in issue order, also drain the ring's
    // prefetches and the E stores at every block.
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) asm volatile("" : "+v"(bop[ks]));
    asm volatile("" : "+v"(lse2), "+v"(dsum));
    // this role's score product of a block: sc = X(block) op^T
    auto score = [&](const unsigned char* tile, f32x16& sc) {
      const int sb = score_base();
      constexpr int NA = 2;  // operands read two k-steps ahead
      OpT xa[NA];
#pragma unroll
      for (int i = 0; i < NA; ++i) xa[i] = *reinterpret_cast<const OpT*>(tile + (sb ^ (32 * i)));
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const OpT x = xa[ks % NA];
        if (ks + NA < KS) xa[ks % NA] = *reinterpret_cast<const OpT*>(tile + (sb ^ (32 * (ks + NA))));
        sc = mma(x, bop[ks], sc);
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    // role 1: dE, E's dE columns and Z for block k (its dP in this wave's
    // dpx, kept in LDS rather than registers until its P arrives in pex[k % 2])
    auto finish_de = [&](int k) {
      f32x16 de;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float4 p4 = pex[k % 2][tile_id][i][lane];
        const float4 d4 = dpx[tile_id][i][lane];
        de[4 * i] = p4.x * (d4.x - dsum);
        de[4 * i + 1] = p4.y * (d4.y - dsum);
        de[4 * i + 2] = p4.z * (d4.z - dsum);
        de[4 * i + 3] = p4.w * (d4.w - dsum);
      }
      store_e(k, de, kLn2);
      const bf16x8 ea[2] = {pack_b(de, 0), pack_b(de, 8)};
      accumulate(ring + (k % STG) * TB, ea);
    };
    int issued = 0;
    for (; issued < AHEAD && issued < nb; ++issued) issue(issued);
    wait_later<PER, AHEAD>(issued - 1);  // block 0 landed
    ring_barrier();
    convert(0);
    for (int k = 0; k < nb; ++k) {
      // block k + 1 landed (later ones may still be in flight); the barrier
      // publishes it, block k's fp16 copy and the P of block k - 1, and every
      // wave is done with block k - 2, whose slot the next load takes
      wait_later<PER, AHEAD>(issued - k - 2);
      ring_barrier();
      if (issued < nb) {
        issue(issued);
        ++issued;
      }
      if (k + 1 < nb) convert(k + 1);
      const unsigned char* tile = ring + (k % STG) * TB;
      // result lane = pair, element v = row 8 (v / 4) + 4 hi + v % 4
      f32x16 sc = {};
      if (ROLE == 0) {
        const unsigned char* tile16 = t16 + (k % 2) * TB;
        score(tile16, sc);
        const int64_t brow = (int64_t)(b0 + k) * 32;
        if (brow >= un.l0 && brow + 32 <= un.l1) {
#pragma unroll
          for (int v = 0; v < 16; ++v) sc[v] = __builtin_amdgcn_exp2f(sc[v] - lse2);
        } else {
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int64_t g = brow + 8 * (v / 4) + 4 * hi + v % 4;
            sc[v] = g >= un.l0 && g < un.l1 ? __builtin_amdgcn_exp2f(sc[v] - lse2) : 0.f;
          }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
          pex[k % 2][tile_id][i][lane] = make_float4(sc[4 * i], sc[4 * i + 1], sc[4 * i + 2], sc[4 * i + 3]);
        store_e(k, sc, 1.f);
        const bf16x8 pa[2] = {pack_b(sc, 0), pack_b(sc, 8)};
        accumulate(tile, pa);
      } else {
        // the previous block first, so that its dP is free before this one's forms
        if (k > 0) finish_de(k - 1);
        score(tile, sc);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          dpx[tile_id][i][lane] = make_float4(sc[4 * i], sc[4 * i + 1], sc[4 * i + 2], sc[4 * i + 3]);
      }
    }
    // the last block's P (every wave passes the barrier: no loads remain)
    wait_loads<0>();
    ring_barrier();
    if (ROLE == 1 && nb > 0) finish_de(nb - 1);
  };
  if (role == 0)
    run(std::integral_constant<int, 0>{});
  else
    run(std::integral_constant<int, 1>{});
  // Z (role 1) or Y (role 0) rows of the tile's pairs: lane = column dim,
  // element v = pair 32 tile_id + 8 (v / 4) + 4 hi + v % 4 = head * M +
  // target slot; a request of several chunks leaves fp32 partials for rb_reduce
  if (A.tchunks[t0] == 1) {
    bf16_bits* __restrict__ out = role == 0 ? A.Y : A.Z;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int pr = 32 * tile_id + 8 * (v / 4) + 4 * hi + v % 4;
        const int hh = pr / M, tt = pr % M;
        if (tt < m) out[((int64_t)hh * A.n_tgt + t0 + tt) * D + 32 * dt + l32] = from_f32<bf16_bits>(acc[dt][v]);
      }
    }
  } else {
    if (un.c == 0 && threadIdx.x == 0) A.first[r] = blockIdx.x;
    float* __restrict__ outp = role == 0 ? A.Yp : A.Zp;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int pr = 32 * tile_id + 8 * (v / 4) + 4 * hi + v % 4;
        outp[((int64_t)blockIdx.x * HM + pr) * D + 32 * dt + l32] = acc[dt][v];
      }
    }
  }
}

// Z, Y (bf16 [head][target][D]) of a request of several chunks: the sum of
// the partials of its units first[r] .. first[r] + chunks - 1
template <int D>
__global__ __launch_bounds__(256) void rb_reduce_kernel(const int32_t* __restrict__ toff, int n_requests,
                                                        const int32_t* __restrict__ tchunks,
                                                        const int32_t* __restrict__ first, const float* __restrict__ Zp,
                                                        const float* __restrict__ Yp, bf16_bits* __restrict__ Z,
                                                        bf16_bits* __restrict__ Y, int64_t n_tgt) {
  constexpr int H = D / DH, M = HM / H;
  const int r = blockIdx.x;
  if (r >= n_requests) return;
  const int64_t t0 = toff[r];
  const int m = static_cast<int>(toff[r + 1] - t0);
  if (m == 0) return;
  const int nch = tchunks[t0];
  if (nch <= 1) return;
  const int u0 = first[r];
  const int64_t cnt = (int64_t)H * m * D;
  for (int64_t e = threadIdx.x; e < cnt; e += blockDim.x) {
    const int hh = static_cast<int>(e / ((int64_t)m * D));
    const int tt = static_cast<int>((e / D) % m);
    const int dd = static_cast<int>(e % D);
    float z = 0.f, y = 0.f;
    for (int c = 0; c < nch; ++c) {
      const int64_t o = ((int64_t)(u0 + c) * HM + hh * M + tt) * D + dd;
      z += Zp[o];
      y += Yp[o];
    }
    const int64_t q = ((int64_t)hh * n_tgt + t0 + tt) * D + dd;
    Z[q] = from_f32<bf16_bits>(z);
    Y[q] = from_f32<bf16_bits>(y);
  }
}

__global__ void rb_zero_rows_kernel(const int32_t* __restrict__ hoff, const int32_t* __restrict__ toff,
                                    int n_requests, float* __restrict__ dst, int cols) {
  const int r = blockIdx.x;
  if (r >= n_requests || toff[r + 1] != toff[r]) return;
  const int64_t cnt = (int64_t)(hoff[r + 1] - hoff[r]) * cols;
  float* p = dst + (int64_t)hoff[r] * cols;
  for (int64_t e = threadIdx.x; e < cnt; e += blockDim.x) p[e] = 0.f;
}

}  // namespace

hipError_t rb_prep(int D, const RbPrep& a, hipStream_t st) {
  if (a.n_requests == 0) return hipSuccess;
#define STCA_RBP(DD) hipLaunchKernelGGL(rb_prep_kernel<DD>, dim3(a.n_requests), dim3(64 * (DD / 32)), 0, st, a)
  if (D == 256) STCA_RBP(256);
  else if (D == 128) STCA_RBP(128);
  else return hipErrorInvalidValue;
#undef STCA_RBP
  return hipGetLastError();
}

hipError_t rb_attn(int D, const RbAttn& a, int grid, hipStream_t st) {
  if (grid == 0) return hipSuccess;
#define STCA_RBA(DD) hipLaunchKernelGGL(rb_attn_kernel<DD>, dim3(grid), dim3(512), 0, st, a)
  if (D == 256) STCA_RBA(256);
  else if (D == 128) STCA_RBA(128);
  else return hipErrorInvalidValue;
#undef STCA_RBA
  return hipGetLastError();
}

hipError_t rb_reduce(int D, const int32_t* tgt_off, int n_requests, const int32_t* tchunks, const int32_t* first,
                     const float* Zp, const float* Yp, bf16_bits* Z, bf16_bits* Y, int64_t n_tgt, hipStream_t st) {
  if (n_requests == 0) return hipSuccess;
#define STCA_RBR(DD)                                                                                              \
  hipLaunchKernelGGL(rb_reduce_kernel<DD>, dim3(n_requests), dim3(256), 0, st, tgt_off, n_requests, tchunks, first, \
                     Zp, Yp, Z, Y, n_tgt)
  if (D == 256) STCA_RBR(256);
  else if (D == 128) STCA_RBR(128);
  else return hipErrorInvalidValue;
#undef STCA_RBR
  return hipGetLastError();
}

hipError_t rb_zero_untargeted(const int32_t* hoff, const int32_t* toff, int n_requests, float* dst, int cols,
                              hipStream_t st) {
  if (n_requests == 0) return hipSuccess;
  hipLaunchKernelGGL(rb_zero_rows_kernel, dim3(n_requests), dim3(256), 0, st, hoff, toff, n_requests, dst, cols);
  return hipGetLastError();
}

}  // namespace stca
