// Attention backward with the history projection fused in (bf16 storage,
// d_h = 32, requests of at most 32 targets): each 32-row history block's K
// and V are formed inside the kernel from X and the layer's W_K, W_V (held in
// registers, one wave per head), as the forward's fused kernel does, so no
// K/V copy exists in HBM.  Per block and head the kernel rebuilds the softmax
// weights from the forward's log-sum-exp and writes the block's dK and dV
// (every target of the request summed; one unit per history chunk, so each
// row is written once) and accumulates the unit's dq.
//
// Per request, layer and head j (targets t, history rows l; queries stored
// pre-scaled by log2(e)/sqrt(d_h), so scores are in log2 units):
//   s_tl = q_t . k_l,  p_tl = 2^(s_tl - lse_t log2(e)),
//   dp_tl = dA_t . v_l,  D_t = dA_t . a_t,  de_tl = p_tl (dp_tl - D_t),
//   dv_l = sum_t p_tl dA_t,  dk_l = ln(2) sum_t de_tl q_t,
//   dq_t = sum_l de_tl k_l / sqrt(d_h)
// (the softmax gradient of Sec. 3.1's single-query attention, d e = p (dp - D)).
//
// v_mfma_f32_32x32x16 operand layout (lane l, hi = l / 32):
//   A: A[i = l%32][k]  B: B[k][j = l%32]  for k in the lane's 8-element set
//   result element v: row i = 8 (v/4) + 4 hi + v%4, column j = l%32
// A result C can feed a later product as an A operand (standing for C^T) or a
// B operand (standing for C) that contracts over C's row index i, with
// element p of k-step s holding index 16 s + 4 hi + (p < 4 ? p : p + 4).
// Every product below is arranged so: K^T and V^T (lane = row, elements =
// head dims) feed S = Q K^T and dP = dA V^T (lane = row, elements =
// targets); P and dE feed dV^T, dK^T (lane = row) and dV, dK (lane = dim) by
// swapping operands; dE^T and K with rows in the elements come from products
// with an identity operand, which then give dQ = dE K.  The score product
// runs on fp16 operands, as in the forward, so the softmax weights match the
// forward's; the gradient products run on bf16 operands with fp32 sums.
#include "common.h"
#include "fast.h"
#include "ring.h"

namespace stca {

namespace {

constexpr int DH = 32;
constexpr int kSegPitch = 1024 + 16;  // one 1 KB LDS segment of the X tile plus padding
constexpr int kXAhead = 2;            // X operands read this many k-steps ahead

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x16 mma(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mma(const f16x8& a, const f16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f16x8 pack_h(const f32x16& a, int off) {
  f16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = static_cast<_Float16>(a[off + i]);
  return r;
}
__device__ __forceinline__ bf16x8 pack_b(const f32x16& a, int off) {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = static_cast<__bf16>(a[off + i]);
  return r;
}

// index (row of a result, or k of an operand) of element p of k-step s
__device__ __forceinline__ int kidx(int s, int p, int hi) { return 16 * s + 4 * hi + (p < 4 ? p : p + 4); }
// row index of result element v
__device__ __forceinline__ int vrow(int v, int hi) { return 8 * (v / 4) + 4 * hi + v % 4; }

// History row (within the block) that MFMA row/column index i stands for: the
// X tile is stored in 1 KB segments of RPS rows, and index i reads segment
// i % (32 / RPS), so that the eight lanes of an LDS read phase hit eight
// segments (distinct banks).
template <int RPS>
__host__ __device__ constexpr int blk_row(int i) {
  return RPS * (i % (32 / RPS)) + i / (32 / RPS);
}

// The value unchanged, but opaque to the compiler.
__device__ __forceinline__ int opaque(int v) {
  asm volatile("" : "+v"(v));
  return v;
}

// keeps the compiler from interleaving the independent products around it
// (each one's result is stored before the next is formed)
__device__ __forceinline__ void fence() { __builtin_amdgcn_sched_barrier(0); }

__device__ __forceinline__ uint32_t pack2(float x, float y) {
  return (uint32_t)from_f32<bf16_bits>(x) | ((uint32_t)from_f32<bf16_bits>(y) << 16);
}

// Per-wave operand slots in LDS (one 16-byte vector per lane each): a unit's
// per-target operands of the wave's head, written once per unit, and the
// identity operand, written once.
enum OpSlot {
  kQa = 0,   // A: Q (i = target, k = head dims), fp16; two k-steps
  kDa = 2,   // A: dA (i = target, k = head dims), bf16
  kQt = 4,   // A: Q^T (i = head dim, k = targets), bf16; as B: Q (k = targets, j = dim)
  kDt = 6,   // A: dA^T (i = head dim, k = targets), bf16; as B: dA
  kSlots = 8
};

template <int D>
__global__ __launch_bounds__(64 * (D / 32)) void bwd_fused_kernel(FastAttnBwd A) {
  constexpr int H = D / DH;
  constexpr int KS = D / 16;
  constexpr int CPR = D / 8;     // 16-byte chunks per history row
  constexpr int RPS = 64 / CPR;  // rows per 1 KB segment
  constexpr int NS = 32 / RPS;   // segments per block (two per wave)
  constexpr int TILE = NS * kSegPitch;
  static_assert(NS == 2 * H, "two segments per wave");
  __shared__ __attribute__((aligned(16))) unsigned char xs[2 * TILE];
  __shared__ __attribute__((aligned(16))) float st_lse[H][32];
  __shared__ __attribute__((aligned(16))) float st_d[H][32];
  __shared__ __attribute__((aligned(16))) u32x4 opnd[H][kSlots][64];
  __shared__ __attribute__((aligned(16))) u32x4 eye[2][64];          // B: identity (k, j = lane column)
  __shared__ __attribute__((aligned(16))) f32x4 dq_acc[H][4][64];     // the unit's dq (result layout)

  const Unit* __restrict__ units = static_cast<const Unit*>(A.units);
  const WsHeader* __restrict__ hdr = static_cast<const WsHeader*>(A.hdr);
  const bf16_bits* __restrict__ X = static_cast<const bf16_bits*>(A.X);
  const int nu = hdr->n_units;
  if (static_cast<int>(blockIdx.x) >= nu) return;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);  // uniform: scalar registers
  // lane quantities; made opaque at every block (below) so that what derives
  // from them is recomputed in the loop rather than kept live across it
  int lane = threadIdx.x % 64, tcol = lane % 32, hi = lane / 32;
  const int64_t n_tgt = A.n_tgt;

  bf16x8 wk[KS], wv[KS];
  {
    const bf16x8* pk = static_cast<const bf16x8*>(A.WkP) + ((int64_t)(A.layer * H + wave) * KS) * 64 + lane;
    const bf16x8* pv = static_cast<const bf16x8*>(A.WvP) + ((int64_t)(A.layer * H + wave) * KS) * 64 + lane;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      wk[ks] = pk[ks * 64];
      wv[ks] = pv[ks * 64];
    }
  }
  auto put_op = [&](int slot, auto v) {
    opnd[wave][slot][lane] = __builtin_bit_cast(u32x4, v);
  };
  auto get_b = [&](int slot) { return __builtin_bit_cast(bf16x8, opnd[wave][slot][lane]); };
  auto get_h = [&](int slot) { return __builtin_bit_cast(f16x8, opnd[wave][slot][lane]); };
  auto get_eye = [&](int s) { return __builtin_bit_cast(bf16x8, eye[s][lane]); };
  // identity B operand: element p of k-step s is 1 where its index is column tcol
  if (wave < 2) {
    bf16x8 e;
#pragma unroll
    for (int p = 0; p < 8; ++p) e[p] = static_cast<__bf16>(kidx(wave, p, hi) == tcol ? 1.f : 0.f);
    eye[wave][lane] = __builtin_bit_cast(u32x4, e);
  }
  // the unit's dq accumulates in LDS (16 floats per lane)
  auto dq_get = [&]() {
    f32x16 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const f32x4 x = dq_acc[wave][i][lane];
      r[4 * i] = x[0], r[4 * i + 1] = x[1], r[4 * i + 2] = x[2], r[4 * i + 3] = x[3];
    }
    return r;
  };
  auto dq_put = [&](const f32x16& r) {
#pragma unroll
    for (int i = 0; i < 4; ++i) dq_acc[wave][i][lane] = f32x4{r[4 * i], r[4 * i + 1], r[4 * i + 2], r[4 * i + 3]};
  };

  // ---- X blocks: this wave's two segments of the next block are loaded into
  // registers while the current block is processed, then written to the
  // other of two LDS tiles; one barrier per block publishes the tile.
  int lu = blockIdx.x;  // load cursor
  Unit lun = units[lu];
  int lb = lun.b0;
  u32x4 xr[2];
  auto fetch = [&]() -> bool {
    if (lu >= nu) return false;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int e = (2 * wave + i) * 64 + lane;  // 16-byte chunk of the block
      const int64_t grow = min((int64_t)lb * 32 + e / CPR, A.n_hist - 1);
      xr[i] = *reinterpret_cast<const u32x4*>(X + grow * D + (e % CPR) * 8);
    }
    if (++lb >= lun.b1) {
      lu += gridDim.x;
      if (lu < nu) {
        lun = units[lu];
        lb = lun.b0;
      }
    }
    return true;
  };
  auto put = [&](int slot) {
    unsigned char* t = xs + slot * TILE;
#pragma unroll
    for (int i = 0; i < 2; ++i) *reinterpret_cast<u32x4*>(t + (2 * wave + i) * kSegPitch + lane * 16) = xr[i];
  };
  auto project = [&](const unsigned char* tile, f32x16& ak, f32x16& av) {
    ak = f32x16{};
    av = f32x16{};
    // MFMA column tcol reads history row blk_row<RPS>(tcol)
    const unsigned char* xp = tile + (tcol % NS) * kSegPitch + (tcol / NS) * (2 * D) + 16 * hi;
    bf16x8 xo[kXAhead];
#pragma unroll
    for (int i = 0; i < kXAhead; ++i) xo[i] = *reinterpret_cast<const bf16x8*>(xp + 32 * i);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const bf16x8 x = xo[ks % kXAhead];
      if (ks + kXAhead < KS) xo[ks % kXAhead] = *reinterpret_cast<const bf16x8*>(xp + 32 * (ks + kXAhead));
      ak = mma(wk[ks], x, ak);  // K^T: rows = head dims, columns = history rows
      av = mma(wv[ks], x, av);  // V^T
    }
  };

  auto init = [&](const Unit& un) {
    const int nt = un.nt;
    const bool tok = tcol < nt;
    const float* qrow = A.Q + (int64_t)(un.t0 + (tok ? tcol : 0)) * D + wave * DH;
    const float* darow = A.da + (int64_t)(un.t0 + (tok ? tcol : 0)) * D + wave * DH;
    const float* arow = A.a + (int64_t)(un.t0 + (tok ? tcol : 0)) * D + wave * DH;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      f16x8 qa;
      bf16x8 da, qt, dt;
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int c = 16 * s + 8 * half + 4 * hi;
        const float4 q4 = tok ? *reinterpret_cast<const float4*>(qrow + c) : make_float4(0.f, 0.f, 0.f, 0.f);
        const float4 d4 = tok ? *reinterpret_cast<const float4*>(darow + c) : make_float4(0.f, 0.f, 0.f, 0.f);
        const float qv[4] = {q4.x, q4.y, q4.z, q4.w}, dv[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          qa[4 * half + e] = static_cast<_Float16>(qv[e]);
          da[4 * half + e] = static_cast<__bf16>(dv[e]);
        }
      }
#pragma unroll
      for (int p = 0; p < 8; ++p) {
        const int tt = kidx(s, p, hi);
        const bool ok = tt < nt;
        const int64_t off = (int64_t)(un.t0 + (ok ? tt : 0)) * D + wave * DH + tcol;
        qt[p] = static_cast<__bf16>(ok ? A.Q[off] : 0.f);
        dt[p] = static_cast<__bf16>(ok ? A.da[off] : 0.f);
      }
      put_op(kQa + s, qa);
      put_op(kDa + s, da);
      put_op(kQt + s, qt);
      put_op(kDt + s, dt);
    }
    // D_t = dA_t . a_t over the head's dims: each lane half sums 16 of them
    float dd = 0.f;
    if (tok) {
#pragma unroll
      for (int c = 0; c < 16; c += 4) {
        const float4 x = *reinterpret_cast<const float4*>(darow + 16 * hi + c);
        const float4 y = *reinterpret_cast<const float4*>(arow + 16 * hi + c);
        dd += x.x * y.x + x.y * y.y + x.z * y.z + x.w * y.w;
      }
    }
    dd += __shfl_xor(dd, 32);
    if (hi == 0) {
      st_lse[wave][tcol] = tok ? A.lse[(int64_t)(un.t0 + tcol) * H + wave] * kLog2e : INFINITY;
      st_d[wave][tcol] = dd;
    }
    dq_put(f32x16{});
    // the statistics are read by other lanes of the wave
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  };

  // stores of this lane's gradient row
  bf16_bits* __restrict__ dKV = A.dKV;
  auto store_rows = [&](const f32x16& g, int col0, int row, bool rok) {
    // g: lane = history row `row`, element v = head dim vrow(v, hi)
    if (!rok) return;
    bf16_bits* p = dKV + (int64_t)row * A.ldkv + col0 + 4 * hi;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint2 w;
      w.x = pack2(g[4 * q], g[4 * q + 1]);
      w.y = pack2(g[4 * q + 2], g[4 * q + 3]);
      *reinterpret_cast<uint2*>(p + 8 * q) = w;
    }
  };

  // ---- walk the workgroup's units block by block
  bool have = fetch();
  if (have) put(0);
  int cu = blockIdx.x;
  Unit cun = units[cu];
  int cb = cun.b0;
  const float scale = rsqrtf(static_cast<float>(DH));
  for (int p = 0; cu < nu; ++p) {
    lane = opaque(lane);
    tcol = opaque(tcol);
    hi = opaque(hi);
    __syncthreads();  // tile p is complete; every wave is done with tile p - 1
    have = fetch();   // block p + 1 into registers
    if (cb == cun.b0) init(cun);
    const unsigned char* tile = xs + (p % 2) * TILE;
    f32x16 ak, av;
    project(tile, ak, av);
    const f16x8 kh[2] = {pack_h(ak, 0), pack_h(ak, 8)};
    const bf16x8 vb[2] = {pack_b(av, 0), pack_b(av, 8)};
    // K with rows in the elements (lane = dim), for dQ: K^T times the identity
    bf16x8 kf[2];
    {
      f32x16 k = mma(pack_b(ak, 0), get_eye(0), f32x16{});
      k = mma(pack_b(ak, 8), get_eye(1), k);
      kf[0] = pack_b(k, 0);
      kf[1] = pack_b(k, 8);
    }
    fence();
    // S = Q K^T and dP = dA V^T: lane = history row, elements = targets
    f32x16 s = mma(get_h(kQa), kh[0], f32x16{});
    s = mma(get_h(kQa + 1), kh[1], s);
    f32x16 dp = mma(get_b(kDa), vb[0], f32x16{});
    dp = mma(get_b(kDa + 1), vb[1], dp);
    const int row = cb * 32 + blk_row<RPS>(tcol);
    const bool rok = row >= cun.l0 && row < cun.l1;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 l4 = *reinterpret_cast<const float4*>(&st_lse[wave][8 * q + 4 * hi]);
      const float4 d4 = *reinterpret_cast<const float4*>(&st_d[wave][8 * q + 4 * hi]);
      const float lv[4] = {l4.x, l4.y, l4.z, l4.w}, dv[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int v = 4 * q + e;
        const float pr = rok ? __builtin_amdgcn_exp2f(s[v] - lv[e]) : 0.f;
        dp[v] = pr * (dp[v] - dv[e]);
        s[v] = pr;
      }
    }
    const bf16x8 pb[2] = {pack_b(s, 0), pack_b(s, 8)};
    const bf16x8 eb[2] = {pack_b(dp, 0), pack_b(dp, 8)};
    fence();
    // dV^T = dA^T P and dK^T = Q^T dE (lane = row): row-major dK | dV
    {
      f32x16 g = mma(get_b(kDt), pb[0], f32x16{});
      g = mma(get_b(kDt + 1), pb[1], g);
      store_rows(g, D + wave * DH, row, rok);
      fence();
      g = mma(get_b(kQt), eb[0], f32x16{});
      g = mma(get_b(kQt + 1), eb[1], g);
      g *= kLn2;
      store_rows(g, wave * DH, row, rok);
    }
    fence();
    // dQ += dE K: dE^T with rows in the elements (lane = target) from dE
    // times the identity
    {
      f32x16 et = mma(eb[0], get_eye(0), f32x16{});
      et = mma(eb[1], get_eye(1), et);
      f32x16 dq = dq_get();
      dq = mma(pack_b(et, 0), kf[0], dq);
      dq = mma(pack_b(et, 8), kf[1], dq);
      dq_put(dq);
    }
    if (cb + 1 == cun.b1) {
      // dq partial of this chunk: lane = dim tcol, element v = target vrow(v, hi)
      const f32x16 dq = dq_get();
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int tt = vrow(v, hi);
        if (tt < cun.nt)
          A.dq_part[((int64_t)cun.c * n_tgt + cun.t0 + tt) * D + wave * DH + tcol] = dq[v] * scale;
      }
      cu += gridDim.x;
      if (cu < nu) {
        cun = units[cu];
        cb = cun.b0;
      }
    } else {
      ++cb;
    }
    if (have) put((p + 1) % 2);
  }
}

// The forward attention recomputed for the backward, also with the history
// projection inside the kernel, but close to fp32: the K, V, query and
// softmax-weight operands are each split into two fp16 terms (hi + lo, about
// 22 significant bits), and every score and P.V product takes the three
// terms hi.hi + hi.lo + lo.hi, so the recomputed attention output (which
// decides the ReLU gates of the update that follows) matches an fp32
// evaluation.  Layout as the forward's fused kernel: S^T = K Q^T (lane =
// target, elements = rows), O^T = V^T P^T (lane = target, elements = head
// dims); the result is the same per-chunk partial (unnormalised O, running
// max in log2 units, sum).
// A unit descriptor read as wave-uniform values: the values are waited for
// where the unit is read, not at their first use inside a loop (where, for a
// kernel whose direct loads the compiler does not see, its wait would also
// drain those loads at every step).
__device__ __forceinline__ Unit uniform_unit(const Unit* units, int i) {
  const Unit u = units[i];
  return Unit{__builtin_amdgcn_readfirstlane(u.r),  __builtin_amdgcn_readfirstlane(u.t0),
              __builtin_amdgcn_readfirstlane(u.nt), __builtin_amdgcn_readfirstlane(u.c),
              __builtin_amdgcn_readfirstlane(u.b0), __builtin_amdgcn_readfirstlane(u.b1),
              __builtin_amdgcn_readfirstlane(u.l0), __builtin_amdgcn_readfirstlane(u.l1)};
}

template <int D>
__global__ __launch_bounds__(64 * (D / 32)) void fwd_precise_kernel(FastAttnFwdPrecise A) {
  constexpr int H = D / DH;
  constexpr int KS = D / 16;
  constexpr int CPR = D / 8;
  constexpr int RPS = 64 / CPR;
  constexpr int NS = 32 / RPS;
  constexpr int TILE = NS * kSegPitch;
  static_assert(NS == 2 * H, "two segments per wave");
  constexpr int STG = 4;  // X blocks in the LDS ring (STG - 1 in flight)
  __shared__ __attribute__((aligned(16))) unsigned char xs[STG * TILE];

  const Unit* __restrict__ units = static_cast<const Unit*>(A.units);
  const WsHeader* __restrict__ hdr = static_cast<const WsHeader*>(A.hdr);
  const bf16_bits* __restrict__ X = static_cast<const bf16_bits*>(A.X);
  const int nu = hdr->n_units;
  if (static_cast<int>(blockIdx.x) >= nu) return;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
  int lane = threadIdx.x % 64, tcol = lane % 32, hi = lane / 32;
  const int64_t n_tgt = A.n_tgt;

  bf16x8 wk[KS], wv[KS];
  {
    const bf16x8* pk = static_cast<const bf16x8*>(A.WkP) + ((int64_t)(A.layer * H + wave) * KS) * 64 + lane;
    const bf16x8* pv = static_cast<const bf16x8*>(A.WvP) + ((int64_t)(A.layer * H + wave) * KS) * 64 + lane;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      wk[ks] = pk[ks * 64];
      wv[ks] = pv[ks * 64];
    }
  }
  // the weights land before the ring's first load (the compiler does not
  // see the ring's direct loads, and would otherwise wait for the weights
  // inside the loop with counts that also drain the ring's prefetches)
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) asm volatile("" : "+v"(wk[ks]), "+v"(wv[ks]));
  // X blocks by direct global-to-LDS loads, each wave two 1 KB segments
  // of every block, STG - 1 blocks ahead
  int lu = blockIdx.x;
  Unit lun = uniform_unit(units, lu);
  int lb = lun.b0;
  int p_load = 0;  // blocks issued so far
  auto issue = [&]() {
    if (lu >= nu) return;
    unsigned char* slot = xs + (p_load % STG) * TILE;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int seg = 2 * wave + i;
      const int e = seg * 64 + lane;
      const int64_t grow = min((int64_t)lb * 32 + e / CPR, A.n_hist - 1);
      dma16(X + grow * D + (e % CPR) * 8, slot + seg * kSegPitch);
    }
    ++p_load;
    if (++lb >= lun.b1) {
      lu += gridDim.x;
      if (lu < nu) {
        lun = uniform_unit(units, lu);
        lb = lun.b0;
      }
    }
  };
  // -1 the compiler cannot fold: the residual a - hi written as
  // fma(hi, -1, a) takes mixed-precision FMAs (an fp16 operand widened
  // inside the instruction, the fp16 result rounded once) instead of a
  // widening conversion and a subtraction per element; the value is the same
  float neg1 = -1.f;
  asm volatile("" : "+s"(neg1));
  // hi and lo fp16 terms of 8 consecutive result elements
  auto split = [&](const f32x16& a, int off, f16x8& h, f16x8& l) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const _Float16 x = static_cast<_Float16>(a[off + i]);
      h[i] = x;
      l[i] = static_cast<_Float16>(__builtin_fmaf(static_cast<float>(x), neg1, a[off + i]));
    }
  };

  f16x8 qh[2], ql[2];  // B: Q^T (k = head dims, j = target tcol)
  f32x16 O;
  float m, l;
  auto init = [&](const Unit& un) {
    const bool tok = tcol < un.nt;
    const float* qrow = A.Q + (int64_t)(un.t0 + (tok ? tcol : 0)) * D + wave * DH;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const float4 q4 = tok ? *reinterpret_cast<const float4*>(qrow + 16 * s + 8 * half + 4 * hi)
                              : make_float4(0.f, 0.f, 0.f, 0.f);
        const float qv[4] = {q4.x, q4.y, q4.z, q4.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const _Float16 x = static_cast<_Float16>(qv[e]);
          qh[s][4 * half + e] = x;
          ql[s][4 * half + e] = static_cast<_Float16>(__builtin_fmaf(static_cast<float>(x), neg1, qv[e]));
        }
      }
    }
    O = f32x16{};
    m = -INFINITY;
    l = 0.f;
  };

#pragma unroll
  for (int i = 0; i < STG - 1; ++i) issue();
  int cu = blockIdx.x;
  Unit cun = uniform_unit(units, cu);
  int cb = cun.b0;
  for (int p = 0; cu < nu; ++p) {
    lane = opaque(lane);
    tcol = opaque(tcol);
    hi = opaque(hi);
    // this wave's parts of block p landed (later ones may be in flight); the
    // barrier publishes everyone's, and the slot of block p - 1 is free
    wait_vm(2 * (p_load - 1 - p));
    ring_barrier();
    if (p_load < p + STG) issue();
    if (cb == cun.b0) init(cun);
    const unsigned char* xp =
        xs + (p % STG) * TILE + (tcol % NS) * kSegPitch + (tcol / NS) * (2 * D) + 16 * hi;
    f32x16 ak = {}, av = {};
    {
      bf16x8 xo[kXAhead];
#pragma unroll
      for (int i = 0; i < kXAhead; ++i) xo[i] = *reinterpret_cast<const bf16x8*>(xp + 32 * i);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 x = xo[ks % kXAhead];
        if (ks + kXAhead < KS) xo[ks % kXAhead] = *reinterpret_cast<const bf16x8*>(xp + 32 * (ks + kXAhead));
        ak = mma(wk[ks], x, ak);  // K^T: lane = history row, elements = head dims
        av = mma(x, wv[ks], av);  // V: lane = head dim, elements = history rows
      }
    }
    fence();
    // S^T = K Q^T: lane = target, elements = history rows
    f32x16 sc = {};
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      f16x8 kh, kl;
      split(ak, 8 * s, kh, kl);
      sc = mma(kh, qh[s], sc);
      sc = mma(kh, ql[s], sc);
      sc = mma(kl, qh[s], sc);
    }
    if (!(cb * 32 >= cun.l0 && cb * 32 + 32 <= cun.l1)) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = cb * 32 + blk_row<RPS>(vrow(v, hi));
        if (row < cun.l0 || row >= cun.l1) sc[v] = -INFINITY;
      }
    }
    float bm = sc[0];
#pragma unroll
    for (int v = 1; v < 16; ++v) bm = fmaxf(bm, sc[v]);
    bm = fmaxf(bm, __shfl_xor(bm, 32));
    const float mn = fmaxf(m, bm);  // finite: every block of a unit holds a row of it
    const float r = __builtin_amdgcn_exp2f(m - mn);
    m = mn;
    l *= r;
    O *= r;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      sc[v] = __builtin_amdgcn_exp2f(sc[v] - mn);
      l += sc[v];
    }
    fence();
    // O^T += V^T P^T
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      f16x8 vh, vl, ph, pl;
      split(av, 8 * s, vh, vl);
      split(sc, 8 * s, ph, pl);
      O = mma(vh, ph, O);
      O = mma(vh, pl, O);
      O = mma(vl, ph, O);
    }
    fence();
    if (cb + 1 == cun.b1) {
      const float lt = l + __shfl_xor(l, 32);
      if (tcol < cun.nt) {
        const int64_t row = (int64_t)cun.c * n_tgt + cun.t0 + tcol;
        float* pa = A.part_acc + row * D + wave * DH + 4 * hi;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          *reinterpret_cast<float4*>(pa + 8 * q) = make_float4(O[4 * q], O[4 * q + 1], O[4 * q + 2], O[4 * q + 3]);
        if (hi == 0) reinterpret_cast<float2*>(A.part_ml)[row * H + wave] = make_float2(m, lt);
      }
      cu += gridDim.x;
      if (cu < nu) {
        cun = uniform_unit(units, cu);
        cb = cun.b0;
      }
    } else {
      ++cb;
    }
  }
}

}  // namespace

hipError_t fast_attn_bwd(int D, const FastAttnBwd& f, int grid, hipStream_t st) {
  if (grid == 0) return hipSuccess;
#define STCA_BWDF(DD) hipLaunchKernelGGL(bwd_fused_kernel<DD>, dim3(grid), dim3(64 * (DD / 32)), 0, st, f)
  switch (D) {
    case 64: STCA_BWDF(64); break;
    case 128: STCA_BWDF(128); break;
    case 256: STCA_BWDF(256); break;
    default: return hipErrorInvalidValue;
  }
#undef STCA_BWDF
  return hipGetLastError();
}

hipError_t fast_attn_fwd_precise(int D, const FastAttnFwdPrecise& f, int grid, hipStream_t st) {
  if (grid == 0) return hipSuccess;
#define STCA_FWDP(DD) hipLaunchKernelGGL(fwd_precise_kernel<DD>, dim3(grid), dim3(64 * (DD / 32)), 0, st, f)
  switch (D) {
    case 64: STCA_FWDP(64); break;
    case 128: STCA_FWDP(128); break;
    case 256: STCA_FWDP(256); break;
    default: return hipErrorInvalidValue;
  }
#undef STCA_FWDP
  return hipGetLastError();
}

}  // namespace stca
