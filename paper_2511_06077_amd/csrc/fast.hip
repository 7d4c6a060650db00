// MFMA path for bf16 storage and d_h = 32 (gfx950 / CDNA4): history K/V
// projection (K1), fused multi-target cross attention (K3) and fused target
// update (K4).
//
// K1 multiplies the bf16 history by the bf16 weights (v_mfma_f32_32x32x16_bf16,
// fp32 accumulate) and stores K and V as fp16: the same two bytes as bf16 with
// three more mantissa bits, which the attention's softmax weights are
// sensitive to.  K3 and K4 run v_mfma_f32_32x32x16_f16 on fp16 operands (Q, K,
// V, the softmax weights P, and the update's activations and weights), always
// accumulating in fp32; the target state stays fp32.  Both instructions have
// the same rate and operand layout.  For them lane l holds
//   A operand: A[i = l%32][k = 8*(l/32) .. +7]           (8 bf16)
//   B operand: B[k = 8*(l/32) .. +7][j = l%32]           (8 bf16)
//   result   : D[i = 8*(v/4) + 4*(l/32) + v%4][j = l%32] for v = 0..15 (fp32)
// The projected history is written in exactly the register order the
// attention kernel's MFMAs consume, so every K/V operand fetch of the
// attention kernel is one fully coalesced 16-byte-per-lane load and no LDS
// round trip is needed:
//
//   KV[layer][block of 32 rows][head][K s=0 | K s=1 | V u=0 | V u=1][64 lanes][8 bf16]
//
//   K, slice s : lane (row l%32, hi = l/32) holds K[row][16s + 4hi + {0,1,2,3,8,9,10,11}]
//   V, slice u : lane (col l%32, hi)        holds V[16u + 4hi + {0,1,2,3,8,9,10,11}][col]
//
// The attention kernel computes S^T = K Q^T (rows = history items, columns =
// targets), so a lane holds 16 scores of one target and the softmax maximum is
// an in-register reduction plus one exchange with lane l^32.  The dimension
// order inside K's slices is a permutation of the head's 32 dimensions; the
// queries are stored with the same permutation (QN below), which leaves q.k
// unchanged.  The item order inside V's slices matches the order in which
// S^T's result registers hold items, so P^T feeds the P.V MFMA as its B
// operand straight from registers.
//
//   QN[target][head][32]: position 16s + 8hi + i holds dimension
//       16s + 4hi + (i < 4 ? i : i + 4), scaled by log2(e)/sqrt(d_h)
//
// Weights are repacked once per call into the same operand order
// ("packed": [N/32][K/16][64 lanes][8 bf16] with lane (n = l%32, hi) holding
// W[16ks + 8hi .. +7][32nb + n]), which serves both as an A operand of D^T and
// as a B operand of D.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "fast.h"
#include "ring.h"

namespace stca {

namespace {

constexpr int DH = 32;
constexpr float kSlack = 8.f;  // log2 units: softmax weights stay <= 256 between rescales

__device__ __forceinline__ f32x16 mfma(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mfma(const f16x8& a, const f16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f16x8 pack8h(const f32x16& a, int off) {
  f16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = static_cast<_Float16>(a[off + i]);
  return r;
}

__device__ __forceinline__ f16x8 zero8h() {
  f16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = static_cast<_Float16>(0.f);
  return r;
}

// 2^x with the hardware instruction alone: the arguments are max-subtracted
// scores (<= 0), whose results below 2^-126 may flush to zero without effect
// on the softmax, so the library's denormal-safe expansion is not needed.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ uint16_t f16_bits(float x) {
  return __builtin_bit_cast(uint16_t, static_cast<_Float16>(x));
}

template <typename V8>
struct elem_of;
template <>
struct elem_of<bf16x8> {
  typedef __bf16 type;
};
template <>
struct elem_of<f16x8> {
  typedef _Float16 type;
};

// ------------------------------------------------------------- repacking
// W: [layers][K][N] bf16 row-major -> P: [layers][N/32][K/16][64][8], kept
// bf16 (V8 = bf16x8) or converted to fp16 (V8 = f16x8, exact for every bf16
// value inside fp16's range).
template <typename V8>
__global__ void pack_kernel(const bf16_bits* __restrict__ W, V8* __restrict__ P, int K, int N,
                            int64_t per_layer_groups) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int layer = blockIdx.y;
  if (g >= per_layer_groups) return;
  const int lane = g % 64;
  const int64_t rest = g / 64;
  const int ks = rest % (K / 16);
  const int nb = rest / (K / 16);
  const int n = nb * 32 + lane % 32;
  const int k0 = ks * 16 + 8 * (lane / 32);
  const bf16_bits* w = W + (int64_t)layer * K * N;
  V8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = static_cast<typename elem_of<V8>::type>(to_f32(w[(int64_t)(k0 + e) * N + n]));
  P[(int64_t)layer * per_layer_groups + g] = r;
}

// Several weights in one launch (blockIdx.z = job): the per-call repacking of
// a forward costs one launch instead of one per weight.
template <typename V8>
__device__ __forceinline__ void pack_one(const bf16_bits* __restrict__ w, V8* __restrict__ P, int K, int N,
                                         int64_t g, bool trans) {
  const int lane = g % 64;
  const int64_t rest = g / 64;
  const int ks = rest % (K / 16);
  const int nb = rest / (K / 16);
  const int n = nb * 32 + lane % 32;
  const int k0 = ks * 16 + 8 * (lane / 32);
  V8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e)
    r[e] = static_cast<typename elem_of<V8>::type>(
        to_f32(w[trans ? (int64_t)n * K + k0 + e : (int64_t)(k0 + e) * N + n]));
  P[g] = r;
}

__global__ void pack_many_kernel(PackJobs J) {
  const int j = blockIdx.z, layer = blockIdx.y;
  const int64_t groups = (int64_t)(J.job[j].N / 32) * (J.job[j].K / 16) * 64;
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= groups) return;
  const PackJob& b = J.job[j];
  const bf16_bits* w = static_cast<const bf16_bits*>(b.src) + (int64_t)layer * b.K * b.N;
  if (b.to_f16)
    pack_one(w, static_cast<f16x8*>(b.dst) + (int64_t)layer * groups, b.K, b.N, g, b.trans != 0);
  else
    pack_one(w, static_cast<bf16x8*>(b.dst) + (int64_t)layer * groups, b.K, b.N, g, b.trans != 0);
}

// ------------------------------------------------------ K1: projection
// Grid: n_layers * parts workgroups, one wave per head.  Each wave keeps its
// head's W_K and W_V columns in registers for the whole kernel; the
// workgroup streams its share of 32-row history blocks through a
// double-buffered LDS tile (one global read of X per block, shared by all
// heads).  Workgroups on the same XCD (id % 8) are given the same history
// rows for all layers, so the re-reads of X by the other layers hit that XCD's L2.
template <int D>
__global__ __launch_bounds__(64 * (D / 32)) void proj_kernel(const bf16_bits* __restrict__ X, int64_t n_hist,
                                                             int64_t n_blocks, const bf16x8* __restrict__ WkP,
                                                             const bf16x8* __restrict__ WvP,
                                                             f16x8* __restrict__ KV, int n_layers, int parts) {
  constexpr int H = D / DH;
  constexpr int KS = D / 16;
  constexpr int ROW = D + 8;             // padded LDS row (bf16): conflict-free 16 B reads
  constexpr int CHUNKS = 32 * D / 8;     // 16-byte chunks per block
  constexpr int NT = 64 * H;
  static_assert(CHUNKS == 2 * NT, "two chunks per thread");
  __shared__ __attribute__((aligned(16))) bf16_bits xs[2][32 * ROW];

  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int id = blockIdx.x;
  const int slot = id / 8;
  const int layer = slot % n_layers;
  const int part = (slot / n_layers) * 8 + id % 8;
  const int64_t bb = (int64_t)part * n_blocks / parts;
  const int64_t be = (int64_t)(part + 1) * n_blocks / parts;
  if (bb >= be) return;

  bf16x8 wk[KS], wv[KS];
  {
    const bf16x8* pk = WkP + ((int64_t)(layer * H + wave) * KS) * 64 + lane;
    const bf16x8* pv = WvP + ((int64_t)(layer * H + wave) * KS) * 64 + lane;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      wk[ks] = pk[ks * 64];
      wv[ks] = pv[ks * 64];
    }
  }

  auto load = [&](int64_t b, uint4 (&r)[2]) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = threadIdx.x + i * NT;
      const int row = c / (D / 8), col8 = c % (D / 8);
      const int64_t grow = b * 32 + row;
      r[i] = grow < n_hist ? *reinterpret_cast<const uint4*>(X + grow * D + col8 * 8) : make_uint4(0, 0, 0, 0);
    }
  };
  auto stash = [&](int buf, const uint4 (&r)[2]) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = threadIdx.x + i * NT;
      const int row = c / (D / 8), col8 = c % (D / 8);
      *reinterpret_cast<uint4*>(&xs[buf][row * ROW + col8 * 8]) = r[i];
    }
  };

  uint4 nxt[2];
  load(bb, nxt);
  stash(0, nxt);
  __syncthreads();
  const int trow = lane % 32, hi = lane / 32;
  for (int64_t b = bb; b < be; ++b) {
    const int cur = (b - bb) & 1;
    if (b + 1 < be) load(b + 1, nxt);
    f32x16 ak = {}, av = {};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const bf16x8 xo = *reinterpret_cast<const bf16x8*>(&xs[cur][trow * ROW + ks * 16 + hi * 8]);
      ak = mfma(wk[ks], xo, ak);  // K^T block: rows = head dims, cols = history rows
      av = mfma(xo, wv[ks], av);  // V block:   rows = history rows, cols = head dims
    }
    f16x8* out = KV + (((int64_t)layer * n_blocks + b) * H + wave) * 4 * 64 + lane;
    out[0] = pack8h(ak, 0);
    out[64] = pack8h(ak, 8);
    out[128] = pack8h(av, 0);
    out[192] = pack8h(av, 8);
    if (b + 1 < be) stash(cur ^ 1, nxt);
    __syncthreads();
  }
}

// Combine a value of lane l with that of lane l ^ 32 (v_permlane32_swap: a
// VALU exchange between the two halves of the wave, no LDS round trip).
__device__ __forceinline__ float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Row order inside a 32-row history block as the fused kernel reads it from
// LDS: MFMA row index i is history row RPS * (i % (32 / RPS)) + i / (32 / RPS)
// (RPS = 1: identity).  With RPS rows per 1 KB LDS segment this sends the
// eight lanes of each LDS read phase to eight different segments, i.e. to
// distinct bank groups.
template <int RPS>
__device__ __forceinline__ int blk_row(int i) {
  return RPS * (i % (32 / RPS)) + i / (32 / RPS);
}

// ------------------------------------------ online softmax over blocks
// State of one wave (one head) for all of a unit's targets (up to 64: two
// 32-wide column groups).  Online softmax in log2 units; the result is an
// unnormalised partial (acc, max, sum) per (chunk, target, head), merged by
// the update kernel.
template <int H, int NG>
struct Online {
  f16x8 qop[NG][2];
  f32x16 O[NG];
  float m[NG], l[NG];

  __device__ __forceinline__ void init(const Unit& un, const f16x8* __restrict__ QN, int j, int tcol, int hi) {
    constexpr int D = H * DH;
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const int tt = g * 32 + tcol;
      const bool ok = tt < un.nt;
      const f16x8* q = QN + ((int64_t)(un.t0 + tt) * D + j * DH) / 8;
      qop[g][0] = ok ? q[hi] : zero8h();
      qop[g][1] = ok ? q[2 + hi] : zero8h();
      O[g] = f32x16{};
      m[g] = -INFINITY;
      l[g] = 0.f;
    }
  }

  // kv: K slices 0, 1 and V slices 0, 1 of history block b (operand order).
  // MFMA row index i of the block holds history row b * 32 + blk_row<RPS>(i).
  // qload(g, qop[g]), when given, fills a column group's query operands right
  // before its MFMAs (so only one group's are live at a time).
  struct KeepQ {
    __device__ __forceinline__ void operator()(int, f16x8 (&)[2]) const {}
  };
  template <int RPS = 1, typename QLoad = KeepQ>
  __device__ __forceinline__ void step(const f16x8 (&kv)[4], int b, const Unit& un, int hi, QLoad qload = {}) {
    const bool full = b * 32 >= un.l0 && b * 32 + 32 <= un.l1;
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      qload(g, qop[g]);
      f32x16 s = mfma(kv[0], qop[g][0], f32x16{});
      s = mfma(kv[1], qop[g][1], s);
      if (!full) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int tok = b * 32 + blk_row<RPS>(8 * (v / 4) + 4 * hi + (v % 4));
          if (tok < un.l0 || tok >= un.l1) s[v] = -INFINITY;
        }
      }
      float bm = s[0];
#pragma unroll
      for (int v = 1; v < 16; ++v) bm = fmaxf(bm, s[v]);
      bm = max_halves(bm);
      // Threshold rescaling: the reference maximum m only moves when some
      // score of the wave exceeds it by more than kSlack (log2 units), so the
      // weights 2^(s - m) stay <= 2^kSlack (fine in fp16 and in the fp32 sums)
      // and the rescale of O and l is skipped for most blocks.
      if (__builtin_amdgcn_ballot_w64(bm > m[g] + kSlack)) {
        const float mn = fmaxf(m[g], bm);
        const float sc = fast_exp2(m[g] - mn);
        m[g] = mn;
        l[g] *= sc;
#pragma unroll
        for (int v = 0; v < 16; ++v) O[g][v] *= sc;
      }
      float ps = 0.f;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        s[v] = fast_exp2(s[v] - m[g]);
        ps += s[v];
      }
      l[g] += ps;
      O[g] = mfma(kv[2], pack8h(s, 0), O[g]);
      O[g] = mfma(kv[3], pack8h(s, 8), O[g]);
    }
  }

  __device__ __forceinline__ void finish(const Unit& un, int j, int tcol, int hi, float* __restrict__ part_acc,
                                         float2* __restrict__ part_ml, int64_t n_tgt) {
    constexpr int D = H * DH;
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const float lt = sum_halves(l[g]);
      const int tt = g * 32 + tcol;
      if (tt < un.nt) {
        const int64_t row = (int64_t)un.c * n_tgt + un.t0 + tt;
        float* pa = part_acc + row * D + j * DH + 4 * hi;
#pragma unroll
        for (int gg = 0; gg < 4; ++gg)
          *reinterpret_cast<float4*>(pa + 8 * gg) =
              make_float4(O[g][4 * gg], O[g][4 * gg + 1], O[g][4 * gg + 2], O[g][4 * gg + 3]);
        if (hi == 0) part_ml[row * H + j] = make_float2(m[g], lt);
      }
    }
  }
};

// ------------------------------------ K3: attention over materialised K/V
// One workgroup per unit (a request's target group x a chunk of its history
// blocks), one wave per head.  All of the unit's targets (up to 128: four
// 32-wide column groups) are held by every wave, so each K/V byte is read
// from HBM once per unit whatever the number of targets.  K/V blocks are double-buffered in registers.
template <int H, int NG>
__device__ __forceinline__ void attn_unit(const Unit& un, const f16x8* __restrict__ QN,
                                          const f16x8* __restrict__ KVl, float* __restrict__ part_acc,
                                          float2* __restrict__ part_ml, int64_t n_tgt) {
  const int j = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int tcol = lane % 32, hi = lane / 32;
  Online<H, NG> st;
  st.init(un, QN, j, tcol, hi);
  const f16x8* base = KVl + (int64_t)j * 4 * 64 + lane;
  auto ld = [&](int64_t b, f16x8 (&r)[4]) {
    const f16x8* p = base + b * (H * 4 * 64);
    r[0] = p[0];
    r[1] = p[64];
    r[2] = p[128];
    r[3] = p[192];
  };
  f16x8 nx[4], cu[4];
  ld(un.b0, nx);
  for (int b = un.b0; b < un.b1; ++b) {
#pragma unroll
    for (int i = 0; i < 4; ++i) cu[i] = nx[i];
    if (b + 1 < un.b1) ld(b + 1, nx);
    st.step(cu, b, un, hi);
  }
  st.finish(un, j, tcol, hi, part_acc, part_ml, n_tgt);
}

template <int H>
__global__ __launch_bounds__(64 * H) void attn_kernel(const Unit* __restrict__ units,
                                                      const WsHeader* __restrict__ hdr,
                                                      const f16x8* __restrict__ QN,
                                                      const f16x8* __restrict__ KVl, float* __restrict__ part_acc,
                                                      float2* __restrict__ part_ml, int64_t n_tgt) {
  const int nu = hdr->n_units;
  for (int u = blockIdx.x; u < nu; u += gridDim.x) {
    const Unit un = units[u];
    if (un.nt > 64)
      attn_unit<H, 4>(un, QN, KVl, part_acc, part_ml, n_tgt);
    else if (un.nt > 32)
      attn_unit<H, 2>(un, QN, KVl, part_acc, part_ml, n_tgt);
    else
      attn_unit<H, 1>(un, QN, KVl, part_acc, part_ml, n_tgt);
  }
}

// ------------------------- K13: projection fused into the attention
// The same attention, but each 32-row history block is projected to this
// layer's K and V inside the kernel and consumed from registers: nothing is
// written to HBM, and the history is read once per layer instead of K and V
// being written once and read back.  One wave per head keeps its W_K and W_V
// columns in registers for the whole (persistent) kernel.  The projection's
// result registers are exactly the attention's operand order (see the layout
// note at the top), so they are converted to fp16 in place and fed to the
// score and P.V MFMAs.
//
// The workgroup walks its units' blocks as one stream.  X blocks arrive by
// direct global-to-LDS loads into a ring of kStages tiles (3 for NG = 2), one fewer blocks
// ahead of the one in use (each wave loads two 1 KB segments of a block and
// waits only for its own older loads; one barrier per block publishes the
// tile and frees the slot read in the previous block).  A unit's queries
// arrive the same way, one block ahead of the unit's first block, into one
// of two LDS areas per wave (its head's slice).  No other global load is
// issued inside the loop, so nothing else waits on the loads in flight.
//
// The per-block work is MFMA-heavy (the projection: 2 KS MFMAs per wave) and
// then VALU-heavy (the softmax).  The two waves that share a SIMD run it
// half a block out of phase: a wave of phase 0 projects block k and attends
// to it; a wave of phase 1 first attends to block k - 1 (its K/V kept in
// registers across the barrier), then projects block k.  So while one wave
// of a SIMD is in its softmax, the other keeps the matrix core busy.  The
// phase comes from each wave's rank among the workgroup's waves on its SIMD
// (hardware SIMD id), whatever order the dispatcher assigned them in.
constexpr int kStages = 4;
constexpr int kSegPitch = 1024 + 16;  // one direct-load segment (64 lanes x 16 B) plus padding

// The value unchanged, but opaque to the compiler: quantities derived from it
// are recomputed where used instead of being hoisted out of the loop and kept
// live (or spilled) across it.
__device__ __forceinline__ int opaque(int v) {
  asm volatile("" : "+v"(v));
  return v;
}

template <int D, int NG>
__global__ __launch_bounds__(64 * (D / 32)) void fused_kernel(const Unit* __restrict__ units,
                                                              const WsHeader* __restrict__ hdr,
                                                              const f16x8* __restrict__ QN,
                                                              const bf16_bits* __restrict__ X, int64_t n_hist,
                                                              const bf16x8* __restrict__ WkP,
                                                              const bf16x8* __restrict__ WvP, int layer,
                                                              float* __restrict__ part_acc,
                                                              float2* __restrict__ part_ml, int64_t n_tgt) {
  constexpr int H = D / DH;
  constexpr int KS = D / 16;
  constexpr int CPR = D / 8;        // 16-byte chunks per history row
  constexpr int RPS = 64 / CPR;     // rows per 1 KB segment
  constexpr int NS = 32 / RPS;      // segments per block (2 per wave)
  constexpr int TILE = NS * kSegPitch;
  constexpr int QA = NG * 32 * DH * 2;  // one wave's query slice of a unit (bytes)
  // NG = 1 keeps the unit's queries in registers from its first block on (two
  // query areas suffice); NG = 2 reads them from LDS at every attention step
  // (16 fewer VGPRs), so a unit's area must outlive its last step: three
  // areas, and a ring of three tiles to stay within the LDS
  constexpr bool QREG = NG == 1;
  constexpr int NQA = QREG ? 2 : 3;
  constexpr int STG = QREG ? kStages : 3;
  static_assert(NS == 2 * H, "two segments per wave");
  __shared__ __attribute__((aligned(16))) unsigned char xs[STG * TILE];
  __shared__ __attribute__((aligned(16))) unsigned char qs[NQA * H * QA];
  __shared__ int simd_waves[4];

  // this width's units: [0, n_narrow) or [n_narrow, n_units)
  const int ub = NG == 1 ? 0 : hdr->n_narrow;
  const int ue = NG == 1 ? hdr->n_narrow : hdr->n_units;
  if (ub + static_cast<int>(blockIdx.x) >= ue) return;
  const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int tcol = lane % 32, hi = lane / 32;

  if (threadIdx.x < 4) simd_waves[threadIdx.x] = 0;
  __syncthreads();
  int phase;
  {
    int simd;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_HW_ID, 4, 2)" : "=s"(simd));
    int rank = 0;
    if (lane == 0) rank = atomicAdd(&simd_waves[simd & 3], 1);
    phase = __shfl(rank, 0) & 1;
  }

  bf16x8 wk[KS], wv[KS];
  {
    const bf16x8* pk = WkP + ((int64_t)(layer * H + wave) * KS) * 64 + lane;
    const bf16x8* pv = WvP + ((int64_t)(layer * H + wave) * KS) * 64 + lane;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      wk[ks] = pk[ks * 64];
      wv[ks] = pv[ks * 64];
    }
  }

  // ---- loads: this wave's parts of the ring's blocks and of the query slices
  int lu = ub + blockIdx.x;  // load cursor: next (unit, block) to bring in
  Unit lun = units[lu];
  int lb = lun.b0;
  int p_load = 0;   // blocks issued so far
  int q_after = 0;  // blocks issued after the latest query slice
  auto issue_x = [&]() {
    if (lu >= ue) return;
    unsigned char* slot = xs + (p_load % STG) * TILE;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int seg = 2 * wave + i;
      const int e = seg * 64 + lane;  // 16-byte chunk of the block
      const int64_t grow = min((int64_t)lb * 32 + e / CPR, n_hist - 1);
      dma16(X + grow * D + (e % CPR) * 8, slot + seg * kSegPitch);
    }
    ++p_load;
    ++q_after;
    if (++lb >= lun.b1) {
      lu += gridDim.x;
      if (lu < ue) {
        lun = units[lu];
        lb = lun.b0;
      }
    }
  };
  // queries of unit un (the ord-th of this workgroup): target rows of 64 bytes
  // (this head's 32 fp16, QN order), 16 targets per wave load
  auto issue_q = [&](const Unit& un, int ord) {
    unsigned char* area = qs + ((ord % NQA) * H + wave) * QA;
    const int ql = QREG ? lane : opaque(lane);
#pragma unroll
    for (int i = 0; i < 2 * NG; ++i) {
      const int64_t t = min((int64_t)un.t0 + i * 16 + ql / 4, n_tgt - 1);
      dma16(reinterpret_cast<const unsigned char*>(QN) + (t * D + wave * DH) * 2 + (ql % 4) * 16, area + i * 1024);
    }
    q_after = 0;
  };
  issue_q(lun, 0);
#pragma unroll
  for (int i = 0; i < STG - 1; ++i) issue_x();
  wait_vm(0);  // the weights are in registers (the loop issues no compiler-visible load)

  // this lane's B operand row: MFMA column tcol reads history row blk_row<RPS>(tcol)
  const int xrow = (tcol % NS) * kSegPitch + (tcol / NS) * (2 * D) + 16 * hi;
  // The X operands are read kXAhead k-steps ahead of their MFMAs (scheduling
  // barriers keep the compiler from sinking the reads next to their use), so
  // an LDS round trip overlaps 2 kXAhead MFMAs of the same wave.
  constexpr int kXAhead = NG == 1 ? 4 : 2;
  auto project = [&](const unsigned char* tile, f16x8 (&kv)[4]) {
    f32x16 ak = {}, av = {};
    const unsigned char* xp = tile + xrow;
    bf16x8 xo[kXAhead];
#pragma unroll
    for (int i = 0; i < kXAhead; ++i) xo[i] = *reinterpret_cast<const bf16x8*>(xp + 32 * i);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const bf16x8 x = xo[ks % kXAhead];
      if (ks + kXAhead < KS) xo[ks % kXAhead] = *reinterpret_cast<const bf16x8*>(xp + 32 * (ks + kXAhead));
      ak = mfma(wk[ks], x, ak);  // K^T block: rows = head dims, cols = history rows
      av = mfma(x, wv[ks], av);  // V block:   rows = history rows, cols = head dims
      __builtin_amdgcn_sched_barrier(0);
    }
    kv[0] = pack8h(ak, 0);
    kv[1] = pack8h(ak, 8);
    kv[2] = pack8h(av, 0);
    kv[3] = pack8h(av, 8);
  };

  // One wave's walk over the stream; PHASE 1 attends to each block one barrier
  // step after projecting it.  Every wave passes the same number of barriers.
  auto run = [&](auto phase_tag) {
    constexpr int PHASE = decltype(phase_tag)::value;
    Online<H, NG> st;
    auto load_q = [&](const Unit& un, int ord) {
      const unsigned char* area = qs + ((ord % NQA) * H + wave) * QA;
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        const int tt = g * 32 + tcol;
        const bool ok = tt < un.nt;
        const f16x8* q = reinterpret_cast<const f16x8*>(area + tt * 64);
        st.qop[g][0] = ok ? q[hi] : zero8h();
        st.qop[g][1] = ok ? q[2 + hi] : zero8h();
      }
    };
    auto init = [&](const Unit& un, int ord) {
      if (QREG) load_q(un, ord);
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        st.O[g] = f32x16{};
        st.m[g] = -INFINITY;
        st.l[g] = 0.f;
      }
    };
    // The matrix core issues the ready MFMA of the oldest wave first, so a
    // projection (32 back-to-back MFMAs at D = 256) would hold off the other
    // wave's few score and P.V MFMAs and leave both waves in their softmax at
    // the same time.  The attention step runs at raised wave priority: its
    // MFMAs go first and its VALU work overlaps the other wave's projection.
    auto attend = [&](const f16x8 (&kv)[4], int b, const Unit& un, int ord) {
      __builtin_amdgcn_s_setprio(1);
      if (QREG) {
        st.template step<RPS>(kv, b, un, hi);
      } else {
        const unsigned char* area = qs + ((ord % NQA) * H + wave) * QA;
        st.template step<RPS>(kv, b, un, hi, [&](int g, f16x8 (&q)[2]) {
          const int tt = g * 32 + opaque(tcol);
          const bool ok = tt < un.nt;
          const f16x8* qp = reinterpret_cast<const f16x8*>(area + tt * 64);
          q[0] = ok ? qp[hi] : zero8h();
          q[1] = ok ? qp[2 + hi] : zero8h();
        });
      }
      __builtin_amdgcn_s_setprio(0);
    };
    auto fin = [&](const Unit& un) {
      if (QREG)
        st.finish(un, wave, tcol, hi, part_acc, part_ml, n_tgt);
      else
        st.finish(un, opaque(wave), opaque(tcol), opaque(hi), part_acc, part_ml, n_tgt);
    };
    int cu = ub + blockIdx.x;  // compute cursor: unit index, its ordinal, block
    int ck = 0;
    Unit cun = units[cu];
    int cb = cun.b0;
    f16x8 held[4];  // PHASE 1: K/V of block hb of unit hun (ordinal hk), attended to in the next step
    Unit hun = cun;
    int hb = -1, hk = 0;
    for (int p_use = 0; cu < ue; ++p_use) {
      const bool first = cb == cun.b0, last = cb + 1 == cun.b1;
      // this wave's part of block p_use (and, at a unit's first block, of its
      // queries, issued one block earlier) has landed
      const int ahead = 2 * (p_load - 1 - p_use);
      wait_vm(first ? min(ahead, 2 * q_after) : ahead);
      ring_barrier();  // everyone's parts; the slot of p_use - 1 is free
      if (last && cu + static_cast<int>(gridDim.x) < ue) issue_q(units[cu + gridDim.x], ck + 1);
      if (p_load < p_use + STG) issue_x();
      const unsigned char* tile = xs + (p_use % STG) * TILE;
      if (PHASE == 0) {
        if (first) init(cun, ck);
        f16x8 kv[4];
        project(tile, kv);
        attend(kv, cb, cun, ck);
        if (last) fin(cun);
      } else {
        if (hb >= 0) {
          attend(held, hb, hun, hk);
          if (hb + 1 == hun.b1) fin(hun);
        }
        if (first) init(cun, ck);
        project(tile, held);
        hun = cun;
        hb = cb;
        hk = ck;
      }
      if (last) {
        cu += gridDim.x;
        ++ck;
        if (cu < ue) {
          cun = units[cu];
          cb = cun.b0;
        }
      } else {
        ++cb;
      }
    }
    if (PHASE == 1 && hb >= 0) {
      attend(held, hb, hun, hk);
      fin(hun);
    }
  };
  if (phase == 0)
    run(std::integral_constant<int, 0>{});
  else
    run(std::integral_constant<int, 1>{});
}

// ------------------------------------------------ K4: target update
// One workgroup per tg = 32 targets (or 16, when 32-target groups would leave
// CUs idle: the MFMA tiles then carry 16 empty target columns, and each CU
// still streams every weight of the layer once), one wave per 32 output
// dimensions.
// mode 0 (init): s^(0) = x_t, Q^(0) = x_t W_Q^0.
// mode 1 (layer i): merge the attention partials into a, then
//   u = s + a W_O;  s' = u + ReLU(u W_1) W_2;  Q' = s' W_Q^{i+1} (if i+1 < n).
// Activations go through LDS as fp16 MFMA operands; the state stays fp32.
struct UpdateArgs {
  int mode, layer, n_layers, F;
  int64_t n_tgt;
  const bf16_bits* tgt;        // mode 0
  const int32_t* tchunks;      // mode 1
  const float* part_acc;       // mode 1
  const float2* part_ml;       // mode 1
  const float* s_in;           // mode 1: layer input state
  float* s_out;                // next state (fp32)
  float* save_a;               // nullable [n_tgt][D]
  float* save_u;               // nullable
  float* save_lse;             // nullable [n_tgt][H]
  bf16_bits* out;              // final layer output, nullable
  f16x8* QN;                   // next queries
  const f16x8 *WoP, *W1P, *W2P, *WqP;  // packed (fp16), all layers
  int tg;                      // targets per workgroup (16 or 32)
  int32_t* range;              // written 1 when a value rounded to fp16 is out of its range
};

template <int D, int NC>
__global__ __launch_bounds__(64 * (D / 32)) void update_kernel(UpdateArgs A) {
  constexpr int NW = D / 32;
  constexpr int H = D / DH;
  constexpr int KS = D / 16;
  constexpr int AROW = D + 8;
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];  // fp16 MFMA operands
  uint16_t* act = lds;                  // [32][AROW]
  uint16_t* hid = lds + 32 * AROW;      // [32][AROW]: D hidden columns at a time
  const int w = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int tcol = lane % 32, hi = lane / 32;
  const int tg = A.tg;  // rows tg..31 of the 32-row tiles stay zero
  const int64_t tb = (int64_t)blockIdx.x * tg;
  const int64_t t = tb + tcol;
  const bool tok = tcol < tg && t < A.n_tgt;
  auto live = [&](int row) { return row < tg && tb + row < A.n_tgt; };
  // fp16 range check of every value this thread rounds to fp16 (and of the
  // merged attention output, where an overflowed K or V shows as a
  // non-finite value); NaN fails the comparison as well
  // (a running maximum of the bits of |x| as an unsigned integer: every
  // finite value orders below the infinity and every NaN above it, so one
  // register remembers the largest and any non-finite value)
  uint32_t big = 0;
  auto chk = [&](float x) { big = max(big, __float_as_uint(fabsf(x))); };
  auto report = [&]() {
    if (big > __float_as_uint(kF16Max)) *A.range = 1;
  };

  // fp32 result of D^T tile: lane holds dims 32w + 4hi + 8g + k for g, k < 4
  auto store_f32 = [&](float* dst, const f32x16& v) {
    float* p = dst + t * D + 32 * w + 4 * hi;
#pragma unroll
    for (int g = 0; g < 4; ++g)
      *reinterpret_cast<float4*>(p + 8 * g) = make_float4(v[4 * g], v[4 * g + 1], v[4 * g + 2], v[4 * g + 3]);
  };
  auto put_act = [&](uint16_t* buf, int col0, const f32x16& v) {
    uint16_t* p = buf + tcol * AROW + col0 + 4 * hi;
#pragma unroll
    for (int i = 0; i < 16; ++i) chk(v[i]);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      uint2 pk;
      pk.x = (uint32_t)f16_bits(v[4 * g]) | ((uint32_t)f16_bits(v[4 * g + 1]) << 16);
      pk.y = (uint32_t)f16_bits(v[4 * g + 2]) | ((uint32_t)f16_bits(v[4 * g + 3]) << 16);
      *reinterpret_cast<uint2*>(p + 8 * g) = pk;
    }
  };
  // Every product of the update is one 32 x 32 tile per wave with KS k-steps:
  // acc = W^T act^T.  With NC (hidden chunks, F / D) known at compile time,
  // its weight operands (one KS-step tile, from L2) are loaded one product
  // ahead into the other of two register sets, so an L2 round trip overlaps
  // the previous product instead of preceding its own; a register set is
  // refilled after an instruction that reads the result of the product that
  // used it.  The chunk loop is then fully unrolled: the same prefetch in a
  // loop with a run-time trip count gave wrong results.  NC = 0 (any other
  // F) loads each product's weights right before it.
  f16x8 wa[KS], wb[KS];
  auto fetch = [&](f16x8 (&r)[KS], const f16x8* Wp) {
#pragma unroll
    for (int k = 0; k < KS; ++k) r[k] = Wp[k * 64 + lane];
  };
  auto gemm = [&](const f16x8 (&r)[KS], const uint16_t* src) {
    const uint16_t* b = src + tcol * AROW + 8 * hi;
    f32x16 acc = {};
#pragma unroll
    for (int k = 0; k < KS; ++k) acc = mfma(r[k], *reinterpret_cast<const f16x8*>(b + k * 16), acc);
    return acc;
  };
  auto gemm_from = [&](const f16x8* Wp, const uint16_t* src) {
    f16x8 r[KS];
    fetch(r, Wp);
    return gemm(r, src);
  };
  constexpr bool PF = NC > 0;
  const int nc = PF ? NC : A.F / D;  // hidden chunks of D columns
  const int KSF = A.F / 16;
  auto w1_tile = [&](int c) { return A.W1P + ((int64_t)A.layer * (A.F / 32) + c * NW + w) * KS * 64; };
  auto w2_tile = [&](int c) { return A.W2P + ((int64_t)(A.layer * NW + w) * KSF + c * KS) * 64; };
  auto wq_tile = [&](int ql) { return A.WqP + ((int64_t)(ql * NW + w) * KS) * 64; };

  if (A.mode == 0) {
    fetch(wb, wq_tile(0));
    // stage x_t rows into LDS (fp16) and write s^(0) (fp32)
    for (int c = threadIdx.x; c < 32 * D / 8; c += 64 * NW) {
      const int row = c / (D / 8), col8 = c % (D / 8);
      uint4 v = make_uint4(0, 0, 0, 0);
      if (live(row)) v = *reinterpret_cast<const uint4*>(A.tgt + (tb + row) * D + col8 * 8);
      const bf16_bits* e = reinterpret_cast<const bf16_bits*>(&v);
      uint16_t* a8 = act + row * AROW + col8 * 8;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        chk(to_f32(e[i]));
        a8[i] = f16_bits(to_f32(e[i]));
      }
      if (live(row)) {
        float* so = A.s_out + (tb + row) * D + col8 * 8;
#pragma unroll
        for (int i = 0; i < 8; ++i) so[i] = to_f32(e[i]);
      }
    }
    __syncthreads();
  } else {
    fetch(wa, A.WoP + ((int64_t)(A.layer * NW + w) * KS) * 64);
    // merge partials: two threads per (target, head), 16 dimensions each.
    // Every chunk's (max, sum) is requested at once and the accumulators four
    // chunks at a time, so the merge costs a few memory round trips.
    {
      const int pair = threadIdx.x >> 1, half = threadIdx.x & 1;
      const int row = pair / H, j = pair % H;
      const int64_t tt = tb + row;
      float av[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) av[i] = 0.f;
      if (live(row)) {
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
            const float wgt = wc[c0 + cc];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              av[4 * q] += wgt * x[cc][q].x;
              av[4 * q + 1] += wgt * x[cc][q].y;
              av[4 * q + 2] += wgt * x[cc][q].z;
              av[4 * q + 3] += wgt * x[cc][q].w;
            }
          }
        }
        const float inv = 1.f / L;
#pragma unroll
        for (int i = 0; i < 16; ++i) av[i] *= inv;
        if (A.save_a) {
          float4* sa = reinterpret_cast<float4*>(A.save_a + tt * D + j * DH + half * 16);
#pragma unroll
          for (int q = 0; q < 4; ++q) sa[q] = make_float4(av[4 * q], av[4 * q + 1], av[4 * q + 2], av[4 * q + 3]);
        }
        if (A.save_lse && half == 0) A.save_lse[tt * H + j] = (M + log2f(L)) * kLn2;
      }
      uint16_t* p = act + row * AROW + j * DH + half * 16;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        chk(av[i]);
        p[i] = f16_bits(av[i]);
      }
    }
    __syncthreads();
    if (PF) fetch(wb, w1_tile(0));  // after the merge, whose registers it would otherwise share
    // u = s + a W_O
    f32x16 u = gemm(wa, act);
    if (tok) {
      const float* sp = A.s_in + t * D + 32 * w + 4 * hi;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const float4 sv = *reinterpret_cast<const float4*>(sp + 8 * g);
        u[4 * g] += sv.x; u[4 * g + 1] += sv.y; u[4 * g + 2] += sv.z; u[4 * g + 3] += sv.w;
      }
      if (A.save_u) store_f32(A.save_u, u);
    }
    __syncthreads();
    put_act(act, 32 * w, u);
    __builtin_amdgcn_sched_barrier(0);
    if (PF) fetch(wa, w2_tile(0));
    __syncthreads();
    // s' = u + ReLU(u W_1) W_2, the hidden layer taken D columns at a time
    f32x16 s_next = u;
    const int ql = A.layer + 1 < A.n_layers ? A.layer + 1 : -1;
#pragma unroll
    for (int c = 0; c < (PF ? NC : nc); ++c) {
      f32x16 h = PF ? gemm(wb, act) : gemm_from(w1_tile(c), act);  // this wave's 32 hidden columns of chunk c
#pragma unroll
      for (int v = 0; v < 16; ++v) h[v] = fmaxf(h[v], 0.f);
      __builtin_amdgcn_sched_barrier(0);
      if (PF) {
        if (c + 1 < nc)
          fetch(wb, w1_tile(c + 1));
        else if (ql >= 0)
          fetch(wb, wq_tile(ql));
      }
      put_act(hid, 32 * w, h);
      __syncthreads();
      const f32x16 y = PF ? gemm(wa, hid) : gemm_from(w2_tile(c), hid);
#pragma unroll
      for (int v = 0; v < 16; ++v) s_next[v] += y[v];
      __builtin_amdgcn_sched_barrier(0);
      if (PF && c + 1 < nc) fetch(wa, w2_tile(c + 1));
      __syncthreads();
    }
    if (tok) {
      if (ql >= 0) {
        store_f32(A.s_out, s_next);
      } else {
        bf16_bits* p = A.out + t * D + 32 * w + 4 * hi;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          uint2 pk;
          pk.x = (uint32_t)from_f32<bf16_bits>(s_next[4 * g]) |
                 ((uint32_t)from_f32<bf16_bits>(s_next[4 * g + 1]) << 16);
          pk.y = (uint32_t)from_f32<bf16_bits>(s_next[4 * g + 2]) |
                 ((uint32_t)from_f32<bf16_bits>(s_next[4 * g + 3]) << 16);
          *reinterpret_cast<uint2*>(p + 8 * g) = pk;
        }
      }
    }
    if (ql < 0) {
      report();
      return;
    }
    put_act(act, 32 * w, s_next);  // act (u) was last read before the previous barrier
    __syncthreads();
  }
  // next queries: Q = s W_Q^{next}, scaled into log2 units, permuted (QN layout)
  f32x16 q = PF || A.mode == 0 ? gemm(wb, act) : gemm_from(wq_tile(A.layer + 1), act);
  const float qs = kLog2e * 0.17677669529663687f;  // log2(e) / sqrt(32)
#pragma unroll
  for (int v = 0; v < 16; ++v) q[v] *= qs;
  if (tok) {
#pragma unroll
    for (int v = 0; v < 16; ++v) chk(q[v]);
    f16x8* qn = A.QN + (t * D + 32 * w) / 8;
    qn[hi] = pack8h(q, 0);
    qn[2 + hi] = pack8h(q, 8);
  }
  report();
}

}  // namespace

// ------------------------------------------------------------ launchers
hipError_t fast_pack(const void* W, void* P, int n_layers, int K, int N, int to_f16, hipStream_t st) {
  const int64_t groups = (int64_t)(N / 32) * (K / 16) * 64;
  dim3 g(static_cast<unsigned>(ceil_div(groups, 256)), n_layers);
  if (to_f16)
    hipLaunchKernelGGL(pack_kernel<f16x8>, g, dim3(256), 0, st, (const bf16_bits*)W, (f16x8*)P, K, N, groups);
  else
    hipLaunchKernelGGL(pack_kernel<bf16x8>, g, dim3(256), 0, st, (const bf16_bits*)W, (bf16x8*)P, K, N, groups);
  return hipGetLastError();
}

hipError_t fast_pack_many(const PackJobs& jobs, int n_jobs, int n_layers, hipStream_t st) {
  if (n_jobs < 1 || n_jobs > kMaxPackJobs) return hipErrorInvalidValue;
  int64_t groups = 0;
  for (int j = 0; j < n_jobs; ++j)
    groups = std::max<int64_t>(groups, (int64_t)(jobs.job[j].N / 32) * (jobs.job[j].K / 16) * 64);
  dim3 g(static_cast<unsigned>(ceil_div(groups, 256)), n_layers, n_jobs);
  hipLaunchKernelGGL(pack_many_kernel, g, dim3(256), 0, st, jobs);
  return hipGetLastError();
}

int fast_proj_parts(int n_layers, int64_t n_blocks, int n_cu) {
  // workgroups = n_layers * parts; parts a multiple of 8 (XCD grouping), about
  // one resident workgroup per CU, and at least one block per part
  int64_t parts = round_up(ceil_div(n_cu, n_layers), 8);
  while (parts > 8 && parts > n_blocks) parts -= 8;
  return static_cast<int>(parts);
}

hipError_t fast_proj(int D, const void* X, int64_t n_hist, int64_t n_blocks, const void* WkP, const void* WvP,
                     void* KV, int n_layers, int parts, hipStream_t st) {
  dim3 g(static_cast<unsigned>(n_layers * parts));
#define STCA_PROJ(DD)                                                                                       \
  hipLaunchKernelGGL(proj_kernel<DD>, g, dim3(64 * (DD / 32)), 0, st, (const bf16_bits*)X, n_hist, n_blocks, \
                     (const bf16x8*)WkP, (const bf16x8*)WvP, (f16x8*)KV, n_layers, parts)
  switch (D) {
    case 64: STCA_PROJ(64); break;
    case 128: STCA_PROJ(128); break;
    case 256: STCA_PROJ(256); break;
    default: return hipErrorInvalidValue;
  }
#undef STCA_PROJ
  return hipGetLastError();
}

hipError_t fast_attn(int D, const Unit* units, const WsHeader* hdr, int grid, const void* QN, const void* KVl,
                     float* part_acc, void* part_ml, int64_t n_tgt, hipStream_t st) {
  if (grid == 0) return hipSuccess;
#define STCA_ATTN(HH)                                                                                \
  hipLaunchKernelGGL(attn_kernel<HH>, dim3(grid), dim3(64 * HH), 0, st, units, hdr, (const f16x8*)QN, \
                     (const f16x8*)KVl, part_acc, (float2*)part_ml, n_tgt)
  switch (D) {
    case 64: STCA_ATTN(2); break;
    case 128: STCA_ATTN(4); break;
    case 256: STCA_ATTN(8); break;
    default: return hipErrorInvalidValue;
  }
#undef STCA_ATTN
  return hipGetLastError();
}

hipError_t fast_fused(int D, int wide, const Unit* units, const WsHeader* hdr, int grid, const void* QN,
                      const void* X, int64_t n_hist, const void* WkP, const void* WvP, int layer, float* part_acc,
                      void* part_ml, int64_t n_tgt, hipStream_t st) {
  if (grid == 0) return hipSuccess;
#define STCA_FUSED1(DD, NG)                                                                                  \
  hipLaunchKernelGGL((fused_kernel<DD, NG>), dim3(grid), dim3(64 * (DD / 32)), 0, st, units, hdr,                \
                     (const f16x8*)QN, (const bf16_bits*)X, n_hist, (const bf16x8*)WkP, (const bf16x8*)WvP, layer, \
                     part_acc, (float2*)part_ml, n_tgt)
#define STCA_FUSED(DD) \
  if (wide) STCA_FUSED1(DD, 2); else STCA_FUSED1(DD, 1)
  switch (D) {
    case 64: STCA_FUSED(64); break;
    case 128: STCA_FUSED(128); break;
    case 256: STCA_FUSED(256); break;
    default: return hipErrorInvalidValue;
  }
#undef STCA_FUSED
#undef STCA_FUSED1
  return hipGetLastError();
}

hipError_t fast_update(int D, const FastUpdate& f, hipStream_t st) {
  UpdateArgs A;
  A.mode = f.mode;
  A.layer = f.layer;
  A.n_layers = f.n_layers;
  A.F = f.F;
  A.n_tgt = f.n_tgt;
  A.tgt = (const bf16_bits*)f.tgt;
  A.tchunks = f.tchunks;
  A.part_acc = f.part_acc;
  A.part_ml = (const float2*)f.part_ml;
  A.s_in = f.s_in;
  A.s_out = f.s_out;
  A.save_a = f.save_a;
  A.save_u = f.save_u;
  A.save_lse = f.save_lse;
  A.out = (bf16_bits*)f.out;
  A.QN = (f16x8*)f.QN;
  A.WoP = (const f16x8*)f.WoP;
  A.W1P = (const f16x8*)f.W1P;
  A.W2P = (const f16x8*)f.W2P;
  A.WqP = (const f16x8*)f.WqP;
  A.tg = f.tg == 16 ? 16 : 32;
  A.range = f.range;
  if (f.n_tgt == 0) return hipSuccess;
  if (!f.range) return hipErrorInvalidValue;
  dim3 g(static_cast<unsigned>(ceil_div(f.n_tgt, A.tg)));
  const size_t lds = (size_t)32 * (D + 8) * 2 * (f.mode == 0 ? 1 : 2);
#define STCA_UPD(DD)                                                                         \
  if (f.F == 4 * (DD))                                                                      \
    hipLaunchKernelGGL((update_kernel<DD, 4>), g, dim3(64 * (DD / 32)), lds, st, A);        \
  else                                                                                      \
    hipLaunchKernelGGL((update_kernel<DD, 0>), g, dim3(64 * (DD / 32)), lds, st, A)
  switch (D) {
    case 64: STCA_UPD(64); break;
    case 128: STCA_UPD(128); break;
    case 256: STCA_UPD(256); break;
    default: return hipErrorInvalidValue;
  }
#undef STCA_UPD
  return hipGetLastError();
}

}  // namespace stca
