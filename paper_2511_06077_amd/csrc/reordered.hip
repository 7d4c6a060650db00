// Reordered single-query attention under RLB (App. A.2.2, Eq. attn-optimized)
// for requests with few targets, bf16 storage, d_h = 32.
//
// Per target t and head j the score of history row x is
//   q_tj . (x W_K^j) = (q_tj W_K^j^T) . x = u_tj . x,
// and the head output is a_tj = (sum_l p_tjl x_l) W_V^j = y_tj W_V^j.  With
// u_tj formed once per (target, head) on the target side, the history is
// read as it is: no K or V exists, and a request's work on its history is
// 4 (m h) L d flop instead of the projection's 4 L d^2 + 4 m L d.  With few
// targets (m h < d) that is far less, and the pass is bound by one read of X
// per layer.
//
//   reord_qu_kernel:    U[t][j][:] = Q[t][head j] W_K^j^T (fp16, scaled as Q)
//   reord_attn_kernel:  per unit, rows (t, j) of up to 32: S^T = X U^T,
//                       online softmax, Y^T += X^T P^T; partial y per chunk
//   reord_merge_kernel: y_tj = merged partials, a_tj = y_tj W_V^j (fp32),
//                       handed to the target update as a single chunk
//
// MFMA lane layouts are those of v_mfma_f32_32x32x16_bf16 (see fast.hip).
// X enters every product as the bf16 it is stored in, with no conversion.
// The other operands, U and the softmax weights P, are fp32 values carried
// as two bf16 terms (hi = bf16(v), lo = bf16(v - hi), about 16 significant
// bits), each product taken twice: more precise than one fp16 operand, and
// cheaper than converting X.
#include "common.h"
#include "fast.h"
#include "ring.h"

namespace stca {

namespace {

constexpr int DH = 32;
constexpr float kSlack = 8.f;  // log2 units: softmax weights stay <= 256 between rescales
constexpr int kWaves = 4;      // X blocks per round of the attention workgroup (two waves each)

// X tile in LDS: the 32 rows in 1 KB segments (512 / D rows each, as one
// wave's direct global-to-LDS load fills them), segments padded by 16 bytes,
// which spreads the rows over the banks while keeping every operand address
// a per-lane base plus a compile-time offset.
constexpr int kSegPitch = 1024 + 16;
__host__ __device__ constexpr size_t reord_tile_bytes(int D) { return (size_t)(D / 16) * kSegPitch; }
// attention kernel LDS: the pairs' double-buffered X tiles (later the merge
// area), then the unit's U rows
__host__ __device__ constexpr size_t reord_main_lds(int D) {
  return (size_t)kWaves * 2 * reord_tile_bytes(D) > (size_t)kWaves * 32 * (D + 2) * 4
             ? (size_t)kWaves * 2 * reord_tile_bytes(D)
             : (size_t)kWaves * 32 * (D + 2) * 4;
}

__device__ __forceinline__ f32x16 mfma16(const f16x8& a, const f16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mfmab(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// v ~ hi + lo, both bf16 (round to nearest even)
__device__ __forceinline__ __bf16 bf_hi(float v) { return static_cast<__bf16>(v); }
__device__ __forceinline__ __bf16 bf_lo(float v, __bf16 hi) { return static_cast<__bf16>(v - static_cast<float>(hi)); }

__device__ __forceinline__ bf16x8 zero8b() {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = static_cast<__bf16>(0.f);
  return r;
}

__device__ __forceinline__ f16x8 pack8(const f32x16& a, int off) {
  f16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = static_cast<_Float16>(a[off + i]);
  return r;
}

__device__ __forceinline__ f16x8 zero8() {
  f16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = static_cast<_Float16>(0.f);
  return r;
}

__device__ __forceinline__ _Float16 bf_to_h(bf16_bits x) { return static_cast<_Float16>(to_f32(x)); }

__device__ __forceinline__ f16x8 bf8_to_h8(const uint4& v) {
  const bf16_bits* e = reinterpret_cast<const bf16_bits*>(&v);
  f16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = bf_to_h(e[i]);
  return r;
}

// ------------------------------------------------------------------- U
// One wave per (32 targets, head j).  U^T tile (32 model dims x 32 targets) =
// W_K^j (dims x head dims) Q_j^T: the B operand is the wave's slice of the
// permuted QN row (k-step s holds head dims 16 s + 4 hi + {0..3, 8..11}), the A
// operand W_K[dim][32 j + the same head dims].
// Targets with a zero chunk count in `tchunks` (requests in the standard form
// when a batch runs both forms) get no U; a wave whose 32 targets have none
// to form exits.
template <int D>
__global__ __launch_bounds__(64) void reord_qu_kernel(const f16x8* __restrict__ QN, const bf16_bits* __restrict__ Wk,
                                                      __bf16* __restrict__ UN, const int32_t* __restrict__ tchunks,
                                                      int64_t n_tgt) {
  constexpr int H = D / DH;
  const int j = blockIdx.y;
  const int lane = threadIdx.x;
  const int tcol = lane % 32, hi = lane / 32;
  const int64_t t = (int64_t)blockIdx.x * 32 + tcol;
  const bool live = t < n_tgt && tchunks[t] > 0;
  if (__builtin_amdgcn_ballot_w64(live) == 0) return;
  f16x8 qb[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) qb[s] = live ? QN[(t * D + 32 * j + 16 * s + 8 * hi) / 8] : zero8();
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt) {
    const int dim = 32 * dt + tcol;
    f32x16 acc = {};
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const bf16_bits* w = Wk + (int64_t)dim * D + 32 * j + 16 * s + 4 * hi;
      const ushort4 lo4 = *reinterpret_cast<const ushort4*>(w);
      const ushort4 hi4 = *reinterpret_cast<const ushort4*>(w + 8);
      f16x8 a;
      a[0] = bf_to_h(lo4.x), a[1] = bf_to_h(lo4.y), a[2] = bf_to_h(lo4.z), a[3] = bf_to_h(lo4.w);
      a[4] = bf_to_h(hi4.x), a[5] = bf_to_h(hi4.y), a[6] = bf_to_h(hi4.z), a[7] = bf_to_h(hi4.w);
      acc = mfma16(a, qb[s], acc);
    }
    // lane holds U[t][j][32 dt + 8 g + 4 hi + k] for g, k < 4; row (t, j) of
    // UN holds the hi terms, then the lo terms
    if (live) {
      __bf16* u = UN + (t * H + j) * 2 * D + 32 * dt + 4 * hi;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        typedef __bf16 b4 __attribute__((ext_vector_type(4)));
        b4 h, l;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          h[k] = bf_hi(acc[4 * g + k]);
          l[k] = bf_lo(acc[4 * g + k], h[k]);
        }
        *reinterpret_cast<b4*>(u + 8 * g) = h;
        *reinterpret_cast<b4*>(u + D + 8 * g) = l;
      }
    }
  }
}

// ------------------------------------------------------------ attention
// One workgroup per unit (request, target group of up to 32 / H targets,
// history chunk): its rows r = t H + j (at most 32) are the 32 columns of
// every tile.  Eight waves in four pairs; in each round the pairs take the
// next four 32-row X blocks (direct global-to-LDS loads into a per-pair
// double buffer, the next round's blocks in flight while this round's are
// used).  Both waves of a pair form
// the block's scores; each accumulates half of the d columns of Y.  Every
// pair keeps its own online-softmax state; the pairs' partials are merged at
// the end.
//   S^T (32 history rows x 32 rows (t, j)) = X U^T, K = d: A = X row operand,
//   B = U rows (staged once in LDS).
//   Y^T (d x 32) += X^T P^T, K = 32 history rows: B = P^T from the S^T
//   registers (k-step s: rows 16 s + 4 hi + {0..3, 8..11}), A = X^T gathered
//   from the LDS tile for the same history rows.
template <int D>
__global__ __launch_bounds__(128 * kWaves) void reord_attn_kernel(const Unit* __restrict__ units,
                                                                  const WsHeader* __restrict__ hdr,
                                                                  const __bf16* __restrict__ UN,
                                                                  const bf16_bits* __restrict__ X, int64_t n_hist,
                                                                  float* __restrict__ part_y,
                                                                  float2* __restrict__ part_ml, int64_t n_tgt) {
  constexpr int H = D / DH;
  constexpr int KS = D / 16;
  constexpr int CPR = D / 8;          // 16-byte chunks per X row
  constexpr int NDT = D / 32;         // 32-dim tiles of Y^T
  constexpr int HALF = NDT / 2;       // tiles per wave of a pair
  constexpr int PER = 32 * CPR / 64;  // 1 KB segments per block
  constexpr int RPS = 512 / D;        // rows per segment
  constexpr int NT = 128 * kWaves;
  constexpr int TB = static_cast<int>(reord_tile_bytes(D));
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int u = blockIdx.x;
  if (u >= hdr->n_units) return;
  const Unit un = units[u];
  const int w = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int pw = w % kWaves, half = w / kWaves;
  const int tcol = lane % 32, hi = lane / 32;
  const int R = un.nt * H;
  unsigned char* xb = smem + (size_t)pw * 2 * TB;
  // byte offset of element (row, col) in a tile
  auto xoff = [](int row, int col) { return (row / RPS) * kSegPitch + (row % RPS) * 2 * D + col * 2; };
  // the unit's U: hi terms in registers (B operand: row tcol, model dims
  // 16 ks + 8 hi ..), lo terms staged in LDS (padded rows) past the X tiles
  // and the merge area
  constexpr int UROW = D + 8;
  __bf16* us = reinterpret_cast<__bf16*>(smem + reord_main_lds(D));
  for (int e = threadIdx.x; e < 32 * (D / 8); e += NT) {
    const int row = e / (D / 8), c8 = e % (D / 8);
    const bf16x8 v = row < R ? *reinterpret_cast<const bf16x8*>(UN + ((int64_t)un.t0 * H + row) * 2 * D + D + c8 * 8)
                             : zero8b();
    *reinterpret_cast<bf16x8*>(us + row * UROW + c8 * 8) = v;
  }
  const __bf16* ulo = us + tcol * UROW + 8 * hi;
  bf16x8 uhi[KS];
  {
    const __bf16* up = UN + ((int64_t)un.t0 * H + tcol) * 2 * D + 8 * hi;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) uhi[ks] = tcol < R ? *reinterpret_cast<const bf16x8*>(up + 16 * ks) : zero8b();
  }
  f32x16 Y[HALF];
#pragma unroll
  for (int dt = 0; dt < HALF; ++dt) Y[dt] = f32x16{};
  float m = -INFINITY, l = 0.f;
  const int rounds = (un.b1 - un.b0 + kWaves - 1) / kWaves;
  // this pair's block of round r: each wave of the pair loads half of it
  auto dma = [&](int r, int buf) {
    const int b = un.b0 + r * kWaves + pw;
    if (b >= un.b1) return;
#pragma unroll
    for (int i = half * (PER / 2); i < (half + 1) * (PER / 2); ++i) {
      const int p = i * 64 + lane;
      const int row = p / CPR, c = p % CPR;
      const int64_t grow = min((int64_t)b * 32 + row, n_hist - 1);
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(X + grow * D + c * 8),
                                       (void __attribute__((address_space(3)))*)(xb + buf * TB + i * kSegPitch), 16,
                                       0, 0);
    }
  };
  dma(0, 0);
  for (int r = 0; r < rounds; ++r) {
    const int cur = r & 1;
    // round r's blocks have landed (every wave waited for its own loads), and
    // every wave is done with the buffers of round r - 1
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (r + 1 < rounds) dma(r + 1, cur ^ 1);
    const int b = un.b0 + r * kWaves + pw;
    if (b >= un.b1) continue;
    const unsigned char* xt = xb + cur * TB;
    f32x16 s = {};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const bf16x8 xr = *reinterpret_cast<const bf16x8*>(xt + xoff(tcol, 16 * ks + 8 * hi));
      s = mfmab(xr, uhi[ks], s);
      s = mfmab(xr, *reinterpret_cast<const bf16x8*>(ulo + 16 * ks), s);
    }
    if (b * 32 < un.l0 || b * 32 + 32 > un.l1) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int tok = b * 32 + 8 * (v / 4) + 4 * hi + (v % 4);
        s[v] = (tok < un.l0 || tok >= un.l1) ? -INFINITY : s[v];
      }
    }
    float bm = s[0];
#pragma unroll
    for (int v = 1; v < 16; ++v) bm = fmaxf(bm, s[v]);
    bm = fmaxf(bm, __shfl_xor(bm, 32));
    // per-lane threshold rescale: the reference max moves only when the block
    // maximum exceeds it by kSlack (every block has a valid row, so bm is finite)
    const float mn = bm > m + kSlack ? bm : m;
    const float sc = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - mn);
    m = mn;
    float ps = 0.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      s[v] = __builtin_amdgcn_exp2f(s[v] - mn);
      ps += s[v];
    }
    l = l * sc + ps;
    bf16x8 ph[2], pl[2];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const __bf16 h = bf_hi(s[i]);
      ph[i / 8][i % 8] = h;
      pl[i / 8][i % 8] = bf_lo(s[i], h);
    }
#pragma unroll
    for (int dt = 0; dt < HALF; ++dt) {
      f32x16 acc = Y[dt] * sc;
      const int dim = 32 * (half * HALF + dt) + tcol;
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        bf16x8 a;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int row = 16 * k2 + 4 * hi + (i < 4 ? i : i + 4);
          a[i] = *reinterpret_cast<const __bf16*>(xt + xoff(row, dim));
        }
        acc = mfmab(a, ph[k2], acc);
        acc = mfmab(a, pl[k2], acc);
      }
      Y[dt] = acc;
      // two gathers in flight at a time: hoisting all of them would take
      // eight registers per element
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  // merge the four pairs (the X tiles are dead: their LDS holds the partials)
  __syncthreads();
  float* red = reinterpret_cast<float*>(smem);  // [kWaves][32][D + 2]
  const float lt = l + __shfl_xor(l, 32);
  float* rw = red + ((size_t)pw * 32 + tcol) * (D + 2);
  if (hi == 0 && half == 0) {
    rw[0] = m;
    rw[1] = lt;
  }
#pragma unroll
  for (int dt = 0; dt < HALF; ++dt)
#pragma unroll
    for (int v = 0; v < 16; ++v) rw[2 + 32 * (half * HALF + dt) + 8 * (v / 4) + 4 * hi + (v % 4)] = Y[dt][v];
  __syncthreads();
  for (int it = threadIdx.x; it < R * (D + 1); it += NT) {
    const int row = it / (D + 1), e = it % (D + 1);  // e == D: (max, sum)
    float M = -INFINITY;
    for (int pp = 0; pp < kWaves; ++pp) M = fmaxf(M, red[((size_t)pp * 32 + row) * (D + 2)]);
    float val = 0.f;
    for (int pp = 0; pp < kWaves; ++pp) {
      const float* rr = red + ((size_t)pp * 32 + row) * (D + 2);
      const float f = rr[0] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(rr[0] - M);
      val += f * (e == D ? rr[1] : rr[2 + e]);
    }
    const int t = row / H, j = row % H;
    const int64_t prow = ((int64_t)un.c * n_tgt + un.t0 + t) * H + j;
    if (e == D)
      part_ml[prow] = make_float2(M, val);
    else
      part_y[prow * D + e] = val;
  }
}

// ----------------------------------------------- attention, wide units
// Units of up to 256 rows (t, j) (up to 256 / H targets of one request, all
// heads), one history chunk each: eight waves, wave w owning the rows
// [32 w, 32 w + 32) as the 32 columns of its tiles (waves past the unit's
// rows only load).  X blocks arrive by direct global-to-LDS loads into a
// ring of four tiles, three blocks ahead; each wave loads a fixed share of
// every block (whole 1 KB segments) and, once its own loads of a block have
// landed, rounds its share from bf16 to fp16 in place, one block ahead of
// its use, so that one barrier per block both publishes a converted tile and
// frees the oldest slot.  Per block and wave:
//   S^T (32 history rows x 32 rows (t, j)) = X U^T on the fp16 MFMA, K = d:
//     A = X rows (16-byte LDS reads, MFMA row i = history row blk_row(i)),
//     B = U of the wave's rows (fp16, registers);
//   online softmax per column, with the reference maximum moved only when a
//     block exceeds it by kSlack (weights <= 2^kSlack, fine in fp16);
//   Y^T (d x 32) += X^T P^T, K = 32 history rows: B = P^T straight from the
//     S^T registers (k-step s: MFMA rows 16 s + 4 hi + {0..3, 8..11}),
//     A = X^T by transposing LDS reads of the same history rows.
// The unit's partials (y per row, running max and sum) go out as chunk c
// of the reordered form's records, merged by reord_merge_kernel.
constexpr int kWideWaves = 8;
constexpr int kWideRows = 32 * kWideWaves;  // (t, j) rows a unit holds
constexpr int kWideStages = 4;

// History row of MFMA row i within a block (RPS rows per 1 KB segment,
// segments 16 bytes apart in the bank order).  The 16-byte row reads of S^T
// send lanes i = 0..15 to sixteen different segments.  At d = 256 the order
// also serves the transposing reads of Y^T: writing i = 16 s + 8 e + 4 h + k,
// the rows k = 0..3 of a read group (fixed s, e, h) lie in segments
// 4 k + 2 e + h, i.e. 64 bytes apart in the bank order, so the two 16-lane
// groups of a half-wave (32-byte column slices side by side) cover the 64
// banks once; with fewer segments per block (d < 256) they share banks.
template <int RPS>
__device__ __forceinline__ int wide_row(int i) {
  if (RPS == 2) return 2 * (4 * (i & 3) + 2 * ((i >> 3) & 1) + ((i >> 2) & 1)) + (i >> 4);
  return RPS * (i % (32 / RPS)) + i / (32 / RPS);
}

template <int D>
__global__ __launch_bounds__(64 * kWideWaves) void reord_wide_kernel(const Unit* __restrict__ units,
                                                                     const WsHeader* __restrict__ hdr,
                                                                     const __bf16* __restrict__ UN,
                                                                     const bf16_bits* __restrict__ X,
                                                                     int64_t n_hist, float* __restrict__ part_y,
                                                                     float2* __restrict__ part_ml, int64_t n_tgt,
                                                                     int32_t* __restrict__ range) {
  constexpr int H = D / DH;
  constexpr int KS = D / 16;
  constexpr int NDT = D / 32;
  constexpr int CPR = D / 8;               // 16-byte chunks per X row
  constexpr int RPS = 64 / CPR;            // rows per 1 KB segment
  constexpr int NSEG = 32 / RPS;           // segments per block
  constexpr int SPW = (NSEG + kWideWaves - 1) / kWideWaves;  // segments a wave loads (the last waves may load none)
  constexpr int TILE = NSEG * kSegPitch;
  __shared__ __attribute__((aligned(16))) unsigned char xs[kWideStages * TILE];
  const int u = blockIdx.x;
  if (u >= hdr->n_units) return;
  const Unit un = units[u];
  const int w = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int tcol = lane % 32, hi = lane / 32;
  const int R = un.nt * H;
  const bool active = 32 * w < R;
  const int nb = un.b1 - un.b0;
  auto rowoff = [](int row) { return (row / RPS) * kSegPitch + (row % RPS) * 2 * D; };

  // U of the wave's rows (bf16 hi + lo terms, combined into one fp16
  // operand): B operand of S^T, lane (row tcol, hi) holds model dims
  // 16 ks + 8 hi .. + 7
  f16x8 ub[KS];
  {
    const int rho = 32 * w + tcol;
    const bool ok = active && rho < R;
    const __bf16* up = UN + ((int64_t)un.t0 * H + (ok ? rho : 0)) * 2 * D + 8 * hi;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const bf16x8 h8 = ok ? *reinterpret_cast<const bf16x8*>(up + 16 * ks) : zero8b();
      const bf16x8 l8 = ok ? *reinterpret_cast<const bf16x8*>(up + D + 16 * ks) : zero8b();
#pragma unroll
      for (int i = 0; i < 8; ++i) ub[ks][i] = static_cast<_Float16>(static_cast<float>(h8[i]) + static_cast<float>(l8[i]));
    }
  }

  // this wave's share of block k: segments w + 8 i
  auto issue = [&](int k) {
    if (k >= nb) return;
    unsigned char* slot = xs + (k % kWideStages) * TILE;
    const int64_t b = un.b0 + k;
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
      const int seg = w + kWideWaves * i;
      if (seg < NSEG) {
        const int e = seg * 64 + lane;
        const int64_t grow = min(b * 32 + e / CPR, n_hist - 1);
        dma16(X + grow * D + (e % CPR) * 8, slot + seg * kSegPitch);
      }
    }
  };
  // round this wave's share of block k from bf16 to fp16 in place (its own
  // loads of the block must have landed); |x| beyond the fp16 range is
  // recorded
  uint32_t big = 0;
  auto conv_ptr = [&](int k, int i) {
    return reinterpret_cast<uint2*>(xs + (k % kWideStages) * TILE + (w + kWideWaves * i) * kSegPitch + 16 * lane);
  };
  // bf16 -> fp16 of four values (two dwords)
  auto conv = [&](const uint2& v) {
    const uint32_t in[2] = {v.x, v.y};
    uint32_t outw[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const float lo = __uint_as_float(in[q] << 16), hv = __uint_as_float(in[q] & 0xffff0000u);
      big = max(big, max(__float_as_uint(fabsf(lo)), __float_as_uint(fabsf(hv))));
      outw[q] = (uint32_t)__builtin_bit_cast(uint16_t, static_cast<_Float16>(lo)) |
                ((uint32_t)__builtin_bit_cast(uint16_t, static_cast<_Float16>(hv)) << 16);
    }
    return make_uint2(outw[0], outw[1]);
  };
  auto convert = [&](int k) {
    if (k >= nb) return;
#pragma unroll
    for (int i = 0; i < SPW; ++i)
      if (w + kWideWaves * i < NSEG)
#pragma unroll
        for (int h = 0; h < 2; ++h) conv_ptr(k, i)[h] = conv(conv_ptr(k, i)[h]);
  };
  // loads in flight after a block's own: SPW per newer block issued
  auto wait_own = [&](int newer) { wait_vm(SPW * newer); };

  f32x16 Y[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) Y[dt] = f32x16{};
  float m = -INFINITY, l = 0.f;

  // lane addresses: S^T A operand (MFMA row tcol, dims 16 ks + 8 hi) and the
  // transposing reads of the Y^T A operand (group g of 16 lanes: model dims
  // 32 dt + 16 (g % 2) + 4 (lane % 4) .. + 3 of MFMA rows 16 s + 4 hi +
  // (lane % 16) / 4, and the same + 8)
  const int xa = rowoff(wide_row<RPS>(tcol)) + 16 * hi;
  const int g16 = lane / 16, sl = lane % 16;
  const int ta0 = 2 * (16 * (g16 % 2) + 4 * (sl % 4));

  wait_vm(0);  // U is in registers: the loop issues no load the compiler counts
  for (int k = 0; k < kWideStages - 1; ++k) issue(k);
  wait_own(min(nb - 1, kWideStages - 2));
  convert(0);
  for (int k = 0; k < nb; ++k) {
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's converted writes are done
    ring_barrier();  // block k converted by every wave; block k - 1 read by every wave
    issue(k + kWideStages - 1);
    // own loads of block k + 1: newer blocks in flight are k + 2 and k + 3
    const int newer = max(0, min(nb - 1, k + kWideStages - 1) - (k + 1));
    if (!active) {
      wait_own(newer);
      convert(k + 1);
      continue;
    }
    const unsigned char* tile = xs + (k % kWideStages) * TILE;
    const int b = un.b0 + k;
    // X operands read kAhead k-steps ahead of their MFMAs (the scheduling
    // barriers keep the compiler from sinking the reads next to their use)
    constexpr int kAhead = 2;
    f32x16 s = {};
    f16x8 xo[kAhead];
#pragma unroll
    for (int i = 0; i < kAhead; ++i) xo[i] = *reinterpret_cast<const f16x8*>(tile + xa + 32 * i);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const f16x8 x = xo[ks % kAhead];
      if (ks + kAhead < KS) xo[ks % kAhead] = *reinterpret_cast<const f16x8*>(tile + xa + 32 * (ks + kAhead));
      s = mfma16(x, ub[ks], s);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (b * 32 < un.l0 || b * 32 + 32 > un.l1) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int tok = b * 32 + wide_row<RPS>(8 * (v / 4) + 4 * hi + (v % 4));
        if (tok < un.l0 || tok >= un.l1) s[v] = -INFINITY;
      }
    }
    float bm = s[0];
#pragma unroll
    for (int v = 1; v < 16; ++v) bm = fmaxf(bm, s[v]);
    bm = fmaxf(bm, __shfl_xor(bm, 32));
    if (__builtin_amdgcn_ballot_w64(bm > m + kSlack)) {
      const float mn = fmaxf(m, bm);
      const float sc = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - mn);
      m = mn;
      l *= sc;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) Y[dt] *= sc;
    }
    float ps = 0.f;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      s[v] = __builtin_amdgcn_exp2f(s[v] - m);
      ps += s[v];
    }
    l += ps;
    const f16x8 p0 = pack8(s, 0), p1 = pack8(s, 8);
    // this wave's share of block k + 1 is rounded to fp16 during the Y^T
    // products (its loads have long landed; the LDS round trips overlap the
    // MFMAs), 8 bytes per lane at a time: part p (segment p / 2, half p % 2)
    // read at product 4 p, converted and written back at product 4 p + 2
    const bool conv_next = k + 1 < nb;
    wait_own(newer);
    uint2 cv = {};
    auto conv_owns = [&](int part) { return conv_next && part < 2 * SPW && w + kWideWaves * (part / 2) < NSEG; };
    // A operands of Y^T: step q = ss NDT + dt, read one step ahead
    auto xt_op = [&](int q) {
      const int dt = q % NDT, ss = q / NDT;
      const int r0 = wide_row<RPS>(16 * ss + 4 * hi + sl / 4);
      const int r1 = wide_row<RPS>(16 * ss + 8 + 4 * hi + sl / 4);
      // (whole-vector casts: casting the four 16-bit elements one by one
      // made this compiler permute them)
      typedef _Float16 h4 __attribute__((ext_vector_type(4)));
      const h4 a0 = __builtin_bit_cast(h4, lds_read_tr16(tile + rowoff(r0) + 64 * dt + ta0));
      const h4 a1 = __builtin_bit_cast(h4, lds_read_tr16(tile + rowoff(r1) + 64 * dt + ta0));
      return __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
    };
    f16x8 an = xt_op(0);
#pragma unroll
    for (int q = 0; q < 2 * NDT; ++q) {
      const f16x8 a = an;
      if (q + 1 < 2 * NDT) an = xt_op(q + 1);
      Y[q % NDT] = mfma16(a, q / NDT ? p1 : p0, Y[q % NDT]);
      if (q % 4 == 0 && q + 2 < 2 * NDT && conv_owns(q / 4)) cv = conv_ptr(k + 1, q / 8)[(q / 4) % 2];
      if (q % 4 == 2 && conv_owns(q / 4)) conv_ptr(k + 1, q / 8)[(q / 4) % 2] = conv(cv);
      __builtin_amdgcn_sched_barrier(0);
    }
    // parts the products did not cover (d = 64)
#pragma unroll
    for (int part = 0; part < 2 * SPW; ++part)
      if (4 * part + 2 >= 2 * NDT && conv_owns(part))
        conv_ptr(k + 1, part / 2)[part % 2] = conv(conv_ptr(k + 1, part / 2)[part % 2]);
  }
  if (big > __float_as_uint(kF16Max)) *range = 1;
  if (!active) return;
  const float lt = l + __shfl_xor(l, 32);
  const int rho = 32 * w + tcol;
  if (rho < R) {
    const int64_t prow = ((int64_t)un.c * n_tgt + un.t0 + rho / H) * H + rho % H;
    float* py = part_y + prow * D + 4 * hi;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *reinterpret_cast<float4*>(py + 32 * dt + 8 * g) =
            make_float4(Y[dt][4 * g], Y[dt][4 * g + 1], Y[dt][4 * g + 2], Y[dt][4 * g + 3]);
    if (hi == 0) part_ml[prow] = make_float2(m, lt);
  }
}

// ---------------------------------------------------------------- merge
// One wave per (32 targets, head j): it merges the chunk partials of y_tj
// into fp16 rows in LDS (two lanes per target, half of the d columns each),
// then forms a_j^T = W_V^j^T y_j^T (A operand: the packed fp16 W_V, whose
// column block j is head j) and writes a (fp32) as the single chunk of the
// update kernel's partials: chunk count 1, (max, sum) = (the scores'
// log2-sum-exp, 1), so the update's merge returns a and the lse unchanged.
// Targets whose chunk count is 0 (requests in the standard form when a
// batch runs both forms) are left alone.
template <int D>
__global__ __launch_bounds__(64) void reord_merge_kernel(const float* __restrict__ part_y,
                                                        const float2* __restrict__ part_ml,
                                                        const int32_t* __restrict__ tchunks,
                                                        const f16x8* __restrict__ WvP16, int layer,
                                                        float* __restrict__ a_out, float2* __restrict__ ml_out,
                                                        int32_t* __restrict__ tch_out, int64_t n_tgt) {
  constexpr int H = D / DH;
  constexpr int KS = D / 16;
  constexpr int YROW = D + 8;  // padded fp16 row
  __shared__ __attribute__((aligned(16))) uint16_t ys[32 * YROW];
  const int64_t tb = (int64_t)blockIdx.x * 32;
  const int j = blockIdx.y;
  const int lane = threadIdx.x;
  {
    const int row = lane / 2, part = lane % 2;  // columns [part D/2, (part + 1) D/2)
    const int64_t t = tb + row;
    uint16_t* y = ys + row * YROW + part * (D / 2);
    const int nch = t < n_tgt ? tchunks[t] : 0;
    if (__builtin_amdgcn_ballot_w64(nch > 0) == 0) return;  // no target of this wave in the reordered form
    if (nch > 0) {
      // every chunk's (max, sum) requested at once, and each chunk's weight
      float2 mlc[kMaxChunks];
#pragma unroll
      for (int c = 0; c < kMaxChunks; ++c)
        mlc[c] = c < nch ? part_ml[((int64_t)c * n_tgt + t) * H + j] : make_float2(-INFINITY, 0.f);
      float M = mlc[0].x;
#pragma unroll
      for (int c = 1; c < kMaxChunks; ++c) M = fmaxf(M, mlc[c].x);
      float L = 0.f;
      float wch[kMaxChunks];
#pragma unroll
      for (int c = 0; c < kMaxChunks; ++c) {
        wch[c] = c < nch ? __builtin_amdgcn_exp2f(mlc[c].x - M) : 0.f;
        L += wch[c] * mlc[c].y;
      }
      const float inv = 1.f / L;
#pragma unroll
      for (int c = 0; c < kMaxChunks; ++c) wch[c] *= inv;
      for (int c0 = 0; c0 < D / 2; c0 += 16) {
        float acc[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[i] = 0.f;
        // four chunks' loads in flight at a time (one memory round trip per
        // four chunks instead of one per chunk)
        for (int cb = 0; cb < nch; cb += 4) {
          float4 v[4][4];
          float wc[4];
#pragma unroll
          for (int cc = 0; cc < 4; ++cc) {
            const int c = cb + cc < nch ? cb + cc : cb;
            wc[cc] = cb + cc < nch ? wch[cb + cc < kMaxChunks ? cb + cc : 0] : 0.f;
            const float4* py = reinterpret_cast<const float4*>(part_y + (((int64_t)c * n_tgt + t) * H + j) * D +
                                                               part * (D / 2) + c0);
#pragma unroll
            for (int q = 0; q < 4; ++q) v[cc][q] = py[q];
          }
#pragma unroll
          for (int cc = 0; cc < 4; ++cc)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              acc[4 * q] += wc[cc] * v[cc][q].x, acc[4 * q + 1] += wc[cc] * v[cc][q].y;
              acc[4 * q + 2] += wc[cc] * v[cc][q].z, acc[4 * q + 3] += wc[cc] * v[cc][q].w;
            }
        }
#pragma unroll
        for (int i = 0; i < 16; ++i) y[c0 + i] = __builtin_bit_cast(uint16_t, static_cast<_Float16>(acc[i]));
      }
      if (part == 0) {
        ml_out[t * H + j] = make_float2(M + log2f(L), 1.f);
        if (j == 0) tch_out[t] = 1;
      }
    } else {
      for (int i = 0; i < D / 2; ++i) y[i] = 0;
    }
  }
  __syncthreads();
  const int tcol = lane % 32, hi = lane / 32;
  const f16x8* wp = WvP16 + ((int64_t)(layer * H + j) * KS) * 64 + lane;
  const uint16_t* yb = ys + tcol * YROW + 8 * hi;
  f16x8 wr[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) wr[ks] = wp[ks * 64];
  f32x16 acc = {};
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) acc = mfma16(wr[ks], *reinterpret_cast<const f16x8*>(yb + 16 * ks), acc);
  // lane holds a[t][32 j + 8 g + 4 hi + k] for g, k < 4
  const int64_t t = tb + tcol;
  if (t < n_tgt && tchunks[t] > 0) {
    float* ap = a_out + t * D + 32 * j + 4 * hi;
#pragma unroll
    for (int g = 0; g < 4; ++g)
      *reinterpret_cast<float4*>(ap + 8 * g) = make_float4(acc[4 * g], acc[4 * g + 1], acc[4 * g + 2], acc[4 * g + 3]);
  }
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

}  // namespace

size_t reord_attn_lds(int D) { return reord_main_lds(D) + (size_t)32 * (D + 8) * 2; }

hipError_t fast_reord_qu(int D, const void* QN, const void* Wk_layer, void* UN, const int32_t* tchunks,
                         int64_t n_tgt, hipStream_t st) {
  if (n_tgt == 0) return hipSuccess;
  dim3 g(static_cast<unsigned>(ceil_div(n_tgt, 32)), D / DH);
#define STCA_QU(DD)                                                                                              \
  hipLaunchKernelGGL(reord_qu_kernel<DD>, g, dim3(64), 0, st, (const f16x8*)QN, (const bf16_bits*)Wk_layer, \
                     (__bf16*)UN, tchunks, n_tgt)
  switch (D) {
    case 64: STCA_QU(64); break;
    case 128: STCA_QU(128); break;
    case 256: STCA_QU(256); break;
    default: return hipErrorInvalidValue;
  }
#undef STCA_QU
  return hipGetLastError();
}

hipError_t fast_reord_attn(int D, const Unit* units, const WsHeader* hdr, int64_t max_units, const void* UN,
                           const void* X, int64_t n_hist, float* part_y, void* part_ml, int64_t n_tgt,
                           hipStream_t st) {
  if (max_units == 0) return hipSuccess;
  const size_t lds = reord_attn_lds(D);
#define STCA_RA(DD)                                                                                               \
  do {                                                                                                            \
    hipError_t e = allow_lds(reord_attn_kernel<DD>, lds);                                                         \
    if (e != hipSuccess) return e;                                                                                \
    hipLaunchKernelGGL(reord_attn_kernel<DD>, dim3(static_cast<unsigned>(max_units)), dim3(128 * kWaves), lds, st, \
                       units, hdr, (const __bf16*)UN, (const bf16_bits*)X, n_hist, part_y, (float2*)part_ml,     \
                       n_tgt);                                                                                    \
  } while (0)
  switch (D) {
    case 64: STCA_RA(64); break;
    case 128: STCA_RA(128); break;
    case 256: STCA_RA(256); break;
    default: return hipErrorInvalidValue;
  }
#undef STCA_RA
  return hipGetLastError();
}

hipError_t fast_reord_wide(int D, const Unit* units, const WsHeader* hdr, int64_t max_units, const void* UN,
                           const void* X, int64_t n_hist, float* part_y, void* part_ml, int64_t n_tgt,
                           int32_t* range, hipStream_t st) {
  if (max_units == 0) return hipSuccess;
  if (!range) return hipErrorInvalidValue;
#define STCA_RW(DD)                                                                                         \
  hipLaunchKernelGGL(reord_wide_kernel<DD>, dim3(static_cast<unsigned>(max_units)), dim3(64 * kWideWaves), 0, \
                     st, units, hdr, (const __bf16*)UN, (const bf16_bits*)X, n_hist, part_y, (float2*)part_ml, \
                     n_tgt, range)
  switch (D) {
    case 64: STCA_RW(64); break;
    case 128: STCA_RW(128); break;
    case 256: STCA_RW(256); break;
    default: return hipErrorInvalidValue;
  }
#undef STCA_RW
  return hipGetLastError();
}

hipError_t fast_reord_merge(int D, const float* part_y, const void* part_ml, const int32_t* tchunks,
                            const void* WvP16, int layer, float* a_out, void* ml_out, int32_t* tch_out,
                            int64_t n_tgt, hipStream_t st) {
  if (n_tgt == 0) return hipSuccess;
  dim3 g(static_cast<unsigned>(ceil_div(n_tgt, 32)), D / DH);
#define STCA_RM(DD)                                                                                             \
  hipLaunchKernelGGL(reord_merge_kernel<DD>, g, dim3(64), 0, st, part_y, (const float2*)part_ml, tchunks,      \
                     (const f16x8*)WvP16, layer, a_out, (float2*)ml_out, tch_out, n_tgt)
  switch (D) {
    case 64: STCA_RM(64); break;
    case 128: STCA_RM(128); break;
    case 256: STCA_RM(256); break;
    default: return hipErrorInvalidValue;
  }
#undef STCA_RM
  return hipGetLastError();
}

}  // namespace stca
