// Launchers of the bf16 MFMA path (fast.hip).
#pragma once

#include "common.h"

namespace stca {

struct FastUpdate {
  int mode;      // 0: s^(0) = x_t and Q^(0); 1: combine + update after `layer`
  int layer, n_layers, F;
  int64_t n_tgt;
  const void* tgt;
  const int32_t* tchunks;
  const float* part_acc;
  const void* part_ml;
  const float* s_in;
  float* s_out;
  float *save_a, *save_u, *save_lse;
  void* out;
  void* QN;
  const void *WoP, *W1P, *W2P, *WqP;
  int tg;  // targets per workgroup: 32, or 16 to spread few targets over more CUs
  int32_t* range;  // set to 1 when a value rounded to fp16 (or the merged attention) is not a finite fp16
};

// Repack W [n_layers][K][N] (bf16) into MFMA operand order, as bf16 or fp16.
hipError_t fast_pack(const void* W, void* P, int n_layers, int K, int N, int to_f16, hipStream_t st);
// The same for up to kMaxPackJobs weights (same layer count) in one launch.
constexpr int kMaxPackJobs = 10;
struct PackJob {
  const void* src;
  void* dst;
  int K, N, to_f16;
  int trans;  // src holds the transpose ([N][K]): pack src^T
};
struct PackJobs {
  PackJob job[kMaxPackJobs];
};
hipError_t fast_pack_many(const PackJobs& jobs, int n_jobs, int n_layers, hipStream_t st);
int fast_proj_parts(int n_layers, int64_t n_blocks, int n_cu);
// K1: history -> K/V of every layer, in the attention kernel's operand layout.
hipError_t fast_proj(int D, const void* X, int64_t n_hist, int64_t n_blocks, const void* WkP, const void* WvP,
                     void* KV, int n_layers, int parts, hipStream_t st);
// K3: one layer's fused multi-target attention over the scheduled units.
hipError_t fast_attn(int D, const Unit* units, const WsHeader* hdr, int grid, const void* QN, const void* KVl,
                     float* part_acc, void* part_ml, int64_t n_tgt, hipStream_t st);
// K13: one layer's attention with the history projected inside the kernel
// (no K/V in HBM); persistent over the scheduled units with `streams`
// workgroup pairs.  wide = 0 runs the units with up to 32 targets, wide = 1
// those with 33..64.
hipError_t fast_fused(int D, int wide, const Unit* units, const WsHeader* hdr, int streams, const void* QN,
                      const void* X, int64_t n_hist, const void* WkP, const void* WvP, int layer, float* part_acc,
                      void* part_ml, int64_t n_tgt, hipStream_t st);
// K4: combine partials, W_O, residual FFN, next queries.
hipError_t fast_update(int D, const FastUpdate& f, hipStream_t st);

// Attention backward with the history projection inside the kernel
// (bwd_fused.hip), for units of at most 32 targets (one unit per history
// chunk of a request): writes this layer's dK | dV rows ([N_hist] rows of
// pitch ldkv, dK in columns [0, D), dV in [D, 2D)) for the history rows of
// every unit, and each unit's dq partial ([chunk][n_tgt][D],
// scaled by 1/sqrt(d_h)).  Q: fp32 queries scaled by log2(e)/sqrt(d_h); a,
// da: attention output and its gradient; lse: the forward's natural
// log-sum-exp per (target, head).
struct FastAttnBwd {
  const void* units;
  const void* hdr;
  const void* X;
  int64_t n_hist;
  const void *WkP, *WvP;
  int layer;
  const float *Q, *a, *da, *lse;
  bf16_bits* dKV;
  int64_t ldkv;
  float* dq_part;
  int64_t n_tgt;
};
hipError_t fast_attn_bwd(int D, const FastAttnBwd& f, int grid, hipStream_t st);
// The forward attention recomputed for the backward (bwd_fused.hip), history
// projected inside the kernel and the attention products evaluated to about
// fp32 accuracy (two-term fp16 operands): the same per-chunk partials as
// fast_fused, for units of at most 32 targets.
struct FastAttnFwdPrecise {
  const void* units;
  const void* hdr;
  const void* X;
  int64_t n_hist;
  const void *WkP, *WvP;
  int layer;
  const float* Q;  // [n_tgt][D], scaled by log2(e)/sqrt(d_h)
  float* part_acc;
  void* part_ml;
  int64_t n_tgt;
};
hipError_t fast_attn_fwd_precise(int D, const FastAttnFwdPrecise& f, int grid, hipStream_t st);
// Attention backward in the reordered form (bwd_reordered.hip): requests of
// at most kRbPairs / n_heads targets; pair j' = head * M + target slot
// (M = kRbPairs / n_heads), zero-padded per request.
constexpr int kRbPairs = 128;
// Per layer and request: U = q W_K^j^T per pair (U16: fp16 [R][kRbPairs][D];
// also bf16 in the request's dX operand), H = da W_V^j^T (bf16), the
// statistics (log2-unit lse, D = da . a per pair; [R][kRbPairs][2]) and bf16
// copies of q and da ([n_tgt][D]).  Wr: [R][n_layers][2][kRbPairs][D], this
// layer's U rows then H rows.
struct RbPrep {
  const int32_t* tgt_off;
  int n_requests, layer, n_layers;
  const float *Q, *da, *a, *lse;  // Q scaled by log2(e)/sqrt(d_h); lse natural, [n_tgt][H]
  const bf16_bits *Wk, *Wv;       // this layer's [D][D]
  _Float16* U16;
  bf16_bits* Wr;
  float* stats;
  bf16_bits *q16, *da16;
};
hipError_t rb_prep(int D, const RbPrep& a, hipStream_t st);
// Per unit (a history chunk of a request, all its targets): E (this layer's
// columns [layer 2 kRbPairs, + 2 kRbPairs) of rows [N_hist][lde], bf16:
// ln(2) dE then P per pair), and the chunk's Z = dE^T X and Y = P^T X: into
// Z, Y (bf16 [n_heads][n_tgt][D]) directly for a request of one chunk
// (tchunks of its first target), else as fp32 partials Zp, Yp
// ([unit][kRbPairs][D]) that rb_reduce sums; `first` records each request's
// first unit.
struct RbAttn {
  const void* units;
  const void* hdr;
  const void* X;
  int64_t n_hist, n_tgt;
  int layer, n_layers;
  const _Float16* U16;
  const bf16_bits* Wr;
  const float* stats;
  bf16_bits* E;
  int64_t lde;
  bf16_bits *Z, *Y;
  const int32_t* tchunks;
  float *Zp, *Yp;
  int32_t* first;
};
hipError_t rb_attn(int D, const RbAttn& a, int grid, hipStream_t st);
// Z, Y of the requests of several chunks: the sum of their units' partials.
hipError_t rb_reduce(int D, const int32_t* tgt_off, int n_requests, const int32_t* tchunks, const int32_t* first,
                     const float* Zp, const float* Yp, bf16_bits* Z, bf16_bits* Y, int64_t n_tgt, hipStream_t st);
// Zero the rows [hoff[r], hoff[r + 1]) x cols (fp32) of every request without targets.
hipError_t rb_zero_untargeted(const int32_t* hoff, const int32_t* toff, int n_requests, float* dst, int cols,
                              hipStream_t st);
// Target-side recomputation for the backward (bwd_update.hip), fp32-accurate
// on the bf16 matrix cores.  mode 0: s^(0) = x_t (s_out), q^(0) (q_out).
// mode 1 (layer): merge the partials into a (a_out) and lse (lse_out), u =
// s_in + a W_O (u_out), h = ReLU(u W_1) (h_out, [n_tgt][F]), s' = u + h W_2
// (s_out) and, before the last layer, q' (q_out).  Queries are scaled by
// log2(e)/sqrt(d_h).  Weights packed as bf16 operand tiles (fast_pack_many
// with to_f16 = 0); F a multiple of D.
// The *16 outputs (nullable) are bf16 copies of a, u, h and s' (s^(0) in
// mode 0) for the weight-gradient products.
struct UpdatePrecise {
  int mode, layer, n_layers, F;
  int64_t n_tgt;
  const bf16_bits* tgt;
  const int32_t* tchunks;
  const float* part_acc;
  const float2* part_ml;
  const float* s_in;
  float *a_out, *lse_out, *u_out, *h_out, *s_out, *q_out;
  bf16_bits *a16_out, *u16_out, *h16_out, *s16_out;
  const void *WoP, *W1P, *W2P, *WqP;
};
hipError_t fast_update_precise(int D, const UpdatePrecise& f, hipStream_t st);
// Reverse of one layer's target-side update (bwd_update.hip), per 32 targets:
// dH = (ds W_2^T) masked where h > 0, du = ds + dH W_1^T, da = du W_O^T, on
// bf16 operands with fp32 sums; writes dH and bf16 copies of ds and du for
// the weight-gradient products.  Weights: the transposes of W_2, W_1, W_O
// packed as bf16 operand tiles (PackJob.trans).
// With dq16 set, the gradient of s' is formed first, ds = du_in + dq16 W_Q^T
// (W_Q of layer q_layer, packed transposed in WqTP; du_in may be du_out:
// each element is read before the same thread writes it), and ds is unused.
// With ds_out set as well, only that ds is formed and written (fp32), and
// nothing else is read or written.
struct UpdateGrad {
  int layer, F;
  int64_t n_tgt;
  const float* ds;  // [n_tgt][D] gradient of s'
  const float* h;   // [n_tgt][F] ReLU(u W_1) of the recomputation
  float *du_out, *da_out;
  bf16_bits *ds16_out, *dh16_out, *du16_out;
  const void *W2TP, *W1TP, *WoTP;
  const float* du_in;      // [n_tgt][D]
  const bf16_bits* dq16;   // [n_tgt][D]
  const void* WqTP;
  int q_layer;
  float* ds_out;
};
hipError_t fast_update_grad(int D, const UpdateGrad& f, hipStream_t st);

// Reordered single-query attention (reordered.hip) for units of at most
// 32 / H targets: U = per-head Q W_K^j^T (bf16 hi and lo terms
// [n_tgt][H][2][D]), the attention
// over X writing per-chunk y partials ([16][n_tgt][H][D] fp32 and (max, sum)
// [16][n_tgt][H]), and the merge that forms a = y W_V^j (fp32 [n_tgt][D]) as
// a single-chunk record for fast_update (ml_out (log2-sum-exp, 1), tch_out 1)
// for every target with a nonzero chunk count in `tchunks`.
size_t reord_attn_lds(int D);
hipError_t fast_reord_qu(int D, const void* QN, const void* Wk_layer, void* UN, const int32_t* tchunks,
                         int64_t n_tgt, hipStream_t st);
hipError_t fast_reord_attn(int D, const Unit* units, const WsHeader* hdr, int64_t max_units, const void* UN,
                           const void* X, int64_t n_hist, float* part_y, void* part_ml, int64_t n_tgt,
                           hipStream_t st);
// Units of up to 256 / H targets (up to 256 rows (t, j)): the same partials
// as fast_reord_attn (reord_wide_kernel, fp16 products on X rounded from
// bf16 in LDS; an X value beyond the fp16 range sets *range).
hipError_t fast_reord_wide(int D, const Unit* units, const WsHeader* hdr, int64_t max_units, const void* UN,
                           const void* X, int64_t n_hist, float* part_y, void* part_ml, int64_t n_tgt,
                           int32_t* range, hipStream_t st);
hipError_t fast_reord_merge(int D, const float* part_y, const void* part_ml, const int32_t* tchunks,
                            const void* WvP16, int layer, float* a_out, void* ml_out, int32_t* tch_out,
                            int64_t n_tgt, hipStream_t st);

}  // namespace stca
