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
};

// Repack W [n_layers][K][N] (bf16) into MFMA operand order, as bf16 or fp16.
hipError_t fast_pack(const void* W, void* P, int n_layers, int K, int N, int to_f16, hipStream_t st);
// The same for up to kMaxPackJobs weights (same layer count) in one launch.
constexpr int kMaxPackJobs = 8;
struct PackJob {
  const void* src;
  void* dst;
  int K, N, to_f16;
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

// Reordered single-query attention (reordered.hip) for units of at most
// 32 / H targets: U = per-head Q W_K^j^T (bf16 hi and lo terms
// [n_tgt][H][2][D]), the attention
// over X writing per-chunk y partials ([16][n_tgt][H][D] fp32 and (max, sum)
// [16][n_tgt][H]), and the merge that forms a = y W_V^j (fp32 [n_tgt][D]) with
// single-chunk records (ml_out (0, 1), tch_out 1) for fast_update.
size_t reord_attn_lds(int D);
hipError_t fast_reord_qu(int D, const void* QN, const void* Wk_layer, void* UN, int64_t n_tgt, hipStream_t st);
hipError_t fast_reord_attn(int D, const Unit* units, const WsHeader* hdr, int64_t max_units, const void* UN,
                           const void* X, int64_t n_hist, float* part_y, void* part_ml, int64_t n_tgt,
                           hipStream_t st);
hipError_t fast_reord_merge(int D, const float* part_y, const void* part_ml, const int32_t* tchunks,
                            const void* WvP16, int layer, float* a_out, void* ml_out, int32_t* tch_out,
                            float* save_lse, int64_t n_tgt, hipStream_t st);

}  // namespace stca
