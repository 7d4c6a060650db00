// C ABI of the STCA library: argument checks, workspace/saved layouts and the
// launch sequences of the forward and backward passes.
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>

#include "common.h"
#include "fast.h"
#include "internal.h"
#include "api_common.h"

using namespace stca;
using namespace stca::api;

namespace {

// Form choices of the bf16 path.  Each follows stca_dims_t's execution
// fields (0 = automatic) and the batch alone, so a workspace sized for a
// (dims, batch) pair fits every call made with the same pair.

// Reordered attention (scores u . x with u = q W_K^j^T, output (P X) W_V^j;
// no K/V at all), which needs the host offsets.  Units of one request's
// targets over all heads: up to 32 rows (t, j) per unit for requests with at
// most 32 / H targets (reord_attn_kernel, four X blocks per round), else up
// to 256 rows (reord_wide_kernel).  Automatic choice, per request: requests
// with at most 32 / H targets take the reordered form and the others the
// standard form, in the same call when the batch holds both kinds (their
// work is cheapest that way: 4 m H L d flop against 4 L d^2 + 4 m L d).
// STCA_ATTN_REORDERED puts every request in the reordered form and is
// unsupported for a batch with a request of more than 256 / H targets.
// Returns 3 (both forms, per request), 2 (every request, wide units), 1
// (every request, narrow units), 0 (standard form) or a negative status.
int reordered_for(const stca_dims_t* dims, const stca_batch_t* b) {
  if (dims->attn_form == STCA_ATTN_STANDARD) return 0;
  const bool dh32 = dims->d_model / dims->n_heads == 32;
  const int64_t narrow_cap = 32 / dims->n_heads, wide_cap = 256 / dims->n_heads;
  int64_t mmax = 0;
  bool any_small = false;
  for (int r = 0; b->tgt_off_host && r < b->n_requests; ++r) {
    const int64_t m = b->tgt_off_host[r + 1] - b->tgt_off_host[r];
    mmax = std::max(mmax, m);
    any_small |= m >= 1 && m <= narrow_cap;
  }
  const bool ok = b->tgt_off_host != nullptr && dh32;
  if (ok && mmax <= narrow_cap) return 1;
  if (dims->attn_form == STCA_ATTN_REORDERED) return ok && mmax <= wide_cap ? 2 : STCA_ERR_UNSUPPORTED;
  return ok && any_small ? 3 : 0;
}

// The target-count bound of requests in the reordered form when a batch runs
// both forms.
inline int mixed_cap(const stca_dims_t* dims) { return 32 / dims->n_heads; }

// Requests with more than kTargetGroup targets: the fused kernel would
// project their history once per 64-target group, so the automatic choice
// writes K/V once instead and runs the attention in units of up to
// kWideGroup targets (K/V read once per 128 targets).  Needs host offsets;
// STCA_KV_FUSED keeps the fused form.
bool wide_groups_for(const stca_dims_t* dims, const stca_batch_t* b) {
  if (dims->kv_form == STCA_KV_FUSED) return false;
  if (!b->tgt_off_host) return false;
  for (int r = 0; r < b->n_requests; ++r)
    if (b->tgt_off_host[r + 1] - b->tgt_off_host[r] > kTargetGroup) return true;
  return false;
}

// The bf16 backward projects the history inside its attention kernels (no
// K/V copy in HBM) and recomputes the target side in one kernel per layer
// when d_h = 32, the FFN width is a multiple of d and every request has at
// most 32 targets, which the host offsets must show; otherwise K | V are
// formed by a GEMM, the attention runs exactly in fp32 and the target side as
// separate GEMMs.  Within the fused conditions, d_model of 128 or 256 and at
// most kRbPairs / n_heads targets per request allow the reordered form (no
// K, V, dK, dV; the automatic choice there when the batch's histories are
// balanced over the CUs).  STCA_BWD_GENERIC forces the
// generic form; STCA_BWD_FUSED and STCA_BWD_REORDERED ask for theirs and are
// unsupported for other batches.  2 (reordered) / 1 (fused) / 0 (generic) /
// negative status.
int fused_bwd_for(const stca_dims_t* dims, const stca_batch_t* b) {
  if (dims->bwd_form == STCA_BWD_GENERIC) return 0;
  bool ok = dims->dtype == STCA_BF16 && dims->d_model / dims->n_heads == 32 &&
            (dims->d_model == 64 || dims->d_model == 128 || dims->d_model == 256) &&
            dims->ffn_hidden % dims->d_model == 0 && b->tgt_off_host != nullptr;
  bool rd = ok && (dims->d_model == 128 || dims->d_model == 256) && b->hist_off_host != nullptr;
  for (int r = 0; ok && r < b->n_requests; ++r) {
    const int64_t m = b->tgt_off_host[r + 1] - b->tgt_off_host[r];
    if (m > 32) ok = false;
    if (m * dims->n_heads > kRbPairs) rd = false;
  }
  rd = rd && ok;
  if (dims->bwd_form == STCA_BWD_FUSED) return ok ? 1 : STCA_ERR_UNSUPPORTED;
  if (dims->bwd_form == STCA_BWD_REORDERED) return rd ? 2 : STCA_ERR_UNSUPPORTED;
  // automatic: the reordered form when no request's history is much longer
  // than one CU's share of the batch (its attention pass streams a request
  // per unit and splits long requests into chunks whose Z, Y partials cost
  // extra traffic; on bimodal stochastic-length batches the fused form is
  // faster)
  if (rd) {
    int64_t total = 0, longest = 0;
    for (int r = 0; r < b->n_requests; ++r) {
      if (b->tgt_off_host[r + 1] == b->tgt_off_host[r]) continue;
      const int64_t nb = ceil_div(b->hist_off_host[r + 1], kBlockTokens) - b->hist_off_host[r] / kBlockTokens;
      total += nb;
      longest = std::max(longest, nb);
    }
    rd = longest <= 2 * ceil_div(total, device_cus());
  }
  return rd ? 2 : ok ? 1 : 0;
}

struct Layout {
  int path;
  int d, h, n, F, dh;
  int64_t nh, nt, nblocks;
  int chunk_blocks;
  int64_t max_units;
  bool any_narrow, any_wide;  // requests with 1..32 / 33+ targets (both true without host offsets)
  bool reord;                 // some requests in the reordered form (bf16 path)
  bool reord_wide;            // ... in units of up to 256 rows (t, j)
  bool mixed;                 // ... and the others in the standard form
  int reord_lo, reord_hi;     // target counts of the requests in the reordered form
  int std_lo;                 // requests with at least this many targets take the standard form
  int chunk_blocks2, group2;  // reordered schedule
  int64_t max_units2;
  bool mat;                   // K/V written to the workspace by one GEMM (bf16 path)
  bool wide;                  // materialised K/V, units of up to kWideGroup targets (bf16 path)
  bool bfused;                // backward with the history projection inside the attention kernels
  bool brd;                   // ... in the reordered form (no K, V, dK, dV)
  int group;                  // targets per attention unit
  // common
  size_t hdr, units, tchunks, part_acc, part_ml, state_a, state_b;
  // fast
  size_t qn, wkp, wvp, wop, w1p, w2p, wqp, kv;
  // reordered: U, the y partials with their (max, sum) and chunk counts, its
  // schedule (its own header and units when both forms run), fp16 W_V
  size_t un, part_y, ml_r, tch_r, hdr2, units2, wvp16;
  // generic forward
  size_t kv32, q32, abuf, ubuf, hid;
  // backward (generic)
  size_t dhid, ds, du, da, dq, ds2, dkv, dq_part, rs, ru, rq, ra, rl, kvs, wkv, dwkv, gpart;
  size_t xt, dkvt, wkvt;
  // fused backward: every layer's weights as bf16 operand tiles (and the
  // transposes of W_2, W_1, W_O), and the region of the recomputed
  // per-layer tensors (RecordLayout)
  size_t fwkp, fwvp, fwop, fw1p, fw2p, fwqp, fw2t, fw1t, fwot, fwqt, rec;
  size_t b_hid, b_dhid, b_ds, b_u, b_du, b_a, b_dq, b_s;  // bf16 copies of backward operands (bf16 path)
  // reordered backward: E, every request's dX operand, U (fp16), pair
  // statistics, Z and Y, bf16 q and da; the per-request schedule and the
  // dX schedule (units of up to 128 rows)
  size_t rb_e, rb_w, rb_u16, rb_st, rb_z, rb_y, rb_q16, rb_da16, rb_hdr, rb_units, rb_hdrx, rb_unitsx, rb_tch;
  size_t rb_tchx, rb_zp, rb_yp, rb_first;
  int64_t rb_maxx, rb_maxu;
  int rb_cb;  // history chunk length (blocks) of the reordered attention's units
  int64_t gpart_floats, nh8;
  size_t total;
};

// The per-layer tensors the fused backward's reverse pass reads (a training
// record): a, lse, the scaled queries and h = ReLU(u W_1) in fp32, and bf16
// copies of a, u, h and the layer input s for the weight-gradient products.
struct RecordLayout {
  size_t a, lse, q, h, a16, u16, h16, s16, total;
};
RecordLayout record_layout(const Layout& L) {
  const size_t d = L.d, h = L.h, F = L.F, n = L.n, nt = L.nt;
  RecordLayout R;
  Bump m;
  R.a = m.take(4 * n * nt * d);
  R.lse = m.take(4 * n * nt * h);
  R.q = m.take(4 * n * nt * d);
  R.h = m.take(4 * n * nt * F);
  R.a16 = m.take(2 * n * nt * d);
  R.u16 = m.take(2 * n * nt * d);
  R.h16 = m.take(2 * n * nt * F);
  R.s16 = m.take(2 * n * nt * d);
  R.total = m.off;
  return R;
}

stca_status_t make_layout(const stca_dims_t* dims, const stca_batch_t* b, int with_backward, bool with_saved,
                          Layout* L) {
  const int p = path_of(dims);
  if (p < 0) return static_cast<stca_status_t>(p);
  const stca_status_t bst = check_batch(b);
  if (bst != STCA_OK) return bst;
  L->path = p;
  L->d = dims->d_model;
  L->h = dims->n_heads;
  L->n = dims->n_layers;
  L->F = dims->ffn_hidden;
  L->dh = L->d / L->h;
  L->nh = b->n_hist;
  L->nt = b->n_tgt;
  L->nblocks = ceil_div(b->n_hist, kBlockTokens);
  L->reord = L->reord_wide = L->mixed = false;
  if (p == 1 && !with_backward) {
    const int r = reordered_for(dims, b);
    if (r < 0) return static_cast<stca_status_t>(r);
    L->reord = r >= 1;
    L->reord_wide = r == 2;
    L->mixed = r == 3;
  }
  // requests [std_lo, inf) targets: standard form; [reord_lo, reord_hi]: reordered
  L->std_lo = L->mixed ? mixed_cap(dims) + 1 : (L->reord ? 1 << 30 : 1);
  L->reord_lo = 1;
  L->reord_hi = L->mixed ? mixed_cap(dims) : (L->reord ? 1 << 30 : 0);
  L->bfused = false;
  const bool std_part = !L->reord || L->mixed;
  L->wide = p == 1 && !with_backward && std_part && wide_groups_for(dims, b);
  L->mat = p == 1 && !with_backward && std_part && (L->wide || dims->kv_form == STCA_KV_MATERIALIZE);
  L->chunk_blocks = chunk_blocks_auto(b, device_cus(), dims->chunk_blocks, L->std_lo);
  L->group = L->wide ? kWideGroup : kTargetGroup;
  L->max_units = std_part ? max_units_for(b, L->chunk_blocks, L->group, L->std_lo) : 0;
  // the reordered schedule spreads its own requests' rows over the chip
  int64_t rows2 = b->n_hist;
  if (L->mixed) {
    rows2 = 0;
    for (int r = 0; r < b->n_requests; ++r) {
      const int64_t m = b->tgt_off_host[r + 1] - b->tgt_off_host[r];
      if (m >= L->reord_lo && m <= L->reord_hi) rows2 += b->hist_off_host[r + 1] - b->hist_off_host[r];
    }
  }
  L->chunk_blocks2 = chunk_blocks_for(b, device_cus(), 1, dims->chunk_blocks, rows2);
  // (a small reordered share of a mixed batch in chunks of at least 512
  // rows: its merge cost grows with the chunk count)
  if (L->mixed && dims->chunk_blocks == 0) L->chunk_blocks2 = std::max(L->chunk_blocks2, 16);
  L->group2 = (L->reord_wide ? 256 : 32) / L->h;
  L->max_units2 = L->reord ? max_units_for(b, L->chunk_blocks2, L->group2, L->reord_lo, L->reord_hi) : 0;
  L->any_narrow = L->any_wide = std_part;
  if (b->tgt_off_host && std_part) {
    L->any_narrow = L->any_wide = false;
    for (int r = 0; r < b->n_requests; ++r) {
      const int64_t m = b->tgt_off_host[r + 1] - b->tgt_off_host[r];
      if (m < L->std_lo) continue;
      // target groups are `group` wide; the last group of a request is what may be narrow
      for (int64_t g0 = 0; g0 < m; g0 += L->group) {
        if (m - g0 > 32) L->any_wide = true;
        else L->any_narrow = true;
      }
    }
  }
  const size_t d = L->d, nt = L->nt, nh = L->nh, F = L->F, n = L->n;
  Bump m;
  L->hdr = m.take(sizeof(WsHeader));
  L->units = m.take(sizeof(Unit) * (L->max_units + 1));
  L->tchunks = m.take(4 * (nt + 1));
  L->state_a = m.take(4 * nt * d);
  L->state_b = m.take(4 * nt * d);
  if (!with_backward) {
    L->part_acc = m.take(4 * kMaxChunks * nt * d);
    L->part_ml = m.take(8 * kMaxChunks * nt * L->h);
    if (p == 1) {
      L->qn = m.take(2 * nt * d);
      L->wkp = m.take(2 * n * d * d);
      L->wvp = m.take(2 * n * d * d);
      L->wop = m.take(2 * n * d * d);
      L->wqp = m.take(2 * n * d * d);
      L->w1p = m.take(2 * n * d * F);
      L->w2p = m.take(2 * n * d * F);
      L->kv = L->mat ? m.take(2 * n * L->nblocks * kBlockTokens * 2 * d) : 0;
      if (L->reord) {
        const size_t h = L->h;
        L->un = m.take(2 * 2 * nt * h * d);  // bf16 hi and lo terms
        L->part_y = m.take(4 * kMaxChunks * nt * h * d);
        L->ml_r = m.take(8 * kMaxChunks * nt * h);
        L->tch_r = m.take(4 * (nt + 1));
        L->wvp16 = m.take(2 * n * d * d);
        L->hdr2 = m.take(sizeof(WsHeader));
        L->units2 = m.take(sizeof(Unit) * (L->max_units2 + 1));
      }
    } else {
      L->kv32 = m.take(4 * nh * 2 * d);
      L->q32 = m.take(4 * nt * d);
      L->abuf = m.take(4 * nt * d);
      L->ubuf = m.take(4 * nt * d);
      L->hid = m.take(4 * nt * F);
    }
  } else {
    const bool bf = dims->dtype == STCA_BF16;
    const int fb = fused_bwd_for(dims, b);
    if (fb < 0) return static_cast<stca_status_t>(fb);
    L->bfused = bf && fb >= 1;
    L->brd = bf && fb == 2;
    L->kvs = L->bfused ? 0 : m.take(4 * n * nh * 2 * d);  // every layer's K | V rows, fp32
    if (L->bfused) {
      L->fwkp = m.take(2 * n * d * d);
      L->fwvp = m.take(2 * n * d * d);
      L->fwop = m.take(2 * n * d * d);
      L->fwqp = m.take(2 * n * d * d);
      L->fw1p = m.take(2 * n * d * F);
      L->fw2p = m.take(2 * n * d * F);
      L->fw2t = m.take(2 * n * d * F);
      L->fw1t = m.take(2 * n * d * F);
      L->fwot = m.take(2 * n * d * d);
      L->fwqt = m.take(2 * n * d * d);
    }
    // dK | dV: fp32 [N_hist][2d] for one layer; bf16 for every layer, rows
    // [N_hist][n 2d] (layer i in columns [2d i, 2d (i + 1)))
    L->dkv = L->brd ? 0 : m.take(bf ? 2 * nh * n * 2 * d : 4 * nh * 2 * d);
    // bf16 history-side products: [W_K | W_V] per layer, and for the
    // unfused form its transpose, X^T and every layer's (dK | dV)^T
    // ([n 2d][nh8]) with the history rows padded to a multiple of 8 (the
    // fused form's [dW_K | dW_V] reads X and dK | dV as they are)
    L->nh8 = round_up(static_cast<int64_t>(nh), 8);
    const size_t nh8 = static_cast<size_t>(L->nh8);
    const bool tcopies = bf && !L->bfused;
    L->wkv = bf && !L->brd ? m.take(2 * n * d * 2 * d) : 0;
    L->wkvt = tcopies ? m.take(2 * n * d * 2 * d) : 0;
    L->xt = tcopies ? m.take(2 * d * nh8) : 0;
    L->dkvt = tcopies ? m.take(2 * n * 2 * d * nh8) : 0;
    L->dwkv = bf && !L->brd ? m.take(4 * d * n * 2 * d) : 0;   // [d][n 2d] fp32
    // split-K partials: the largest of [dW_K | dW_V] (K = history rows) and
    // the target-side weight gradients (K = targets)
    L->gpart_floats = 0;
    if (bf) {
      const int di = static_cast<int>(d), Fi = static_cast<int>(F), nti = static_cast<int>(nt);
      // (the fused form runs the target-side weight gradients of a layer,
      // with dW_Q of the layer above, as one group whose splits share it)
      L->gpart_floats = std::max({L->brd ? 2 * L->h * gemm_mfma_part_floats(di, 32, nti)
                                         : gemm_ring_part_floats(di, 2 * di * static_cast<int>(n),
                                                                 static_cast<int>(nh8), device_cus()),
                                  gemm_mfma_part_floats(Fi, di, nti) + gemm_mfma_part_floats(di, Fi, nti) +
                                      2 * gemm_mfma_part_floats(di, di, nti)});
    }
    L->gpart = bf ? m.take(4 * L->gpart_floats) : 0;
    if (L->bfused) {
      L->rec = m.take(record_layout(*L).total);
    } else {
      L->rq = m.take(4 * n * nt * d);  // per-layer queries, attention outputs, lse
      L->ra = m.take(4 * n * nt * d);
      L->rl = m.take(4 * n * nt * L->h);
      L->hid = m.take(4 * n * nt * F);  // every layer's ReLU(u W_1) from the recomputation
    }
    L->dhid = m.take(4 * nt * F);
    L->ds = m.take(4 * nt * d);
    L->du = m.take(4 * nt * d);
    L->da = m.take(4 * nt * d);
    L->dq = m.take(4 * nt * d);
    L->ds2 = m.take(4 * nt * d);
    L->dq_part = m.take(4 * kMaxChunks * nt * d);
    L->part_acc = m.take(4 * kMaxChunks * nt * d);
    L->part_ml = m.take(8 * kMaxChunks * nt * L->h);
    L->rs = m.take(4 * (n + 1) * nt * d);  // recomputed s^(0..n)
    L->ru = m.take(4 * n * nt * d);        // recomputed u^(0..n-1)
    if (bf) {
      L->b_hid = m.take(2 * nt * F);
      L->b_dhid = m.take(2 * nt * F);
      L->b_ds = m.take(2 * nt * d);
      L->b_u = m.take(2 * nt * d);
      L->b_du = m.take(2 * nt * d);
      L->b_a = m.take(2 * nt * d);
      L->b_dq = m.take(2 * nt * d);
      L->b_s = m.take(2 * nt * d);
    }
    if (L->brd) {
      const size_t R = static_cast<size_t>(b->n_requests), hm = kRbPairs;
      L->rb_e = m.take(2 * nh * n * 2 * hm);
      L->rb_w = m.take(2 * R * n * 2 * hm * d);
      L->rb_u16 = m.take(2 * R * hm * d);
      L->rb_st = m.take(8 * R * hm);
      L->rb_z = m.take(2 * L->h * nt * d);
      L->rb_y = m.take(2 * L->h * nt * d);
      L->rb_q16 = m.take(2 * nt * d);
      L->rb_da16 = m.take(2 * nt * d);
      L->rb_hdr = m.take(sizeof(WsHeader));
      // about one unit per CU over the whole batch: long requests are cut into
      // history chunks whose Z, Y partials are summed afterwards
      L->rb_cb = chunk_blocks_for(b, device_cus(), 1, dims->chunk_blocks);
      L->rb_maxu = std::max<int64_t>(1, host_count_units(b->hist_off_host, b->tgt_off_host, b->n_requests,
                                                         L->rb_cb, 32));
      L->rb_units = m.take(sizeof(Unit) * static_cast<size_t>(L->rb_maxu));
      L->rb_zp = m.take(4 * static_cast<size_t>(L->rb_maxu) * hm * d);
      L->rb_yp = m.take(4 * static_cast<size_t>(L->rb_maxu) * hm * d);
      L->rb_first = m.take(4 * std::max<size_t>(R, 1));
      L->rb_tchx = m.take(4 * std::max<size_t>(nt, 1));
      L->rb_hdrx = m.take(sizeof(WsHeader));
      L->rb_maxx = std::max<int64_t>(1, host_count_units(b->hist_off_host, b->tgt_off_host, b->n_requests, 4, 32));
      L->rb_unitsx = m.take(sizeof(Unit) * static_cast<size_t>(L->rb_maxx));
      L->rb_tch = m.take(4 * std::max<size_t>(nt, 1));
    }
  }
  L->total = m.off;
  return STCA_OK;
}

bool saved_layout(const stca_dims_t* dims, const stca_batch_t* b, stca_saved_layout_t* s) {
  const int p = path_of(dims);
  if (p < 0 || check_batch(b) != STCA_OK) return false;
  const size_t d = dims->d_model, nt = b->n_tgt, n = dims->n_layers, h = dims->n_heads;
  Bump m;
  s->s = m.take(4 * n * nt * d);
  s->a = m.take(4 * n * nt * d);
  s->u = m.take(4 * n * nt * d);
  s->lse = m.take(4 * n * nt * h);
  s->total = m.off;
  return true;
}

stca_status_t check_common(const stca_dims_t* dims, const stca_batch_t* b, const void* hist, const void* tgt,
                           const stca_weights_t* w, void* ws) {
  const int p = path_of(dims);
  if (p < 0) return static_cast<stca_status_t>(p);
  stca_status_t st = check_batch(b);
  if (st != STCA_OK) return st;
  if (!w || !ws || (b->n_hist > 0 && !hist) || (b->n_tgt > 0 && !tgt)) return STCA_ERR_INVALID_ARG;
  const void* ptrs[] = {hist, tgt, w->wq, w->wk, w->wv, w->wo, w->w1, w->w2, ws};
  for (const void* q : ptrs)
    if (q && !aligned16(q)) return STCA_ERR_INVALID_ARG;
  if (!w->wq || !w->wk || !w->wv || !w->wo || !w->w1 || !w->w2) return STCA_ERR_INVALID_ARG;
  return STCA_OK;
}

// ---------------------------------------------------------------- forward
// The bf16 path.  Requests in the standard form: per layer the history
// projected to K/V inside the attention kernel (or K/V written once and
// streamed), partials per history chunk.  Requests in the reordered form
// (App. A.2.2): per layer U = Q W_K^j^T, attention over X itself, merge with
// W_V^j into a single-chunk partial.  Each form has its own schedule; then
// one target update per layer merges every target's partials.
stca_status_t forward_fast(const Layout& L, const stca_batch_t* b, const void* hist, const void* tgt,
                           const stca_weights_t* w, void* out, void* saved, const stca_saved_layout_t& SL,
                           void* ws, hipStream_t st, Rec& rec) {
  HIPCHK(rec.start());
  const int d = L.d, n = L.n, F = L.F;
  const bool std_part = !L.reord || L.mixed, reo_part = L.reord;
  WsHeader* hdr = at<WsHeader>(ws, L.hdr);
  Unit* units = at<Unit>(ws, L.units);
  int32_t* tch = at<int32_t>(ws, L.tchunks);
  // the reordered schedule: its own header and units when both forms run,
  // else the workspace's
  WsHeader* hdr2 = L.mixed ? at<WsHeader>(ws, L.hdr2) : hdr;
  Unit* units2 = reo_part ? at<Unit>(ws, L.units2) : nullptr;
  int32_t* tch_r = reo_part ? at<int32_t>(ws, L.tch_r) : nullptr;
  if (std_part)
    HIPCHK(launch_sched(b->hist_off, b->tgt_off, b->n_requests, L.nh, L.nt, L.chunk_blocks, L.group, units,
                        L.max_units, tch, hdr, st, L.std_lo, 1 << 30, device_cus()));
  if (std_part) HIPCHK(rec.mark("sched"));
  if (reo_part)
    HIPCHK(launch_sched(b->hist_off, b->tgt_off, b->n_requests, L.nh, L.nt, L.chunk_blocks2, L.group2, units2,
                        L.max_units2, tch_r, hdr2, st, L.reord_lo, L.reord_hi, device_cus()));
  if (reo_part) HIPCHK(rec.mark("sched"));
  {
    PackJobs pj{};
    int nj = 0;
    if (std_part) {
      pj.job[nj++] = {w->wk, at<char>(ws, L.wkp), d, d, 0};
      pj.job[nj++] = {w->wv, at<char>(ws, L.wvp), d, d, 0};
    }
    if (reo_part) pj.job[nj++] = {w->wv, at<char>(ws, L.wvp16), d, d, 1};
    pj.job[nj++] = {w->wo, at<char>(ws, L.wop), d, d, 1};
    pj.job[nj++] = {w->wq, at<char>(ws, L.wqp), d, d, 1};
    pj.job[nj++] = {w->w1, at<char>(ws, L.w1p), d, F, 1};
    pj.job[nj++] = {w->w2, at<char>(ws, L.w2p), F, d, 1};
    HIPCHK(fast_pack_many(pj, nj, n, st));
    HIPCHK(rec.mark("pack"));
  }
  char* kv = at<char>(ws, L.kv);
  if (L.mat) {
    if (L.nh > 0)
      HIPCHK(fast_proj(d, hist, L.nh, L.nblocks, at<char>(ws, L.wkp), at<char>(ws, L.wvp), kv, n,
                       fast_proj_parts(n, L.nblocks, device_cus()), st));
    HIPCHK(rec.mark("proj"));
  }
  const size_t kv_layer = (size_t)L.nblocks * kBlockTokens * 2 * d * 2;
  const size_t wlayer = (size_t)d * d * 2;  // bytes of one layer's bf16 W_K
  FastUpdate f{};
  f.tg = ceil_div(static_cast<int64_t>(L.nt), 32) < device_cus() ? 16 : 32;
  f.n_layers = n;
  f.F = F;
  f.n_tgt = L.nt;
  f.tgt = tgt;
  f.tchunks = tch;
  f.part_acc = at<float>(ws, L.part_acc);
  f.part_ml = at<char>(ws, L.part_ml);
  f.QN = at<char>(ws, L.qn);
  f.WoP = at<char>(ws, L.wop);
  f.W1P = at<char>(ws, L.w1p);
  f.W2P = at<char>(ws, L.w2p);
  f.WqP = at<char>(ws, L.wqp);
  f.out = out;
  f.range = &hdr->range;
  // s^(i) lives in saved.s[i] when saving, else alternates between two buffers
  auto state = [&](int i) -> float* {
    if (saved) return at<float>(saved, SL.s) + (size_t)i * L.nt * d;
    return at<float>(ws, (i % 2) ? L.state_b : L.state_a);
  };
  f.mode = 0;
  f.layer = 0;
  f.s_out = state(0);
  HIPCHK(fast_update(d, f, st)); HIPCHK(rec.mark("update"));
  const int grid = static_cast<int>(std::min<int64_t>(L.max_units, 8 * (int64_t)device_cus()));
  // the fused kernel is persistent: one workgroup per CU, looping over its
  // units with its weight columns loaded once
  const int fgrid = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(L.max_units, device_cus())));
  for (int i = 0; i < n; ++i) {
    if (reo_part) {
      HIPCHK(fast_reord_qu(d, f.QN, static_cast<const char*>(w->wk) + i * wlayer, at<char>(ws, L.un), tch_r, L.nt,
                           st));
      HIPCHK(rec.mark("reord_u"));
    }
    if (std_part && L.mat) {
      HIPCHK(fast_attn(d, units, hdr, grid, f.QN, kv + i * kv_layer, at<float>(ws, L.part_acc),
                       at<char>(ws, L.part_ml), L.nt, st));
      HIPCHK(rec.mark("attn"));
    } else if (std_part) {
      for (int wide = 0; wide < 2; ++wide) {
        if (!(wide ? L.any_wide : L.any_narrow)) {  // no request of this width: nothing to launch
          HIPCHK(rec.mark(wide ? "fused_wide" : "fused"));
          continue;
        }
        HIPCHK(fast_fused(d, wide, units, hdr, fgrid, f.QN, hist, L.nh, at<char>(ws, L.wkp), at<char>(ws, L.wvp), i,
                          at<float>(ws, L.part_acc), at<char>(ws, L.part_ml), L.nt, st));
        HIPCHK(rec.mark(wide ? "fused_wide" : "fused"));
      }
    }
    if (reo_part) {
      if (L.reord_wide)
        HIPCHK(fast_reord_wide(d, units2, hdr2, L.max_units2, at<char>(ws, L.un), hist, L.nh,
                               at<float>(ws, L.part_y), at<char>(ws, L.ml_r), L.nt, &hdr->range, st));
      else
        HIPCHK(fast_reord_attn(d, units2, hdr2, L.max_units2, at<char>(ws, L.un), hist, L.nh,
                               at<float>(ws, L.part_y), at<char>(ws, L.ml_r), L.nt, st));
      HIPCHK(rec.mark("reord_attn"));
      // a of the reordered requests as their single chunk of the update's partials
      HIPCHK(fast_reord_merge(d, at<float>(ws, L.part_y), at<char>(ws, L.ml_r), tch_r, at<char>(ws, L.wvp16), i,
                              at<float>(ws, L.part_acc), at<char>(ws, L.part_ml), tch, L.nt, st));
      HIPCHK(rec.mark("reord_merge"));
    }
    f.mode = 1;
    f.layer = i;
    f.s_in = state(i);
    f.s_out = i + 1 < n ? state(i + 1) : nullptr;
    f.save_a = saved ? at<float>(saved, SL.a) + (size_t)i * L.nt * d : nullptr;
    f.save_u = saved ? at<float>(saved, SL.u) + (size_t)i * L.nt * d : nullptr;
    f.save_lse = saved ? at<float>(saved, SL.lse) + (size_t)i * L.nt * L.h : nullptr;
    HIPCHK(fast_update(d, f, st)); HIPCHK(rec.mark("update"));
  }
  return STCA_OK;
}

stca_status_t forward_generic(const Layout& L, int bf, const stca_batch_t* b, const void* hist, const void* tgt,
                              const stca_weights_t* w, void* out, void* saved, const stca_saved_layout_t& SL,
                              void* ws, hipStream_t st, Rec& rec) {
  HIPCHK(rec.start());
  const int d = L.d, n = L.n, F = L.F, h = L.h;
  const size_t es = bf ? 2 : 4;
  WsHeader* hdr = at<WsHeader>(ws, L.hdr);
  Unit* units = at<Unit>(ws, L.units);
  int32_t* tch = at<int32_t>(ws, L.tchunks);
  HIPCHK(launch_sched(b->hist_off, b->tgt_off, b->n_requests, L.nh, L.nt, L.chunk_blocks, L.group, units, L.max_units,
                      tch, hdr, st, 1, 1 << 30, device_cus())); HIPCHK(rec.mark("sched"));
  float* kv = at<float>(ws, L.kv32);
  float* q = at<float>(ws, L.q32);
  float* hid = at<float>(ws, L.hid);
  float* pacc = at<float>(ws, L.part_acc);
  float* pml = at<float>(ws, L.part_ml);
  auto state = [&](int i) -> float* {
    if (saved && i < n) return at<float>(saved, SL.s) + (size_t)i * L.nt * d;
    return at<float>(ws, (i % 2) ? L.state_b : L.state_a);
  };
  auto W = [&](const void* base, int i, size_t per) { return static_cast<const char*>(base) + i * per * es; };
  HIPCHK(convert(bf, 0, tgt, state(0), L.nt * d, st)); HIPCHK(rec.mark("convert_in"));
  const float qscale = kLog2e / std::sqrt(static_cast<float>(L.dh));
  for (int i = 0; i < n; ++i) {
    float* s = state(i);
    float* a = saved ? at<float>(saved, SL.a) + (size_t)i * L.nt * d : at<float>(ws, L.abuf);
    float* u = saved ? at<float>(saved, SL.u) + (size_t)i * L.nt * d : at<float>(ws, L.ubuf);
    float* lse = saved ? at<float>(saved, SL.lse) + (size_t)i * L.nt * h : nullptr;
    HIPCHK(gemm_generic(bf, bf, L.nh, d, d, hist, d, 0, W(w->wk, i, (size_t)d * d), d, 0, kv, 2 * d, 1.f,
                        kEpiStore, nullptr, 0, nullptr, 0, st)); HIPCHK(rec.mark("gemm_k"));
    HIPCHK(gemm_generic(bf, bf, L.nh, d, d, hist, d, 0, W(w->wv, i, (size_t)d * d), d, 0, kv + d, 2 * d, 1.f,
                        kEpiStore, nullptr, 0, nullptr, 0, st)); HIPCHK(rec.mark("gemm_v"));
    HIPCHK(gemm_generic(0, bf, L.nt, d, d, s, d, 0, W(w->wq, i, (size_t)d * d), d, 0, q, d, qscale, kEpiStore,
                        nullptr, 0, nullptr, 0, st)); HIPCHK(rec.mark("gemm_q"));
    HIPCHK(attn_generic(L.dh, h, units, L.max_units, hdr, q, kv, d, pacc, pml, L.nt, st)); HIPCHK(rec.mark("attn"));
    HIPCHK(merge_generic(L.dh, h, L.nt, tch, pacc, pml, a, lse, st)); HIPCHK(rec.mark("merge"));
    HIPCHK(gemm_generic(0, bf, L.nt, d, d, a, d, 0, W(w->wo, i, (size_t)d * d), d, 0, u, d, 1.f, kEpiAddRes, s, d,
                        nullptr, 0, st)); HIPCHK(rec.mark("gemm_o"));
    HIPCHK(gemm_generic(0, bf, L.nt, F, d, u, d, 0, W(w->w1, i, (size_t)d * F), F, 0, hid, F, 1.f, kEpiRelu,
                        nullptr, 0, nullptr, 0, st)); HIPCHK(rec.mark("gemm_ffn1"));
    HIPCHK(gemm_generic(0, bf, L.nt, d, F, hid, F, 0, W(w->w2, i, (size_t)d * F), d, 0, state(i + 1), d, 1.f,
                        kEpiAddRes, u, d, nullptr, 0, st)); HIPCHK(rec.mark("gemm_ffn2"));
  }
  HIPCHK(convert(0, bf, state(n), out, L.nt * d, st)); HIPCHK(rec.mark("convert_out"));
  return STCA_OK;
}

// --------------------------------------------------------------- backward
// Activation recomputation: the layer states are rebuilt in fp32 from the
// inputs first, so every ReLU gate and softmax weight of the backward follows
// fp32 states whatever arithmetic the forward call used.
// rec_out (fused form only): stop after the recomputation, which writes the
// training record there and the output into `out` (the forward of a
// training step).  rec_in (fused form only): skip the recomputation and read
// the record written by such a call.
stca_status_t backward_generic(const Layout& L, int bf, const stca_batch_t* b, const void* hist, const void* tgt,
                               const stca_weights_t* w, const void* dout, float* dhist, float* dtgt,
                               const stca_wgrads_t* dw, void* ws, hipStream_t st, Rec& rec,
                               const void* rec_in = nullptr, void* rec_out = nullptr, void* out = nullptr) {
  const int d = L.d, n = L.n, F = L.F, h = L.h;
  const int64_t nt = L.nt, nh = L.nh;
  const size_t es = bf ? 2 : 4;
  WsHeader* hdr = at<WsHeader>(ws, L.hdr);
  Unit* units = at<Unit>(ws, L.units);
  int32_t* tch = at<int32_t>(ws, L.tchunks);
  HIPCHK(rec.start());
  HIPCHK(launch_sched(b->hist_off, b->tgt_off, b->n_requests, nh, nt, L.chunk_blocks, L.group, units, L.max_units, tch,
                      hdr, st, 1, 1 << 30, device_cus()));
  if (L.brd) {
    // history chunks of the requests for the reordered attention backward,
    // units of at most 128 rows for dX
    HIPCHK(launch_sched(b->hist_off, b->tgt_off, b->n_requests, nh, nt, L.rb_cb, 32, at<Unit>(ws, L.rb_units),
                        L.rb_maxu, at<int32_t>(ws, L.rb_tch), at<WsHeader>(ws, L.rb_hdr), st));
    HIPCHK(launch_sched(b->hist_off, b->tgt_off, b->n_requests, nh, nt, 4, 32, at<Unit>(ws, L.rb_unitsx), L.rb_maxx,
                        at<int32_t>(ws, L.rb_tchx), at<WsHeader>(ws, L.rb_hdrx), st));
  }
  HIPCHK(rec.mark("sched"));
  void* dkv = L.brd ? nullptr : at<char>(ws, L.dkv);
  // the recomputed per-layer tensors: in the workspace, or the training record
  const RecordLayout R = L.bfused ? record_layout(L) : RecordLayout{};
  char* rb = !L.bfused ? nullptr
                       : rec_in ? const_cast<char*>(static_cast<const char*>(rec_in))
                                : rec_out ? static_cast<char*>(rec_out) : at<char>(ws, L.rec);
  auto rec32 = [&](size_t off, int i, size_t per) { return reinterpret_cast<float*>(rb + off) + (size_t)i * per; };
  auto rec16 = [&](size_t off, int i, size_t per) { return reinterpret_cast<bf16_bits*>(rb + off) + (size_t)i * per; };
  auto RH = [&](int i) { return L.bfused ? rec32(R.h, i, nt * F) : at<float>(ws, L.hid) + (size_t)i * nt * F; };
  auto FA16 = [&](int i) { return rec16(R.a16, i, nt * d); };
  auto FU16 = [&](int i) { return rec16(R.u16, i, nt * d); };
  auto FH16 = [&](int i) { return rec16(R.h16, i, nt * F); };
  auto FS16 = [&](int i) { return rec16(R.s16, i, nt * d); };
  float* dhid = at<float>(ws, L.dhid);
  float* ds = at<float>(ws, L.ds);
  float* du = at<float>(ws, L.du);
  float* da = at<float>(ws, L.da);
  float* dq = at<float>(ws, L.dq);
  float* ds2 = at<float>(ws, L.ds2);
  float* dqp = at<float>(ws, L.dq_part);
  auto W = [&](const void* base, int i, size_t per) { return static_cast<const char*>(base) + i * per * es; };
  auto per_layer = [&](size_t off, int i, size_t per) { return at<float>(ws, off) + (size_t)i * per; };
  auto RS = [&](int i) { return per_layer(L.rs, i, nt * d); };
  auto RU = [&](int i) { return per_layer(L.ru, i, nt * d); };
  auto RQ = [&](int i) { return L.bfused ? rec32(R.q, i, nt * d) : per_layer(L.rq, i, nt * d); };
  auto RA = [&](int i) { return L.bfused ? rec32(R.a, i, nt * d) : per_layer(L.ra, i, nt * d); };
  auto RL = [&](int i) { return L.bfused ? rec32(R.lse, i, nt * h) : per_layer(L.rl, i, nt * h); };
  auto KVS = [&](int i) { return per_layer(L.kvs, i, nh * 2 * d); };
  // [W_K^0 | W_V^0 | W_K^1 | ...]: [d][n 2d], B operand of dX for every layer at once
  bf16_bits* wkv_all = bf ? at<bf16_bits>(ws, L.wkv) : nullptr;
  auto WKVT = [&](int i) { return at<bf16_bits>(ws, L.wkvt) + (size_t)i * d * 2 * d; };
  bf16_bits* xt = bf && !L.bfused ? at<bf16_bits>(ws, L.xt) : nullptr;
  bf16_bits* dkvt = bf && !L.bfused ? at<bf16_bits>(ws, L.dkvt) : nullptr;
  const int nh8 = static_cast<int>(L.nh8);
  auto gemm = [&](int a_bf, int b_bf, int M, int N, int K, const void* A, int64_t lda, int tA, const void* B,
                  int64_t ldb, int tB, float* C, int64_t ldc, float alpha, GemmEpi epi, const float* R,
                  int64_t ldr, float* C2) {
    return gemm_generic(a_bf, b_bf, M, N, K, A, lda, tA, B, ldb, tB, C, ldc, alpha, epi, R, ldr, C2, 0, st);
  };
  const float qscale = kLog2e / std::sqrt(static_cast<float>(L.dh));
  // History-side products (rows = history items) on bf16 inputs run on the
  // MFMA GEMM with [W_K | W_V] packed side by side, so K and V of a layer come
  // from one product, and every operand arranged with k contiguous (copies
  // of X^T, [W_K | W_V]^T and (dK | dV)^T); fp32 inputs keep fp32 products.
  if (bf) {
    const bf16_bits* X = static_cast<const bf16_bits*>(hist);
    if (!rec_out && !L.brd)
      HIPCHK(pack_wkv(static_cast<const bf16_bits*>(w->wk), static_cast<const bf16_bits*>(w->wv), n, d, wkv_all,
                      st));
    for (int i = 0; i < n && !rec_out; ++i) {
      const bf16_bits* Wk = reinterpret_cast<const bf16_bits*>(W(w->wk, i, (size_t)d * d));
      const bf16_bits* Wv = reinterpret_cast<const bf16_bits*>(W(w->wv, i, (size_t)d * d));
      if (!L.bfused) {
        HIPCHK(transpose_bf16(Wk, d, d, d, WKVT(i), d, d, st));
        HIPCHK(transpose_bf16(Wv, d, d, d, WKVT(i) + (size_t)d * d, d, d, st));
      }
    }
    if (!rec_out && !L.bfused) HIPCHK(transpose_bf16(X, d, static_cast<int>(nh), d, xt, nh8, nh8, st));
    if (L.bfused) {
      PackJobs pj{};
      pj.job[0] = {w->wk, at<char>(ws, L.fwkp), d, d, 0};
      pj.job[1] = {w->wv, at<char>(ws, L.fwvp), d, d, 0};
      pj.job[2] = {w->wo, at<char>(ws, L.fwop), d, d, 0};
      pj.job[3] = {w->wq, at<char>(ws, L.fwqp), d, d, 0};
      pj.job[4] = {w->w1, at<char>(ws, L.fw1p), d, F, 0};
      pj.job[5] = {w->w2, at<char>(ws, L.fw2p), F, d, 0};
      pj.job[6] = {w->w2, at<char>(ws, L.fw2t), d, F, 0, 1};
      pj.job[7] = {w->w1, at<char>(ws, L.fw1t), F, d, 0, 1};
      pj.job[8] = {w->wo, at<char>(ws, L.fwot), d, d, 0, 1};
      pj.job[9] = {w->wq, at<char>(ws, L.fwqt), d, d, 0, 1};
      HIPCHK(fast_pack_many(pj, 10, n, st));
    }
  }
  // persistent grid of the fused kernels: one workgroup per CU
  const int fgrid = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(L.max_units, device_cus())));
  HIPCHK(rec.mark("prep"));
  // forward recomputation in fp32: s^(i), u^(i), and per layer K|V, the
  // scaled queries, the attention output and its lse
  UpdatePrecise up{};
  if (L.bfused && !rec_in) {
    up.n_layers = n;
    up.F = F;
    up.n_tgt = nt;
    up.tgt = static_cast<const bf16_bits*>(tgt);
    up.tchunks = tch;
    up.part_acc = at<float>(ws, L.part_acc);
    up.part_ml = at<float2>(ws, L.part_ml);
    up.WoP = at<char>(ws, L.fwop);
    up.W1P = at<char>(ws, L.fw1p);
    up.W2P = at<char>(ws, L.fw2p);
    up.WqP = at<char>(ws, L.fwqp);
    up.mode = 0;
    up.s_out = RS(0);
    up.q_out = RQ(0);
    up.s16_out = FS16(0);
    HIPCHK(fast_update_precise(d, up, st));
    HIPCHK(rec.mark("target_gemm"));
  } else {
    HIPCHK(convert(bf, 0, tgt, RS(0), nt * d, st));
  }
  for (int i = 0; i < n && L.bfused && !rec_in; ++i) {
    FastAttnFwdPrecise f{};
    f.units = units;
    f.hdr = hdr;
    f.X = hist;
    f.n_hist = nh;
    f.WkP = at<char>(ws, L.fwkp);
    f.WvP = at<char>(ws, L.fwvp);
    f.layer = i;
    f.Q = RQ(i);
    f.part_acc = at<float>(ws, L.part_acc);
    f.part_ml = at<char>(ws, L.part_ml);
    f.n_tgt = nt;
    HIPCHK(fast_attn_fwd_precise(d, f, fgrid, st));
    HIPCHK(rec.mark("attn_fwd"));
    up.mode = 1;
    up.layer = i;
    up.s_in = RS(i);
    up.a_out = RA(i);
    up.lse_out = RL(i);
    up.u_out = RU(i);
    up.h_out = RH(i);
    up.s_out = RS(i + 1);
    up.q_out = i + 1 < n ? RQ(i + 1) : nullptr;
    up.a16_out = FA16(i);
    up.u16_out = FU16(i);
    up.h16_out = FH16(i);
    up.s16_out = i + 1 < n ? FS16(i + 1) : nullptr;
    HIPCHK(fast_update_precise(d, up, st));
    HIPCHK(rec.mark("target_gemm"));
  }
  for (int i = 0; i < n && !L.bfused; ++i) {
    float* kv = KVS(i);
    if (bf) {
      HIPCHK(gemm_mfma(static_cast<int>(nh), 2 * d, d, static_cast<const bf16_bits*>(hist), d, 0, WKVT(i), d, 1,
                       kv, 2 * d, 1.f, 0, nullptr, 0, st));
    } else {
      HIPCHK(gemm(0, 0, nh, d, d, hist, d, 0, W(w->wk, i, (size_t)d * d), d, 0, kv, 2 * d, 1.f, kEpiStore,
                  nullptr, 0, nullptr));
      HIPCHK(gemm(0, 0, nh, d, d, hist, d, 0, W(w->wv, i, (size_t)d * d), d, 0, kv + d, 2 * d, 1.f, kEpiStore,
                  nullptr, 0, nullptr));
    }
    HIPCHK(rec.mark("kv_gemm"));
    HIPCHK(gemm(0, bf, nt, d, d, RS(i), d, 0, W(w->wq, i, (size_t)d * d), d, 0, RQ(i), d, qscale, kEpiStore,
                nullptr, 0, nullptr));
    HIPCHK(rec.mark("target_gemm"));
    HIPCHK(attn_generic(L.dh, h, units, L.max_units, hdr, RQ(i), kv, d, at<float>(ws, L.part_acc),
                        at<float>(ws, L.part_ml), nt, st));
    HIPCHK(merge_generic(L.dh, h, nt, tch, at<float>(ws, L.part_acc), at<float>(ws, L.part_ml), RA(i), RL(i),
                         st));
    HIPCHK(rec.mark("attn_fwd"));
    HIPCHK(gemm(0, bf, nt, d, d, RA(i), d, 0, W(w->wo, i, (size_t)d * d), d, 0, RU(i), d, 1.f, kEpiAddRes, RS(i),
                d, nullptr));
    HIPCHK(gemm(0, bf, nt, F, d, RU(i), d, 0, W(w->w1, i, (size_t)d * F), F, 0, RH(i), F, 1.f, kEpiRelu, nullptr, 0,
                nullptr));
    HIPCHK(gemm(0, bf, nt, d, F, RH(i), F, 0, W(w->w2, i, (size_t)d * F), d, 0, RS(i + 1), d, 1.f, kEpiAddRes,
                RU(i), d, nullptr));
    HIPCHK(rec.mark("target_gemm"));
  }
  if (rec_out) {
    // the forward of a training step: Y = s^(n) in the storage dtype
    HIPCHK(convert(0, bf, RS(n), out, nt * d, st));
    HIPCHK(rec.mark("out"));
    return STCA_OK;
  }
  HIPCHK(convert(bf, 0, dout, ds, nt * d, st));
  // rows of requests without targets keep a zero gradient (and dK|dV^T's
  // padding columns stay zero)
  if (L.brd) {
    HIPCHK(rb_zero_untargeted(b->hist_off, b->tgt_off, b->n_requests, dhist, d, st));
  } else if (bf) {
    HIPCHK(zero_untargeted(b->hist_off, b->tgt_off, b->n_requests, nh, static_cast<bf16_bits*>(dkv), n * 2 * d,
                           n * 2 * d, dkvt, nh8, st));
  } else {
    HIPCHK(fill_f32(static_cast<float*>(dkv), 0.f, nh * 2 * d, st));
    HIPCHK(fill_f32(dhist, 0.f, nh * d, st));
  }
  HIPCHK(rec.mark("prep"));
  for (int i = n - 1; i >= 0; --i) {
    const float* s = RS(i);
    const float* u = RU(i);
    const float* a = RA(i);
    const float* kv = L.bfused ? nullptr : KVS(i);
    const void* W1 = W(w->w1, i, (size_t)d * F);
    const void* W2 = W(w->w2, i, (size_t)d * F);
    const void* Wo = W(w->wo, i, (size_t)d * d);
    const void* Wq = W(w->wq, i, (size_t)d * d);
    // s' = u + ReLU(u W1) W2.  The ReLU gates are those of the fp32
    // recomputation (hid > 0 exactly where u W1 > 0); on the bf16 path the
    // products that only carry gradients take bf16 copies of their fp32
    // operands on the bf16 MFMA (fp32 sums), the others stay fp32.
    const float* hid = RH(i);
    if (L.bfused) {
      const int nti = static_cast<int>(nt);
      float* gp = at<float>(ws, L.gpart);
      const int64_t gpf = L.gpart_floats;
      auto B = [&](size_t off) { return at<bf16_bits>(ws, off); };
      UpdateGrad ug{};
      ug.layer = i;
      ug.F = F;
      ug.n_tgt = nt;
      ug.ds = ds;
      ug.h = hid;
      ug.du_out = du;
      ug.da_out = da;
      ug.ds16_out = B(L.b_ds);
      ug.dh16_out = B(L.b_dhid);
      ug.du16_out = B(L.b_du);
      ug.W2TP = at<char>(ws, L.fw2t);
      ug.W1TP = at<char>(ws, L.fw1t);
      ug.WoTP = at<char>(ws, L.fwot);
      if (i + 1 < n) {
        // ds = du + dq W_Q^T of layer i + 1, formed inside the update
        ug.du_in = du;
        ug.dq16 = at<bf16_bits>(ws, L.b_dq);
        ug.WqTP = at<char>(ws, L.fwqt);
        ug.q_layer = i + 1;
      }
      HIPCHK(fast_update_grad(d, ug, st));
      // dW_2 = h^T ds, dW_1 = u^T dH, dW_O = a^T du, and dW_Q = s^T dq of
      // layer i + 1: one grouped launch
      const GemmSpec wg[4] = {
          {F, d, nti, FH16(i), F, 1, B(L.b_ds), d, 0, dw->dw2 + (size_t)i * F * d, d, 1.f, 0},
          {d, F, nti, FU16(i), d, 1, B(L.b_dhid), F, 0, dw->dw1 + (size_t)i * d * F, F, 1.f, 0},
          {d, d, nti, FA16(i), d, 1, B(L.b_du), d, 0, dw->dwo + (size_t)i * d * d, d, 1.f, 0},
          {d, d, nti, FS16(i + 1 < n ? i + 1 : i), d, 1, B(L.b_dq), d, 0, dw->dwq + (size_t)(i + 1) * d * d, d, 1.f,
           0}};
      HIPCHK(gemm_mfma_group(wg, i + 1 < n ? 4 : 3, gp, gpf, st));
    } else if (bf) {
      const int nti = static_cast<int>(nt);
      float* gp = at<float>(ws, L.gpart);
      const int64_t gpf = L.gpart_floats;
      auto bcopy = [&](const float* src, size_t off, int64_t count) {
        return convert(0, 1, src, at<bf16_bits>(ws, off), count, st);
      };
      auto B = [&](size_t off) { return at<bf16_bits>(ws, off); };
      auto WB = [&](const void* p) { return static_cast<const bf16_bits*>(p); };
      HIPCHK(bcopy(hid, L.b_hid, nt * F));
      HIPCHK(bcopy(ds, L.b_ds, nt * d));
      HIPCHK(bcopy(u, L.b_u, nt * d));
      HIPCHK(bcopy(a, L.b_a, nt * d));
      HIPCHK(gemm_mfma(F, d, nti, B(L.b_hid), F, 1, B(L.b_ds), d, 0, dw->dw2 + (size_t)i * F * d, d, 1.f, 0, gp, gpf,
                       st));
      HIPCHK(gemm_mfma(nti, F, d, B(L.b_ds), d, 0, WB(W2), d, 1, dhid, F, 1.f, 0, nullptr, 0, st));
      HIPCHK(relu_mask_mul(dhid, hid, nt * F, st));
      HIPCHK(bcopy(dhid, L.b_dhid, nt * F));
      HIPCHK(gemm_mfma(d, F, nti, B(L.b_u), d, 1, B(L.b_dhid), F, 0, dw->dw1 + (size_t)i * d * F, F, 1.f, 0, gp, gpf,
                       st));
      HIPCHK(hipMemcpyAsync(du, ds, 4 * nt * d, hipMemcpyDeviceToDevice, st));
      HIPCHK(gemm_mfma(nti, d, F, B(L.b_dhid), F, 0, WB(W1), F, 1, du, d, 1.f, 1, nullptr, 0, st));
      // u = s + a Wo
      HIPCHK(bcopy(du, L.b_du, nt * d));
      HIPCHK(gemm_mfma(d, d, nti, B(L.b_a), d, 1, B(L.b_du), d, 0, dw->dwo + (size_t)i * d * d, d, 1.f, 0, gp, gpf,
                       st));
      HIPCHK(gemm_mfma(nti, d, d, B(L.b_du), d, 0, WB(Wo), d, 1, da, d, 1.f, 0, nullptr, 0, st));
    } else {
      HIPCHK(gemm(0, 0, F, d, nt, hid, F, 1, ds, d, 0, dw->dw2 + (size_t)i * F * d, d, 1.f, kEpiStore, nullptr, 0,
                  nullptr));
      HIPCHK(gemm(0, 0, nt, F, d, ds, d, 0, W2, d, 1, dhid, F, 1.f, kEpiStore, nullptr, 0, nullptr));
      HIPCHK(relu_mask_mul(dhid, hid, nt * F, st));
      HIPCHK(gemm(0, 0, d, F, nt, u, d, 1, dhid, F, 0, dw->dw1 + (size_t)i * d * F, F, 1.f, kEpiStore, nullptr, 0,
                  nullptr));
      HIPCHK(gemm(0, 0, nt, d, F, dhid, F, 0, W1, F, 1, du, d, 1.f, kEpiAddRes, ds, d, nullptr));
      // u = s + a Wo
      HIPCHK(gemm(0, 0, d, d, nt, a, d, 1, du, d, 0, dw->dwo + (size_t)i * d * d, d, 1.f, kEpiStore, nullptr, 0,
                  nullptr));
      HIPCHK(gemm(0, 0, nt, d, d, du, d, 0, Wo, d, 1, da, d, 1.f, kEpiStore, nullptr, 0, nullptr));
    }
    HIPCHK(rec.mark("target_gemm"));
    // attention (softmax weights rebuilt from the same q, K, V and lse that
    // gave a, so rowsum(dA * A) matches them)
    void* dkv_i = L.brd ? nullptr : bf ? static_cast<void*>(static_cast<bf16_bits*>(dkv) + (size_t)i * 2 * d) : dkv;
    if (L.brd) {
      // reordered form: U, H and statistics per request, then one pass over
      // the history (E, Z, Y), then dW_K^j, dW_V^j and dq^j from Z and Y
      const bf16_bits* Wk = reinterpret_cast<const bf16_bits*>(W(w->wk, i, (size_t)d * d));
      const bf16_bits* Wv = reinterpret_cast<const bf16_bits*>(W(w->wv, i, (size_t)d * d));
      bf16_bits* q16 = at<bf16_bits>(ws, L.rb_q16);
      bf16_bits* da16 = at<bf16_bits>(ws, L.rb_da16);
      bf16_bits* Z = at<bf16_bits>(ws, L.rb_z);
      bf16_bits* Y = at<bf16_bits>(ws, L.rb_y);
      RbPrep pp{};
      pp.tgt_off = b->tgt_off;
      pp.n_requests = b->n_requests;
      pp.layer = i;
      pp.n_layers = n;
      pp.Q = RQ(i);
      pp.da = da;
      pp.a = a;
      pp.lse = RL(i);
      pp.Wk = Wk;
      pp.Wv = Wv;
      pp.U16 = at<_Float16>(ws, L.rb_u16);
      pp.Wr = at<bf16_bits>(ws, L.rb_w);
      pp.stats = at<float>(ws, L.rb_st);
      pp.q16 = q16;
      pp.da16 = da16;
      HIPCHK(rb_prep(d, pp, st));
      RbAttn ra{};
      ra.units = at<Unit>(ws, L.rb_units);
      ra.hdr = at<WsHeader>(ws, L.rb_hdr);
      ra.X = hist;
      ra.n_hist = nh;
      ra.n_tgt = nt;
      ra.layer = i;
      ra.n_layers = n;
      ra.U16 = pp.U16;
      ra.Wr = pp.Wr;
      ra.stats = pp.stats;
      ra.E = at<bf16_bits>(ws, L.rb_e);
      ra.lde = (int64_t)n * 2 * kRbPairs;
      ra.Z = Z;
      ra.Y = Y;
      ra.tchunks = at<int32_t>(ws, L.rb_tch);
      ra.Zp = at<float>(ws, L.rb_zp);
      ra.Yp = at<float>(ws, L.rb_yp);
      ra.first = at<int32_t>(ws, L.rb_first);
      HIPCHK(rb_attn(d, ra, static_cast<int>(L.rb_maxu), st));
      HIPCHK(rb_reduce(d, b->tgt_off, b->n_requests, ra.tchunks, ra.first, ra.Zp, ra.Yp, Z, Y, nt, st));
      HIPCHK(rec.mark("attn_bwd"));
      const int nti = static_cast<int>(nt);
      GemmSpec g[2 * 8], gq[8];
      for (int j = 0; j < h; ++j) {
        const size_t zo = (size_t)j * nt * d;
        g[j] = {d, 32, nti, Z + zo, d, 1, q16 + 32 * j, d, 0, dw->dwk + (size_t)i * d * d + 32 * j, d, kLn2, 0};
        g[h + j] = {d, 32, nti, Y + zo, d, 1, da16 + 32 * j, d, 0, dw->dwv + (size_t)i * d * d + 32 * j, d, 1.f, 0};
        gq[j] = {nti, 32, d, Z + zo, d, 0, Wk + 32 * j, d, 0, dq + 32 * j, d, 1.f / std::sqrt(32.f), 0};
      }
      HIPCHK(gemm_mfma_group(g, 2 * h, at<float>(ws, L.gpart), L.gpart_floats, st));
      HIPCHK(gemm_mfma_group(gq, h, nullptr, 0, st));
      HIPCHK(convert(0, 1, dq, at<bf16_bits>(ws, L.b_dq), nt * d, st));
      HIPCHK(rec.mark("kv_grads"));
    } else if (L.bfused) {
      FastAttnBwd f{};
      f.units = units;
      f.hdr = hdr;
      f.X = hist;
      f.n_hist = nh;
      f.WkP = at<char>(ws, L.fwkp);
      f.WvP = at<char>(ws, L.fwvp);
      f.layer = i;
      f.Q = RQ(i);
      f.a = a;
      f.da = da;
      f.lse = RL(i);
      f.dKV = static_cast<bf16_bits*>(dkv_i);
      f.ldkv = n * 2 * d;
      f.dq_part = dqp;
      f.n_tgt = nt;
      HIPCHK(fast_attn_bwd(d, f, fgrid, st));
    } else {
      HIPCHK(attn_bwd_generic(L.dh, h, units, L.max_units, hdr, b->tgt_off, RQ(i), kv, d, a, da, RL(i), dqp, dkv_i,
                              bf ? n * 2 * d : 2 * d, bf, bf ? dkvt + (size_t)i * 2 * d * nh8 : nullptr, nh8, nt,
                              st));
    }
    // dq: fp32 for the fp32 products, else only its bf16 copy
    if (!L.brd) {
      HIPCHK(reduce_chunks(nt, d, tch, dqp, bf ? nullptr : dq, bf ? at<bf16_bits>(ws, L.b_dq) : nullptr, 1.f, st));
      HIPCHK(rec.mark("attn_bwd"));
    }
    // q = s Wq
    if (bf) {
      const int nti = static_cast<int>(nt);
      const bf16_bits* s16 = L.bfused ? FS16(i) : at<bf16_bits>(ws, L.b_s);
      if (!L.bfused) HIPCHK(convert(0, 1, s, at<bf16_bits>(ws, L.b_s), nt * d, st));
      // dW_Q = s^T dq: in the fused form it joins the next layer's group of
      // weight gradients (its operands stay until the next attention
      // backward), the last one runs alone
      if (!L.bfused || i == 0)
        HIPCHK(gemm_mfma(d, d, nti, s16, d, 1, at<bf16_bits>(ws, L.b_dq), d, 0,
                         dw->dwq + (size_t)i * d * d, d, 1.f, 0, at<float>(ws, L.gpart), L.gpart_floats, st));
      // ds of the layer below = du + dq W_Q^T: the fused form's next update
      // forms it; the last one (the target gradient) is a product here
      if (L.bfused && i == 0) {
        UpdateGrad fin{};
        fin.layer = 0;
        fin.W2TP = at<char>(ws, L.fw2t);  // valid but unread in this mode
        fin.W1TP = at<char>(ws, L.fw1t);
        fin.WoTP = at<char>(ws, L.fwot);
        fin.F = F;
        fin.n_tgt = nt;
        fin.du_in = du;
        fin.dq16 = at<bf16_bits>(ws, L.b_dq);
        fin.WqTP = at<char>(ws, L.fwqt);
        fin.q_layer = 0;
        fin.ds_out = ds2;
        HIPCHK(fast_update_grad(d, fin, st));
      } else if (!L.bfused) {
        HIPCHK(hipMemcpyAsync(ds2, du, 4 * nt * d, hipMemcpyDeviceToDevice, st));
        HIPCHK(gemm_mfma(nti, d, d, at<bf16_bits>(ws, L.b_dq), d, 0, static_cast<const bf16_bits*>(Wq), d, 1, ds2,
                         d, 1.f, 1, nullptr, 0, st));
      }
    } else {
      HIPCHK(gemm(0, 0, d, d, nt, s, d, 1, dq, d, 0, dw->dwq + (size_t)i * d * d, d, 1.f, kEpiStore, nullptr, 0,
                  nullptr));
      HIPCHK(gemm(0, 0, nt, d, d, dq, d, 0, Wq, d, 1, ds2, d, 1.f, kEpiAddRes, du, d, nullptr));
    }
    HIPCHK(rec.mark("target_gemm"));
    // [K | V] = X [W_K | W_V]: on the bf16 path every layer's dK | dV is kept
    // and the history-side gradients are formed once after the loop
    if (!bf) {
      const float* dKV = static_cast<const float*>(dkv);
      const void* Wk = W(w->wk, i, (size_t)d * d);
      const void* Wv = W(w->wv, i, (size_t)d * d);
      HIPCHK(gemm(0, 0, d, d, nh, hist, d, 1, dKV, 2 * d, 0, dw->dwk + (size_t)i * d * d, d, 1.f, kEpiStore,
                  nullptr, 0, nullptr));
      HIPCHK(gemm(0, 0, d, d, nh, hist, d, 1, dKV + d, 2 * d, 0, dw->dwv + (size_t)i * d * d, d, 1.f, kEpiStore,
                  nullptr, 0, nullptr));
      HIPCHK(rec.mark("dw_kv"));
      HIPCHK(gemm_generic(0, 0, nh, d, d, dKV, 2 * d, 0, Wk, d, 1, dhist, d, 1.f, kEpiStore, nullptr, 0, nullptr, 1,
                          st));
      HIPCHK(gemm_generic(0, 0, nh, d, d, dKV + d, 2 * d, 0, Wv, d, 1, dhist, d, 1.f, kEpiStore, nullptr, 0,
                          nullptr, 1, st));
      HIPCHK(rec.mark("dx"));
    }
    std::swap(ds, ds2);
  }
  if (L.brd) {
    // dX = E W_r over every layer's pairs (K = n 2 kRbPairs), per request
    const int64_t kr = (int64_t)n * 2 * kRbPairs;
    HIPCHK(gemm_ring_units(d, static_cast<int>(kr), at<bf16_bits>(ws, L.rb_e), kr, at<bf16_bits>(ws, L.rb_w), d,
                           kr * d, dhist, d, at<Unit>(ws, L.rb_unitsx), at<WsHeader>(ws, L.rb_hdrx), device_cus(),
                           st));
    HIPCHK(rec.mark("dx"));
  } else if (bf) {
    // [dW_K^i | dW_V^i] for every layer = X^T [dK^i | dV^i] (one product over
    // the history rows: the fused form reads X and dK | dV row-major, the
    // unfused one their transposed copies), then
    // dX = sum_i [dK^i | dV^i] [W_K^i | W_V^i]^T as one product with
    // K = n 2d, written once
    float* dwkv = at<float>(ws, L.dwkv);
    const int n_cu = device_cus();
    if (L.bfused)
      HIPCHK(gemm_ring(d, n * 2 * d, static_cast<int>(nh), static_cast<const bf16_bits*>(hist), d, 1,
                       static_cast<const bf16_bits*>(dkv), n * 2 * d, 0, dwkv, n * 2 * d, 1.f, 0,
                       at<float>(ws, L.gpart), L.gpart_floats, n_cu, st));
    else
      HIPCHK(gemm_ring(d, n * 2 * d, nh8, xt, nh8, 0, dkvt, nh8, 1, dwkv, n * 2 * d, 1.f, 0, at<float>(ws, L.gpart),
                       L.gpart_floats, n_cu, st));
    HIPCHK(split_dwkv(dwkv, n, d, dw->dwk, dw->dwv, st));
    HIPCHK(rec.mark("dw_kv"));
    HIPCHK(gemm_ring(static_cast<int>(nh), d, n * 2 * d, static_cast<const bf16_bits*>(dkv), n * 2 * d, 0, wkv_all,
                     n * 2 * d, 1, dhist, d, 1.f, 0, nullptr, 0, n_cu, st));
    HIPCHK(rec.mark("dx"));
  }
  HIPCHK(convert(0, 0, ds, dtgt, nt * d, st));
  HIPCHK(rec.mark("out"));
  return STCA_OK;
}

}  // namespace

extern "C" {

int stca_path(const stca_dims_t* dims) { return path_of(dims); }

size_t stca_workspace_size(const stca_dims_t* dims, const stca_batch_t* batch, int with_backward) {
  Layout L;
  if (make_layout(dims, batch, with_backward, false, &L) != STCA_OK) return 0;
  return L.total;
}

size_t stca_saved_size(const stca_dims_t* dims, const stca_batch_t* batch) {
  stca_saved_layout_t s;
  if (!saved_layout(dims, batch, &s)) return 0;
  return s.total;
}

stca_status_t stca_saved_layout(const stca_dims_t* dims, const stca_batch_t* batch, stca_saved_layout_t* layout) {
  if (!layout) return STCA_ERR_INVALID_ARG;
  const int p = path_of(dims);
  if (p < 0) return static_cast<stca_status_t>(p);
  stca_status_t st = check_batch(batch);
  if (st != STCA_OK) return st;
  saved_layout(dims, batch, layout);
  return STCA_OK;
}

stca_status_t stca_forward(const stca_dims_t* dims, const stca_batch_t* batch, const void* hist, const void* tgt,
                           const stca_weights_t* w, void* out, void* saved, void* ws, size_t ws_bytes,
                           hipStream_t stream) {
  stca_status_t st = check_common(dims, batch, hist, tgt, w, ws);
  if (st != STCA_OK) return st;
  if ((batch->n_tgt > 0 && !out) || (out && !aligned16(out)) || (saved && !aligned16(saved)))
    return STCA_ERR_INVALID_ARG;
  Layout L;
  st = make_layout(dims, batch, 0, saved != nullptr, &L);
  if (st != STCA_OK) return st;
  if (ws_bytes < L.total) return STCA_ERR_WORKSPACE;
  stca_saved_layout_t SL{};
  saved_layout(dims, batch, &SL);
  Rec rec;
  if (L.path == 1) return forward_fast(L, batch, hist, tgt, w, out, saved, SL, ws, stream, rec);
  return forward_generic(L, dims->dtype == STCA_BF16, batch, hist, tgt, w, out, saved, SL, ws, stream, rec);
}

int stca_forward_launch_count(const stca_dims_t* dims, const stca_batch_t* batch) {
  Layout L;
  if (make_layout(dims, batch, 0, false, &L) != STCA_OK) return -1;
  // sched, one repack launch, the initial update, then per layer
  if (L.path == 1) {
    const bool std_part = !L.reord || L.mixed, reo_part = L.reord;
    // schedules, one repack launch, the initial update, the K/V GEMM; per
    // layer: U, the standard form's attention (two fused launches or one
    // over materialised K/V), the reordered attention and merge, the update
    const int per_layer = (reo_part ? 3 : 0) + (std_part ? (L.mat ? 1 : 2) : 0) + 1;
    return (std_part ? 1 : 0) + (reo_part ? 1 : 0) + 1 + 1 + (L.mat ? 1 : 0) + per_layer * L.n;
  }
  return 1 + 1 + 8 * L.n + 1;
}

stca_status_t stca_forward_profiled(const stca_dims_t* dims, const stca_batch_t* batch, const void* hist,
                                    const void* tgt, const stca_weights_t* w, void* out, void* saved, void* ws,
                                    size_t ws_bytes, hipStream_t stream, hipEvent_t* events, int n_events,
                                    const char** labels) {
  stca_status_t st = check_common(dims, batch, hist, tgt, w, ws);
  if (st != STCA_OK) return st;
  if ((batch->n_tgt > 0 && !out) || (out && !aligned16(out)) || (saved && !aligned16(saved)) || !events)
    return STCA_ERR_INVALID_ARG;
  Layout L;
  st = make_layout(dims, batch, 0, saved != nullptr, &L);
  if (st != STCA_OK) return st;
  if (ws_bytes < L.total) return STCA_ERR_WORKSPACE;
  if (n_events < stca_forward_launch_count(dims, batch) + 1) return STCA_ERR_INVALID_ARG;
  stca_saved_layout_t SL{};
  saved_layout(dims, batch, &SL);
  Rec rec;
  rec.ev = events;
  rec.n = n_events;
  rec.labels = labels;
  rec.st = stream;
  if (L.path == 1) return forward_fast(L, batch, hist, tgt, w, out, saved, SL, ws, stream, rec);
  return forward_generic(L, dims->dtype == STCA_BF16, batch, hist, tgt, w, out, saved, SL, ws, stream, rec);
}

stca_status_t stca_backward(const stca_dims_t* dims, const stca_batch_t* batch, const void* hist, const void* tgt,
                            const stca_weights_t* w, const void* dout, float* dhist, float* dtgt,
                            const stca_wgrads_t* dw, void* ws, size_t ws_bytes, hipStream_t stream) {
  stca_status_t st = check_common(dims, batch, hist, tgt, w, ws);
  if (st != STCA_OK) return st;
  if (!dw || (batch->n_tgt > 0 && (!dout || !dtgt)) || (batch->n_hist > 0 && !dhist))
    return STCA_ERR_INVALID_ARG;
  if (!dw->dwq || !dw->dwk || !dw->dwv || !dw->dwo || !dw->dw1 || !dw->dw2) return STCA_ERR_INVALID_ARG;
  const void* ptrs[] = {dout, dhist, dtgt, dw->dwq, dw->dwk, dw->dwv, dw->dwo, dw->dw1, dw->dw2};
  for (const void* q : ptrs)
    if (q && !aligned16(q)) return STCA_ERR_INVALID_ARG;
  Layout L;
  st = make_layout(dims, batch, 1, true, &L);
  if (st != STCA_OK) return st;
  if (ws_bytes < L.total) return STCA_ERR_WORKSPACE;
  Rec none;
  return backward_generic(L, dims->dtype == STCA_BF16, batch, hist, tgt, w, dout, dhist, dtgt, dw, ws, stream, none);
}

int stca_backward_launch_count(const stca_dims_t* dims, const stca_batch_t* batch) {
  Layout L;
  if (make_layout(dims, batch, 1, true, &L) != STCA_OK) return -1;
  // sched, prep, 4 per layer (recomputation), prep, then per layer 5 (fp32)
  // or 3 plus the two history-side products of every layer (bf16), out
  // fused: sched, prep, the initial update, 2 per layer (attention, update), prep,
  // 3 per layer, dW_KV, dX, out
  // reordered: ... 4 per layer (target side, attention, K/V-side gradients,
  // target side), dX, out
  if (L.brd) return 6 + 6 * L.n;
  if (L.bfused) return 7 + 5 * L.n;
  return dims->dtype == STCA_BF16 ? 6 + 7 * L.n : 4 + 9 * L.n;
}

stca_status_t stca_backward_profiled(const stca_dims_t* dims, const stca_batch_t* batch, const void* hist,
                                     const void* tgt, const stca_weights_t* w, const void* dout, float* dhist,
                                     float* dtgt, const stca_wgrads_t* dw, void* ws, size_t ws_bytes,
                                     hipStream_t stream, hipEvent_t* events, int n_events, const char** labels) {
  if (!events || n_events < stca_backward_launch_count(dims, batch) + 1) return STCA_ERR_INVALID_ARG;
  stca_status_t st = check_common(dims, batch, hist, tgt, w, ws);
  if (st != STCA_OK) return st;
  if (!dw || (batch->n_tgt > 0 && (!dout || !dtgt)) || (batch->n_hist > 0 && !dhist))
    return STCA_ERR_INVALID_ARG;
  if (!dw->dwq || !dw->dwk || !dw->dwv || !dw->dwo || !dw->dw1 || !dw->dw2) return STCA_ERR_INVALID_ARG;
  const void* ptrs[] = {dout, dhist, dtgt, dw->dwq, dw->dwk, dw->dwv, dw->dwo, dw->dw1, dw->dw2};
  for (const void* q : ptrs)
    if (q && !aligned16(q)) return STCA_ERR_INVALID_ARG;
  Layout L;
  st = make_layout(dims, batch, 1, true, &L);
  if (st != STCA_OK) return st;
  if (ws_bytes < L.total) return STCA_ERR_WORKSPACE;
  Rec rec;
  rec.ev = events;
  rec.n = n_events;
  rec.labels = labels;
  rec.st = stream;
  return backward_generic(L, dims->dtype == STCA_BF16, batch, hist, tgt, w, dout, dhist, dtgt, dw, ws, stream, rec);
}

size_t stca_train_record_size(const stca_dims_t* dims, const stca_batch_t* batch) {
  Layout L;
  if (make_layout(dims, batch, 1, true, &L) != STCA_OK || !L.bfused) return 0;
  return record_layout(L).total;
}

stca_status_t stca_forward_train(const stca_dims_t* dims, const stca_batch_t* batch, const void* hist,
                                 const void* tgt, const stca_weights_t* w, void* out, void* record, void* ws,
                                 size_t ws_bytes, hipStream_t stream) {
  stca_status_t st = check_common(dims, batch, hist, tgt, w, ws);
  if (st != STCA_OK) return st;
  if ((batch->n_tgt > 0 && !out) || (out && !aligned16(out)) || !record || !aligned16(record))
    return STCA_ERR_INVALID_ARG;
  Layout L;
  st = make_layout(dims, batch, 1, true, &L);
  if (st != STCA_OK) return st;
  if (!L.bfused) return STCA_ERR_UNSUPPORTED;
  if (ws_bytes < L.total) return STCA_ERR_WORKSPACE;
  Rec none;
  return backward_generic(L, 1, batch, hist, tgt, w, nullptr, nullptr, nullptr, nullptr, ws, stream, none, nullptr,
                          record, out);
}

stca_status_t stca_backward_record(const stca_dims_t* dims, const stca_batch_t* batch, const void* hist,
                                   const void* tgt, const stca_weights_t* w, const void* record, const void* dout,
                                   float* dhist, float* dtgt, const stca_wgrads_t* dw, void* ws, size_t ws_bytes,
                                   hipStream_t stream) {
  stca_status_t st = check_common(dims, batch, hist, tgt, w, ws);
  if (st != STCA_OK) return st;
  if (!dw || (batch->n_tgt > 0 && (!dout || !dtgt)) || (batch->n_hist > 0 && !dhist) || !record ||
      !aligned16(record))
    return STCA_ERR_INVALID_ARG;
  if (!dw->dwq || !dw->dwk || !dw->dwv || !dw->dwo || !dw->dw1 || !dw->dw2) return STCA_ERR_INVALID_ARG;
  const void* ptrs[] = {dout, dhist, dtgt, dw->dwq, dw->dwk, dw->dwv, dw->dwo, dw->dw1, dw->dw2};
  for (const void* q : ptrs)
    if (q && !aligned16(q)) return STCA_ERR_INVALID_ARG;
  Layout L;
  st = make_layout(dims, batch, 1, true, &L);
  if (st != STCA_OK) return st;
  if (!L.bfused) return STCA_ERR_UNSUPPORTED;
  if (ws_bytes < L.total) return STCA_ERR_WORKSPACE;
  Rec none;
  return backward_generic(L, 1, batch, hist, tgt, w, dout, dhist, dtgt, dw, ws, stream, none, record);
}

stca_status_t stca_device_status(const void* ws, hipStream_t stream) {
  if (!ws) return STCA_ERR_INVALID_ARG;
  WsHeader h;
  if (hipMemcpyAsync(&h, ws, sizeof(h), hipMemcpyDeviceToHost, stream) != hipSuccess) return STCA_ERR_HIP;
  if (hipStreamSynchronize(stream) != hipSuccess) return STCA_ERR_HIP;
  if (h.status != STCA_OK) return static_cast<stca_status_t>(h.status);
  return h.range ? STCA_ERR_RANGE : STCA_OK;
}

const char* stca_status_string(stca_status_t s) {
  switch (s) {
    case STCA_OK: return "ok";
    case STCA_ERR_INVALID_ARG: return "invalid argument";
    case STCA_ERR_UNSUPPORTED: return "unsupported shape or dtype";
    case STCA_ERR_WORKSPACE: return "workspace or saved buffer too small";
    case STCA_ERR_HIP: return "HIP runtime error";
    case STCA_ERR_RANGE: return "an fp16 intermediate overflowed or a value was not finite";
  }
  return "unknown status";
}

}  // extern "C"
