// C ABI of the paper-exact layer stack (Sec. 3.1): per layer the history is
// transformed by its own SwiGLU block and LayerNorm, the target query starts
// as LN(SwiGLUFFN^(1)(x_t)), each later query is the LayerNorm'd SwiGLU of the
// compressed concatenation of the layer summaries and x_t (Eq. fuse), and the
// stack ends in the head token z (the Eq. of z).  The attention itself is the
// same target-to-history cross attention as stca_forward, computed once per
// request for all its targets (Sec. 3.2).
#include <algorithm>
#include <cmath>

#include "api_common.h"
#include "common.h"
#include "fast.h"
#include "internal.h"
#include "paper.h"

using namespace stca;
using namespace stca::api;

namespace {

struct PaperLayout {
  int path;  // 1: bf16 MFMA kernels, 0: generic fp32 kernels
  int d, h, n, F, dh;
  int64_t nh, nt;
  int chunk_blocks;
  int64_t max_units;
  bool any_narrow, any_wide;
  size_t hdr, units, tchunks, part_acc, part_ml;
  size_t q, a, cat, f, hu, hv, y, qs;  // target side, fp32
  size_t qn, wsp, wkp, wvp, xt16;      // bf16 MFMA path
  size_t hhu, hhv, hy, xt32, kv32;     // generic path: history side
  size_t total;
};

bool paper_saved_layout(const stca_dims_t* dims, const stca_batch_t* b, stca_paper_saved_layout_t* s) {
  if (path_of(dims) < 0 || check_batch(b) != STCA_OK) return false;
  const size_t d = dims->d_model, nt = b->n_tgt, nh = b->n_hist, n = dims->n_layers, h = dims->n_heads;
  Bump m;
  s->q = m.take(4 * n * nt * d);
  s->a = m.take(4 * n * nt * d);
  s->o = m.take(4 * nt * n * d);
  s->lse = m.take(4 * n * nt * h);
  s->xt = m.take(4 * n * nh * d);
  s->total = m.off;
  return true;
}

bool make_paper_layout(const stca_dims_t* dims, const stca_batch_t* b, PaperLayout* L) {
  const int p = path_of(dims);
  if (p < 0 || check_batch(b) != STCA_OK) return false;
  L->path = p;
  L->d = dims->d_model;
  L->h = dims->n_heads;
  L->n = dims->n_layers;
  L->F = dims->ffn_hidden;
  L->dh = L->d / L->h;
  L->nh = b->n_hist;
  L->nt = b->n_tgt;
  L->chunk_blocks = chunk_blocks_auto(b, device_cus(), dims->chunk_blocks);
  L->max_units = max_units_for(b, L->chunk_blocks, kTargetGroup);
  L->any_narrow = L->any_wide = true;
  if (b->tgt_off_host) {
    L->any_narrow = L->any_wide = false;
    for (int r = 0; r < b->n_requests; ++r) {
      const int64_t m = b->tgt_off_host[r + 1] - b->tgt_off_host[r];
      for (int64_t g0 = 0; g0 < m; g0 += kTargetGroup) {
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
  L->part_acc = m.take(4 * kMaxChunks * nt * d);
  L->part_ml = m.take(8 * kMaxChunks * nt * L->h);
  L->q = m.take(4 * nt * d);
  L->a = m.take(4 * nt * d);
  L->cat = m.take(4 * nt * n * d);
  L->f = m.take(4 * nt * d);
  L->hu = m.take(4 * nt * F);
  L->hv = m.take(4 * nt * F);
  L->y = m.take(4 * nt * d);
  L->qs = m.take(4 * nt * d);
  if (p == 1) {
    L->qn = m.take(2 * nt * d);
    L->wsp = m.take(n * swiglu_packed_bytes(L->d, L->F));
    L->wkp = m.take(2 * n * d * d);
    L->wvp = m.take(2 * n * d * d);
    L->xt16 = m.take(2 * nh * d);
  } else {
    L->hhu = m.take(4 * nh * F);
    L->hhv = m.take(4 * nh * F);
    L->hy = m.take(4 * nh * d);
    L->xt32 = m.take(4 * nh * d);
    L->kv32 = m.take(4 * nh * 2 * d);
  }
  L->total = m.off;
  return true;
}

int paper_launch_count(const PaperLayout& L) {
  // q^(1): block (4) + LN; per layer the history transform, the query, the
  // attention, the merge and W_O; per fusion two GEMMs, the block and LN; the
  // head: two GEMMs, the block and the output conversion
  if (L.path == 1) return 4 + 5 + 7 * L.n + 7 * (L.n - 1) + 7;
  return 1 + 5 + 11 * L.n + 7 * (L.n - 1) + 7;
}

stca_status_t check_paper(const stca_dims_t* dims, const stca_batch_t* b, const void* hist, const void* tgt,
                          const stca_paper_weights_t* w, void* z, void* saved, void* ws) {
  const int p = path_of(dims);
  if (p < 0) return static_cast<stca_status_t>(p);
  stca_status_t st = check_batch(b);
  if (st != STCA_OK) return st;
  if (!w || !ws || (b->n_hist > 0 && !hist) || (b->n_tgt > 0 && (!tgt || !z))) return STCA_ERR_INVALID_ARG;
  if (!w->ffn_u || !w->ffn_v || !w->ffn_o || !w->wq || !w->wk || !w->wv || !w->wo || !w->wz || !w->z_u ||
      !w->z_v || !w->z_o || (dims->n_layers > 1 && !w->wc))
    return STCA_ERR_INVALID_ARG;
  const void* ptrs[] = {hist, tgt, z, saved, ws, w->ffn_u, w->ffn_v, w->ffn_o, w->wq, w->wk, w->wv,
                        w->wo, w->wc, w->wz, w->z_u, w->z_v, w->z_o};
  for (const void* q : ptrs)
    if (q && !aligned16(q)) return STCA_ERR_INVALID_ARG;
  return STCA_OK;
}

stca_status_t forward_paper(const PaperLayout& L, int bf, const stca_batch_t* b, const void* hist, const void* tgt,
                            const stca_paper_weights_t* w, void* z, void* saved,
                            const stca_paper_saved_layout_t& SL, void* ws, hipStream_t st, Rec& rec) {
  HIPCHK(rec.start());
  const int d = L.d, n = L.n, F = L.F, h = L.h;
  const int64_t nt = L.nt, nh = L.nh;
  const size_t es = bf ? 2 : 4;
  WsHeader* hdr = at<WsHeader>(ws, L.hdr);
  Unit* units = at<Unit>(ws, L.units);
  int32_t* tch = at<int32_t>(ws, L.tchunks);
  float* pacc = at<float>(ws, L.part_acc);
  float* pml = at<float>(ws, L.part_ml);
  float* hu = at<float>(ws, L.hu);
  float* hv = at<float>(ws, L.hv);
  float* y = at<float>(ws, L.y);
  float* f = at<float>(ws, L.f);
  float* qs = at<float>(ws, L.qs);
  // row t of `cat` is [o^(1) || ... || o^(n)]
  float* cat = saved ? at<float>(saved, SL.o) : at<float>(ws, L.cat);
  const int64_t ldcat = (int64_t)n * d;
  auto W = [&](const void* base, size_t elems) { return static_cast<const char*>(base) + elems * es; };
  auto qbuf = [&](int i) { return saved ? at<float>(saved, SL.q) + (size_t)i * nt * d : at<float>(ws, L.q); };
  HIPCHK(launch_sched(b->hist_off, b->tgt_off, b->n_requests, nh, nt, L.chunk_blocks, kTargetGroup, units,
                      L.max_units, tch, hdr, st, 1, 1 << 30, device_cus()));
  HIPCHK(rec.mark("sched"));
  if (L.path == 1) {
    HIPCHK(swiglu_pack(w->ffn_u, w->ffn_v, w->ffn_o, n, d, F, at<char>(ws, L.wsp), st));
    HIPCHK(rec.mark("pack_swiglu"));
    HIPCHK(fast_pack(w->wk, at<char>(ws, L.wkp), n, d, d, 0, st)); HIPCHK(rec.mark("pack_wk"));
    HIPCHK(fast_pack(w->wv, at<char>(ws, L.wvp), n, d, d, 0, st)); HIPCHK(rec.mark("pack_wv"));
  }
  // y = SwiGLUFFN(x) on the target rows (Eq. swigluffn), fp32 result
  auto target_block = [&](const void* x, int x_bf16, const void* wu, const void* wv, const void* wo) -> hipError_t {
    hipError_t e;
    if ((e = gemm_generic(x_bf16, bf, (int)nt, F, d, x, d, 0, wu, F, 0, hu, F, 1.f, kEpiStore, nullptr, 0, nullptr,
                          0, st)) != hipSuccess || (e = rec.mark("gemm_up")) != hipSuccess)
      return e;
    if ((e = gemm_generic(x_bf16, bf, (int)nt, F, d, x, d, 0, wv, F, 0, hv, F, 1.f, kEpiStore, nullptr, 0, nullptr,
                          0, st)) != hipSuccess || (e = rec.mark("gemm_up")) != hipSuccess)
      return e;
    if ((e = swiglu_gate_f32(hu, hv, nt * F, st)) != hipSuccess || (e = rec.mark("gate")) != hipSuccess) return e;
    if ((e = gemm_generic(0, bf, (int)nt, d, F, hu, F, 0, wo, d, 0, y, d, 1.f, kEpiStore, nullptr, 0, nullptr, 0,
                          st)) != hipSuccess)
      return e;
    return rec.mark("gemm_down");
  };
  // q^(1) = LN(SwiGLUFFN^(1)(x_t))
  HIPCHK(target_block(tgt, bf, w->ffn_u, w->ffn_v, w->ffn_o));
  HIPCHK(layer_norm_rows(y, nt, d, qbuf(0), st)); HIPCHK(rec.mark("ln"));
  const float qscale = kLog2e / std::sqrt(static_cast<float>(L.dh));
  const size_t dF = (size_t)d * F, dd = (size_t)d * d;
  size_t wc_off = 0;  // rows of W_C^(2), ..., W_C^(i+1) before W_C^(i+2)
  for (int i = 0; i < n; ++i) {
    float* q = qbuf(i);
    float* a = saved ? at<float>(saved, SL.a) + (size_t)i * nt * d : at<float>(ws, L.a);
    float* lse = saved ? at<float>(saved, SL.lse) + (size_t)i * nt * h : nullptr;
    float* xt32 = saved ? at<float>(saved, SL.xt) + (size_t)i * nh * d : nullptr;
    // X~^(i) = LN(SwiGLUFFN^(i)(X)), then the layer's attention over it
    if (L.path == 1) {
      HIPCHK(swiglu_ln(d, hist, nh, at<char>(ws, L.wsp) + i * swiglu_packed_bytes(d, F), F, at<char>(ws, L.xt16),
                       xt32, st));
      HIPCHK(rec.mark("swiglu_ln"));
      HIPCHK(gemm_generic(0, bf, (int)nt, d, d, q, d, 0, W(w->wq, i * dd), d, 0, qs, d, qscale, kEpiStore, nullptr,
                          0, nullptr, 0, st));
      HIPCHK(rec.mark("gemm_q"));
      HIPCHK(qn_pack(qs, at<char>(ws, L.qn), nt, d, st)); HIPCHK(rec.mark("qn_pack"));
      const int fgrid = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(L.max_units, device_cus())));
      for (int wide = 0; wide < 2; ++wide) {
        if (wide ? L.any_wide : L.any_narrow)
          HIPCHK(fast_fused(d, wide, units, hdr, fgrid, at<char>(ws, L.qn), at<char>(ws, L.xt16), nh,
                            at<char>(ws, L.wkp), at<char>(ws, L.wvp), i, pacc, pml, nt, st));
        HIPCHK(rec.mark(wide ? "fused_wide" : "fused"));
      }
    } else {
      float* xt = xt32 ? xt32 : at<float>(ws, L.xt32);
      float* hhu = at<float>(ws, L.hhu);
      float* hhv = at<float>(ws, L.hhv);
      float* hy = at<float>(ws, L.hy);
      float* kv = at<float>(ws, L.kv32);
      HIPCHK(gemm_generic(bf, bf, (int)nh, F, d, hist, d, 0, W(w->ffn_u, i * dF), F, 0, hhu, F, 1.f, kEpiStore,
                          nullptr, 0, nullptr, 0, st));
      HIPCHK(rec.mark("hist_up"));
      HIPCHK(gemm_generic(bf, bf, (int)nh, F, d, hist, d, 0, W(w->ffn_v, i * dF), F, 0, hhv, F, 1.f, kEpiStore,
                          nullptr, 0, nullptr, 0, st));
      HIPCHK(rec.mark("hist_up"));
      HIPCHK(swiglu_gate_f32(hhu, hhv, nh * F, st)); HIPCHK(rec.mark("hist_gate"));
      HIPCHK(gemm_generic(0, bf, (int)nh, d, F, hhu, F, 0, W(w->ffn_o, i * dF), d, 0, hy, d, 1.f, kEpiStore,
                          nullptr, 0, nullptr, 0, st));
      HIPCHK(rec.mark("hist_down"));
      HIPCHK(layer_norm_rows(hy, nh, d, xt, st)); HIPCHK(rec.mark("hist_ln"));
      HIPCHK(gemm_generic(0, bf, (int)nh, d, d, xt, d, 0, W(w->wk, i * dd), d, 0, kv, 2 * d, 1.f, kEpiStore, nullptr,
                          0, nullptr, 0, st));
      HIPCHK(rec.mark("gemm_k"));
      HIPCHK(gemm_generic(0, bf, (int)nh, d, d, xt, d, 0, W(w->wv, i * dd), d, 0, kv + d, 2 * d, 1.f, kEpiStore,
                          nullptr, 0, nullptr, 0, st));
      HIPCHK(rec.mark("gemm_v"));
      HIPCHK(gemm_generic(0, bf, (int)nt, d, d, q, d, 0, W(w->wq, i * dd), d, 0, qs, d, qscale, kEpiStore, nullptr,
                          0, nullptr, 0, st));
      HIPCHK(rec.mark("gemm_q"));
      HIPCHK(attn_generic(L.dh, h, units, L.max_units, hdr, qs, kv, d, pacc, pml, nt, st));
      HIPCHK(rec.mark("attn"));
    }
    HIPCHK(merge_generic(L.dh, h, nt, tch, pacc, pml, a, lse, st)); HIPCHK(rec.mark("merge"));
    // o^(i) = [heads] W_O^(i) (Eq. layer-output), into column block i of cat
    HIPCHK(gemm_generic(0, bf, (int)nt, d, d, a, d, 0, W(w->wo, i * dd), d, 0, cat + (size_t)i * d, ldcat, 1.f,
                        kEpiStore, nullptr, 0, nullptr, 0, st));
    HIPCHK(rec.mark("gemm_o"));
    if (i + 1 < n) {
      // q^(i+2) = LN(SwiGLUFFN^(i+2)([o^(1) .. o^(i+1) || x_t] W_C^(i+2))), the
      // product split at the x_t block
      const int kc = (i + 1) * d;
      HIPCHK(gemm_generic(0, bf, (int)nt, d, kc, cat, ldcat, 0, W(w->wc, wc_off * d), d, 0, f, d, 1.f, kEpiStore,
                          nullptr, 0, nullptr, 0, st));
      HIPCHK(rec.mark("gemm_fuse"));
      HIPCHK(gemm_generic(bf, bf, (int)nt, d, d, tgt, d, 0, W(w->wc, (wc_off + kc) * d), d, 0, f, d, 1.f,
                          kEpiStore, nullptr, 0, nullptr, 1, st));
      HIPCHK(rec.mark("gemm_fuse"));
      wc_off += (size_t)kc + d;
      HIPCHK(target_block(f, 0, W(w->ffn_u, (i + 1) * dF), W(w->ffn_v, (i + 1) * dF), W(w->ffn_o, (i + 1) * dF)));
      HIPCHK(layer_norm_rows(y, nt, d, qbuf(i + 1), st)); HIPCHK(rec.mark("ln"));
    }
  }
  // z = SwiGLUFFN_z([o^(1) .. o^(n) || x_t] W_Z)
  HIPCHK(gemm_generic(0, bf, (int)nt, d, n * d, cat, ldcat, 0, w->wz, d, 0, f, d, 1.f, kEpiStore, nullptr, 0,
                      nullptr, 0, st));
  HIPCHK(rec.mark("gemm_head"));
  HIPCHK(gemm_generic(bf, bf, (int)nt, d, d, tgt, d, 0, W(w->wz, (size_t)n * d * d), d, 0, f, d, 1.f, kEpiStore,
                      nullptr, 0, nullptr, 1, st));
  HIPCHK(rec.mark("gemm_head"));
  HIPCHK(target_block(f, 0, w->z_u, w->z_v, w->z_o));
  HIPCHK(convert(0, bf, y, z, nt * d, st)); HIPCHK(rec.mark("convert_out"));
  return STCA_OK;
}

stca_status_t run_paper(const stca_dims_t* dims, const stca_batch_t* b, const void* hist, const void* tgt,
                        const stca_paper_weights_t* w, void* z, void* saved, void* ws, size_t ws_bytes,
                        hipStream_t st, Rec& rec) {
  stca_status_t s = check_paper(dims, b, hist, tgt, w, z, saved, ws);
  if (s != STCA_OK) return s;
  PaperLayout L;
  make_paper_layout(dims, b, &L);
  if (ws_bytes < L.total) return STCA_ERR_WORKSPACE;
  if (rec.ev && rec.n < paper_launch_count(L) + 1) return STCA_ERR_INVALID_ARG;
  stca_paper_saved_layout_t SL{};
  paper_saved_layout(dims, b, &SL);
  return forward_paper(L, dims->dtype == STCA_BF16, b, hist, tgt, w, z, saved, SL, ws, st, rec);
}

}  // namespace

extern "C" {

size_t stca_paper_workspace_size(const stca_dims_t* dims, const stca_batch_t* batch) {
  PaperLayout L;
  if (!make_paper_layout(dims, batch, &L)) return 0;
  return L.total;
}

size_t stca_paper_saved_size(const stca_dims_t* dims, const stca_batch_t* batch) {
  stca_paper_saved_layout_t s;
  if (!paper_saved_layout(dims, batch, &s)) return 0;
  return s.total;
}

stca_status_t stca_paper_saved_layout(const stca_dims_t* dims, const stca_batch_t* batch,
                                      stca_paper_saved_layout_t* layout) {
  if (!layout) return STCA_ERR_INVALID_ARG;
  const int p = path_of(dims);
  if (p < 0) return static_cast<stca_status_t>(p);
  stca_status_t st = check_batch(batch);
  if (st != STCA_OK) return st;
  paper_saved_layout(dims, batch, layout);
  return STCA_OK;
}

int stca_paper_launch_count(const stca_dims_t* dims, const stca_batch_t* batch) {
  PaperLayout L;
  if (!make_paper_layout(dims, batch, &L)) return -1;
  return paper_launch_count(L);
}

stca_status_t stca_forward_paper(const stca_dims_t* dims, const stca_batch_t* batch, const void* hist,
                                 const void* tgt, const stca_paper_weights_t* w, void* z, void* saved, void* ws,
                                 size_t ws_bytes, hipStream_t stream) {
  Rec none;
  return run_paper(dims, batch, hist, tgt, w, z, saved, ws, ws_bytes, stream, none);
}

stca_status_t stca_forward_paper_profiled(const stca_dims_t* dims, const stca_batch_t* batch, const void* hist,
                                          const void* tgt, const stca_paper_weights_t* w, void* z, void* saved,
                                          void* ws, size_t ws_bytes, hipStream_t stream, hipEvent_t* events,
                                          int n_events, const char** labels) {
  if (!events) return STCA_ERR_INVALID_ARG;
  Rec rec;
  rec.ev = events;
  rec.n = n_events;
  rec.labels = labels;
  rec.st = stream;
  return run_paper(dims, batch, hist, tgt, w, z, saved, ws, ws_bytes, stream, rec);
}

}  // extern "C"
