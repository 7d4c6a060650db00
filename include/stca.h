/*
 * stca.h - C ABI of the MI355X (gfx950) STCA library.
 *
 * Stacked Target-to-History Cross Attention under Request Level Batching:
 * every target (candidate item) of a request attends, with a single query per
 * head, to that request's whole history, layer after layer (paper Sec. 3.1,
 * "Multi-head target-to-history cross attention" and Eq. layer-output).
 * The history of a request is projected to the per-layer K/V once and the
 * projection is shared by all of that request's targets (Sec. 3.2, App. A.3).
 * Ragged batches are packed without padding; per-request offset arrays mark
 * the segments (App. A.4, the index-based ragged target attention).
 *
 * Layer (the benchmark workloads' form of the stacked update, Sec. 3.1
 * "Stacking" replaced by a residual FFN; biases omitted as in the paper):
 *   s^(0)   = x_t
 *   q       = s^(i) W_Q^i                          head j: columns [j d_h, (j+1) d_h)
 *   a_j     = softmax(q_j (X W_K^i)_j^T / sqrt(d_h)) (X W_V^i)_j      over the request's history X
 *   u       = s^(i) + [a_1 | ... | a_h] W_O^i
 *   s^(i+1) = u + ReLU(u W_1^i) W_2^i
 *   out     = s^(n)
 *
 * Conventions shared by every entry point:
 *  - All tensor pointers are device pointers unless named *_host, and must be
 *    16-byte aligned.  Matrices are row-major; y = x W (W is [d_in][d_out]).
 *  - Weights are stacked per layer: wq, wk, wv, wo [n_layers][d][d],
 *    w1 [n_layers][d][ffn_hidden], w2 [n_layers][ffn_hidden][d].
 *  - Storage dtype (STCA_F32 or STCA_BF16) applies to hist, tgt, the weights,
 *    out and dout; accumulation is always fp32; gradients are fp32.
 *  - Range of the bf16 path.  bf16 storage keeps two bytes per value inside
 *    the kernels as well, but in fp16 (three more mantissa bits, which the
 *    attention's accuracy needs): the projected K and V, the queries, the
 *    softmax weights and the target update's activations are fp16 MFMA
 *    operands (fp32 accumulation), so each must stay below 65504 in
 *    magnitude (the fp32 state and the fp32 sums have no such limit).  The
 *    inputs themselves may use the whole bf16 range.  The forward's target
 *    update checks every value it rounds to fp16 (input targets, merged
 *    attention output, activations, next queries); an overflowed V, or a K
 *    whose overflow drives a score to plus infinity, reaches it as a
 *    non-finite attention output.  A violation is recorded in the workspace
 *    and stca_device_status() then returns STCA_ERR_RANGE; outputs of such a
 *    call are undefined.  A K entry whose overflow drives its score to minus
 *    infinity only removes that history row from the softmax and is not
 *    detected.  The backward's fp16 operands (two-term, hi + lo) have the same
 *    range and are not checked.  Non-finite inputs propagate.
 *  - Request r owns hist rows [hist_off[r], hist_off[r+1]) and tgt rows
 *    [tgt_off[r], tgt_off[r+1]).  offsets[0] = 0, non-decreasing,
 *    offsets[R] = n_hist / n_tgt.  A request with targets must have at least
 *    one history row; a request with no targets is legal and produces nothing.
 *  - The caller owns every buffer.  The library never allocates, frees or
 *    synchronises: all work is enqueued on `stream`, and calls return before it
 *    runs.  Calls on different streams need distinct workspaces.
 *  - Errors found on the host are returned before anything is enqueued.
 *    Offsets are checked on the host when the *_host copies are given;
 *    otherwise the device scheduler checks them, produces no work for a bad
 *    request and records STCA_ERR_INVALID_ARG in the workspace, readable with
 *    stca_device_status().  No exception crosses the ABI.
 */
#ifndef STCA_H_
#define STCA_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  STCA_OK = 0,
  STCA_ERR_INVALID_ARG = -1, /* bad pointer, size or offsets */
  STCA_ERR_UNSUPPORTED = -2, /* valid but not implemented shape/dtype/form */
  STCA_ERR_WORKSPACE = -3,   /* workspace or saved buffer too small */
  STCA_ERR_HIP = -4,         /* a HIP runtime call or launch failed */
  STCA_ERR_RANGE = -5        /* (device status only) an fp16 intermediate of the bf16 path
                                overflowed or a non-finite value appeared; see below */
} stca_status_t;

typedef enum { STCA_F32 = 0, STCA_BF16 = 1 } stca_dtype_t;

/* Execution forms of the bf16 MFMA path (0 = automatic everywhere).  The
 * generic fp32-arithmetic path has one form of each and ignores them.
 *
 * kv_form  STCA_KV_AUTO: each layer's K/V is projected inside the attention
 *          kernel and never stored, except when the host offsets show a
 *          request with more than 64 targets: then one GEMM writes every
 *          layer's K/V to the workspace once and the attention reads it once
 *          per 128 targets.  STCA_KV_FUSED: always the former.
 *          STCA_KV_MATERIALIZE: always the latter.
 * attn_form STCA_ATTN_AUTO: with d_h = 32 and host offsets, the requests
 *          with at most 32 / n_heads targets run in the reordered
 *          single-query form of App. A.2.2 (Eq. attn-optimized: scores
 *          u . x with u = q W_K^T, output (P X) W_V; no K/V) and the others
 *          in the standard form, in the same call; without host offsets the
 *          standard form.
 *          STCA_ATTN_STANDARD: always the standard form.
 *          STCA_ATTN_REORDERED: every request in the reordered form, for
 *          requests of up to 256 / n_heads targets (d_h = 32, host offsets
 *          given); STCA_ERR_UNSUPPORTED for other batches.
 * bwd_form STCA_BWD_AUTO: with d_h = 32, ffn_hidden a multiple of d_model and
 *          host offsets showing at most 32 targets per request, the
 *          backward on bf16 storage runs in the reordered form (the
 *          attention gradients through u = q W_K^T and h = da W_V^T per
 *          target and head, no K, V, dK or dV; Sec. 3.1's reordering applied
 *          to the backward) when d_model is 128 or 256, every request has
 *          at most 128 / n_heads targets and no request's history is longer
 *          than twice one compute unit's share of the batch's history
 *          blocks, else in the fused form (K/V formed
 *          inside the attention kernels, dK | dV written for the
 *          history-side products); otherwise K | V are formed by a GEMM and
 *          the attention runs in exact fp32 (generic).
 *          STCA_BWD_GENERIC: always the generic form.  STCA_BWD_FUSED: the
 *          fused form.  STCA_BWD_REORDERED: the reordered form.  Each is
 *          STCA_ERR_UNSUPPORTED for a batch outside its conditions.
 * chunk_blocks: history chunk length, in 32-row blocks, of the attention's
 *          split over a request's history (at most 16 chunks per request, so
 *          long histories get longer chunks); 0 = chosen from the batch size
 *          and the number of compute units.
 * Out-of-range values are STCA_ERR_INVALID_ARG. */
typedef enum { STCA_KV_AUTO = 0, STCA_KV_FUSED = 1, STCA_KV_MATERIALIZE = 2 } stca_kv_form_t;
typedef enum { STCA_ATTN_AUTO = 0, STCA_ATTN_STANDARD = 1, STCA_ATTN_REORDERED = 2 } stca_attn_form_t;
typedef enum { STCA_BWD_AUTO = 0, STCA_BWD_FUSED = 1, STCA_BWD_GENERIC = 2, STCA_BWD_REORDERED = 3 } stca_bwd_form_t;

/* Model shape and execution forms.  d_model % n_heads == 0 and ffn_hidden a
 * multiple of 32.  STCA_BF16 with d_head = d_model / n_heads = 32, d_model in
 * {64, 128, 256} and ffn_hidden a multiple of 256 runs on the bf16 MFMA
 * kernels; every other shape with d_head in {8, 16, 32, 64} (either dtype)
 * runs on the generic fp32-arithmetic kernels (stca_path tells which).
 * Every size and launch decision depends only on this structure and the
 * batch, so a workspace sized for a (dims, batch) pair fits every call with
 * the same pair.  Zero-initialise the structure to get the automatic forms. */
typedef struct {
  int32_t d_model;
  int32_t n_heads;
  int32_t n_layers;
  int32_t ffn_hidden;
  int32_t dtype;        /* stca_dtype_t */
  int32_t kv_form;      /* stca_kv_form_t */
  int32_t attn_form;    /* stca_attn_form_t */
  int32_t bwd_form;     /* stca_bwd_form_t */
  int32_t chunk_blocks; /* >= 0 */
} stca_dims_t;

/* A packed ragged batch (App. A.4: flattened rows plus segment boundaries). */
typedef struct {
  int32_t n_requests;           /* R >= 1 */
  int64_t n_hist;               /* total history rows, < 2^31 */
  int64_t n_tgt;                /* total target rows, < 2^31 */
  const int32_t* hist_off;      /* device [R+1] */
  const int32_t* tgt_off;       /* device [R+1] */
  const int32_t* hist_off_host; /* optional host copy [R+1]: enables host checks and exact sizing */
  const int32_t* tgt_off_host;  /* optional host copy [R+1] */
} stca_batch_t;

/* Per-layer weights (paper Sec. 3.1: W_Q, W_K, W_V, W_O; the FFN W_1, W_2). */
typedef struct {
  const void* wq;
  const void* wk;
  const void* wv;
  const void* wo;
  const void* w1;
  const void* w2;
} stca_weights_t;

/* Weight gradients, fp32, same shapes as the weights; overwritten. */
typedef struct {
  float* dwq;
  float* dwk;
  float* dwv;
  float* dwo;
  float* dw1;
  float* dw2;
} stca_wgrads_t;

/* Byte offsets into the `saved` buffer (all fp32 unless stated), for reading
 * per-layer intermediates back.  Each per-layer tensor is stacked on a leading
 * layer axis: s [n][n_tgt][d] (layer input state), a [n][n_tgt][d] (head
 * concatenation before W_O), u [n][n_tgt][d] (state after the attention
 * residual), lse [n][n_tgt][h] (natural log-sum-exp of each head's scores). */
typedef struct {
  size_t s, a, u, lse;
  size_t total;
} stca_saved_layout_t;

/* Workspace bytes needed by stca_forward (with_backward = 0) or stca_backward
 * (with_backward = 1).  Returns 0 for invalid or unsupported arguments. */
size_t stca_workspace_size(const stca_dims_t* dims, const stca_batch_t* batch, int with_backward);

/* Bytes of the optional `saved` buffer that stca_forward fills. */
size_t stca_saved_size(const stca_dims_t* dims, const stca_batch_t* batch);

/* Offsets of the saved tensors; returns STCA_ERR_INVALID_ARG / UNSUPPORTED
 * like the other calls. */
stca_status_t stca_saved_layout(const stca_dims_t* dims, const stca_batch_t* batch,
                                stca_saved_layout_t* layout);

/* Forward pass: out[n_tgt][d] (storage dtype) = s^(n) for every target.
 *  hist  [n_hist][d], tgt [n_tgt][d]  storage dtype, device
 *  saved nullable; when given (stca_saved_size bytes) the per-layer
 *        intermediates (see stca_saved_layout_t) are written there
 *  ws    device workspace of ws_bytes >= stca_workspace_size(dims, batch, 0)
 * The bf16 MFMA path's forms of K/V and of the attention follow
 * dims->kv_form and dims->attn_form. */
stca_status_t stca_forward(const stca_dims_t* dims, const stca_batch_t* batch,
                           const void* hist, const void* tgt, const stca_weights_t* w,
                           void* out, void* saved, void* ws, size_t ws_bytes,
                           hipStream_t stream);

/* Backward pass: the gradients of f = sum_t <dout_t, out_t> with respect to
 * hist, tgt and every weight, for the same inputs as a forward call.  The
 * layer states are recomputed from the inputs in fp32 (activation
 * recomputation), so every ReLU gate and softmax weight of the backward
 * follows fp32 states.  Writes (overwrites) dhist [n_hist][d], dtgt [n_tgt][d]
 * and all weight gradients, fp32.  dout is [n_tgt][d] in the storage dtype.
 * ws_bytes >= stca_workspace_size(dims, batch, 1). */
stca_status_t stca_backward(const stca_dims_t* dims, const stca_batch_t* batch,
                            const void* hist, const void* tgt, const stca_weights_t* w,
                            const void* dout, float* dhist, float* dtgt,
                            const stca_wgrads_t* dw, void* ws, size_t ws_bytes,
                            hipStream_t stream);

/* Forward without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation).  The same computation and results as
 * stca_forward, with the workspace in a device array of the library of
 * STCA_NOALLOC_SCRATCH_BYTES bytes, one per GPU, set up on the first call on
 * that GPU (with it current) and held until the process ends; nothing is
 * allocated by any call.  Returns STCA_ERR_WORKSPACE, before anything is
 * launched, when stca_workspace_size(dims, batch, 0) exceeds that size; other
 * errors as stca_forward.  Every call on a GPU uses that GPU's one array:
 * calls that may overlap on the same GPU (other streams, other threads) race
 * and must be serialised by the caller.  Nothing in the array needs to start
 * at zero; the device-side status of such a call (stca_device_status) is not
 * readable, so give host offsets to have them checked. */
#define STCA_NOALLOC_SCRATCH_BYTES ((size_t)256 << 20)
stca_status_t stca_forward_noalloc(const stca_dims_t* dims, const stca_batch_t* batch, const void* hist,
                                   const void* tgt, const stca_weights_t* w, void* out, void* saved,
                                   hipStream_t stream);

/* Training step in two calls, for batches the fused backward takes (bf16,
 * d_h = 32, FFN width a multiple of d, host offsets showing at most 32
 * targets per request): the forward writes, besides out, a training record
 * of the per-layer tensors the backward needs, computed to fp32 accuracy (so
 * the ReLU gates follow fp32 states), and the backward reads it instead of
 * recomputing them.
 *
 * stca_train_record_size: bytes of the record; 0 when the batch does not
 * qualify or the arguments are invalid.
 * stca_forward_train: out as stca_forward (evaluated to fp32 accuracy before
 * the final rounding to the storage dtype); record (device, 16-byte aligned,
 * stca_train_record_size bytes) is overwritten; ws as for stca_backward
 * (ws_bytes >= stca_workspace_size(dims, batch, 1)).
 * stca_backward_record: the same gradients as stca_backward for the inputs
 * that produced `record` (which must not change in between), without the
 * recomputation.  Both return STCA_ERR_UNSUPPORTED for batches that do not
 * qualify; other errors as stca_forward / stca_backward. */
size_t stca_train_record_size(const stca_dims_t* dims, const stca_batch_t* batch);
stca_status_t stca_forward_train(const stca_dims_t* dims, const stca_batch_t* batch,
                                 const void* hist, const void* tgt, const stca_weights_t* w,
                                 void* out, void* record, void* ws, size_t ws_bytes, hipStream_t stream);
stca_status_t stca_backward_record(const stca_dims_t* dims, const stca_batch_t* batch,
                                   const void* hist, const void* tgt, const stca_weights_t* w,
                                   const void* record, const void* dout, float* dhist, float* dtgt,
                                   const stca_wgrads_t* dw, void* ws, size_t ws_bytes,
                                   hipStream_t stream);

/* Measurement variant of stca_forward: the same work, plus hipEventRecord on
 * `stream` around every kernel launch so a caller can time each kernel on the
 * stream it runs on.  events[0] is recorded before the first launch and
 * events[k+1] right after launch k; n_events must be at least
 * stca_forward_launch_count(dims, batch) + 1.  labels (nullable, n_events - 1
 * entries) receive static kernel names ("proj", "attn", "update", ...).
 * The events must have been created by the caller (hipEventCreate). */
int stca_forward_launch_count(const stca_dims_t* dims, const stca_batch_t* batch);
stca_status_t stca_forward_profiled(const stca_dims_t* dims, const stca_batch_t* batch,
                                    const void* hist, const void* tgt, const stca_weights_t* w,
                                    void* out, void* saved, void* ws, size_t ws_bytes,
                                    hipStream_t stream, hipEvent_t* events, int n_events,
                                    const char** labels);

/* Measurement variant of stca_backward: the same work, plus hipEventRecord on
 * `stream` at phase boundaries.  events[0] is recorded before the first
 * launch and events[k+1] at the end of phase k; labels (nullable) receive the
 * phase names ("sched", "prep", "kv_gemm", "attn_fwd", "target_gemm",
 * "attn_bwd", "dw_kv", "dx", "out").  n_events must be at least
 * stca_backward_launch_count(dims, batch) + 1; the events are the caller's. */
int stca_backward_launch_count(const stca_dims_t* dims, const stca_batch_t* batch);
stca_status_t stca_backward_profiled(const stca_dims_t* dims, const stca_batch_t* batch,
                                     const void* hist, const void* tgt, const stca_weights_t* w,
                                     const void* dout, float* dhist, float* dtgt,
                                     const stca_wgrads_t* dw, void* ws, size_t ws_bytes,
                                     hipStream_t stream, hipEvent_t* events, int n_events,
                                     const char** labels);

/* ---- Stochastic-length training batches (Sec. 3.3; App. "Extrapolation
 * details": Beta sampling, Eq. beta-scale and Eq. beta; batch-level load
 * balancing).  Host functions on host arrays; no GPU involved.
 *
 * stca_sl_beta: the Beta shape beta that makes E[L_raw] = l_avg (Eq. beta):
 * alpha (l_max - l_avg) / (l_avg - l_min).  NaN unless alpha > 0 and
 * 0 <= l_min < l_avg < l_max.
 *
 * stca_sl_sample: per request r, s ~ Beta(alpha, beta) from a counter-based
 * stream keyed by (seed, r), L_raw = l_min + s (l_max - l_min) (written to
 * l_raw[r] when l_raw is not NULL), and l_train[r] = L_raw rounded to the
 * nearest multiple of 8, clamped to [max(8, l_min rounded), l_max].
 *
 * stca_sl_allocate: global length allocation under a token budget (the paper
 * uses B * l_avg): l_keep[r] = min(l_full[r], l_train[r]); if their sum
 * exceeds `budget`, every l_keep is capped at the largest multiple of 8 that
 * brings the sum within it (at least 8).
 *
 * stca_sl_pack: sequence compaction with temporal-suffix selection.  full_off
 * [n+1] segments the full histories; request r keeps its last l_keep[r] rows.
 * Writes hist_off [n+1] of the packed layout and, when src_rows is not NULL,
 * src_rows [hist_off[n]]: the full-history row each packed row comes from.
 *
 * All return STCA_ERR_INVALID_ARG on inconsistent arguments. */
double stca_sl_beta(double alpha, int32_t l_min, int32_t l_avg, int32_t l_max);
stca_status_t stca_sl_sample(uint64_t seed, int32_t n, double alpha, int32_t l_min, int32_t l_avg,
                             int32_t l_max, double* l_raw, int32_t* l_train);
stca_status_t stca_sl_allocate(int32_t n, const int32_t* l_full, const int32_t* l_train, int64_t budget,
                               int32_t* l_keep);
stca_status_t stca_sl_pack(int32_t n, const int32_t* full_off, const int32_t* l_keep, int32_t* hist_off,
                           int32_t* src_rows);

/* ---- Paper-exact layer stack (Sec. 3.1, "Input encoding", "Multi-head
 * target-to-history cross attention", "Stacking and target-conditioned
 * fusion", "Prediction head and objective").  With M = n_layers, F =
 * ffn_hidden (= r d, the SwiGLU width) and SwiGLUFFN(x) = ((x W_u) *
 * (x W_v * sigmoid(x W_v))) W_o (Eq. swigluffn, no biases):
 *   X~^(i)    = LN(SwiGLUFFN^(i)(X))                          every history row, i = 1..M
 *   q^(1)     = LN(SwiGLUFFN^(1)(x_t))
 *   o^(i)     = [heads of the cross attention of q^(i) onto X~^(i)] W_O^(i)   (Eq. layer-output)
 *   q^(i+1)   = LN(SwiGLUFFN^(i+1)([o^(1) || ... || o^(i) || x_t] W_C^(i+1)))  (Eq. fuse)
 *   z         = SwiGLUFFN_z([o^(1) || ... || o^(M) || x_t] W_Z)
 * LN normalises each row over its d features (biased variance, eps 1e-5,
 * unit scale, zero shift).  SwiGLUFFN^(i) is one block per layer, used for
 * both the history and the query input of layer i.  The attention heads,
 * scale and per-request sharing are those of stca_forward.
 *
 * Weights (storage dtype, row-major, y = x W):
 *   ffn_u, ffn_v [M][d][F], ffn_o [M][F][d]   SwiGLUFFN^(1..M)
 *   wq, wk, wv, wo [M][d][d]
 *   wc   W_C^(2), ..., W_C^(M) one after the other, W_C^(k) being k d rows
 *        x d (rows in concatenation order, x_t's block last); NULL when M = 1
 *   wz   [(M+1) d][d]
 *   z_u, z_v [d][F], z_o [F][d]              the head's SwiGLU block
 * Shapes: as stca_forward (stca_path tells the kernel family); on the bf16
 * MFMA path the history transform runs as one fused SwiGLU + LayerNorm kernel
 * per layer (the hidden activations never leave the registers) and the
 * transformed history is stored in bf16 for the attention; the generic path
 * keeps everything in fp32.  The target-side blocks run on fp32 arithmetic. */
typedef struct {
  const void* ffn_u;
  const void* ffn_v;
  const void* ffn_o;
  const void* wq;
  const void* wk;
  const void* wv;
  const void* wo;
  const void* wc;
  const void* wz;
  const void* z_u;
  const void* z_v;
  const void* z_o;
} stca_paper_weights_t;

/* Byte offsets into the optional `saved` buffer of stca_forward_paper, fp32:
 * q [M][n_tgt][d] (the layer queries q^(i)), a [M][n_tgt][d] (head
 * concatenation before W_O), o [n_tgt][M d] (row t = o^(1) || ... || o^(M)),
 * lse [M][n_tgt][h] (natural log-sum-exp of each head's scores) and xt
 * [M][n_hist][d] (the transformed histories X~^(i)). */
typedef struct {
  size_t q, a, o, lse, xt;
  size_t total;
} stca_paper_saved_layout_t;

size_t stca_paper_workspace_size(const stca_dims_t* dims, const stca_batch_t* batch);
size_t stca_paper_saved_size(const stca_dims_t* dims, const stca_batch_t* batch);
stca_status_t stca_paper_saved_layout(const stca_dims_t* dims, const stca_batch_t* batch,
                                      stca_paper_saved_layout_t* layout);

/* Forward pass of the paper-exact stack: z [n_tgt][d] (storage dtype) for
 * every target.  hist, tgt, z, saved and ws as in stca_forward, with
 * ws_bytes >= stca_paper_workspace_size(dims, batch) and saved (nullable)
 * of stca_paper_saved_size bytes.  Errors as for stca_forward. */
stca_status_t stca_forward_paper(const stca_dims_t* dims, const stca_batch_t* batch,
                                 const void* hist, const void* tgt, const stca_paper_weights_t* w,
                                 void* z, void* saved, void* ws, size_t ws_bytes, hipStream_t stream);

/* Measurement variant of stca_forward_paper (events and labels as in
 * stca_forward_profiled; n_events >= stca_paper_launch_count + 1). */
int stca_paper_launch_count(const stca_dims_t* dims, const stca_batch_t* batch);
stca_status_t stca_forward_paper_profiled(const stca_dims_t* dims, const stca_batch_t* batch,
                                          const void* hist, const void* tgt, const stca_paper_weights_t* w,
                                          void* z, void* saved, void* ws, size_t ws_bytes, hipStream_t stream,
                                          hipEvent_t* events, int n_events, const char** labels);

/* Reads (synchronising on `stream`) the status the kernels recorded in `ws`
 * during the last call that used it: STCA_ERR_INVALID_ARG when the device
 * scheduler found bad offsets, else STCA_ERR_RANGE when the forward's target
 * update found an fp16 intermediate out of range or a non-finite attention
 * output (bf16 path, see "Range of the bf16 path"), else STCA_OK. */
stca_status_t stca_device_status(const void* ws, hipStream_t stream);

/* Static description of a status code. */
const char* stca_status_string(stca_status_t status);

/* Which kernel family a shape runs on: 1 = bf16 MFMA path, 0 = generic fp32
 * path, negative = a status code for invalid or unsupported dims. */
int stca_path(const stca_dims_t* dims);

#ifdef __cplusplus
}
#endif

#endif /* STCA_H_ */
