"""fp64 CPU oracle for the paper-exact STCA layer stack.

TEST INFRASTRUCTURE.  Only the tests, the package's smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code with
the HIP path and never calls it.

It evaluates, in float64 and one request at a time, the layer stack exactly as
Sec. 3.1 writes it:

* the dimension-preserving SwiGLU block, Eq. swigluffn:
  SwiGLUFFN(x) = ((x W_u) * (x W_v * sigmoid(x W_v))) W_o, W_u, W_v in
  R^{d x r d}, W_o in R^{r d x d}, no biases;
* per layer i, the history X~^(i) = LN(SwiGLUFFN^(i)(X)) and the first query
  q^(1) = LN(SwiGLUFFN^(1)(x_t));
* multi-head single-query cross attention of q^(i) onto X~^(i) (W_Q, W_K,
  W_V per head, head concatenation then W_O, Eq. layer-output), computed in
  the standard form (project K and V, max-subtracted softmax), once per
  request (Sec. 3.2);
* the target-conditioned fusion, Eq. fuse:
  q^(i+1) = LN(SwiGLUFFN^(i+1)([o^(1) || ... || o^(i) || x_t] W_C^(i+1)));
* the head token z = SwiGLUFFN_z([o^(1) || ... || o^(M) || x_t] W_Z), the
  output of the stack (what the prediction head consumes).

Readings where the paper leaves details open (each stated, none pinned by a
printed value):

P1. r = 4 (the paper's setting for its SwiGLU blocks).
P2. LayerNorm normalises each row over its d features with the biased
    variance and eps = 1e-5; its affine scale and shift are the identity.
P3. SwiGLUFFN^(i) is one block per layer: the same weights transform the
    history of layer i and the query input of layer i (q^(1) from x_t, q^(i)
    from the fused concatenation), as the shared superscript reads.
P4. The rows of W_C^(i+1) (and of W_Z) follow the concatenation order
    [o^(1) || ... || o^(i) || x_t]; the head block SwiGLUFFN_z has its own
    weights and no LayerNorm after it (the equation has none).
P5. Heads, scale, masking and empty segments as in the configuration mode
    (column blocks of W_Q/W_K/W_V, 1/sqrt(d_h), every history row visible to
    every target of its request, a request with targets has history).

Pins (tests/test_oracle_paper.py): the SwiGLU block's closed form at
identity-like weights; LayerNorm's moments and torch's layer_norm; an
independent float64 evaluation of the whole stack on torch's layer_norm, silu
and scaled_dot_product_attention; L = 1 (the output is the transformed item's
V row whatever the query); W_Q = 0 (mean of the V rows, lse = ln L); W_v = 0
for one layer (every gate closed: that layer's history, query and output are
zero); fusion and head weights that keep a single block of the concatenation
(the target block last, block k = layer k's summary); target permutation and
request independence; and planted mistakes, each caught by some pin.
"""
from __future__ import annotations

import math
from typing import Dict, List

import numpy as np

EPS = 1e-5


def layer_norm(x: np.ndarray) -> np.ndarray:
    """Row-wise normalisation over the last axis (reading P2)."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + EPS)


def swiglu_ffn(x: np.ndarray, wu: np.ndarray, wv: np.ndarray, wo: np.ndarray) -> np.ndarray:
    """Eq. swigluffn, applied row-wise."""
    g = x @ wv
    return ((x @ wu) * (g / (1.0 + np.exp(-g)))) @ wo


def wc_block(wc: np.ndarray, d: int, i: int) -> np.ndarray:
    """W_C^(i+1) (for i = 1 .. M-1) out of the stacked array holding W_C^(2),
    W_C^(3), ... one after the other: (i+1) d rows each."""
    start = sum((k + 1) * d for k in range(1, i))
    return wc[start:start + (i + 1) * d]


def summaries_with_target(outs: List[np.ndarray], xt: np.ndarray) -> np.ndarray:
    """[o^(1) || ... || o^(k) || x_t] for the fusion and head inputs (Eq. fuse,
    Eq. of z): the layer summaries in layer order, the target embedding last."""
    return np.concatenate(list(outs) + [xt], axis=1)


def attend(q: np.ndarray, Xt: np.ndarray, wq: np.ndarray, wk: np.ndarray, wv: np.ndarray, n_heads: int):
    """Head concatenation a [m, d] and lse [m, h] of the queries q onto the
    transformed history Xt (standard form: K, V projected, max subtracted)."""
    Q, K, V = q @ wq, Xt @ wk, Xt @ wv
    m, d = Q.shape
    dh = d // n_heads
    a = np.zeros((m, d))
    lse = np.zeros((m, n_heads))
    for j in range(n_heads):
        J = slice(j * dh, (j + 1) * dh)
        e = Q[:, J] @ K[:, J].T / math.sqrt(dh)
        mu = e.max(axis=1, keepdims=True)
        w = np.exp(e - mu)
        Z = w.sum(axis=1, keepdims=True)
        a[:, J] = (w / Z) @ V[:, J]
        lse[:, j] = (mu + np.log(Z))[:, 0]
    return a, lse


def forward_paper(inp: Dict[str, np.ndarray], keep: bool = True) -> Dict[str, np.ndarray]:
    """Paper-exact stack over a packed batch.

    ``inp`` holds float64 arrays: hist [N_hist, d], tgt [N_tgt, d], offsets
    hist_off / tgt_off [R+1], n_heads, and the weights
    ffn_u, ffn_v [M, d, r d], ffn_o [M, r d, d] (SwiGLUFFN^(i)),
    wq, wk, wv, wo [M, d, d], wc [sum_{i=2..M} i d, d] (W_C^(2), ... stacked),
    wz [(M + 1) d, d], z_u, z_v [d, r d], z_o [r d, d].
    Returns z [N_tgt, d] and, with ``keep``, per layer q, a (head
    concatenation), o, lse and the transformed history xt.
    """
    X, T = inp["hist"], inp["tgt"]
    hoff, toff = np.asarray(inp["hist_off"]), np.asarray(inp["tgt_off"])
    h = int(inp["n_heads"])
    M = inp["wq"].shape[0]
    Nt, d = T.shape
    Z = np.zeros((Nt, d))
    rec = {"q": np.zeros((M, Nt, d)), "a": np.zeros((M, Nt, d)), "o": np.zeros((M, Nt, d)),
           "lse": np.zeros((M, Nt, h)), "xt": np.zeros((M,) + X.shape)} if keep else None
    # the transformed histories do not depend on the targets: every row once per layer
    Xt = [layer_norm(swiglu_ffn(X, inp["ffn_u"][i], inp["ffn_v"][i], inp["ffn_o"][i])) for i in range(M)]
    if keep:
        for i in range(M):
            rec["xt"][i] = Xt[i]
    for r in range(len(hoff) - 1):
        t0, t1 = toff[r], toff[r + 1]
        if t1 == t0:
            continue
        h0, h1 = hoff[r], hoff[r + 1]
        if h1 == h0:
            raise ValueError(f"request {r} has targets but an empty history")
        xt = T[t0:t1]
        q = layer_norm(swiglu_ffn(xt, inp["ffn_u"][0], inp["ffn_v"][0], inp["ffn_o"][0]))
        outs: List[np.ndarray] = []
        for i in range(M):
            a, lse = attend(q, Xt[i][h0:h1], inp["wq"][i], inp["wk"][i], inp["wv"][i], h)
            o = a @ inp["wo"][i]
            outs.append(o)
            if keep:
                rec["q"][i, t0:t1], rec["a"][i, t0:t1], rec["o"][i, t0:t1], rec["lse"][i, t0:t1] = q, a, o, lse
            if i + 1 < M:
                fused = summaries_with_target(outs, xt) @ wc_block(inp["wc"], d, i + 1)
                q = layer_norm(swiglu_ffn(fused, inp["ffn_u"][i + 1], inp["ffn_v"][i + 1], inp["ffn_o"][i + 1]))
        Z[t0:t1] = swiglu_ffn(summaries_with_target(outs, xt) @ inp["wz"], inp["z_u"], inp["z_v"], inp["z_o"])
    out = {"z": Z}
    if keep:
        out.update(rec)
    return out
