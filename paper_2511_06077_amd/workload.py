"""Seeded synthetic STCA workloads under Request Level Batching.

This module only draws and lays out inputs: it holds none of the method's
arithmetic, and it is the one module that both the HIP path's callers and the
fp64 oracle read their inputs from.

Shapes follow the paper's workloads: d = 256, h = 8 heads (d_h = 32) and four
stacked layers (Sec. 4.2 compute/quality study; App. A.2.2 worked FLOP example),
histories up to the 10k serving length with a ~2k training window (Sec. 3.3),
and several targets per request sharing one history (Sec. 3.2, App. A.3).
The Douyin logs the paper trains on are not public; i.i.d. normal embeddings
with the same shapes stand in for them.

Recipe (one ``numpy.random.default_rng`` stream per purpose, keyed by the
workload seed so that any subset of requests can be regenerated alone):

* ragged batches: ``default_rng([seed, 0])`` draws the history lengths
  ``L_r ~ U{L_lo..L_hi}`` and then the target counts ``m_r ~ U{m_lo..m_hi}``
  (both inclusive);
* weights: ``default_rng([seed, 1])`` draws, layer by layer,
  ``W_Q, W_K, W_V, W_O ~ N(0, 1/d)`` (each d x d), ``W_1 ~ N(0, 1/d)``
  (d x 4d) and ``W_2 ~ N(0, 1/(4d))`` (4d x d);
* request r: ``default_rng([seed, 2, r])`` draws its history rows
  ``X_r ~ N(0, 1)`` (L_r x d) and then its target rows ``x_t ~ N(0, 1)``
  (m_r x d);
* upstream gradient of request r: ``default_rng([seed, 3, r])`` draws
  ``G_r ~ N(0, 1)`` (m_r x d);
* weights of the paper-exact stack (Sec. 3.1): ``default_rng([seed, 4])``
  draws, layer by layer, the SwiGLU block ``W_u, W_v ~ N(0, 1/d)`` (d x rd)
  and ``W_o ~ N(0, 1/(rd))`` (rd x d) with r = ffn_mult, then
  ``W_Q, W_K, W_V, W_O ~ N(0, 1/d)``; then ``W_C^(k) ~ N(0, 1/(k d))``
  (k d x d) for k = 2..M, ``W_Z ~ N(0, 1/((M+1) d))`` and the head block's
  ``W_u, W_v ~ N(0, 1/d)``, ``W_o ~ N(0, 1/(rd))``.

All draws are float32 (``standard_normal(dtype=float32)``); bf16 workloads then
round every value to bfloat16 with round-to-nearest-even.  The exact stored
values (decoded to float64) are what the oracle consumes, so a parity error
measures only the kernels' arithmetic.
"""
from __future__ import annotations

import dataclasses
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, Optional, Sequence

import numpy as np

WEIGHT_NAMES = ("wq", "wk", "wv", "wo", "w1", "w2")
# weights of the paper-exact stack, in the order of the C structure
PAPER_WEIGHT_NAMES = ("ffn_u", "ffn_v", "ffn_o", "wq", "wk", "wv", "wo", "wc", "wz", "z_u", "z_v", "z_o")


@dataclasses.dataclass(frozen=True)
class Workload:
    """One batch shape: R requests, m targets and L history items each."""

    name: str
    n_requests: int
    d_model: int
    n_heads: int
    n_layers: int
    dtype: str  # "f32" or "bf16": storage of inputs, weights and output
    seed: int
    hist_len: int = 0  # uniform history length (0 when ragged)
    n_targets: int = 0  # uniform targets per request (0 when ragged)
    hist_range: Optional[tuple] = None  # (lo, hi) inclusive, ragged batches
    tgt_range: Optional[tuple] = None  # (lo, hi) inclusive, ragged batches
    backward: bool = False
    ffn_mult: int = 4

    @property
    def d_head(self) -> int:
        return self.d_model // self.n_heads

    @property
    def ffn_hidden(self) -> int:
        return self.ffn_mult * self.d_model


WORKLOADS: Dict[str, Workload] = {
    w.name: w
    for w in (
        Workload("tiny_f32_R4_m4_L256_d64", 4, 64, 2, 2, "f32", seed=1,
                 hist_len=256, n_targets=4, backward=True),
        Workload("uniform_bf16_R64_m16_L1024_d128", 64, 128, 4, 2, "bf16", seed=2,
                 hist_len=1024, n_targets=16),
        Workload("long_bf16_R128_m32_L10240_d256", 128, 256, 8, 4, "bf16", seed=3,
                 hist_len=10240, n_targets=32),
        Workload("long_bf16_R128_m1_L10240_d256", 128, 256, 8, 4, "bf16", seed=3,
                 hist_len=10240, n_targets=1),
        Workload("ragged_bf16_R256_L512-10240_m1-64_d256", 256, 256, 8, 4, "bf16",
                 seed=4, hist_range=(512, 10240), tgt_range=(1, 64)),
        Workload("train_bf16_R256_m16_L2048_d256", 256, 256, 8, 4, "bf16", seed=5,
                 hist_len=2048, n_targets=16, backward=True),
    )
}

# The workload whose forward throughput is the headline number.
HEADLINE = "long_bf16_R128_m32_L10240_d256"


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclasses.dataclass
class Batch:
    """A packed RLB batch.

    ``hist`` is [N_hist, d] and ``tgt`` is [N_tgt, d]; request r owns history
    rows ``hist_off[r]:hist_off[r+1]`` and target rows ``tgt_off[r]:tgt_off[r+1]``.
    Arrays hold the storage encoding: float32, or uint16 bfloat16 bits.
    Weights are stacked ``[n_layers, d_in, d_out]`` with ``y = x @ W``; head j of
    W_Q/W_K/W_V uses columns ``[j*d_h, (j+1)*d_h)``.
    """

    wl: Workload
    requests: np.ndarray  # int64 [R]: the workload request ids held here
    hist_len: np.ndarray  # int64 [R]
    n_tgt: np.ndarray  # int64 [R]
    hist_off: np.ndarray  # int32 [R+1]
    tgt_off: np.ndarray  # int32 [R+1]
    hist: np.ndarray
    tgt: np.ndarray
    weights: Dict[str, np.ndarray]
    grad_out: Optional[np.ndarray] = None  # [N_tgt, d], storage encoding

    @property
    def n_requests(self) -> int:
        return int(self.hist_len.shape[0])

    @property
    def n_hist(self) -> int:
        return int(self.hist_off[-1])

    @property
    def n_tgt_total(self) -> int:
        return int(self.tgt_off[-1])

    def decode(self, a: np.ndarray) -> np.ndarray:
        """Storage array -> the exact float64 values it holds."""
        if a.dtype == np.uint16:
            return bf16_bits_to_f32(a).astype(np.float64)
        return np.asarray(a, dtype=np.float64)

    def f64(self) -> dict:
        """Exact float64 view of every input, as the oracle takes it."""
        out = {
            "hist": self.decode(self.hist),
            "tgt": self.decode(self.tgt),
            "hist_off": self.hist_off.astype(np.int64),
            "tgt_off": self.tgt_off.astype(np.int64),
            "n_heads": self.wl.n_heads,
        }
        for k in WEIGHT_NAMES:
            out[k] = self.decode(self.weights[k])
        if self.grad_out is not None:
            out["grad_out"] = self.decode(self.grad_out)
        return out


def _store(x: np.ndarray, dtype: str) -> np.ndarray:
    return to_bf16_bits(x) if dtype == "bf16" else np.ascontiguousarray(x, dtype=np.float32)


def request_shapes(wl: Workload):
    """Per-request (history length, target count) for the whole workload."""
    if wl.hist_range is None:
        L = np.full(wl.n_requests, wl.hist_len, dtype=np.int64)
        m = np.full(wl.n_requests, wl.n_targets, dtype=np.int64)
        return L, m
    rng = np.random.default_rng([wl.seed, 0])
    L = rng.integers(wl.hist_range[0], wl.hist_range[1], wl.n_requests, endpoint=True)
    m = rng.integers(wl.tgt_range[0], wl.tgt_range[1], wl.n_requests, endpoint=True)
    return L.astype(np.int64), m.astype(np.int64)


def make_weights(wl: Workload, scale_q: float = 1.0) -> Dict[str, np.ndarray]:
    d, f, n = wl.d_model, wl.ffn_hidden, wl.n_layers
    rng = np.random.default_rng([wl.seed, 1])
    ws = {k: [] for k in WEIGHT_NAMES}
    for _ in range(n):
        for k in ("wq", "wk", "wv", "wo"):
            ws[k].append(rng.standard_normal((d, d), dtype=np.float32) / np.float32(np.sqrt(d)))
        ws["w1"].append(rng.standard_normal((d, f), dtype=np.float32) / np.float32(np.sqrt(d)))
        ws["w2"].append(rng.standard_normal((f, d), dtype=np.float32) / np.float32(np.sqrt(f)))
    out = {k: np.stack(v) for k, v in ws.items()}
    if scale_q != 1.0:
        out["wq"] = out["wq"] * np.float32(scale_q)
    return {k: _store(v, wl.dtype) for k, v in out.items()}


def make_paper_weights(wl: Workload) -> Dict[str, np.ndarray]:
    """Seeded weights of the paper-exact stack (storage encoding)."""
    d, rd, M = wl.d_model, wl.ffn_hidden, wl.n_layers
    rng = np.random.default_rng([wl.seed, 4])

    def n(rows, cols, fan_in):
        return rng.standard_normal((rows, cols), dtype=np.float32) / np.float32(np.sqrt(fan_in))
    ws = {k: [] for k in ("ffn_u", "ffn_v", "ffn_o", "wq", "wk", "wv", "wo")}
    for _ in range(M):
        ws["ffn_u"].append(n(d, rd, d))
        ws["ffn_v"].append(n(d, rd, d))
        ws["ffn_o"].append(n(rd, d, rd))
        for k in ("wq", "wk", "wv", "wo"):
            ws[k].append(n(d, d, d))
    out = {k: np.stack(v) for k, v in ws.items()}
    wc = [n(k * d, d, k * d) for k in range(2, M + 1)]
    out["wc"] = np.concatenate(wc) if wc else np.zeros((0, d), dtype=np.float32)
    out["wz"] = n((M + 1) * d, d, (M + 1) * d)
    out["z_u"] = n(d, rd, d)
    out["z_v"] = n(d, rd, d)
    out["z_o"] = n(rd, d, rd)
    return {k: _store(v, wl.dtype) for k, v in out.items()}


def paper_f64(b: "Batch", weights: Dict[str, np.ndarray]) -> dict:
    """Exact float64 view of a batch with paper-exact weights, as the oracle
    takes it."""
    out = {
        "hist": b.decode(b.hist),
        "tgt": b.decode(b.tgt),
        "hist_off": b.hist_off.astype(np.int64),
        "tgt_off": b.tgt_off.astype(np.int64),
        "n_heads": b.wl.n_heads,
    }
    for k in PAPER_WEIGHT_NAMES:
        out[k] = b.decode(weights[k])
    return out


def _request_rows(wl: Workload, r: int, L: int, m: int):
    rng = np.random.default_rng([wl.seed, 2, int(r)])
    x = rng.standard_normal((L, wl.d_model), dtype=np.float32)
    t = rng.standard_normal((m, wl.d_model), dtype=np.float32)
    return _store(x, wl.dtype), _store(t, wl.dtype)


def _request_grad(wl: Workload, r: int, m: int):
    rng = np.random.default_rng([wl.seed, 3, int(r)])
    return _store(rng.standard_normal((m, wl.d_model), dtype=np.float32), wl.dtype)


def offsets(counts: np.ndarray) -> np.ndarray:
    off = np.zeros(len(counts) + 1, dtype=np.int64)
    np.cumsum(counts, out=off[1:])
    if off[-1] >= 2**31:
        raise ValueError("packed size exceeds int32 offsets")
    return off.astype(np.int32)


def make_batch(wl: Workload, requests: Optional[Sequence[int]] = None, *,
               with_grad: Optional[bool] = None, threads: int = 8,
               scale_q: float = 1.0) -> Batch:
    """Generate the workload, or only the listed requests of it (same values)."""
    L_all, m_all = request_shapes(wl)
    req = np.arange(wl.n_requests) if requests is None else np.asarray(requests, dtype=np.int64)
    L, m = L_all[req], m_all[req]
    hoff, toff = offsets(L), offsets(m)
    d = wl.d_model
    sdt = np.uint16 if wl.dtype == "bf16" else np.float32
    hist = np.empty((int(hoff[-1]), d), dtype=sdt)
    tgt = np.empty((int(toff[-1]), d), dtype=sdt)
    want_grad = wl.backward if with_grad is None else with_grad
    grad = np.empty((int(toff[-1]), d), dtype=sdt) if want_grad else None

    def fill(i):
        x, t = _request_rows(wl, req[i], int(L[i]), int(m[i]))
        hist[hoff[i]:hoff[i + 1]] = x
        tgt[toff[i]:toff[i + 1]] = t
        if grad is not None:
            grad[toff[i]:toff[i + 1]] = _request_grad(wl, req[i], int(m[i]))

    if threads > 1 and len(req) > 1:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(fill, range(len(req))))
    else:
        for i in range(len(req)):
            fill(i)
    return Batch(wl, req, L, m, hoff, toff, hist, tgt, make_weights(wl, scale_q), grad)


def replicate_per_target(b: Batch) -> Batch:
    """Instance-wise (non-RLB) layout of the same samples: every target becomes
    its own request carrying a physical copy of its request's history
    (App. A.3's triplet batching)."""
    reps = b.n_tgt
    rows = []
    for r in range(b.n_requests):
        for _ in range(int(reps[r])):
            rows.append(np.arange(b.hist_off[r], b.hist_off[r + 1]))
    idx = np.concatenate(rows) if rows else np.zeros(0, dtype=np.int64)
    L = np.repeat(b.hist_len, reps)
    ones = np.ones(int(reps.sum()), dtype=np.int64)
    return Batch(b.wl, np.repeat(b.requests, reps), L, ones, offsets(L), offsets(ones),
                 b.hist[idx], b.tgt.copy(), b.weights, None if b.grad_out is None else b.grad_out.copy())


def make_custom_batch(name: str, hist_len: Sequence[int], n_tgt: Sequence[int], *, d_model: int, n_heads: int,
                      n_layers: int, dtype: str, seed: int, scale_q: float = 1.0, with_grad: bool = False,
                      ffn_mult: int = 4) -> Batch:
    """A batch with explicitly listed per-request history lengths and target
    counts (edge cases: tails, empty target segments, single-row histories),
    drawn with the same per-request streams as the named workloads."""
    L = np.asarray(hist_len, dtype=np.int64)
    m = np.asarray(n_tgt, dtype=np.int64)
    wl = Workload(name, len(L), d_model, n_heads, n_layers, dtype, seed, backward=with_grad, ffn_mult=ffn_mult)
    hoff, toff = offsets(L), offsets(m)
    sdt = np.uint16 if dtype == "bf16" else np.float32
    hist = np.empty((int(hoff[-1]), d_model), dtype=sdt)
    tgt = np.empty((int(toff[-1]), d_model), dtype=sdt)
    grad = np.empty((int(toff[-1]), d_model), dtype=sdt) if with_grad else None
    for r in range(len(L)):
        x, t = _request_rows(wl, r, int(L[r]), int(m[r]))
        hist[hoff[r]:hoff[r + 1]] = x
        tgt[toff[r]:toff[r + 1]] = t
        if grad is not None:
            grad[toff[r]:toff[r + 1]] = _request_grad(wl, r, int(m[r]))
    return Batch(wl, np.arange(len(L)), L, m, hoff, toff, hist, tgt, make_weights(wl, scale_q), grad)
