"""Algorithmic work of the STCA forward, per stage, for roofline reporting.

Counts what the method must do, not what an implementation happens to move:
flop = 2 x multiply-accumulates; bytes = compulsory HBM traffic.

Per request r and layer (history length L, m targets, width d, storage s bytes):
  history K/V projection  flop 4 L d^2        bytes 2 L d (read X, once for all
                          layers when the projection of every layer is one GEMM)
                                             + 2 s L d (write K and V)
  cross attention         flop 4 m L d        bytes 2 s L d (read K and V once,
                                             whatever m is: request level batching)
  target update           flop 20 m d^2       (W_O, the 4x FFN and the next W_Q)
"""
from __future__ import annotations

import numpy as np


def stage_costs(hist_len, n_tgt, d: int, n_layers: int, elem_bytes: int = 2):
    L = np.asarray(hist_len, dtype=np.float64)
    m = np.asarray(n_tgt, dtype=np.float64)
    act = m > 0
    L, m = L[act], m[act]
    n = n_layers
    return {
        "proj": {"flop": 4.0 * L.sum() * d * d * n,
                 "bytes": elem_bytes * L.sum() * d + 2.0 * elem_bytes * L.sum() * d * n},
        "attn": {"flop": 4.0 * (m * L).sum() * d * n,
                 "bytes": 2.0 * elem_bytes * L.sum() * d * n},
        "update": {"flop": 20.0 * m.sum() * d * d * n,
                   "bytes": 0.0},
    }


def transformer_macs_per_sample(L: float, d: int, n_layers: int) -> float:
    """Self-attention Transformer over the history, the paper's baseline."""
    return n_layers * (12.0 * d * d * L + 2.0 * L * L * d)
