"""Stochastic-length training batches (Sec. 3.3; App. "Extrapolation
details"): a batch of full histories is cut to Beta-sampled temporal suffixes
under a token budget and packed without padding, by the library's host
functions (stca_sl_sample, stca_sl_allocate, stca_sl_pack); the result is an
ordinary ragged batch for stca_forward / stca_backward.

The row gather that assembles the packed batch (the kept suffix rows of the
full histories, by the index stca_sl_pack returns) is data preparation on
the host, as a data loader would do it; no computation of the method takes
place in it."""
from __future__ import annotations

from dataclasses import replace

import numpy as np

from . import stca
from . import workload as W


def sl_batch(full: W.Batch, seed: int, *, alpha: float = 0.02, l_min: int = 8, l_avg: int = 2048,
             l_max: int = 10240, budget: int | None = None):
    """The packed stochastic-length batch drawn from `full`, and a record of
    the draw (raw and rounded lengths, budget, kept lengths, sequence
    sparsity)."""
    R = full.n_requests
    raw, l_train = stca.sl_sample(seed, R, alpha, l_min, l_avg, l_max)
    budget = R * l_avg if budget is None else budget
    keep = stca.sl_allocate(full.hist_len, l_train, budget)
    hoff, src = stca.sl_pack(full.hist_off, keep)
    b = W.Batch(replace(full.wl, name=full.wl.name + "_sl"), full.requests.copy(), keep.astype(np.int64),
                full.n_tgt.copy(), hoff, full.tgt_off.copy(), full.hist[src], full.tgt, full.weights, full.grad_out)
    info = {"alpha": alpha, "beta": stca.sl_beta(alpha, l_min, l_avg, l_max), "l_min": l_min, "l_avg": l_avg,
            "l_max": l_max, "budget": int(budget), "l_raw_mean": float(raw.mean()),
            "l_train_mean": float(l_train.mean()), "kept_tokens": int(keep.sum()),
            "sequence_sparsity": float(keep.mean() / l_max)}
    return b, info
