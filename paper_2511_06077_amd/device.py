"""Device-resident STCA batch: uploads a packed workload batch into torch
device memory and calls the C ABI on it.  Plumbing only (allocation, copies,
pointer marshalling); all computation happens in libstca.so.
"""
from __future__ import annotations

from typing import Optional

import numpy as np

from . import stca
from .workload import WEIGHT_NAMES, Batch


def _torch():
    import torch
    return torch


def to_device(a: np.ndarray, device):
    torch = _torch()
    if a.dtype == np.uint16:
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(device)


class DeviceBatch:
    """One batch on the GPU plus its workspace (and, optionally, the saved
    buffer the backward pass needs)."""

    def __init__(self, b: Batch, device="cuda", keep_saved: bool = False, backward: bool = False,
                 host_offsets: bool = True, **forms):
        """forms: kv, attn, bwd (names of stca.FORMS) and chunk_blocks, passed
        through stca_dims_t."""
        self._setup(b, to_device(b.hist, device), to_device(b.tgt, device),
                    {k: to_device(b.weights[k], device) for k in WEIGHT_NAMES}, device, keep_saved, backward,
                    host_offsets, forms)

    @classmethod
    def from_tensors(cls, b: Batch, hist, tgt, weights: dict, device="cuda", keep_saved: bool = False,
                     backward: bool = False, host_offsets: bool = True, **forms):
        """A batch whose rows are already device tensors (b supplies the shapes
        and offsets; its row arrays are not read)."""
        self = cls.__new__(cls)
        self._setup(b, hist, tgt, weights, device, keep_saved, backward, host_offsets, forms)
        return self

    def _setup(self, b, hist, tgt, weights, device, keep_saved, backward, host_offsets, forms):
        torch = _torch()
        self.b = b
        wl = b.wl
        self.device = torch.device(device)
        self.bf16 = wl.dtype == "bf16"
        self.sdtype = torch.bfloat16 if self.bf16 else torch.float32
        self.hist = hist
        self.tgt = tgt
        self.w = weights
        self.hoff_h = np.ascontiguousarray(b.hist_off, dtype=np.int32)
        self.toff_h = np.ascontiguousarray(b.tgt_off, dtype=np.int32)
        self.hoff = torch.from_numpy(self.hoff_h).to(device)
        self.toff = torch.from_numpy(self.toff_h).to(device)
        self.dims = stca.dims(wl.d_model, wl.n_heads, wl.n_layers, wl.ffn_hidden,
                              stca.STCA_BF16 if self.bf16 else stca.STCA_F32, **forms)
        self.batch = stca.batch(b.n_requests, b.n_hist, b.n_tgt_total, self.hoff, self.toff,
                                self.hoff_h if host_offsets else None, self.toff_h if host_offsets else None)
        self.weights = stca.weights(*(self.w[k] for k in WEIGHT_NAMES))
        self.out = torch.empty((b.n_tgt_total, wl.d_model), dtype=self.sdtype, device=device)
        self.ws_bytes = stca.stca_workspace_size(self.dims, self.batch, False)
        if self.ws_bytes == 0:
            raise stca.StcaError(stca.STCA_ERR_INVALID_ARG, "stca_workspace_size")
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        self.saved = None
        if keep_saved:
            self.saved_bytes = stca.stca_saved_size(self.dims, self.batch)
            self.saved = torch.empty(self.saved_bytes, dtype=torch.uint8, device=device)
            self.layout = stca.stca_saved_layout(self.dims, self.batch)
        self.bws = None
        self.record = None
        if backward:
            self.bws_bytes = stca.stca_workspace_size(self.dims, self.batch, True)
            self.bws = torch.empty(self.bws_bytes, dtype=torch.uint8, device=device)
            # training record for stca_forward_train / stca_backward_record
            # (batches the fused backward takes)
            rec = stca.stca_train_record_size(self.dims, self.batch)
            if rec:
                self.record = torch.empty(rec, dtype=torch.uint8, device=device)

    def stream(self):
        return _torch().cuda.current_stream(self.device).cuda_stream

    def forward(self, stream: Optional[int] = None):
        stca.stca_forward(self.dims, self.batch, self.hist, self.tgt, self.weights, self.out, self.saved,
                          self.ws, self.ws_bytes, self.stream() if stream is None else stream)
        return self.out

    def device_status(self) -> int:
        return stca.stca_device_status(self.ws, self.stream())

    def saved_tensor(self, name: str):
        """Per-layer saved intermediate: s, a, u -> [n, N_tgt, d]; lse -> [n, N_tgt, h] (fp32)."""
        torch = _torch()
        wl = self.b.wl
        n, nt = wl.n_layers, self.b.n_tgt_total
        cols = wl.n_heads if name == "lse" else wl.d_model
        off = getattr(self.layout, name)
        count = n * nt * cols
        flat = self.saved[off:off + 4 * count].view(torch.float32)
        return flat.view(n, nt, cols)

    def forward_train(self, stream: Optional[int] = None):
        """Forward of a training step: out and the training record."""
        stca.stca_forward_train(self.dims, self.batch, self.hist, self.tgt, self.weights, self.out, self.record,
                                self.bws, self.bws_bytes, self.stream() if stream is None else stream)
        return self.out

    def backward(self, dout, stream: Optional[int] = None, use_record: bool = False):
        """Gradients of sum <dout, out>; with use_record, from the record of the
        last forward_train call instead of a recomputation."""
        torch = _torch()
        wl = self.b.wl
        d, F, n = wl.d_model, wl.ffn_hidden, wl.n_layers
        f32 = dict(dtype=torch.float32, device=self.device)
        g = {
            "dhist": torch.empty((self.b.n_hist, d), **f32),
            "dtgt": torch.empty((self.b.n_tgt_total, d), **f32),
            "dwq": torch.empty((n, d, d), **f32), "dwk": torch.empty((n, d, d), **f32),
            "dwv": torch.empty((n, d, d), **f32), "dwo": torch.empty((n, d, d), **f32),
            "dw1": torch.empty((n, d, F), **f32), "dw2": torch.empty((n, F, d), **f32),
        }
        dw = stca.wgrads(g["dwq"], g["dwk"], g["dwv"], g["dwo"], g["dw1"], g["dw2"])
        if use_record:
            stca.stca_backward_record(self.dims, self.batch, self.hist, self.tgt, self.weights, self.record, dout,
                                      g["dhist"], g["dtgt"], dw, self.bws, self.bws_bytes,
                                      self.stream() if stream is None else stream)
        else:
            stca.stca_backward(self.dims, self.batch, self.hist, self.tgt, self.weights, dout,
                               g["dhist"], g["dtgt"], dw, self.bws, self.bws_bytes,
                               self.stream() if stream is None else stream)
        return g


class PaperDeviceBatch:
    """A batch with paper-exact weights on the GPU, for stca_forward_paper."""

    def __init__(self, b: Batch, weights: dict, device="cuda", keep_saved: bool = False,
                 host_offsets: bool = True, chunk_blocks: int = 0):
        torch = _torch()
        self.b = b
        wl = b.wl
        self.device = torch.device(device)
        self.bf16 = wl.dtype == "bf16"
        self.sdtype = torch.bfloat16 if self.bf16 else torch.float32
        self.hist = to_device(b.hist, device)
        self.tgt = to_device(b.tgt, device)
        self.w = {k: (to_device(v, device) if v.size else None) for k, v in weights.items()}
        self.hoff_h = np.ascontiguousarray(b.hist_off, dtype=np.int32)
        self.toff_h = np.ascontiguousarray(b.tgt_off, dtype=np.int32)
        self.hoff = torch.from_numpy(self.hoff_h).to(device)
        self.toff = torch.from_numpy(self.toff_h).to(device)
        self.dims = stca.dims(wl.d_model, wl.n_heads, wl.n_layers, wl.ffn_hidden,
                              stca.STCA_BF16 if self.bf16 else stca.STCA_F32, chunk_blocks=chunk_blocks)
        self.batch = stca.batch(b.n_requests, b.n_hist, b.n_tgt_total, self.hoff, self.toff,
                                self.hoff_h if host_offsets else None, self.toff_h if host_offsets else None)
        self.weights = stca.paper_weights(**self.w)
        self.z = torch.empty((b.n_tgt_total, wl.d_model), dtype=self.sdtype, device=device)
        self.ws_bytes = stca.stca_paper_workspace_size(self.dims, self.batch)
        if self.ws_bytes == 0:
            raise stca.StcaError(stca.STCA_ERR_INVALID_ARG, "stca_paper_workspace_size")
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        self.saved = None
        if keep_saved:
            self.saved = torch.empty(stca.stca_paper_saved_size(self.dims, self.batch), dtype=torch.uint8,
                                     device=device)
            self.layout = stca.stca_paper_saved_layout(self.dims, self.batch)

    def stream(self):
        return _torch().cuda.current_stream(self.device).cuda_stream

    def forward(self, stream: Optional[int] = None):
        stca.stca_forward_paper(self.dims, self.batch, self.hist, self.tgt, self.weights, self.z, self.saved,
                                self.ws, self.ws_bytes, self.stream() if stream is None else stream)
        return self.z

    def saved_tensor(self, name: str):
        """q, a -> [n, N_tgt, d]; o -> [N_tgt, n, d]; lse -> [n, N_tgt, h];
        xt -> [n, N_hist, d] (fp32)."""
        torch = _torch()
        wl = self.b.wl
        n, nt, nh, d = wl.n_layers, self.b.n_tgt_total, self.b.n_hist, wl.d_model
        shape = {"q": (n, nt, d), "a": (n, nt, d), "o": (nt, n, d), "lse": (n, nt, wl.n_heads),
                 "xt": (n, nh, d)}[name]
        off = getattr(self.layout, name)
        count = int(np.prod(shape))
        return self.saved[off:off + 4 * count].view(torch.float32).view(*shape)
