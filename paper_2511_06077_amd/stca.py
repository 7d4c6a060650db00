"""Thin ctypes binding of libstca.so (the C ABI in include/stca.h).

Argument marshalling only: torch tensors supply device memory and the stream;
every step of the computation runs in the library's HIP kernels.  There is no
fallback: if the library is missing, loading it raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libstca.so")

STCA_OK, STCA_ERR_INVALID_ARG, STCA_ERR_UNSUPPORTED, STCA_ERR_WORKSPACE, STCA_ERR_HIP = 0, -1, -2, -3, -4
STCA_ERR_RANGE = -5
STCA_F32, STCA_BF16 = 0, 1
# execution forms (stca_dims_t.kv_form / attn_form / bwd_form); 0 = automatic
STCA_KV_AUTO, STCA_KV_FUSED, STCA_KV_MATERIALIZE = 0, 1, 2
STCA_ATTN_AUTO, STCA_ATTN_STANDARD, STCA_ATTN_REORDERED = 0, 1, 2
STCA_BWD_AUTO, STCA_BWD_FUSED, STCA_BWD_GENERIC, STCA_BWD_REORDERED = 0, 1, 2, 3
FORMS = {
    "kv": {"auto": STCA_KV_AUTO, "fused": STCA_KV_FUSED, "materialize": STCA_KV_MATERIALIZE},
    "attn": {"auto": STCA_ATTN_AUTO, "standard": STCA_ATTN_STANDARD, "reordered": STCA_ATTN_REORDERED},
    "bwd": {"auto": STCA_BWD_AUTO, "fused": STCA_BWD_FUSED, "generic": STCA_BWD_GENERIC,
            "reordered": STCA_BWD_REORDERED},
}

EXPORTED = ("stca_workspace_size", "stca_saved_size", "stca_saved_layout", "stca_forward", "stca_backward",
            "stca_device_status", "stca_status_string", "stca_path", "stca_forward_launch_count",
            "stca_forward_profiled", "stca_backward_launch_count", "stca_backward_profiled",
            "stca_sl_beta", "stca_sl_sample", "stca_sl_allocate", "stca_sl_pack",
            "stca_paper_workspace_size", "stca_paper_saved_size", "stca_paper_saved_layout", "stca_forward_paper",
            "stca_paper_launch_count", "stca_forward_paper_profiled", "stca_train_record_size", "stca_forward_train",
            "stca_backward_record", "stca_forward_noalloc")
NOALLOC_SCRATCH_BYTES = 256 << 20  # STCA_NOALLOC_SCRATCH_BYTES
PAPER_WEIGHT_FIELDS = ("ffn_u", "ffn_v", "ffn_o", "wq", "wk", "wv", "wo", "wc", "wz", "z_u", "z_v", "z_o")


class stca_dims_t(ctypes.Structure):
    _fields_ = [("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32), ("n_layers", ctypes.c_int32),
                ("ffn_hidden", ctypes.c_int32), ("dtype", ctypes.c_int32), ("kv_form", ctypes.c_int32),
                ("attn_form", ctypes.c_int32), ("bwd_form", ctypes.c_int32), ("chunk_blocks", ctypes.c_int32)]


class stca_batch_t(ctypes.Structure):
    _fields_ = [("n_requests", ctypes.c_int32), ("n_hist", ctypes.c_int64), ("n_tgt", ctypes.c_int64),
                ("hist_off", ctypes.c_void_p), ("tgt_off", ctypes.c_void_p),
                ("hist_off_host", ctypes.c_void_p), ("tgt_off_host", ctypes.c_void_p)]


class stca_weights_t(ctypes.Structure):
    _fields_ = [(k, ctypes.c_void_p) for k in ("wq", "wk", "wv", "wo", "w1", "w2")]


class stca_wgrads_t(ctypes.Structure):
    _fields_ = [(k, ctypes.c_void_p) for k in ("dwq", "dwk", "dwv", "dwo", "dw1", "dw2")]


class stca_saved_layout_t(ctypes.Structure):
    _fields_ = [(k, ctypes.c_size_t) for k in ("s", "a", "u", "lse", "total")]


class stca_paper_weights_t(ctypes.Structure):
    _fields_ = [(k, ctypes.c_void_p) for k in PAPER_WEIGHT_FIELDS]


class stca_paper_saved_layout_t(ctypes.Structure):
    _fields_ = [(k, ctypes.c_size_t) for k in ("q", "a", "o", "lse", "xt", "total")]


class StcaError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {status_string(status)} ({status})")
        self.status = status


_lib = None


def lib():
    """Load libstca.so (built in-tree by paper_2511_06077_amd.build)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2511_06077_amd.build`")
        # torch ships its own HIP runtime (soname libamdhip64.so.7, needed by
        # torch as libamdhip64.so): load it first so that libstca binds to the
        # same runtime instead of pulling in a second copy.
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER
        L.stca_workspace_size.restype = ctypes.c_size_t
        L.stca_workspace_size.argtypes = [P(stca_dims_t), P(stca_batch_t), ctypes.c_int]
        L.stca_saved_size.restype = ctypes.c_size_t
        L.stca_saved_size.argtypes = [P(stca_dims_t), P(stca_batch_t)]
        L.stca_saved_layout.restype = ctypes.c_int
        L.stca_saved_layout.argtypes = [P(stca_dims_t), P(stca_batch_t), P(stca_saved_layout_t)]
        L.stca_forward.restype = ctypes.c_int
        L.stca_forward.argtypes = [P(stca_dims_t), P(stca_batch_t), ctypes.c_void_p, ctypes.c_void_p,
                                   P(stca_weights_t), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                   ctypes.c_size_t, ctypes.c_void_p]
        L.stca_backward.restype = ctypes.c_int
        L.stca_backward.argtypes = [P(stca_dims_t), P(stca_batch_t), ctypes.c_void_p, ctypes.c_void_p,
                                    P(stca_weights_t), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                    P(stca_wgrads_t), ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
        L.stca_device_status.restype = ctypes.c_int
        L.stca_device_status.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        L.stca_status_string.restype = ctypes.c_char_p
        L.stca_status_string.argtypes = [ctypes.c_int]
        L.stca_path.restype = ctypes.c_int
        L.stca_path.argtypes = [P(stca_dims_t)]
        L.stca_forward_launch_count.restype = ctypes.c_int
        L.stca_forward_launch_count.argtypes = [P(stca_dims_t), P(stca_batch_t)]
        L.stca_forward_profiled.restype = ctypes.c_int
        L.stca_forward_profiled.argtypes = [P(stca_dims_t), P(stca_batch_t), ctypes.c_void_p, ctypes.c_void_p,
                                            P(stca_weights_t), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                            ctypes.c_size_t, ctypes.c_void_p, P(ctypes.c_void_p), ctypes.c_int,
                                            P(ctypes.c_char_p)]
        L.stca_backward_launch_count.restype = ctypes.c_int
        L.stca_backward_launch_count.argtypes = [P(stca_dims_t), P(stca_batch_t)]
        L.stca_backward_profiled.restype = ctypes.c_int
        L.stca_backward_profiled.argtypes = [P(stca_dims_t), P(stca_batch_t), ctypes.c_void_p, ctypes.c_void_p,
                                             P(stca_weights_t), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                             P(stca_wgrads_t), ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                             P(ctypes.c_void_p), ctypes.c_int, P(ctypes.c_char_p)]
        L.stca_train_record_size.restype = ctypes.c_size_t
        L.stca_train_record_size.argtypes = [P(stca_dims_t), P(stca_batch_t)]
        L.stca_forward_train.restype = ctypes.c_int
        L.stca_forward_train.argtypes = [P(stca_dims_t), P(stca_batch_t), ctypes.c_void_p, ctypes.c_void_p,
                                         P(stca_weights_t), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                         ctypes.c_size_t, ctypes.c_void_p]
        L.stca_backward_record.restype = ctypes.c_int
        L.stca_backward_record.argtypes = [P(stca_dims_t), P(stca_batch_t), ctypes.c_void_p, ctypes.c_void_p,
                                           P(stca_weights_t), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                           ctypes.c_void_p, P(stca_wgrads_t), ctypes.c_void_p, ctypes.c_size_t,
                                           ctypes.c_void_p]
        L.stca_forward_noalloc.restype = ctypes.c_int
        L.stca_forward_noalloc.argtypes = [P(stca_dims_t), P(stca_batch_t), ctypes.c_void_p, ctypes.c_void_p,
                                           P(stca_weights_t), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        I32P = P(ctypes.c_int32)
        L.stca_sl_beta.restype = ctypes.c_double
        L.stca_sl_beta.argtypes = [ctypes.c_double, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]
        L.stca_sl_sample.restype = ctypes.c_int
        L.stca_sl_sample.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_double, ctypes.c_int32, ctypes.c_int32,
                                     ctypes.c_int32, P(ctypes.c_double), I32P]
        L.stca_sl_allocate.restype = ctypes.c_int
        L.stca_sl_allocate.argtypes = [ctypes.c_int32, I32P, I32P, ctypes.c_int64, I32P]
        L.stca_sl_pack.restype = ctypes.c_int
        L.stca_sl_pack.argtypes = [ctypes.c_int32, I32P, I32P, I32P, I32P]
        L.stca_paper_workspace_size.restype = ctypes.c_size_t
        L.stca_paper_workspace_size.argtypes = [P(stca_dims_t), P(stca_batch_t)]
        L.stca_paper_saved_size.restype = ctypes.c_size_t
        L.stca_paper_saved_size.argtypes = [P(stca_dims_t), P(stca_batch_t)]
        L.stca_paper_saved_layout.restype = ctypes.c_int
        L.stca_paper_saved_layout.argtypes = [P(stca_dims_t), P(stca_batch_t), P(stca_paper_saved_layout_t)]
        L.stca_forward_paper.restype = ctypes.c_int
        L.stca_forward_paper.argtypes = [P(stca_dims_t), P(stca_batch_t), ctypes.c_void_p, ctypes.c_void_p,
                                         P(stca_paper_weights_t), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                         ctypes.c_size_t, ctypes.c_void_p]
        L.stca_paper_launch_count.restype = ctypes.c_int
        L.stca_paper_launch_count.argtypes = [P(stca_dims_t), P(stca_batch_t)]
        L.stca_forward_paper_profiled.restype = ctypes.c_int
        L.stca_forward_paper_profiled.argtypes = [P(stca_dims_t), P(stca_batch_t), ctypes.c_void_p, ctypes.c_void_p,
                                                  P(stca_paper_weights_t), ctypes.c_void_p, ctypes.c_void_p,
                                                  ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                                  P(ctypes.c_void_p), ctypes.c_int, P(ctypes.c_char_p)]
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().stca_status_string(int(status)).decode()


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def dims(d_model: int, n_heads: int, n_layers: int, ffn_hidden: int, dtype: int, kv: str = "auto",
         attn: str = "auto", bwd: str = "auto", chunk_blocks: int = 0) -> stca_dims_t:
    """Model shape and execution forms (names as in FORMS; chunk_blocks 0 =
    automatic)."""
    return stca_dims_t(d_model, n_heads, n_layers, ffn_hidden, dtype, FORMS["kv"][kv], FORMS["attn"][attn],
                       FORMS["bwd"][bwd], chunk_blocks)


def batch(n_requests: int, n_hist: int, n_tgt: int, hist_off, tgt_off, hist_off_host=None,
          tgt_off_host=None) -> stca_batch_t:
    """hist_off / tgt_off: device int32 tensors; *_host: optional contiguous
    int32 numpy arrays (kept alive by the caller)."""
    def host(a):
        return None if a is None else a.ctypes.data
    return stca_batch_t(n_requests, n_hist, n_tgt, _ptr(hist_off), _ptr(tgt_off), host(hist_off_host),
                        host(tgt_off_host))


def weights(wq, wk, wv, wo, w1, w2) -> stca_weights_t:
    return stca_weights_t(*(_ptr(t) for t in (wq, wk, wv, wo, w1, w2)))


def wgrads(dwq, dwk, dwv, dwo, dw1, dw2) -> stca_wgrads_t:
    return stca_wgrads_t(*(_ptr(t) for t in (dwq, dwk, dwv, dwo, dw1, dw2)))


def stca_path(d: stca_dims_t) -> int:
    return lib().stca_path(ctypes.byref(d))


def stca_workspace_size(d: stca_dims_t, b: stca_batch_t, with_backward: bool = False) -> int:
    return lib().stca_workspace_size(ctypes.byref(d), ctypes.byref(b), int(with_backward))


def stca_saved_size(d: stca_dims_t, b: stca_batch_t) -> int:
    return lib().stca_saved_size(ctypes.byref(d), ctypes.byref(b))


def stca_saved_layout(d: stca_dims_t, b: stca_batch_t) -> stca_saved_layout_t:
    out = stca_saved_layout_t()
    st = lib().stca_saved_layout(ctypes.byref(d), ctypes.byref(b), ctypes.byref(out))
    if st != STCA_OK:
        raise StcaError(st, "stca_saved_layout")
    return out


def stca_forward(d, b, hist, tgt, w, out, saved, ws, ws_bytes: int, stream=None, check: bool = True) -> int:
    st = lib().stca_forward(ctypes.byref(d), ctypes.byref(b), _ptr(hist), _ptr(tgt), ctypes.byref(w), _ptr(out),
                            _ptr(saved), _ptr(ws), int(ws_bytes), _ptr(stream))
    if check and st != STCA_OK:
        raise StcaError(st, "stca_forward")
    return st


def stca_backward(d, b, hist, tgt, w, dout, dhist, dtgt, dw, ws, ws_bytes: int, stream=None,
                  check: bool = True) -> int:
    st = lib().stca_backward(ctypes.byref(d), ctypes.byref(b), _ptr(hist), _ptr(tgt), ctypes.byref(w),
                             _ptr(dout), _ptr(dhist), _ptr(dtgt), ctypes.byref(dw), _ptr(ws), int(ws_bytes),
                             _ptr(stream))
    if check and st != STCA_OK:
        raise StcaError(st, "stca_backward")
    return st


def stca_forward_noalloc(d, b, hist, tgt, w, out, saved, stream=None, check: bool = True) -> int:
    """stca_forward with the library's own per-GPU scratch array as the
    workspace (no workspace argument, nothing allocated)."""
    st = lib().stca_forward_noalloc(ctypes.byref(d), ctypes.byref(b), _ptr(hist), _ptr(tgt), ctypes.byref(w),
                                    _ptr(out), _ptr(saved), _ptr(stream))
    if check and st != STCA_OK:
        raise StcaError(st, "stca_forward_noalloc")
    return st


def stca_train_record_size(d: stca_dims_t, b: stca_batch_t) -> int:
    return lib().stca_train_record_size(ctypes.byref(d), ctypes.byref(b))


def stca_forward_train(d, b, hist, tgt, w, out, record, ws, ws_bytes: int, stream=None, check: bool = True) -> int:
    st = lib().stca_forward_train(ctypes.byref(d), ctypes.byref(b), _ptr(hist), _ptr(tgt), ctypes.byref(w),
                                  _ptr(out), _ptr(record), _ptr(ws), int(ws_bytes), _ptr(stream))
    if check and st != STCA_OK:
        raise StcaError(st, "stca_forward_train")
    return st


def stca_backward_record(d, b, hist, tgt, w, record, dout, dhist, dtgt, dw, ws, ws_bytes: int, stream=None,
                         check: bool = True) -> int:
    st = lib().stca_backward_record(ctypes.byref(d), ctypes.byref(b), _ptr(hist), _ptr(tgt), ctypes.byref(w),
                                    _ptr(record), _ptr(dout), _ptr(dhist), _ptr(dtgt), ctypes.byref(dw), _ptr(ws),
                                    int(ws_bytes), _ptr(stream))
    if check and st != STCA_OK:
        raise StcaError(st, "stca_backward_record")
    return st


def stca_device_status(ws, stream=None) -> int:
    return lib().stca_device_status(_ptr(ws), _ptr(stream))


def stca_forward_launch_count(d: stca_dims_t, b: stca_batch_t) -> int:
    return lib().stca_forward_launch_count(ctypes.byref(d), ctypes.byref(b))


def stca_forward_profiled(d, b, hist, tgt, w, out, saved, ws, ws_bytes: int, stream, events, labels=None) -> int:
    """events: a ctypes array of hipEvent_t (see HipEvents); labels: optional
    ctypes array of c_char_p receiving kernel names."""
    st = lib().stca_forward_profiled(ctypes.byref(d), ctypes.byref(b), _ptr(hist), _ptr(tgt), ctypes.byref(w),
                                     _ptr(out), _ptr(saved), _ptr(ws), int(ws_bytes), _ptr(stream), events,
                                     len(events), labels)
    if st != STCA_OK:
        raise StcaError(st, "stca_forward_profiled")
    return st


def stca_backward_launch_count(d: stca_dims_t, b: stca_batch_t) -> int:
    return lib().stca_backward_launch_count(ctypes.byref(d), ctypes.byref(b))


def stca_backward_profiled(d, b, hist, tgt, w, dout, dhist, dtgt, dw, ws, ws_bytes: int, stream, events,
                           labels=None) -> int:
    """As stca_backward, with events recorded at phase boundaries (see HipEvents)."""
    st = lib().stca_backward_profiled(ctypes.byref(d), ctypes.byref(b), _ptr(hist), _ptr(tgt), ctypes.byref(w),
                                      _ptr(dout), _ptr(dhist), _ptr(dtgt), ctypes.byref(dw), _ptr(ws), int(ws_bytes),
                                      _ptr(stream), events, len(events), labels)
    if st != STCA_OK:
        raise StcaError(st, "stca_backward_profiled")
    return st


# ---- paper-exact stack
def paper_weights(**w) -> stca_paper_weights_t:
    """Keyword arguments named as PAPER_WEIGHT_FIELDS (wc may be None for one layer)."""
    return stca_paper_weights_t(*(_ptr(w.get(k)) for k in PAPER_WEIGHT_FIELDS))


def stca_paper_workspace_size(d: stca_dims_t, b: stca_batch_t) -> int:
    return lib().stca_paper_workspace_size(ctypes.byref(d), ctypes.byref(b))


def stca_paper_saved_size(d: stca_dims_t, b: stca_batch_t) -> int:
    return lib().stca_paper_saved_size(ctypes.byref(d), ctypes.byref(b))


def stca_paper_saved_layout(d: stca_dims_t, b: stca_batch_t) -> stca_paper_saved_layout_t:
    out = stca_paper_saved_layout_t()
    st = lib().stca_paper_saved_layout(ctypes.byref(d), ctypes.byref(b), ctypes.byref(out))
    if st != STCA_OK:
        raise StcaError(st, "stca_paper_saved_layout")
    return out


def stca_forward_paper(d, b, hist, tgt, w, z, saved, ws, ws_bytes: int, stream=None, check: bool = True) -> int:
    st = lib().stca_forward_paper(ctypes.byref(d), ctypes.byref(b), _ptr(hist), _ptr(tgt), ctypes.byref(w), _ptr(z),
                                  _ptr(saved), _ptr(ws), int(ws_bytes), _ptr(stream))
    if check and st != STCA_OK:
        raise StcaError(st, "stca_forward_paper")
    return st


def stca_paper_launch_count(d: stca_dims_t, b: stca_batch_t) -> int:
    return lib().stca_paper_launch_count(ctypes.byref(d), ctypes.byref(b))


def stca_forward_paper_profiled(d, b, hist, tgt, w, z, saved, ws, ws_bytes: int, stream, events, labels=None) -> int:
    st = lib().stca_forward_paper_profiled(ctypes.byref(d), ctypes.byref(b), _ptr(hist), _ptr(tgt), ctypes.byref(w),
                                           _ptr(z), _ptr(saved), _ptr(ws), int(ws_bytes), _ptr(stream), events,
                                           len(events), labels)
    if st != STCA_OK:
        raise StcaError(st, "stca_forward_paper_profiled")
    return st


class HipEvents:
    """A set of HIP events created through the HIP runtime (for timing kernels
    on the stream the library launches them on)."""

    def __init__(self, n: int):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.ev = (ctypes.c_void_p * n)()
        for i in range(n):
            e = ctypes.c_void_p()
            # timing-only events: no system-scope fence (cache writeback and
            # invalidate) when recorded, which would otherwise slow the
            # kernels around every marker
            if self.hip.hipEventCreateWithFlags(ctypes.byref(e), 0x20000000) != 0:  # hipEventDisableSystemFence
                raise RuntimeError("hipEventCreateWithFlags failed")
            self.ev[i] = e
        self.labels = (ctypes.c_char_p * max(1, n - 1))()

    def elapsed_ms(self, i: int, j: int) -> float:
        if self.hip.hipEventSynchronize(self.ev[j]) != 0:
            raise RuntimeError("hipEventSynchronize failed")
        ms = ctypes.c_float()
        if self.hip.hipEventElapsedTime(ctypes.byref(ms), self.ev[i], self.ev[j]) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(ms.value)

    def label(self, k: int) -> str:
        v = self.labels[k]
        return v.decode() if v else "?"

    def close(self):
        for i in range(len(self.ev)):
            if self.ev[i]:
                self.hip.hipEventDestroy(self.ev[i])
                self.ev[i] = None


# ---- stochastic-length batches (host functions)
def _i32p(a):
    return None if a is None else a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def sl_beta(alpha: float, l_min: int, l_avg: int, l_max: int) -> float:
    return lib().stca_sl_beta(alpha, l_min, l_avg, l_max)


def sl_sample(seed: int, n: int, alpha: float, l_min: int, l_avg: int, l_max: int):
    """(l_raw float64 [n], l_train int32 [n])"""
    import numpy as np
    raw = np.empty(n, dtype=np.float64)
    out = np.empty(n, dtype=np.int32)
    st = lib().stca_sl_sample(seed, n, alpha, l_min, l_avg, l_max,
                              raw.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), _i32p(out))
    if st != STCA_OK:
        raise StcaError(st, "stca_sl_sample")
    return raw, out


def sl_allocate(l_full, l_train, budget: int):
    import numpy as np
    l_full = np.ascontiguousarray(l_full, dtype=np.int32)
    l_train = np.ascontiguousarray(l_train, dtype=np.int32)
    out = np.empty_like(l_full)
    st = lib().stca_sl_allocate(len(l_full), _i32p(l_full), _i32p(l_train), int(budget), _i32p(out))
    if st != STCA_OK:
        raise StcaError(st, "stca_sl_allocate")
    return out


def sl_pack(full_off, l_keep):
    """(hist_off int32 [n+1], src_rows int32 [sum l_keep])"""
    import numpy as np
    full_off = np.ascontiguousarray(full_off, dtype=np.int32)
    l_keep = np.ascontiguousarray(l_keep, dtype=np.int32)
    hoff = np.empty(len(l_keep) + 1, dtype=np.int32)
    src = np.empty(int(l_keep.sum()), dtype=np.int32)
    st = lib().stca_sl_pack(len(l_keep), _i32p(full_off), _i32p(l_keep), _i32p(hoff), _i32p(src))
    if st != STCA_OK:
        raise StcaError(st, "stca_sl_pack")
    return hoff, src
