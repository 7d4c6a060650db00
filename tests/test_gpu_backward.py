"""GPU parity of the STCA backward (through the C ABI) against the oracle's
hand-derived gradients.  Metric per gradient tensor: |g_gpu - g|_inf / |g|_inf.
Bars: 1e-4 for fp32 storage, 2e-2 for bf16 storage."""
import numpy as np
import pytest

from oracle import stca_oracle as O
from paper_2511_06077_amd import workload as W

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}
GRADS = ("dhist", "dtgt", "dwq", "dwk", "dwv", "dwo", "dw1", "dw2")


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available(), "GPU tests need a GPU"
    return t


def tensor_err(g, ref):
    return float(np.abs(g - ref).max() / max(np.abs(ref).max(), 1e-30))


def gpu_grads(torch, b, **forms):
    from paper_2511_06077_amd.device import DeviceBatch, to_device
    db = DeviceBatch(b, backward=True, **forms)
    db.forward()
    g = db.backward(to_device(b.grad_out, "cuda"))
    torch.cuda.synchronize()
    return {k: v.cpu().numpy().astype(np.float64) for k, v in g.items()}


def check(b, g, tol, keys=GRADS, rows=None):
    f = b.f64()
    ref = O.backward(f, f["grad_out"])
    errs = {}
    for k in keys:
        got = g[k]
        if rows is not None and k in rows:
            got = got[rows[k]]
        errs[k] = tensor_err(got, ref[k])
    print(f"[grad] {b.wl.name}: " + " ".join(f"{k}={v:.1e}" for k, v in errs.items()), flush=True)
    for k, v in errs.items():
        assert v <= tol, (k, v)


@pytest.mark.parametrize("chunk", [0, 1])
def test_tiny_f32_gradients(torch, chunk):
    b = W.make_batch(W.WORKLOADS["tiny_f32_R4_m4_L256_d64"])
    check(b, gpu_grads(torch, b, chunk_blocks=chunk), TOL["f32"])


@pytest.mark.parametrize("dtype,d,h", [("bf16", 256, 8), ("bf16", 128, 4), ("f32", 64, 2)])
def test_ragged_tail_gradients(torch, dtype, d, h):
    b = W.make_custom_batch("gtail", [1, 33, 130, 64, 7], [2, 65, 0, 17, 1], d_model=d, n_heads=h, n_layers=2,
                            dtype=dtype, seed=31, with_grad=True)
    check(b, gpu_grads(torch, b, chunk_blocks=2), TOL[dtype])


@pytest.mark.parametrize("d,h", [(256, 8), (128, 4), (64, 2)])
def test_fused_projection_gradients(torch, d, h):
    """Requests of at most 32 targets: the backward projects the history
    inside its attention kernels.  Ragged histories (one row, block tails,
    blocks shared by two requests, a request without targets), several
    history chunks per request, every gradient against the oracle."""
    b = W.make_custom_batch("gfused", [1, 33, 130, 64, 7, 300], [2, 31, 0, 17, 1, 32], d_model=d, n_heads=h,
                            n_layers=2, dtype="bf16", seed=37, with_grad=True)
    check(b, gpu_grads(torch, b, bwd="fused", chunk_blocks=2), TOL["bf16"])


@pytest.mark.parametrize("d,h,mult", [(128, 4, 2), (64, 2, 3)])
def test_fused_other_ffn_width(torch, d, h, mult):
    """An FFN width other than 4 d (still a multiple of d, so the fused
    backward takes the batch): the update kernels' path without the
    compile-time chunk count.  The fast forward's output, stca_forward_train's
    output and every gradient against the oracle."""
    from paper_2511_06077_amd.device import DeviceBatch, to_device
    b = W.make_custom_batch("gffn", [1, 33, 130, 64, 7, 300], [2, 31, 0, 17, 1, 32], d_model=d, n_heads=h,
                            n_layers=2, dtype="bf16", seed=43, with_grad=True, ffn_mult=mult)
    db = DeviceBatch(b, backward=True, bwd="fused", chunk_blocks=2)
    y_fast = db.forward().float().cpu().numpy().astype(np.float64)
    y_train = db.forward_train().float().cpu().numpy().astype(np.float64)
    g = db.backward(to_device(b.grad_out, "cuda"), use_record=True)
    torch.cuda.synchronize()
    ref_y = O.forward(b.f64(), keep=False)["out"]
    for name, y in (("forward", y_fast), ("forward_train", y_train)):
        err = float(np.max(np.abs(y - ref_y).max(axis=1) / np.abs(ref_y).max(axis=1)))
        print(f"[grad] F = {mult} d {name} y err {err:.1e}", flush=True)
        assert err <= TOL["bf16"], (name, err)
    check(b, {k: v.cpu().numpy().astype(np.float64) for k, v in g.items()}, TOL["bf16"])


def test_fused_and_generic_backward_agree(torch):
    """The same batch through the fused backward and through the K|V product
    with the exact fp32 attention (bwd_form STCA_BWD_GENERIC): both within the
    bar of the oracle, and within the bar of each other."""
    b = W.make_custom_batch("gboth", [512, 77, 1024, 5], [16, 3, 32, 1], d_model=256, n_heads=8, n_layers=4,
                            dtype="bf16", seed=41, with_grad=True)
    g_fused = gpu_grads(torch, b, bwd="fused")
    g_gen = gpu_grads(torch, b, bwd="generic")
    check(b, g_fused, TOL["bf16"])
    check(b, g_gen, TOL["bf16"])
    for k in GRADS:
        e = tensor_err(g_fused[k], g_gen[k])
        print(f"[grad] fused vs generic {k}: {e:.1e}", flush=True)
        assert e <= TOL["bf16"], (k, e)


def test_training_record(torch):
    """Training step in two calls: stca_forward_train's output against the
    oracle, and stca_backward_record's gradients identical to the recomputing
    stca_backward's (the same kernels on the same inputs), also after the
    workspace was reused in between."""
    from paper_2511_06077_amd.device import DeviceBatch, to_device
    b = W.make_custom_batch("grec", [1, 33, 130, 64, 7, 300], [2, 31, 0, 17, 1, 32], d_model=256, n_heads=8,
                            n_layers=2, dtype="bf16", seed=43, with_grad=True)
    db = DeviceBatch(b, backward=True, chunk_blocks=3)
    assert db.record is not None
    y = db.forward_train().float().cpu().numpy().astype(np.float64)
    dout = to_device(b.grad_out, "cuda")
    g_rec = db.backward(dout, use_record=True)
    g_full = db.backward(dout)
    g_rec2 = db.backward(dout, use_record=True)
    torch.cuda.synchronize()
    f = b.f64()
    ref_y = O.forward(f, keep=False)["out"]
    err = float(np.max(np.abs(y - ref_y).max(axis=1) / np.abs(ref_y).max(axis=1)))
    print(f"[grad] forward_train y err {err:.1e}", flush=True)
    assert err <= TOL["bf16"], err
    for k in GRADS:
        a, r, a2 = g_rec[k].cpu().numpy(), g_full[k].cpu().numpy(), g_rec2[k].cpu().numpy()
        assert np.array_equal(a, r), k
        assert np.array_equal(a, a2), k
    check(b, {k: v.cpu().numpy().astype(np.float64) for k, v in g_rec.items()}, TOL["bf16"])


def test_training_window_gradients(torch):
    """256 requests x 16 targets, L = 2048, d = 256, 4 layers (the training
    window).  History and target gradients are per request: checked on a
    seeded sample of 16 requests of the full-batch run.  Weight gradients sum
    over all requests: those of a 16-request sub-batch (4096 history rows per
    chunk, split-K products over 32768 history and 256 target rows) are
    checked against the oracle, and on the full batch they must equal
    (linearity) the sum of the gradients of two disjoint halves.  The
    chunking of the history is pinned so that every request's work is the
    same in the full and the half batches: with different chunkings the fp32
    states differ in the last bits and the few ReLU gates that sit within
    that distance of zero flip, each moving a weight gradient by ~1e-4
    relative."""
    wl = W.WORKLOADS["train_bf16_R256_m16_L2048_d256"]
    b = W.make_batch(wl)
    g = gpu_grads(torch, b, chunk_blocks=16)
    req = np.sort(np.random.default_rng(3).choice(wl.n_requests, 16, replace=False))
    sub = W.make_batch(wl, requests=req)
    rows = {
        "dhist": np.concatenate([np.arange(b.hist_off[r], b.hist_off[r + 1]) for r in req]),
        "dtgt": np.concatenate([np.arange(b.tgt_off[r], b.tgt_off[r + 1]) for r in req]),
    }
    check(sub, g, TOL["bf16"], keys=("dhist", "dtgt"), rows=rows)
    # every gradient of the 16-request sub-batch against the oracle
    gs = gpu_grads(torch, sub, chunk_blocks=16)
    check(sub, gs, TOL["bf16"])
    # linearity over requests on the full batch
    half = wl.n_requests // 2
    ga = gpu_grads(torch, W.make_batch(wl, requests=range(half)), chunk_blocks=16)
    gb = gpu_grads(torch, W.make_batch(wl, requests=range(half, wl.n_requests)), chunk_blocks=16)
    for k in ("dwq", "dwk", "dwv", "dwo", "dw1", "dw2"):
        e = tensor_err(g[k], ga[k] + gb[k])
        print(f"[grad] linearity {k}: {e:.1e}", flush=True)
        assert e <= 1e-3, (k, e)


@pytest.mark.parametrize("n_layers", [2])
def test_fused_backward_split_k_weight_gradients(torch, n_layers):
    """128 requests x 16 targets (2048 targets) with 64-row histories: the
    target-side weight-gradient products have K = 2048 target rows, so they
    split over K in the grouped launches (the layer's dW_2, dW_1, dW_O with
    dW_Q of the layer above) and in the lone dW_Q of layer 0, and their
    split sums run.  Every gradient against the oracle."""
    L = [64] * 128
    M = [16] * 128
    b = W.make_custom_batch("gsplit", L, M, d_model=256, n_heads=8, n_layers=n_layers, dtype="bf16", seed=47,
                            with_grad=True)
    check(b, gpu_grads(torch, b, bwd="fused"), TOL["bf16"])


def test_stochastic_length_batch(torch):
    """A stochastic-length training batch (Beta lengths with alpha = 0.02,
    temporal suffixes, token budget, packed): bimodal ragged histories from
    8 rows to the full length.  Forward and every gradient against the oracle."""
    from paper_2511_06077_amd import sl
    from test_gpu_forward import check_against_oracle, run_gpu
    full = W.make_custom_batch("slfull", [2048] * 12, [4, 16, 1, 33, 8, 2, 16, 5, 64, 3, 1, 9], d_model=256,
                               n_heads=8, n_layers=2, dtype="bf16", seed=42, with_grad=True)
    b, info = sl.sl_batch(full, 17, alpha=0.02, l_min=8, l_avg=256, l_max=2048)
    print(f"[sl] kept {info['kept_tokens']} of budget {info['budget']}, lengths {b.hist_len.tolist()}", flush=True)
    assert info["kept_tokens"] <= info["budget"]
    y, a, lse, _ = run_gpu(torch, b)
    check_against_oracle(b, y, a, lse, TOL["bf16"])
    check(b, gpu_grads(torch, b), TOL["bf16"])
