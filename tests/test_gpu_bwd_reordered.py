"""GPU parity of the backward in the reordered form (bwd_form
STCA_BWD_REORDERED: the attention gradients through u = q W_K^T and
h = da W_V^T per target and head, Sec. 3.1's reordering applied to the
gradients; no K, V, dK or dV) against the oracle's hand-derived gradients.
Metric and bars as in test_gpu_backward (|g - g_ref|_inf / |g_ref|_inf,
2e-2 for bf16 storage)."""
import numpy as np
import pytest

from paper_2511_06077_amd import workload as W
from test_gpu_backward import GRADS, TOL, check, gpu_grads, tensor_err

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available(), "GPU tests need a GPU"
    return t


def edge_batch(d, h, seed, scale_q=1.0, n_layers=2):
    """Ragged histories (one row, block tails, blocks shared by two requests,
    a long request, a request without targets) and target counts up to the
    form's limit of 128 / n_heads per request."""
    mmax = 128 // h
    return W.make_custom_batch("grd", [1, 33, 130, 64, 7, 700, 45], [2, mmax, 0, mmax - 1, 1, 5, 3], d_model=d,
                               n_heads=h, n_layers=n_layers, dtype="bf16", seed=seed, with_grad=True,
                               scale_q=scale_q)


@pytest.mark.parametrize("d,h", [(256, 8), (128, 4)])
def test_reordered_gradients(torch, d, h):
    """Every gradient against the oracle; the rows of the request without
    targets get an exactly zero history gradient."""
    b = edge_batch(d, h, 71)
    g = gpu_grads(torch, b, bwd="reordered")
    check(b, g, TOL["bf16"])
    r = 2  # no targets
    assert not np.any(g["dhist"][b.hist_off[r]:b.hist_off[r + 1]])


def test_reordered_and_fused_agree(torch):
    """The same batch through the reordered and the fused backward: both
    within the bar of the oracle and of each other."""
    b = edge_batch(256, 8, 73, n_layers=3)
    g_rd = gpu_grads(torch, b, bwd="reordered")
    g_fu = gpu_grads(torch, b, bwd="fused")
    check(b, g_rd, TOL["bf16"])
    check(b, g_fu, TOL["bf16"])
    for k in GRADS:
        e = tensor_err(g_rd[k], g_fu[k])
        print(f"[grad] reordered vs fused {k}: {e:.1e}", flush=True)
        assert e <= TOL["bf16"], (k, e)


def test_reordered_peaked_softmax(torch):
    """W_Q scaled by 8: sharply peaked softmax weights, where the scores'
    rounding matters most (the recomputed weights use fp16 X and U)."""
    b = edge_batch(256, 8, 79, scale_q=8.0)
    check(b, gpu_grads(torch, b, bwd="reordered"), TOL["bf16"])


def test_reordered_training_record(torch):
    """stca_forward_train then stca_backward_record: identical to the
    recomputing backward, and against the oracle."""
    from paper_2511_06077_amd.device import DeviceBatch, to_device
    b = edge_batch(256, 8, 83)
    db = DeviceBatch(b, backward=True, bwd="reordered")
    assert db.record is not None
    db.forward_train()
    dout = to_device(b.grad_out, "cuda")
    g_rec = db.backward(dout, use_record=True)
    g_full = db.backward(dout)
    torch.cuda.synchronize()
    for k in GRADS:
        a, r = g_rec[k].cpu().numpy(), g_full[k].cpu().numpy()
        assert np.array_equal(a, r), k
    check(b, {k: v.cpu().numpy().astype(np.float64) for k, v in g_rec.items()}, TOL["bf16"])


def test_reordered_is_the_automatic_choice(torch):
    """16 targets x 8 heads = 128 pairs per request and histories balanced
    over the CUs (the training window's shape, here 64 rows each) take the
    reordered form by itself (no dK | dV phase); every gradient against the
    oracle.  The ragged edge batch, with one history much longer than a CU's
    share, takes the fused form."""
    from paper_2511_06077_amd import stca
    from paper_2511_06077_amd.device import DeviceBatch
    b = W.make_custom_batch("gauto", [64] * 12, [16, 3, 16, 1, 9, 16, 16, 2, 16, 7, 16, 16], d_model=256,
                            n_heads=8, n_layers=2, dtype="bf16", seed=89, with_grad=True)
    db = DeviceBatch(b, backward=True)
    n = b.wl.n_layers
    assert stca.stca_backward_launch_count(db.dims, db.batch) == 6 + 6 * n
    check(b, gpu_grads(torch, b), TOL["bf16"])
    e = edge_batch(256, 8, 89)
    de = DeviceBatch(e, backward=True)
    assert stca.stca_backward_launch_count(de.dims, de.batch) == 7 + 5 * e.wl.n_layers


def test_reordered_long_history(torch):
    """A history of 3000 rows: the attention pass cuts it into chunks whose Z,
    Y partials are summed, and the dX product's units (at most 16 history
    chunks per request) span several 128-row tiles.  Every gradient against
    the oracle."""
    b = W.make_custom_batch("glong", [3000, 64, 517], [16, 5, 9], d_model=256, n_heads=8, n_layers=2,
                            dtype="bf16", seed=97, with_grad=True)
    check(b, gpu_grads(torch, b, bwd="reordered"), TOL["bf16"])
