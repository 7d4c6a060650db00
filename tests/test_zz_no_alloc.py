"""stca_forward_noalloc (the forward with the library's per-GPU scratch array
as its workspace) against stca_forward on the same inputs: two calls in a
row, the second on a smaller batch (the array keeps the first call's
contents), and the size limit checked on the host before any launch."""
import numpy as np
import pytest

from paper_2511_06077_amd import workload as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available(), "GPU tests need a GPU"
    return t


def _noalloc(torch, db):
    from paper_2511_06077_amd import stca
    out = torch.empty_like(db.out)
    saved = torch.empty_like(db.saved)
    stca.stca_forward_noalloc(db.dims, db.batch, db.hist, db.tgt, db.weights, out, saved, db.stream())
    return out, saved


def _check(torch, db, out, saved):
    y = db.forward()
    torch.cuda.synchronize()
    n, nt, d, h = db.b.wl.n_layers, db.b.n_tgt_total, db.b.wl.d_model, db.b.wl.n_heads
    assert torch.equal(out, y)
    for name, cols in (("s", d), ("a", d), ("u", d), ("lse", h)):
        off, cnt = getattr(db.layout, name), 4 * n * nt * cols
        assert torch.equal(saved[off:off + cnt], db.saved[off:off + cnt]), name


@pytest.mark.parametrize("forms", [{}, {"kv": "materialize"}])
def test_noalloc_matches_forward_twice(torch, forms):
    from paper_2511_06077_amd.device import DeviceBatch
    big = W.make_batch(W.WORKLOADS["uniform_bf16_R64_m16_L1024_d128"])
    small = W.make_custom_batch("noalloc_small", [1, 7, 300, 65], [3, 0, 17, 33], d_model=256, n_heads=8,
                                n_layers=2, dtype="bf16", seed=71)
    dbs = [DeviceBatch(bb, keep_saved=True, **forms) for bb in (big, small)]
    for db in dbs:  # the second call is the smaller one
        out, saved = _noalloc(torch, db)
        torch.cuda.synchronize()
        _check(torch, db, out, saved)
        print(f"[noalloc] {db.b.wl.name} {forms}: equal to stca_forward ({db.ws_bytes} workspace bytes)",
              flush=True)


def test_noalloc_rejects_what_does_not_fit(torch):
    """A batch whose workspace exceeds the array: STCA_ERR_WORKSPACE on the
    host (the sizes alone decide; nothing is launched)."""
    from paper_2511_06077_amd import stca
    L = np.full(4096, 2048, dtype=np.int32)
    m = np.full(4096, 32, dtype=np.int32)
    ho, to = W.offsets(L), W.offsets(m)
    d = stca.dims(256, 8, 4, 1024, stca.STCA_BF16)
    b = stca.batch(len(L), int(ho[-1]), int(to[-1]), 0x10000, 0x20000, ho, to)
    assert stca.stca_workspace_size(d, b) > stca.NOALLOC_SCRATCH_BYTES
    w = stca.weights(*([0x100000] * 6))
    st = stca.stca_forward_noalloc(d, b, 0x200000, 0x300000, w, 0x400000, None, None, check=False)
    assert st == stca.STCA_ERR_WORKSPACE
