"""The C-ABI library loads, exports every declared entry point, and rejects
bad arguments on the host before any launch (runs without a GPU)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2511_06077_amd import stca

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "stca.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(stca_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert "stca_forward" in names and "stca_backward" in names
    lib = stca.lib()
    for n in names:
        assert hasattr(lib, n), n
    assert set(stca.EXPORTED) <= set(names)


def test_status_strings():
    for s in (0, -1, -2, -3, -4, -5):
        assert stca.status_string(s)


def fake_batch(hoff, toff):
    hoff = np.asarray(hoff, dtype=np.int32)
    toff = np.asarray(toff, dtype=np.int32)
    # device pointers are never dereferenced on these paths
    return stca.batch(len(hoff) - 1, int(hoff[-1]), int(toff[-1]), 0x10000, 0x20000, hoff, toff), (hoff, toff)


GOOD_DIMS = dict(d_model=256, n_heads=8, n_layers=4, ffn_hidden=1024, dtype=stca.STCA_BF16)


def dims(**kw):
    forms = {k: kw.pop(k) for k in ("kv", "attn", "bwd", "chunk_blocks") if k in kw}
    a = dict(GOOD_DIMS)
    a.update(kw)
    return stca.dims(a["d_model"], a["n_heads"], a["n_layers"], a["ffn_hidden"], a["dtype"], **forms)


def fake_weights():
    return stca.weights(*([0x100000] * 6))


def call_forward(d, b, ws_bytes=1 << 40, hist=0x200000, tgt=0x300000, out=0x400000, ws=0x500000):
    return stca.stca_forward(d, b, hist, tgt, fake_weights(), out, None, ws, ws_bytes, None, check=False)


def test_path_selection():
    assert stca.stca_path(dims()) == 1
    assert stca.stca_path(dims(d_model=128, n_heads=4)) == 1
    assert stca.stca_path(dims(dtype=stca.STCA_F32)) == 0
    assert stca.stca_path(dims(d_model=64, n_heads=2, dtype=stca.STCA_F32)) == 0
    assert stca.stca_path(dims(n_heads=16)) == 0  # bf16, d_h = 16: generic kernels
    assert stca.stca_path(dims(n_heads=7)) == stca.STCA_ERR_INVALID_ARG
    assert stca.stca_path(dims(ffn_hidden=100)) == stca.STCA_ERR_UNSUPPORTED
    assert stca.stca_path(dims(ffn_hidden=96)) == 0  # not a multiple of 256: generic kernels
    assert stca.stca_path(dims(ffn_hidden=768)) == 1
    assert stca.stca_path(dims(n_heads=2)) == stca.STCA_ERR_UNSUPPORTED  # d_h = 128
    assert stca.stca_path(dims(dtype=7)) == stca.STCA_ERR_INVALID_ARG


@pytest.mark.parametrize("hoff,toff", [
    ([0, 5, 3, 8], [0, 1, 2, 3]),       # decreasing history offsets
    ([0, 5, 5, 8], [0, 1, 2, 3]),       # request 1 has a target but no history
    ([1, 5, 6, 8], [0, 1, 2, 3]),       # offsets[0] != 0
    ([0, 5, 6, 8], [0, 2, 1, 3]),       # decreasing target offsets
])
def test_invalid_host_offsets_rejected(hoff, toff):
    b, keep = fake_batch(hoff, toff)
    assert stca.stca_workspace_size(dims(), b) == 0
    assert call_forward(dims(), b) == stca.STCA_ERR_INVALID_ARG


def test_empty_target_segments_are_legal():
    b, keep = fake_batch([0, 5, 5, 8], [0, 1, 1, 3])
    assert stca.stca_workspace_size(dims(), b) > 0


def test_workspace_too_small_and_bad_pointers():
    b, keep = fake_batch([0, 40, 100], [0, 3, 9])
    need = stca.stca_workspace_size(dims(), b)
    assert need > 0
    assert call_forward(dims(), b, ws_bytes=need - 1) == stca.STCA_ERR_WORKSPACE
    assert call_forward(dims(), b, hist=0x200004) == stca.STCA_ERR_INVALID_ARG  # misaligned
    assert call_forward(dims(), b, tgt=0) == stca.STCA_ERR_INVALID_ARG
    assert call_forward(dims(), b, out=0) == stca.STCA_ERR_INVALID_ARG
    assert call_forward(dims(), b, ws=0) == stca.STCA_ERR_INVALID_ARG
    assert call_forward(dims(n_heads=7), b) == stca.STCA_ERR_INVALID_ARG
    assert call_forward(dims(n_heads=2), b) == stca.STCA_ERR_UNSUPPORTED


def test_backward_argument_checks():
    b, keep = fake_batch([0, 40, 100], [0, 3, 9])
    dw = stca.wgrads(*([0x600000] * 6))
    args = (dims(), b, 0x200000, 0x300000, fake_weights())
    st = stca.stca_backward(*args, 0, 0x800000, 0x900000, dw, 0x500000, 1 << 40, check=False)
    assert st == stca.STCA_ERR_INVALID_ARG  # dout is required when there are targets
    need = stca.stca_workspace_size(dims(), b, True)
    st = stca.stca_backward(*args, 0x700000, 0x800000, 0x900000, dw, 0x500000, need - 1, check=False)
    assert st == stca.STCA_ERR_WORKSPACE
    bad_dw = stca.wgrads(0x600000, 0, 0x600000, 0x600000, 0x600000, 0x600000)
    st = stca.stca_backward(*args, 0x700000, 0x800000, 0x900000, bad_dw, 0x500000, need, check=False)
    assert st == stca.STCA_ERR_INVALID_ARG
    st = stca.stca_backward(*args, 0x700008, 0x800000, 0x900000, dw, 0x500000, need, check=False)
    assert st == stca.STCA_ERR_INVALID_ARG  # misaligned


def test_saved_layout_is_disjoint_and_sized():
    b, keep = fake_batch([0, 40, 100], [0, 3, 9])
    lay = stca.stca_saved_layout(dims(), b)
    nt, d, n, h = 9, 256, 4, 8
    assert lay.a >= lay.s + 4 * n * nt * d
    assert lay.u >= lay.a + 4 * n * nt * d
    assert lay.lse >= lay.u + 4 * n * nt * d
    assert lay.total >= lay.lse + 4 * n * nt * h
    assert lay.total == stca.stca_saved_size(dims(), b)


def test_materialized_kv_needs_workspace_for_every_layer():
    b, keep = fake_batch([0, 40, 100], [0, 3, 9])
    fused = stca.stca_workspace_size(dims(), b)
    mat = stca.stca_workspace_size(dims(kv="materialize"), b)
    assert mat >= fused + 2 * 4 * 128 * 2 * 256  # 100 rows -> 4 blocks of 32, K and V, 4 layers, fp16


def test_reordered_form_selection():
    """Requests with at most 32 / h targets (host offsets known) run the
    reordered attention: its launch sequence is 3 + 4 n launches against the
    standard form's 3 + 3 n; a batch with both kinds of request runs each in
    its own form."""
    n = GOOD_DIMS["n_layers"]
    small, keep1 = fake_batch([0, 40, 100, 101], [0, 4, 5, 8])   # m = 4, 1, 3 <= 32 / 8
    wide, keep2 = fake_batch([0, 40, 100], [0, 5, 9])            # m = 5
    assert stca.stca_forward_launch_count(dims(), small) == 3 + 4 * n
    # m = 5 and m = 4: each request in its own form (two schedules; per layer
    # U, two fused launches, the reordered attention and merge, the update)
    assert stca.stca_forward_launch_count(dims(), wide) == 4 + 6 * n
    big, keep5 = fake_batch([0, 40, 100], [0, 5, 14])
    assert stca.stca_forward_launch_count(dims(), big) == 3 + 3 * n
    assert stca.stca_forward_launch_count(dims(d_model=128, n_heads=4), wide) == 3 + 4 * n  # 32 / 4 = 8
    nohost = stca.batch(3, 101, 8, 0x10000, 0x20000, None, None)
    assert stca.stca_forward_launch_count(dims(), nohost) == 3 + 3 * n
    assert stca.stca_forward_launch_count(dims(attn="standard"), small) == 3 + 3 * n
    assert stca.stca_forward_launch_count(dims(attn="reordered"), small) == 3 + 4 * n
    # asked for, the reordered form takes up to 256 / h targets per request
    # (wide units of up to 256 rows (t, j)); more is unsupported
    assert stca.stca_forward_launch_count(dims(attn="reordered"), wide) == 3 + 4 * n
    top, keep3 = fake_batch([0, 40, 100], [0, 32, 40])
    over, keep4 = fake_batch([0, 40, 100], [0, 33, 40])
    assert stca.stca_forward_launch_count(dims(attn="reordered"), top) == 3 + 4 * n
    assert stca.stca_forward_launch_count(dims(attn="reordered"), over) == -1
    assert call_forward(dims(attn="reordered"), over) == stca.STCA_ERR_UNSUPPORTED
    assert stca.stca_workspace_size(dims(attn="reordered"), over) == 0
    assert stca.stca_forward_launch_count(dims(attn="reordered", d_model=64, n_heads=2), over) == 3 + 4 * n


def test_wide_groups_selection():
    """A request with more than 64 targets switches the bf16 path to K/V
    written once (4 + 2 n launches); kv_form STCA_KV_FUSED keeps the fused form."""
    n = GOOD_DIMS["n_layers"]
    many, keep = fake_batch([0, 400, 500], [0, 65, 70])
    few, keep2 = fake_batch([0, 400, 500], [0, 64, 70])
    assert stca.stca_forward_launch_count(dims(), many) == 4 + 2 * n
    assert stca.stca_forward_launch_count(dims(), few) == 3 + 3 * n
    assert stca.stca_forward_launch_count(dims(kv="fused"), many) == 3 + 3 * n
    assert stca.stca_forward_launch_count(dims(kv="materialize"), few) == 4 + 2 * n


def test_fused_backward_selection():
    """The bf16 backward keeps K | V inside its attention kernels (7 + 5 n
    phases, no K|V product per layer) when the host offsets show at most 32
    targets per request, and runs in the reordered form (6 + 6 n) when d is
    128 or 256, every request has at most 128 / n_heads targets and the
    histories are balanced over the CUs; more
    targets, no host offsets, fp32 storage, an FFN
    width that is not a multiple of d or bwd_form STCA_BWD_GENERIC take the K|V product and the exact fp32 attention
    (6 + 7 n, 4 + 9 n for fp32), and only that form sizes the fp32 K|V
    buffer of every layer into the workspace."""
    n = GOOD_DIMS["n_layers"]
    small, keep1 = fake_batch([0, 40, 100, 101], [0, 32, 33, 40])   # m = 32, 1, 7
    big, keep2 = fake_batch([0, 40, 100], [0, 33, 40])               # m = 33
    nohost = stca.batch(3, 101, 40, 0x10000, 0x20000, None, None)
    assert stca.stca_backward_launch_count(dims(), small) == 7 + 5 * n
    # d = 128: 32 targets x 4 heads fit the reordered form's 128 pairs; the
    # automatic rule takes it for histories balanced over the CUs (here at
    # most two 32-row blocks per request), the fused form for the ragged batch
    even, keep4 = fake_batch([0, 64, 128, 192], [0, 32, 33, 40])
    assert stca.stca_backward_launch_count(dims(d_model=128, n_heads=4), even) == 6 + 6 * n
    assert stca.stca_backward_launch_count(dims(d_model=128, n_heads=4), small) == 7 + 5 * n
    assert stca.stca_backward_launch_count(dims(d_model=128, n_heads=4, bwd="reordered"), small) == 6 + 6 * n
    assert stca.stca_backward_launch_count(dims(d_model=128, n_heads=4, bwd="fused"), even) == 7 + 5 * n
    assert stca.stca_backward_launch_count(dims(d_model=64, n_heads=2), small) == 7 + 5 * n
    assert stca.stca_backward_launch_count(dims(), big) == 6 + 7 * n
    assert stca.stca_backward_launch_count(dims(), nohost) == 6 + 7 * n
    assert stca.stca_backward_launch_count(dims(d_model=256, n_heads=4), small) == 6 + 7 * n  # d_h = 64
    assert stca.stca_backward_launch_count(dims(dtype=stca.STCA_F32), small) == 4 + 9 * n
    assert stca.stca_backward_launch_count(dims(ffn_hidden=3 * 128), small) == 6 + 7 * n  # F not a multiple of d
    # the training record exists exactly for the batches the fused form takes
    assert stca.stca_train_record_size(dims(), small) > 0
    assert stca.stca_train_record_size(dims(), big) == 0
    assert stca.stca_train_record_size(dims(), nohost) == 0
    assert stca.stca_train_record_size(dims(dtype=stca.STCA_F32), small) == 0
    long, keep3 = fake_batch([0, 60000, 100000], [0, 32, 40])
    d, F = GOOD_DIMS["d_model"], GOOD_DIMS["ffn_hidden"]
    fused = stca.stca_workspace_size(dims(), long, True)
    assert stca.stca_backward_launch_count(dims(bwd="generic"), small) == 6 + 7 * n
    assert stca.stca_backward_launch_count(dims(bwd="fused"), small) == 7 + 5 * n
    assert stca.stca_backward_launch_count(dims(bwd="fused"), big) == -1  # unsupported there
    assert stca.stca_backward_launch_count(dims(bwd="reordered"), small) == -1  # 32 targets x 8 heads > 128
    assert stca.stca_workspace_size(dims(bwd="fused"), big, True) == 0
    generic = stca.stca_workspace_size(dims(bwd="generic"), long, True)
    # the fp32 K|V of every layer and the bf16 transposed copies of X and of
    # every layer's dK|dV, less the fused form's packed weights (W_K, W_V,
    # W_O, W_Q, W_O^T; W_1, W_2, W_1^T, W_2^T) and bf16 copies of a, u, h, s
    rows = 100000
    assert generic - fused >= (4 * n * rows * 2 * d + 2 * rows * d + 2 * n * 2 * d * rows
                               - 2 * n * (5 * d * d + 4 * d * F) - 2 * n * 40 * (3 * d + F))


def test_form_fields_are_validated():
    """Out-of-range execution forms and negative chunk lengths are invalid
    arguments, reported by every call before anything is launched."""
    b, keep = fake_batch([0, 40, 100], [0, 3, 9])
    for bad in (dict(kv_form=3), dict(attn_form=-1), dict(bwd_form=7), dict(chunk_blocks=-2)):
        d = dims()
        for k, v in bad.items():
            setattr(d, k, v)
        assert stca.stca_path(d) == stca.STCA_ERR_INVALID_ARG, bad
        assert stca.stca_workspace_size(d, b) == 0, bad
        assert call_forward(d, b) == stca.STCA_ERR_INVALID_ARG, bad


def test_workspace_depends_only_on_arguments(monkeypatch):
    """Sizes and launch plans follow the arguments alone: the same (dims,
    batch) gives the same size whatever the process environment holds, and a
    forced chunk length changes the plan only through dims."""
    b, keep = fake_batch([0, 4000, 10000], [0, 3, 9])
    sizes = [stca.stca_workspace_size(dims(), b), stca.stca_workspace_size(dims(), b, True)]
    for k in ("STCA_KV", "STCA_ATTN", "STCA_BWD", "STCA_CHUNK_BLOCKS"):
        monkeypatch.setenv(k, "1")
    assert [stca.stca_workspace_size(dims(), b), stca.stca_workspace_size(dims(), b, True)] == sizes
    # chunks longer than any history: one unit per request instead of the
    # default's chunks of 8 blocks
    assert stca.stca_workspace_size(dims(chunk_blocks=1000), b) < sizes[0]


def _chunk_for(n_hist, per_cu, n_cu=256):
    """The library's chunk length for `per_cu` units per CU (blocks of 32 rows, at least 8)."""
    nb = -(-n_hist // 32)
    return max(8, -(-nb // (per_cu * n_cu)))


def test_chunk_rule_equal_histories_take_one_unit_per_cu():
    # 128 requests x 10240 rows, 32 targets each: two chunks of 160 blocks per
    # request give one unit per CU, which the makespan estimate prefers to
    # the finer cuts (same balance, fewer units); the workspace (its unit
    # table and chunk partials) follows the chosen chunk length
    b, keep = fake_batch(np.arange(129) * 10240, np.arange(129) * 32)
    auto = stca.stca_workspace_size(dims(), b)
    assert auto == stca.stca_workspace_size(dims(chunk_blocks=_chunk_for(10240 * 128, 1)), b)
    assert auto < stca.stca_workspace_size(dims(chunk_blocks=_chunk_for(10240 * 128, 4)), b)


def test_chunk_rule_ragged_histories_take_finer_cuts():
    # unequal histories balance better in smaller chunks: the choice is one of
    # the finer candidates, never one unit per CU
    rng = np.random.default_rng(7)
    L = [int(x) for x in rng.integers(512, 10241, size=256)]
    m = [int(x) for x in rng.integers(5, 65, size=256)]  # above the reordered form's 4 targets
    b, keep = fake_batch(np.concatenate([[0], np.cumsum(L)]), np.concatenate([[0], np.cumsum(m)]))
    auto = stca.stca_workspace_size(dims(), b)
    sizes = {p: stca.stca_workspace_size(dims(chunk_blocks=_chunk_for(sum(L), p)), b) for p in (1, 2, 4, 8)}
    assert auto in (sizes[4], sizes[8])
    assert auto != sizes[1]
