"""Stochastic-length training batches (Sec. 3.3; App. "Extrapolation
details"): the library's host sampler, allocator and packer, checked against
the Beta distribution (scipy), the expectation constraint, and the
definitions of the budget cap and the temporal suffix.  Runs without a GPU."""
import numpy as np
import pytest
from scipy import stats

from paper_2511_06077_amd import sl, stca
from paper_2511_06077_amd import workload as W

CASES = [(0.02, 8, 2048, 10240), (0.5, 0, 1000, 4000), (2.0, 64, 5000, 10240), (0.02, 8, 500, 2048)]


@pytest.mark.parametrize("alpha,l_min,l_avg,l_max", CASES)
def test_beta_meets_the_expectation_constraint(alpha, l_min, l_avg, l_max):
    """The Beta mean alpha / (alpha + beta) mapped by Eq. beta-scale gives l_avg."""
    b = stca.sl_beta(alpha, l_min, l_avg, l_max)
    assert b > 0
    assert np.isclose(l_min + (l_max - l_min) * alpha / (alpha + b), l_avg, rtol=1e-12)


def test_beta_rejects_bad_lengths():
    assert np.isnan(stca.sl_beta(0.02, 100, 50, 1000))
    assert np.isnan(stca.sl_beta(0.0, 8, 50, 1000))
    assert np.isnan(stca.sl_beta(0.02, 8, 1000, 1000))


@pytest.mark.parametrize("alpha,l_min,l_avg,l_max", CASES)
def test_sampled_ratio_follows_the_beta_distribution(alpha, l_min, l_avg, l_max):
    b = stca.sl_beta(alpha, l_min, l_avg, l_max)
    raw, _ = stca.sl_sample(7, 40000, alpha, l_min, l_avg, l_max)
    s = (raw - l_min) / (l_max - l_min)
    assert ((s >= 0) & (s <= 1)).all()
    # Empirical CDF against the Beta CDF on a grid down to 1e-12 (below ~1e-16
    # the ratio is lost in L_raw's float64 rounding, far below one length
    # step).  By the Dvoretzky-Kiefer-Wolfowitz inequality the sup distance
    # exceeds eps with probability at most 2 exp(-2 n eps^2): 1e-6 here.
    grid = np.concatenate([np.logspace(-12, -1, 45), np.linspace(0.1, 1.0, 46)])
    emp = np.searchsorted(np.sort(s), grid, side="right") / s.size
    eps = np.sqrt(np.log(2e6) / (2 * s.size))
    dev = np.abs(emp - stats.beta(alpha, b).cdf(grid)).max()
    assert dev < eps, (dev, eps)
    # the mean within 4 standard errors of l_avg
    var = alpha * b / ((alpha + b) ** 2 * (alpha + b + 1)) * (l_max - l_min) ** 2
    assert abs(raw.mean() - l_avg) < 4 * np.sqrt(var / raw.size)


def test_u_shape_and_sequence_sparsity():
    """alpha = 0.02 puts most draws at the short end and the rest near the
    maximum, with mean l_avg: sequence sparsity l_avg / l_max."""
    raw, lt = stca.sl_sample(3, 100000, 0.02, 8, 2048, 10240)
    s = (raw - 8) / (10240 - 8)
    assert (s < 0.05).mean() > 0.6 and (s > 0.95).mean() > 0.1 and ((s > 0.2) & (s < 0.8)).mean() < 0.05
    assert abs(lt.mean() / 10240 - 0.2) < 0.01


def test_lengths_are_rounded_multiples_of_eight():
    raw, lt = stca.sl_sample(5, 5000, 0.5, 0, 1000, 4000)
    assert (lt % 8 == 0).all() and lt.min() >= 8 and lt.max() <= 4000
    expect = np.clip(np.floor(raw / 8 + 0.5) * 8, 8, 4000)
    np.testing.assert_array_equal(lt, expect.astype(np.int32))


def test_streams_are_deterministic_and_per_request():
    a = stca.sl_sample(11, 100, 0.02, 8, 2048, 10240)[0]
    b = stca.sl_sample(11, 100, 0.02, 8, 2048, 10240)[0]
    c = stca.sl_sample(12, 100, 0.02, 8, 2048, 10240)[0]
    d = stca.sl_sample(11, 50, 0.02, 8, 2048, 10240)[0]
    np.testing.assert_array_equal(a, b)
    assert not np.array_equal(a, c)
    np.testing.assert_array_equal(a[:50], d)  # request r's draw does not depend on the batch size


def test_allocation_under_budget_keeps_lengths():
    l_full = np.array([100, 5000, 40, 3000])
    l_train = np.array([64, 2048, 80, 10240])
    keep = stca.sl_allocate(l_full, l_train, 10 ** 6)
    np.testing.assert_array_equal(keep, np.minimum(l_full, l_train))


def test_allocation_caps_the_longest_to_fit_the_budget():
    rng = np.random.default_rng(0)
    l_full = rng.integers(1, 10241, 64)
    l_train = (rng.integers(1, 1281, 64) * 8).astype(np.int64)
    base = np.minimum(l_full, l_train)
    budget = int(base.sum() * 0.6)
    keep = stca.sl_allocate(l_full, l_train, budget)
    assert keep.sum() <= budget
    cap = keep.max()
    assert cap % 8 == 0
    np.testing.assert_array_equal(keep, np.minimum(base, cap))   # only the longest are cut, to one cap
    assert np.minimum(base, cap + 8).sum() > budget               # the cap is the largest that fits


def test_pack_keeps_the_temporal_suffix():
    full_off = np.array([0, 10, 10, 25, 26], dtype=np.int32)
    keep = np.array([4, 0, 15, 1], dtype=np.int32)
    hoff, src = stca.sl_pack(full_off, keep)
    np.testing.assert_array_equal(hoff, [0, 4, 4, 19, 20])
    np.testing.assert_array_equal(src, np.concatenate([np.arange(6, 10), np.arange(10, 25), [25]]))
    with pytest.raises(stca.StcaError):
        stca.sl_pack(full_off, np.array([11, 0, 0, 0], dtype=np.int32))


def test_sl_batch_packs_suffix_rows_of_the_full_batch():
    full = W.make_custom_batch("slfull", [512, 300, 700, 64], [3, 0, 5, 2], d_model=64, n_heads=2, n_layers=1,
                               dtype="bf16", seed=41)
    b, info = sl.sl_batch(full, 9, alpha=0.5, l_min=8, l_avg=128, l_max=512)
    assert b.hist_off[-1] == b.hist.shape[0] == info["kept_tokens"] <= info["budget"] == 4 * 128
    for r in range(4):
        k = int(b.hist_len[r])
        f1 = int(full.hist_off[r + 1])
        np.testing.assert_array_equal(b.hist[b.hist_off[r]:b.hist_off[r + 1]], full.hist[f1 - k:f1])
    np.testing.assert_array_equal(b.tgt, full.tgt)
    np.testing.assert_array_equal(b.tgt_off, full.tgt_off)
