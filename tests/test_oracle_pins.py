"""Pins of the fp64 oracle to facts outside it (CPU only).

Each test checks the oracle against something the paper or mathematics fixes:
special cases with closed forms, invariances the method guarantees, the paper's
second evaluation order, a library attention routine, a hand-derived two-item
case, and (for gradients) autograd and finite differences.
"""
import math

import numpy as np
import pytest

from oracle import stca_oracle as O
from paper_2511_06077_amd import workload as W


def small_inputs(R=3, m=(2, 3, 1), L=(5, 1, 7), d=8, h=2, n=2, seed=0, f=None):
    rng = np.random.default_rng(seed)
    f = f or 4 * d
    hoff = np.concatenate([[0], np.cumsum(L)])
    toff = np.concatenate([[0], np.cumsum(m)])
    return {
        "hist": rng.standard_normal((hoff[-1], d)),
        "tgt": rng.standard_normal((toff[-1], d)),
        "hist_off": hoff, "tgt_off": toff, "n_heads": h,
        "wq": rng.standard_normal((n, d, d)) / math.sqrt(d),
        "wk": rng.standard_normal((n, d, d)) / math.sqrt(d),
        "wv": rng.standard_normal((n, d, d)) / math.sqrt(d),
        "wo": rng.standard_normal((n, d, d)) / math.sqrt(d),
        "w1": rng.standard_normal((n, d, f)) / math.sqrt(d),
        "w2": rng.standard_normal((n, f, d)) / math.sqrt(f),
    }


def with_(inp, **kw):
    out = dict(inp)
    out.update(kw)
    return out


# ---------------------------------------------------------------- P1: L = 1
def test_single_history_item_gives_projected_v_row():
    """With one history item the softmax weight is exactly 1, so every target's
    head concatenation equals that item's V row, at every layer."""
    inp = small_inputs(R=2, m=(3, 2), L=(1, 1))
    fw = O.forward(inp)
    for r in range(2):
        x0 = inp["hist"][inp["hist_off"][r]]
        for i in range(2):
            v = x0 @ inp["wv"][i]
            t0, t1 = inp["tgt_off"][r], inp["tgt_off"][r + 1]
            np.testing.assert_allclose(fw["a"][i, t0:t1], np.broadcast_to(v, (t1 - t0, v.size)),
                                       rtol=0, atol=1e-14)
            # log-sum-exp of a single score is the score itself
            q = fw["s"][i, t0:t1] @ inp["wq"][i]
            k = x0 @ inp["wk"][i]
            dh = 4
            for j in range(2):
                J = slice(j * dh, (j + 1) * dh)
                np.testing.assert_allclose(fw["lse"][i, t0:t1, j], q[:, J] @ k[J] / math.sqrt(dh),
                                           rtol=1e-13, atol=1e-13)


# ---------------------------------------------------------- P2: zero scores
@pytest.mark.parametrize("zero", ["wq", "wk"])
def test_zero_scores_give_mean_of_v(zero):
    """All-zero scores make the softmax uniform: a = mean_l V_l."""
    inp = small_inputs()
    inp = with_(inp, **{zero: np.zeros_like(inp[zero])})
    fw = O.forward(inp)
    for r in range(3):
        Xr = inp["hist"][inp["hist_off"][r]:inp["hist_off"][r + 1]]
        t0, t1 = inp["tgt_off"][r], inp["tgt_off"][r + 1]
        L = Xr.shape[0]
        for i in range(2):
            mean_v = (Xr @ inp["wv"][i]).mean(axis=0)
            np.testing.assert_allclose(fw["a"][i, t0:t1], np.broadcast_to(mean_v, (t1 - t0, 8)),
                                       rtol=0, atol=1e-14)
            np.testing.assert_allclose(fw["lse"][i, t0:t1], math.log(L), rtol=0, atol=1e-14)


# -------------------------------------------------------- P3: RLB invariants
def test_target_permutation_within_request():
    inp = small_inputs(R=2, m=(5, 4), L=(9, 6))
    fw = O.forward(inp)
    perm = np.concatenate([np.random.default_rng(3).permutation(5), 5 + np.arange(4)[::-1]])
    fp = O.forward(with_(inp, tgt=inp["tgt"][perm]))
    np.testing.assert_allclose(fp["out"], fw["out"][perm], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(fp["a"], fw["a"][:, perm], rtol=1e-13, atol=1e-13)


def test_rlb_grouping_equals_one_target_per_request():
    """RLB only regroups samples (Sec. 3.2): each target's result equals the
    result of a batch in which it is alone with its own copy of the history."""
    wl = W.Workload("t", 3, 16, 2, 2, "f32", seed=9, hist_range=(1, 12), tgt_range=(0, 4))
    b = W.make_batch(wl)
    nb = W.replicate_per_target(b)
    fw = O.forward(b.f64())
    fn = O.forward(nb.f64())
    np.testing.assert_allclose(fn["out"], fw["out"], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(fn["a"], fw["a"], rtol=1e-13, atol=1e-13)


def test_requests_are_independent():
    inp = small_inputs()
    fw = O.forward(inp)
    for r in range(3):
        h0, h1 = inp["hist_off"][r], inp["hist_off"][r + 1]
        t0, t1 = inp["tgt_off"][r], inp["tgt_off"][r + 1]
        one = with_(inp, hist=inp["hist"][h0:h1], tgt=inp["tgt"][t0:t1],
                    hist_off=np.array([0, h1 - h0]), tgt_off=np.array([0, t1 - t0]))
        np.testing.assert_allclose(O.forward(one)["out"], fw["out"][t0:t1], rtol=1e-13, atol=1e-13)


def test_empty_target_segment_and_empty_history_rules():
    inp = small_inputs(R=3, m=(2, 0, 1), L=(4, 0, 3))
    fw = O.forward(inp)
    assert fw["out"].shape == (3, 8)
    bad = small_inputs(R=2, m=(1, 1), L=(3, 0))
    with pytest.raises(ValueError):
        O.forward(bad)


# ---------------------------------------------------- P4: history symmetries
def test_history_permutation_invariance():
    inp = small_inputs(R=1, m=(4,), L=(11,))
    perm = np.random.default_rng(5).permutation(11)
    a = O.forward(inp)
    b = O.forward(with_(inp, hist=inp["hist"][perm]))
    np.testing.assert_allclose(b["out"], a["out"], rtol=1e-12, atol=1e-12)


def test_history_duplication_invariance():
    inp = small_inputs(R=1, m=(4,), L=(11,))
    a = O.forward(inp)
    b = O.forward(with_(inp, hist=np.concatenate([inp["hist"], inp["hist"]]),
                        hist_off=np.array([0, 22])))
    np.testing.assert_allclose(b["out"], a["out"], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(b["lse"], a["lse"] + math.log(2), rtol=1e-12, atol=1e-12)


# ------------------------------------- P5: the paper's reordered evaluation
def test_reordered_single_query_form_matches():
    """Eq. attn-optimized: softmax(((q W_Q) W_K^T) X^T / sqrt(d_h)) X W_V, per
    head, without forming K or V, equals the standard form."""
    inp = small_inputs(R=2, m=(3, 2), L=(13, 6), d=12, h=3)
    fw = O.forward(inp)
    dh = 4
    for r in range(2):
        X = inp["hist"][inp["hist_off"][r]:inp["hist_off"][r + 1]]
        t0, t1 = inp["tgt_off"][r], inp["tgt_off"][r + 1]
        for i in range(2):
            s = fw["s"][i, t0:t1]
            for j in range(3):
                J = slice(j * dh, (j + 1) * dh)
                Wq, Wk, Wv = (inp[k][i][:, J] for k in ("wq", "wk", "wv"))
                u = (s @ Wq) @ Wk.T
                e = u @ X.T / math.sqrt(dh)
                alpha = np.exp(e - e.max(1, keepdims=True))
                alpha /= alpha.sum(1, keepdims=True)
                o = (alpha @ X) @ Wv
                np.testing.assert_allclose(o, fw["a"][i, t0:t1, J], rtol=1e-12, atol=1e-12)


# ------------------------------------------------ P6: library attention call
def test_matches_torch_scaled_dot_product_attention():
    torch = pytest.importorskip("torch")
    inp = small_inputs(R=2, m=(4, 3), L=(17, 9), d=64, h=2)
    fw = O.forward(inp)
    dh = 32
    for r in range(2):
        X = torch.from_numpy(inp["hist"][inp["hist_off"][r]:inp["hist_off"][r + 1]])
        t0, t1 = inp["tgt_off"][r], inp["tgt_off"][r + 1]
        for i in range(2):
            q = torch.from_numpy(fw["s"][i, t0:t1]) @ torch.from_numpy(inp["wq"][i])
            K = X @ torch.from_numpy(inp["wk"][i])
            V = X @ torch.from_numpy(inp["wv"][i])
            qh = q.view(-1, 2, dh).transpose(0, 1).contiguous()
            Kh = K.view(-1, 2, dh).transpose(0, 1).contiguous()
            Vh = V.view(-1, 2, dh).transpose(0, 1).contiguous()
            o = torch.nn.functional.scaled_dot_product_attention(qh, Kh, Vh)
            o = o.transpose(0, 1).reshape(t1 - t0, 64).numpy()
            np.testing.assert_allclose(o, fw["a"][i, t0:t1], rtol=1e-12, atol=1e-12)


# --------------------------------------------------- P7: two items by hand
def test_two_item_attention_by_hand():
    """L = 2, d = 2, h = 1: alpha = (sigma(e1 - e2), sigma(e2 - e1))."""
    x1, x2 = np.array([0.3, -1.2]), np.array([1.1, 0.4])
    t = np.array([0.7, 0.2])
    Wq = np.array([[1.0, 0.5], [-0.3, 2.0]])
    Wk = np.array([[0.2, -1.0], [0.8, 0.1]])
    Wv = np.array([[1.5, 0.0], [-0.5, 1.0]])
    I, Z = np.eye(2), np.zeros((2, 8))
    inp = {"hist": np.stack([x1, x2]), "tgt": t[None], "hist_off": np.array([0, 2]),
           "tgt_off": np.array([0, 1]), "n_heads": 1, "wq": Wq[None], "wk": Wk[None],
           "wv": Wv[None], "wo": I[None], "w1": Z[None], "w2": Z.T[None]}
    q = [t[0] * Wq[0, c] + t[1] * Wq[1, c] for c in range(2)]
    k1 = [x1[0] * Wk[0, c] + x1[1] * Wk[1, c] for c in range(2)]
    k2 = [x2[0] * Wk[0, c] + x2[1] * Wk[1, c] for c in range(2)]
    v1 = [x1[0] * Wv[0, c] + x1[1] * Wv[1, c] for c in range(2)]
    v2 = [x2[0] * Wv[0, c] + x2[1] * Wv[1, c] for c in range(2)]
    e1 = (q[0] * k1[0] + q[1] * k1[1]) / math.sqrt(2)
    e2 = (q[0] * k2[0] + q[1] * k2[1]) / math.sqrt(2)
    sig = lambda z: 1.0 / (1.0 + math.exp(-z))
    a = [sig(e1 - e2) * v1[c] + sig(e2 - e1) * v2[c] for c in range(2)]
    fw = O.forward(inp)
    np.testing.assert_allclose(fw["a"][0, 0], a, rtol=1e-14, atol=1e-15)
    # W_O = I and a zero FFN leave Y = x_t + a
    np.testing.assert_allclose(fw["out"][0], t + np.array(a), rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(fw["lse"][0, 0, 0], max(e1, e2) + math.log1p(math.exp(-abs(e1 - e2))),
                               rtol=1e-14)


def test_layer_update_special_case():
    """With L = 1 the attention output is known exactly (x_0 W_V), so one layer
    reduces to u = x_t + (x_0 W_V) W_O and Y = u + ReLU(u W_1) W_2; checked with
    a non-symmetric W_O and a W_2 that is not W_1^T."""
    inp = small_inputs(R=1, m=(3,), L=(1,), n=1, d=6, h=2)
    fw = O.forward(inp)
    x0, T = inp["hist"][0], inp["tgt"]
    u = T + (x0 @ inp["wv"][0]) @ inp["wo"][0]
    y = u + np.maximum(u @ inp["w1"][0], 0) @ inp["w2"][0]
    np.testing.assert_allclose(fw["out"], y, rtol=1e-13, atol=1e-13)


# ------------------------------------------------ gradients: autograd and FD
def torch_forward(torch, p, hoff, toff, h):
    """An independent float64 torch evaluation of the same definition, for autograd."""
    outs = []
    d = p["hist"].shape[1]
    dh = d // h
    for r in range(len(hoff) - 1):
        t0, t1 = int(toff[r]), int(toff[r + 1])
        if t1 == t0:
            continue
        X = p["hist"][int(hoff[r]):int(hoff[r + 1])]
        s = p["tgt"][t0:t1]
        for i in range(p["wq"].shape[0]):
            q = (s @ p["wq"][i]).view(t1 - t0, h, dh).transpose(0, 1)
            K = (X @ p["wk"][i]).view(-1, h, dh).transpose(0, 1)
            V = (X @ p["wv"][i]).view(-1, h, dh).transpose(0, 1)
            att = torch.softmax(q @ K.transpose(1, 2) / math.sqrt(dh), dim=-1)
            a = (att @ V).transpose(0, 1).reshape(t1 - t0, d)
            u = s + a @ p["wo"][i]
            s = u + torch.relu(u @ p["w1"][i]) @ p["w2"][i]
        outs.append(s)
    return torch.cat(outs)


def test_gradients_match_torch_autograd():
    torch = pytest.importorskip("torch")
    inp = small_inputs(R=3, m=(2, 3, 1), L=(5, 1, 7), d=8, h=2, n=2)
    G = np.random.default_rng(11).standard_normal(inp["tgt"].shape)
    g = O.backward(inp, G)
    names = ["hist", "tgt"] + list(O.LAYER_WEIGHTS)
    p = {k: torch.tensor(inp[k], requires_grad=True) for k in names}
    Y = torch_forward(torch, p, inp["hist_off"], inp["tgt_off"], 2)
    np.testing.assert_allclose(Y.detach().numpy(), O.forward(inp)["out"], rtol=1e-12, atol=1e-12)
    (Y * torch.from_numpy(G)).sum().backward()
    for k in names:
        np.testing.assert_allclose(g["d" + k], p[k].grad.numpy(), rtol=1e-10, atol=1e-11, err_msg=k)


def test_gradients_central_finite_differences():
    inp = small_inputs(R=2, m=(2, 3), L=(6, 4), d=8, h=2, n=2, seed=4)
    G = np.random.default_rng(12).standard_normal(inp["tgt"].shape)
    g = O.backward(inp, G)
    rng = np.random.default_rng(13)
    eps = 1e-6
    for k in ["hist", "tgt"] + list(O.LAYER_WEIGHTS):
        flat = inp[k].reshape(-1)
        for idx in rng.choice(flat.size, size=min(40, flat.size), replace=False):
            plus, minus = inp[k].copy(), inp[k].copy()
            plus.reshape(-1)[idx] += eps
            minus.reshape(-1)[idx] -= eps
            fp = O.forward(with_(inp, **{k: plus}), keep=True)
            fm = O.forward(with_(inp, **{k: minus}), keep=True)
            # skip coordinates whose step flips a ReLU
            if np.any(np.sign(fp["pre"]) != np.sign(fm["pre"])):
                continue
            num = ((fp["out"] - fm["out"]) * G).sum() / (2 * eps)
            ana = g["d" + k].reshape(-1)[idx]
            assert abs(num - ana) <= 1e-6 * max(1.0, abs(ana)), (k, idx, num, ana)


C1 = "tiny_f32_R4_m4_L256_d64"  # R = 4, m = 4, L = 256, d = 64, h = 2, n = 2, F = 4 d


def _c1_inputs():
    b = W.make_batch(W.WORKLOADS[C1], with_grad=True)
    inp = b.f64()
    return inp, inp.pop("grad_out")


def test_gradients_central_finite_differences_c1_shape():
    """Central differences (eps = 1e-6, fp64) of f = sum <G, Y> at the tiny
    workload's shape (4 requests x 4 targets, L = 256, d = 64, 2 heads,
    2 layers, FFN width 4 d) on 200 random coordinates of every input and
    weight tensor.  A coordinate is skipped (and replaced by another) when
    the step moves any FFN pre-activation across zero, i.e. when the
    function is not differentiable inside [x - eps, x + eps].  Per tensor,
    max |fd - g| over the checked coordinates must stay within 1e-6 of the
    tensor's largest gradient entry (rounding of f alone puts central
    differences near 1e-8 of it here)."""
    inp, G = _c1_inputs()
    g = O.backward(inp, G)
    base = O.forward(inp, keep=True)
    rng = np.random.default_rng(2024)
    eps = 1e-6
    for k in ["hist", "tgt"] + list(O.LAYER_WEIGHTS):
        flat = inp[k].reshape(-1)
        order = rng.permutation(flat.size)
        worst, checked, skipped = 0.0, 0, 0
        scale = float(np.abs(g["d" + k]).max())
        for idx in order:
            plus, minus = inp[k].copy(), inp[k].copy()
            plus.reshape(-1)[idx] += eps
            minus.reshape(-1)[idx] -= eps
            fp = O.forward(with_(inp, **{k: plus}), keep=True)
            fm = O.forward(with_(inp, **{k: minus}), keep=True)
            sb = np.sign(base["pre"])
            if np.any(np.sign(fp["pre"]) != sb) or np.any(np.sign(fm["pre"]) != sb):
                skipped += 1
                continue
            num = ((fp["out"] - fm["out"]) * G).sum() / (2 * eps)
            worst = max(worst, abs(num - g["d" + k].reshape(-1)[idx]))
            checked += 1
            if checked == 200:
                break
        print(f"[fd c1] {k}: {checked} coordinates ({skipped} skipped at a ReLU kink), "
              f"max |fd - g| / max |g| = {worst / scale:.1e}")
        assert checked == 200, (k, checked)
        assert worst <= 1e-6 * scale, (k, worst / scale)


def _autograd_check(inp, G, h):
    torch = pytest.importorskip("torch")
    g = O.backward(inp, G)
    names = ["hist", "tgt"] + list(O.LAYER_WEIGHTS)
    p = {k: torch.tensor(inp[k], requires_grad=True) for k in names}
    Y = torch_forward(torch, p, inp["hist_off"], inp["tgt_off"], h)
    ref_y = O.forward(inp, keep=False)["out"]
    assert np.abs(Y.detach().numpy() - ref_y).max() <= 1e-12 * np.abs(ref_y).max()
    (Y * torch.from_numpy(G)).sum().backward()
    for k in names:
        ref = p[k].grad.numpy()
        err = np.abs(g["d" + k] - ref).max() / np.abs(ref).max()
        print(f"[autograd] {k}: {err:.1e}")
        assert err <= 1e-11, (k, err)


def test_gradients_match_torch_autograd_c1_shape():
    """Every gradient of the hand-derived reverse mode against torch float64
    autograd through an independent forward, at the tiny workload's shape."""
    inp, G = _c1_inputs()
    _autograd_check(inp, G, 2)


def test_gradients_match_torch_autograd_c2_shape_short_history():
    """The same at the uniform bf16 workload's shape (64 requests x 16
    targets, d = 128, 4 heads, 2 layers) with the history cut from 1024 to
    64 rows so that the fp64 evaluation stays short; inputs are the bf16
    workload's exact values."""
    b = W.make_custom_batch("c2_short", [64] * 64, [16] * 64, d_model=128, n_heads=4, n_layers=2, dtype="bf16",
                            seed=2, with_grad=True)
    inp = b.f64()
    G = inp.pop("grad_out")
    _autograd_check(inp, G, 4)


# --------------------------- planted mistakes must be caught by some pin
def _mutant_cross_attention(kind):
    orig = O.cross_attention

    def f(q, K, V, n_heads):
        if kind == "scale_sqrt_d":
            return orig(q * math.sqrt(n_heads), K, V, n_heads)
        if kind == "v_uses_k":
            return orig(q, K, K, n_heads)
        if kind == "head_order":
            a, al, lse = orig(q, K, V, n_heads)
            dh = q.shape[1] // n_heads
            a = np.concatenate([a[:, j * dh:(j + 1) * dh] for j in reversed(range(n_heads))], axis=1)
            return a, al, lse
        if kind == "no_normalise":
            a, al, lse = orig(q, K, V, n_heads)
            return a * np.exp(lse.max()), al, lse
        raise AssertionError(kind)
    return f


@pytest.mark.parametrize("kind", ["scale_sqrt_d", "v_uses_k", "head_order", "no_normalise"])
def test_planted_attention_mistakes_are_caught(kind, monkeypatch):
    monkeypatch.setattr(O, "cross_attention", _mutant_cross_attention(kind))
    pins = [test_single_history_item_gives_projected_v_row, test_reordered_single_query_form_matches,
            test_matches_torch_scaled_dot_product_attention, test_two_item_attention_by_hand]
    caught = 0
    for pin in pins:
        try:
            pin()
        except AssertionError:
            caught += 1
    assert caught >= 1, kind


def test_planted_update_mistake_is_caught(monkeypatch):
    """Using W_O^T in place of W_O (square, so shapes do not catch it)."""
    orig = O.forward

    def mutant(inp, keep=True):
        inp2 = dict(inp)
        inp2["wo"] = np.ascontiguousarray(np.transpose(inp["wo"], (0, 2, 1)))
        return orig(inp2, keep)
    monkeypatch.setattr(O, "forward", mutant)
    with pytest.raises(AssertionError):
        test_layer_update_special_case()
