"""Pins that tie the fp64 oracle to the paper and to mathematics, not to itself.

Each test checks an oracle function against something independent of its
code: a hand-derived value (tests/golden, with its derivation), torch autograd
in float64 on the CPU, central finite differences, a closed-form identity, or
brute force. The identity-layer toy is the definition of the pseudogradient
(Sec. 2.1, eq. decomp): with every layer after the target acting as the
identity, the true gradient of the mean cross-entropy equals the oracle's
pseudogradient.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle as O

GOLD = os.path.join(os.path.dirname(__file__), "golden")



def toy(seed=0, T=4, d=6, V=16, d_ff=10, L=2):
    r = np.random.default_rng(seed)
    return dict(
        x=r.standard_normal((T, d)),
        gamma=1.0 + 0.1 * r.standard_normal(d),
        W_U=0.5 * r.standard_normal((V, d)),
        y=r.integers(0, V, T).astype(np.int32),
        a=[r.standard_normal((T, d_ff)) for _ in range(L)],
        W=[0.3 * r.standard_normal((d, d_ff)) for _ in range(L)],
    )


def torch_rmsnorm(x, gamma, eps):
    rho = torch.sqrt((x * x).mean(dim=1, keepdim=True) + eps)
    return gamma * x / rho


# ------------------------------------------------------------ golden (hand)
def test_golden_rmsnorm_vjp_hand():
    data = json.load(open(os.path.join(GOLD, "rmsnorm_vjp_hand.json")))
    for c in data["cases"]:
        got = O.rmsnorm_vjp(np.array([c["g"]]), np.array([c["x"]]), np.array(c["gamma"]),
                            eps=c["eps"], min_rms=c["min_rms"])[0]
        np.testing.assert_allclose(got, c["g_tilde"], rtol=0, atol=1e-14)


def test_golden_output_error_hand():
    data = json.load(open(os.path.join(GOLD, "output_error_hand.json")))
    for c in data["cases"]:
        x = np.array([c["x"]])
        W = np.array(c["W_U"])
        out = O.output_error(x, np.ones(2), W, np.array([c["target"]]), eps=0.0, min_rms=0.0)
        np.testing.assert_allclose(out["g_pre"][0], c["g_pre"], atol=1e-14)
        assert abs(out["lse"][0] - c["lse"]) < 1e-14
        assert abs(out["loss"][0] - c["loss"]) < 1e-14
        assert int(out["argmax"][0]) == c["argmax"]
        e = O.error_rows(x, np.ones(2), W, np.array([c["target"]]), eps=0.0)[0]
        np.testing.assert_allclose(e, c["e"], atol=1e-15)


# ------------------------------------------------------------ output error
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_g_is_autograd_gradient_of_ce_wrt_unembedding_input(seed):
    """eq. gproj: g is the exact gradient of the CE loss w.r.t. the unembedding input."""
    t = toy(seed)
    rho, u = O.rmsnorm_forward(t["x"], t["gamma"], 1e-6)
    U = torch.tensor(u, requires_grad=True)
    W = torch.tensor(t["W_U"])
    loss = torch.nn.functional.cross_entropy(U @ W.T, torch.tensor(t["y"]).long(), reduction="sum")
    (gu,) = torch.autograd.grad(loss, U)
    out = O.output_error(t["x"], t["gamma"], t["W_U"], t["y"], eps=1e-6, min_rms=0.5, vocab_chunk=5)
    np.testing.assert_allclose(out["g_pre"], gu.numpy(), rtol=1e-10, atol=1e-13)
    # loss and lse
    ce = torch.nn.functional.cross_entropy(U @ W.T, torch.tensor(t["y"]).long(), reduction="none")
    np.testing.assert_allclose(out["loss"], ce.detach().numpy(), rtol=1e-12)
    np.testing.assert_allclose(out["lse"], torch.logsumexp(U @ W.T, 1).detach().numpy(), rtol=1e-12)


def test_g_matches_central_finite_differences():
    t = toy(3, T=2, d=4, V=7)
    _, u = O.rmsnorm_forward(t["x"], t["gamma"], 1e-6)
    W = t["W_U"]
    y = t["y"]

    def ce(uu):
        z = uu @ W.T
        m = z.max(axis=1, keepdims=True)
        lse = (m + np.log(np.exp(z - m).sum(axis=1, keepdims=True)))[:, 0]
        return float(np.sum(lse - z[np.arange(len(y)), y]))

    h = 1e-6
    fd = np.zeros_like(u)
    for i in range(u.shape[0]):
        for k in range(u.shape[1]):
            up, dn = u.copy(), u.copy()
            up[i, k] += h
            dn[i, k] -= h
            fd[i, k] = (ce(up) - ce(dn)) / (2 * h)
    out = O.output_error(t["x"], t["gamma"], W, y)
    np.testing.assert_allclose(out["g_pre"], fd, rtol=1e-7, atol=1e-8)


def test_error_row_invariants_and_brute_force_lse():
    t = toy(4, T=5, V=33)
    e = O.error_rows(t["x"], t["gamma"], t["W_U"], t["y"])
    np.testing.assert_allclose(e.sum(axis=1), 0.0, atol=1e-14)
    for r in range(e.shape[0]):
        yv = t["y"][r]
        assert -1.0 <= e[r, yv] < 0.0
        others = np.delete(e[r], yv)
        assert np.all((others >= 0) & (others < 1))
        p_y = e[r, yv] + 1.0
        assert abs(np.abs(e[r]).sum() - 2 * (1 - p_y)) < 1e-14
    # lse by math.fsum brute force
    _, u = O.rmsnorm_forward(t["x"], t["gamma"], 1e-6)
    out = O.output_error(t["x"], t["gamma"], t["W_U"], t["y"])
    for r in range(u.shape[0]):
        z = [float(np.dot(u[r], t["W_U"][v])) for v in range(t["W_U"].shape[0])]
        lse = math.log(math.fsum(math.exp(v) for v in z))
        assert abs(out["lse"][r] - lse) < 1e-13
        assert int(out["argmax"][r]) == int(np.argmax(z))


def test_two_way_vocabulary_reduces_to_logistic():
    t = toy(5, T=3, V=2)
    _, u = O.rmsnorm_forward(t["x"], t["gamma"], 1e-6)
    e = O.error_rows(t["x"], t["gamma"], t["W_U"], t["y"])
    dz = u @ (t["W_U"][1] - t["W_U"][0])
    sig = 1.0 / (1.0 + np.exp(-dz))
    onehot1 = (t["y"] == 1).astype(float)
    np.testing.assert_allclose(e[:, 1], sig - onehot1, atol=1e-15)


def test_unembedding_common_shift_leaves_g_unchanged():
    t = toy(6, V=12)
    c = np.random.default_rng(9).standard_normal(t["W_U"].shape[1])
    g0 = O.output_error(t["x"], t["gamma"], t["W_U"], t["y"])["g_pre"]
    g1 = O.output_error(t["x"], t["gamma"], t["W_U"] + c[None, :], t["y"])["g_pre"]
    np.testing.assert_allclose(g1, g0, rtol=1e-12, atol=1e-12)
    same = np.repeat(t["W_U"][:1], t["W_U"].shape[0], axis=0)
    g2 = O.output_error(t["x"], t["gamma"], same, t["y"])["g_pre"]
    np.testing.assert_allclose(g2, 0.0, atol=1e-15)


def test_chunking_does_not_change_result():
    t = toy(7, T=3, V=50)
    a = O.output_error(t["x"], t["gamma"], t["W_U"], t["y"], vocab_chunk=50)
    b = O.output_error(t["x"], t["gamma"], t["W_U"], t["y"], vocab_chunk=7)
    for k in ("g_pre", "g_tilde", "lse", "loss"):
        np.testing.assert_allclose(a[k], b[k], rtol=1e-13, atol=1e-15)
    assert np.array_equal(a["argmax"], b["argmax"])


@pytest.mark.parametrize("eps", [1e-6, 0.3])
def test_single_logit_matches_torch_forward(eps):
    """oracle.logit (the argmax tie-margin check of the parity tests) against
    an independent float64 torch forward z = RMSNorm_gamma(x) W_U^T, on every
    (token, vocabulary entry) of a toy whose gain is far from 1 and, in the
    second case, whose eps is large enough that dropping it (or the gain, or
    taking another token's row) moves every logit by far more than rounding;
    also from bf16 storage (the bits upcast exactly)."""
    t = toy(11, T=5, V=13)
    gam = t["gamma"] * 1.7
    Z = (torch_rmsnorm(torch.tensor(t["x"]), torch.tensor(gam), eps) @ torch.tensor(t["W_U"]).T).numpy()
    for r in range(Z.shape[0]):
        for v in range(Z.shape[1]):
            assert abs(O.logit(t["x"], gam, t["W_U"], r, v, eps=eps) - Z[r, v]) <= 1e-13 * (1 + abs(Z[r, v]))
    # bf16 storage arrays: the oracle reads the bit patterns exactly
    to_bits = lambda a: (np.asarray(a, np.float32).view(np.uint32) >> 16).astype(np.uint16)  # noqa: E731
    xb, gb, wb = to_bits(t["x"]), to_bits(gam), to_bits(t["W_U"])
    up = lambda b: torch.tensor((b.astype(np.uint32) << 16).view(np.float32).astype(np.float64))  # noqa: E731
    Zb = (torch_rmsnorm(up(xb), up(gb), eps) @ up(wb).T).numpy()
    for r, v in [(0, 0), (2, 7), (4, 12)]:
        assert abs(O.logit(xb, gb, wb, r, v, eps=eps) - Zb[r, v]) <= 1e-13 * (1 + abs(Zb[r, v]))
    # the mistakes the pin must catch change the value far beyond the tolerance
    Z_nogain = (torch_rmsnorm(torch.tensor(t["x"]), torch.ones(len(gam), dtype=torch.float64), eps)
                @ torch.tensor(t["W_U"]).T).numpy()
    assert np.min(np.abs(Z_nogain - Z)) > 1e-6
    if eps > 0.1:
        Z_noeps = (torch_rmsnorm(torch.tensor(t["x"]), torch.tensor(gam), 0.0) @ torch.tensor(t["W_U"]).T).numpy()
        assert np.min(np.abs(Z_noeps - Z)) > 1e-6


def test_bad_targets_zero_row_and_counted():
    t = toy(8, T=4, V=9)
    y = t["y"].copy()
    y[1] = 9
    y[3] = -1
    out = O.output_error(t["x"], t["gamma"], t["W_U"], y)
    assert out["bad"] == 2
    np.testing.assert_array_equal(out["g_pre"][[1, 3]], 0.0)
    np.testing.assert_array_equal(out["g_tilde"][[1, 3]], 0.0)
    assert out["loss"][1] == 0 and out["loss"][3] == 0


# ------------------------------------------------------------ RMSNorm VJP
@pytest.mark.parametrize("seed", [0, 1])
def test_vjp_matches_autograd_unclamped(seed):
    r = np.random.default_rng(seed)
    x = r.standard_normal((5, 7)) * 2
    gam = 1 + 0.1 * r.standard_normal(7)
    g = r.standard_normal((5, 7))
    X = torch.tensor(x, requires_grad=True)
    (gx,) = torch.autograd.grad((torch_rmsnorm(X, torch.tensor(gam), 1e-6) * torch.tensor(g)).sum(), X)
    got = O.rmsnorm_vjp(g, x, gam, eps=1e-6, min_rms=0.5)
    np.testing.assert_allclose(got, gx.numpy(), rtol=1e-12, atol=1e-14)


def test_vjp_matches_finite_differences():
    r = np.random.default_rng(11)
    x = r.standard_normal((2, 5))
    gam = 1 + 0.1 * r.standard_normal(5)
    g = r.standard_normal((2, 5))

    def f(xx):
        _, y = O.rmsnorm_forward(xx, gam, 1e-6)
        return float(np.sum(g * y))

    h = 1e-6
    fd = np.zeros_like(x)
    for i in range(2):
        for k in range(5):
            a, b = x.copy(), x.copy()
            a[i, k] += h
            b[i, k] -= h
            fd[i, k] = (f(a) - f(b)) / (2 * h)
    np.testing.assert_allclose(O.rmsnorm_vjp(g, x, gam, 1e-6, 0.5), fd, rtol=1e-7, atol=1e-9)


def test_vjp_scale_invariance_identity():
    """<x, g~> = eps <x, gamma*g> / rho^3 (RMSNorm is scale invariant up to eps)."""
    r = np.random.default_rng(12)
    x = r.standard_normal((6, 9))
    gam = 1 + 0.1 * r.standard_normal(9)
    g = r.standard_normal((6, 9))
    eps = 1e-3
    gt = O.rmsnorm_vjp(g, x, gam, eps=eps, min_rms=0.0)
    rho = np.sqrt((x * x).mean(1) + eps)
    lhs = (x * gt).sum(1)
    rhs = eps * (x * gam * g).sum(1) / rho ** 3
    np.testing.assert_allclose(lhs, rhs, rtol=1e-9, atol=1e-15)


def test_vjp_clamp_inactive_is_bit_identical_and_active_rows_use_floor():
    r = np.random.default_rng(13)
    x = r.standard_normal((8, 16))
    x[2] *= 0.05     # rho ~ 0.05: clamp active
    gam = 1 + 0.1 * r.standard_normal(16)
    g = r.standard_normal((8, 16))
    a = O.rmsnorm_vjp(g, x, gam, 1e-6, 0.5)
    b = O.rmsnorm_vjp(g, x, gam, 1e-6, 0.0)
    keep = [i for i in range(8) if i != 2]
    assert np.array_equal(a[keep], b[keep])
    # clamped row: plain formula with rho replaced by 0.5 everywhere
    xh = x[2] / 0.5
    c = np.dot(xh, gam * g[2]) / 16
    np.testing.assert_allclose(a[2], (gam * g[2] - xh * c) / 0.5, rtol=1e-14)


def test_vjp_clamp_branch_is_the_vjp_of_an_rmsnorm_lifted_to_the_floor():
    """Rows whose RMS is below the floor: the clamped VJP equals the exact
    (autograd) VJP of a plain RMSNorm whose epsilon is raised, for that row, to
    floor^2 - mean(x^2), so that its RMS is exactly the floor. This definition
    does not use the VJP formula, so it pins the rho < min_rms branch; the other
    rows keep the ordinary epsilon and match too."""
    r = np.random.default_rng(21)
    x = r.standard_normal((6, 12))
    x[[1, 4]] *= 0.05  # RMS ~0.05: below the floor
    gam = 1 + 0.1 * r.standard_normal(12)
    g = r.standard_normal((6, 12))
    eps, floor = 1e-6, 0.5
    ms = (x * x).mean(1)
    rho = np.sqrt(ms + eps)
    assert np.all(rho[[1, 4]] < floor) and np.all(rho[[0, 2, 3, 5]] > floor)
    eps_row = np.where(rho < floor, floor ** 2 - ms, eps)
    X = torch.tensor(x, requires_grad=True)
    Y = torch.tensor(gam) * X / torch.sqrt((X * X).mean(1, keepdim=True) + torch.tensor(eps_row)[:, None])
    (gx,) = torch.autograd.grad((Y * torch.tensor(g)).sum(), X)
    got = O.rmsnorm_vjp(g, x, gam, eps=eps, min_rms=floor)
    np.testing.assert_allclose(got, gx.numpy(), rtol=1e-12, atol=1e-14)


# ------------------------------------------------------------ pseudograd
def test_pseudograd_single_token_is_exact_outer_product():
    r = np.random.default_rng(14)
    g = r.standard_normal((1, 6))
    a = r.standard_normal((1, 10))
    D = O.pseudograd(g, a)
    assert np.array_equal(D, np.outer(g[0], a[0]))
    s = np.linalg.svd(D, compute_uv=False)
    assert s[1] / s[0] < 1e-15


def test_pseudograd_linear_and_additive_over_token_splits():
    r = np.random.default_rng(15)
    g = r.standard_normal((7, 5))
    a = r.standard_normal((7, 9))
    b = r.standard_normal((7, 9))
    np.testing.assert_allclose(O.pseudograd(g, a + 2 * b), O.pseudograd(g, a) + 2 * O.pseudograd(g, b), atol=1e-14)
    D = O.pseudograd(g, a)
    D1 = O.pseudograd(g[:3], a[:3])
    D2 = O.pseudograd(g[3:], a[3:])
    np.testing.assert_allclose(D, (3 * D1 + 4 * D2) / 7, atol=1e-14)


def _identity_toy_loss(x_res, a_list, W_list, gamma, W_U, y, eps):
    h = x_res
    for a, W in zip(a_list, W_list):
        h = h + a @ W.T
    u = torch_rmsnorm(h, gamma, eps)
    return torch.nn.functional.cross_entropy(u @ W_U.T, y, reduction="mean"), h


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_identity_layer_toy_pseudograd_is_true_gradient(seed):
    """Sec. 2.1: with identity layers after the targets, g~ (x) a is the gradient."""
    t = toy(seed, T=5, d=6, V=16, d_ff=10, L=2)
    Ws = [torch.tensor(W, requires_grad=True) for W in t["W"]]
    As = [torch.tensor(a) for a in t["a"]]
    loss, h = _identity_toy_loss(torch.tensor(t["x"]), As, Ws, torch.tensor(t["gamma"]),
                                 torch.tensor(t["W_U"]), torch.tensor(t["y"]).long(), 1e-6)
    grads = torch.autograd.grad(loss, Ws)
    hf = h.detach().numpy()
    assert np.all(np.sqrt((hf ** 2).mean(1)) > 0.5)
    out = O.output_error(hf, t["gamma"], t["W_U"], t["y"], eps=1e-6, min_rms=0.5)
    for a, gW in zip(t["a"], grads):
        np.testing.assert_allclose(O.pseudograd(out["g_tilde"], a), gW.numpy(), rtol=1e-10, atol=1e-13)


def test_identity_layer_toy_directional_finite_difference():
    t = toy(21, T=3, d=5, V=8, d_ff=7, L=1)
    r = np.random.default_rng(22)
    dirn = r.standard_normal(t["W"][0].shape)

    def L_of(W):
        h = t["x"] + t["a"][0] @ W.T
        _, u = O.rmsnorm_forward(h, t["gamma"], 1e-6)
        z = u @ t["W_U"].T
        m = z.max(1, keepdims=True)
        lse = (m + np.log(np.exp(z - m).sum(1, keepdims=True)))[:, 0]
        return float(np.mean(lse - z[np.arange(3), t["y"]]))

    hstep = 1e-6
    fd = (L_of(t["W"][0] + hstep * dirn) - L_of(t["W"][0] - hstep * dirn)) / (2 * hstep)
    h = t["x"] + t["a"][0] @ t["W"][0].T
    D = O.pseudograd(O.output_error(h, t["gamma"], t["W_U"], t["y"])["g_tilde"], t["a"][0])
    assert abs(float(np.sum(D * dirn)) - fd) < 1e-7 * max(1.0, abs(fd))


@pytest.mark.parametrize("seed", [3, 4])
def test_post_ffn_toy_composed_signal_is_true_gradient(seed):
    """Sec. 3.2 post-feedforward RMSNorm (App. A pseudocode): each target layer
    adds postnorm_l(a_l W_l^T) to the residual; with identity layers after the
    targets, the gradient of the mean cross-entropy w.r.t. W_l is
    (1/T) [VJP of postnorm_l at the MLP output applied to g~]^T a_l, i.e. the
    oracle's post_ffn_signal followed by pseudograd (clamp inactive)."""
    t = toy(seed, T=5, d=6, V=16, d_ff=10, L=2)
    r = np.random.default_rng(100 + seed)
    gp = [0.3 * (1 + 0.1 * r.standard_normal(6)) for _ in range(2)]
    Ws = [torch.tensor(3.0 * W, requires_grad=True) for W in t["W"]]  # MLP-output RMS well above 0.5
    As = [torch.tensor(a) for a in t["a"]]
    h = torch.tensor(t["x"])
    mlp_out = []
    for a, W, g in zip(As, Ws, gp):
        m = a @ W.T
        mlp_out.append(m.detach().numpy())
        h = h + torch_rmsnorm(m, torch.tensor(g), 1e-6)
    U = torch_rmsnorm(h, torch.tensor(t["gamma"]), 1e-6)
    loss = torch.nn.functional.cross_entropy(U @ torch.tensor(t["W_U"]).T, torch.tensor(t["y"]).long(),
                                             reduction="mean")
    grads = torch.autograd.grad(loss, Ws)
    hf = h.detach().numpy()
    for m in mlp_out:
        assert np.all(np.sqrt((m ** 2).mean(1)) > 0.5)  # clamp inactive: the composition is exact
    out = O.output_error(hf, t["gamma"], t["W_U"], t["y"], eps=1e-6, min_rms=0.5)
    for l in range(2):
        gl = O.post_ffn_signal(out["g_tilde"], mlp_out[l], gp[l], eps=1e-6, min_rms=0.5)
        np.testing.assert_allclose(O.pseudograd(gl, t["a"][l]), grads[l].numpy(), rtol=1e-10, atol=1e-13)
        # and the composition differs from skipping the post-FFN VJP
        assert not np.allclose(O.pseudograd(out["g_tilde"], t["a"][l]), grads[l].numpy(), rtol=1e-3)


def test_post_ffn_signal_scale_and_gain_properties():
    """Scaling the MLP output by k (RMS stays above the clamp) divides the
    composed signal by k; the signal is linear in the gain."""
    r = np.random.default_rng(41)
    g = r.standard_normal((4, 8))
    x = 2.0 * r.standard_normal((4, 8))
    gam = 0.3 + 0.05 * r.standard_normal(8)
    base = O.post_ffn_signal(g, x, gam, eps=0.0, min_rms=0.5)
    np.testing.assert_allclose(O.post_ffn_signal(g, 3.0 * x, gam, eps=0.0, min_rms=0.5), base / 3.0, rtol=1e-12)
    np.testing.assert_allclose(O.post_ffn_signal(g, x, 2.0 * gam, eps=0.0, min_rms=0.5), 2.0 * base, rtol=1e-12)


def _rmsnorm_vjp_autograd(g, x, gam, eps, floor):
    """The VJP of a plain RMSNorm at x by torch autograd, with a row's epsilon
    raised to floor^2 - mean(x^2) where its RMS is below the floor (the clamp,
    as pinned above)."""
    ms = (x * x).mean(1)
    rho = np.sqrt(ms + eps)
    eps_row = np.where(rho < floor, floor ** 2 - ms, eps)
    X = torch.tensor(x, requires_grad=True)
    Y = torch.tensor(gam) * X / torch.sqrt((X * X).mean(1, keepdim=True) + torch.tensor(eps_row)[:, None])
    (gx,) = torch.autograd.grad((Y * torch.tensor(g)).sum(), X)
    return gx.numpy()


@pytest.mark.parametrize("post", [False, True], ids=["pre-MLP only (Qwen3)", "post-FFN then pre-MLP (Gemma 3)"])
def test_layer_signal_is_the_chain_of_rmsnorm_vjps(post):
    """Sec. 3.2 pre-MLP RMSNorm: layer_signal applies the VJP of the pre-MLP
    norm at its own cached input and gain after the post-FFN one, each an
    exact RMSNorm VJP (autograd), clamp active on some rows of each norm. A
    swapped order or swapped inputs / gains do not match."""
    r = np.random.default_rng(51)
    T, d = 7, 10
    g = r.standard_normal((T, d))
    x_post = 2.0 * r.standard_normal((T, d))
    x_post[2] *= 0.1                      # RMS ~0.2: clamp active on this row of the post-FFN norm
    x_pre = 4.0 * r.standard_normal((T, d))
    x_pre[5] *= 0.05                      # RMS ~0.2: clamp active on this row of the pre-MLP norm
    gp = 0.3 + 0.05 * r.standard_normal(d)
    gq = 1.0 + 0.1 * r.standard_normal(d)
    eps, floor = 1e-6, 0.5
    want = _rmsnorm_vjp_autograd(g, x_post, gp, eps, floor) if post else g
    want = _rmsnorm_vjp_autograd(want, x_pre, gq, eps, floor)
    got = O.layer_signal(g, x_post if post else None, gp if post else None, x_pre, gq, eps=eps, min_rms=floor)
    np.testing.assert_allclose(got, want, rtol=1e-11, atol=1e-13)
    if post:
        swapped = _rmsnorm_vjp_autograd(_rmsnorm_vjp_autograd(g, x_pre, gq, eps, floor), x_post, gp, eps, floor)
        assert not np.allclose(got, swapped, rtol=1e-3)
        np.testing.assert_allclose(O.layer_signal(g, x_post, gp, eps=eps, min_rms=floor),
                                   O.post_ffn_signal(g, x_post, gp, eps=eps, min_rms=floor), rtol=0, atol=0)
    assert not np.allclose(got, O.layer_signal(g, x_post if post else None, gp if post else None, x_pre, gp,
                                               eps=eps, min_rms=floor), rtol=1e-3)
    np.testing.assert_array_equal(O.layer_signal(g), g)


def test_pre_mlp_signal_scale_invariance():
    """The pre-MLP norm's output does not depend on the scale of its input, so
    its VJP at k x is the VJP at x divided by k (RMS above the clamp): the
    composed signal shrinks as the residual stream grows; eps = 0."""
    r = np.random.default_rng(52)
    g = r.standard_normal((4, 8))
    x = 3.0 * r.standard_normal((4, 8))
    gam = 1.0 + 0.1 * r.standard_normal(8)
    base = O.layer_signal(g, pre_in=x, gamma_pre=gam, eps=0.0, min_rms=0.5)
    np.testing.assert_allclose(O.layer_signal(g, pre_in=5.0 * x, gamma_pre=gam, eps=0.0, min_rms=0.5), base / 5.0,
                               rtol=1e-12)
    # the signal is orthogonal to its own input row (scale invariance of RMSNorm, eps = 0)
    np.testing.assert_allclose(np.sum(base * x, axis=1), 0.0, atol=1e-12)


def test_full_mlp_step0_feedback_is_exact_gradient():
    """eq. errh: at step 0 (W3 = W3_init) the W1/W2 signals are the exact gradients."""
    r = np.random.default_rng(31)
    T, d, d_ff, V = 5, 6, 10, 12
    x_res = r.standard_normal((T, d))
    x_in = r.standard_normal((T, d))
    W1 = 0.4 * r.standard_normal((d_ff, d))
    W2 = 0.4 * r.standard_normal((d_ff, d))
    W3 = 0.4 * r.standard_normal((d, d_ff))
    gam = 1 + 0.1 * r.standard_normal(d)
    W_U = 0.5 * r.standard_normal((V, d))
    y = r.integers(0, V, T)
    tW1, tW2, tW3 = (torch.tensor(w, requires_grad=True) for w in (W1, W2, W3))
    X = torch.tensor(x_in)
    q = X @ tW1.T
    u = X @ tW2.T
    m = torch.nn.functional.silu(q) * u
    h = torch.tensor(x_res) + m @ tW3.T
    U = torch_rmsnorm(h, torch.tensor(gam), 1e-6)
    loss = torch.nn.functional.cross_entropy(U @ torch.tensor(W_U).T, torch.tensor(y), reduction="mean")
    g1, g2, g3 = torch.autograd.grad(loss, (tW1, tW2, tW3))
    hf = h.detach().numpy()
    assert np.all(np.sqrt((hf ** 2).mean(1)) > 0.5)
    gt = O.output_error(hf, gam, W_U, y)["g_tilde"]
    D1, D2 = O.full_mlp_grads(gt, W3, q.detach().numpy(), u.detach().numpy(), x_in)
    np.testing.assert_allclose(D1, g1.numpy(), rtol=1e-10, atol=1e-13)
    np.testing.assert_allclose(D2, g2.numpy(), rtol=1e-10, atol=1e-13)
    np.testing.assert_allclose(O.pseudograd(gt, m.detach().numpy()), g3.numpy(), rtol=1e-10, atol=1e-13)


def test_silu_derivative_matches_autograd():
    z = np.linspace(-8, 8, 101)
    Z = torch.tensor(z, requires_grad=True)
    (gz,) = torch.autograd.grad(torch.nn.functional.silu(Z).sum(), Z)
    np.testing.assert_allclose(O.silu_prime(z), gz.numpy(), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(O.silu(z), torch.nn.functional.silu(torch.tensor(z)).numpy(), rtol=1e-14)


# ------------------------------------------------------------ clip + optimizers
def test_clip_bounds_norm():
    r = np.random.default_rng(41)
    for scale in (1e-4, 1.0, 1e3):
        D = scale * r.standard_normal((7, 9))
        W = r.standard_normal((7, 9))
        s = O.clip_scale(float((D * D).sum()), float((W * W).sum()), 0.01)
        nD, nW = np.linalg.norm(D), np.linalg.norm(W)
        assert abs(np.linalg.norm(s * D) - min(nD, 0.01 * nW)) < 1e-12 * max(nD, 1)
    assert O.clip_scale(1e-6, 1.0, 1.0) == 1.0
    assert O.clip_scale(0.0, 1.0, 0.01) == 1.0
    assert O.clip_scale(5.0, 1.0, 0.0) == 1.0


def test_sgd_momentum_matches_torch_three_steps():
    r = np.random.default_rng(42)
    W = r.standard_normal((4, 5))
    Gs = [r.standard_normal((4, 5)) for _ in range(3)]
    P = torch.nn.Parameter(torch.tensor(W))
    opt = torch.optim.SGD([P], lr=1e-2, momentum=0.9)
    Wo, b = W.copy(), np.zeros_like(W)
    for k, G in enumerate(Gs, start=1):
        P.grad = torch.tensor(G)
        opt.step()
        Wo, b = O.sgd_momentum(Wo, b, G, 1e-2, 0.9, step=k)
    np.testing.assert_allclose(Wo, P.detach().numpy(), rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(b, opt.state[P]["momentum_buffer"].numpy(), rtol=1e-14)


def test_adamw_matches_torch_three_steps():
    r = np.random.default_rng(43)
    W = r.standard_normal((4, 5))
    Gs = [r.standard_normal((4, 5)) * 1e-3 for _ in range(3)]
    P = torch.nn.Parameter(torch.tensor(W))
    opt = torch.optim.AdamW([P], lr=1e-3, betas=(0.9, 0.999), eps=1e-8, weight_decay=0.01)
    Wo, m, v = W.copy(), np.zeros_like(W), np.zeros_like(W)
    for k, G in enumerate(Gs, start=1):
        P.grad = torch.tensor(G)
        opt.step()
        Wo, m, v = O.adamw(Wo, m, v, G, 1e-3, k)
    np.testing.assert_allclose(Wo, P.detach().numpy(), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(m, opt.state[P]["exp_avg"].numpy(), rtol=1e-13)
    np.testing.assert_allclose(v, opt.state[P]["exp_avg_sq"].numpy(), rtol=1e-13)


@pytest.mark.parametrize("kind", ["sgd", "adamw"])
@pytest.mark.parametrize("frac", [1e-4, 10.0])
def test_update_clip_variant_against_torch(kind, frac):
    """The clip-the-update reading: torch.optim's own step from the current
    (clipped) weights gives the unclipped update delta; the oracle must apply
    W + s * delta with s = min(1, frac ||W|| / ||delta||) and keep torch's
    (unclipped) optimizer state, over three steps. frac 10 leaves the clip
    idle, so the result is torch's trajectory itself."""
    r = np.random.default_rng(44)
    W = r.standard_normal((4, 5))
    Gs = [r.standard_normal((4, 5)) * (1e-3 if kind == "adamw" else 1.0) for _ in range(3)]
    P = torch.nn.Parameter(torch.tensor(W))
    opt = (torch.optim.SGD([P], lr=1e-2, momentum=0.9) if kind == "sgd" else
           torch.optim.AdamW([P], lr=1e-3, betas=(0.9, 0.999), eps=1e-8, weight_decay=0.01))
    Wo, b1, b2 = W.copy(), np.zeros_like(W), np.zeros_like(W)
    for k, G in enumerate(Gs, start=1):
        with torch.no_grad():
            P.copy_(torch.tensor(Wo))
        P.grad = torch.tensor(G)
        opt.step()
        delta = P.detach().numpy() - Wo
        s_exp = min(1.0, frac * np.linalg.norm(Wo) / np.linalg.norm(delta))
        if kind == "sgd":
            W2, b1, s = O.sgd_momentum_update_clip(Wo, b1, G, 1e-2, 0.9, step=k, frac=frac)
            np.testing.assert_allclose(b1, opt.state[P]["momentum_buffer"].numpy(), rtol=1e-14)
        else:
            W2, b1, b2, s = O.adamw_update_clip(Wo, b1, b2, G, 1e-3, k, frac=frac)
            np.testing.assert_allclose(b1, opt.state[P]["exp_avg"].numpy(), rtol=1e-13)
            np.testing.assert_allclose(b2, opt.state[P]["exp_avg_sq"].numpy(), rtol=1e-13)
        assert abs(s - s_exp) <= 1e-12 * s_exp
        np.testing.assert_allclose(W2 - Wo, s_exp * delta, rtol=1e-9, atol=1e-15)
        if frac < 1.0:
            assert s < 1.0
            assert abs(np.linalg.norm(W2 - Wo) - frac * np.linalg.norm(Wo)) <= 1e-9 * frac * np.linalg.norm(Wo)
        else:
            assert s == 1.0
            np.testing.assert_allclose(W2, P.detach().numpy(), rtol=1e-13, atol=1e-15)
        Wo = W2


# ------------------------------------------------------------ cosine
def test_cosine_closed_forms():
    r = np.random.default_rng(51)
    A = r.standard_normal((30, 40))
    assert abs(O.cosine(A, A)[3] - 1) < 1e-14
    assert abs(O.cosine(A, -A)[3] + 1) < 1e-14
    B = r.standard_normal((30, 40))
    Bp = B - (np.sum(A * B) / np.sum(A * A)) * A
    assert abs(O.cosine(A, Bp)[3]) < 1e-13
    assert O.cosine(np.zeros_like(A), B)[3] == 0.0
    dot, na, nb, _ = O.cosine(A, B)
    assert abs(dot - math.fsum((A * B).ravel())) < 1e-10
    assert abs(na - math.fsum((A * A).ravel())) < 1e-10


def test_cosine_noise_recipe_gives_half():
    """R = D + sigma N with sigma = sqrt(3) ||D|| / sqrt(n) has E[cos] = 1/2."""
    r = np.random.default_rng(52)
    n = 1_000_000
    D = r.standard_normal(n) * 0.3 + 0.1
    sigma = math.sqrt(3) * np.linalg.norm(D) / math.sqrt(n)
    R = D + sigma * r.standard_normal(n)
    assert abs(O.cosine(D, R)[3] - 0.5) < 3e-3


def test_layer_summary_last_quarter():
    assert O.layer_summary(list(range(36))) == np.mean(range(27, 36))
    assert O.layer_summary(list(range(28))) == np.mean(range(21, 28))
    assert O.layer_summary(list(range(32))) == np.mean(range(24, 32))
