"""Pins of the end-to-end diagnostic oracle (oracle/transformer.py).

The pseudogradient is defined as the gradient the target layer would see if
every later layer acted as the identity (Sec. 2.1, eq. decomp). So on a real
transformer, run by the oracle in float64 with autograd:
  * at the last layer the pseudogradient IS the true gradient (R = 0), in
    both norm layouts (the post-FFN one through its composition, Sec. 3.2);
  * at an earlier layer it becomes the true gradient once the later blocks
    are made identity maps (zero output projections, or zero post-norm
    gains), and is not the true gradient otherwise;
  * the W1/W2 pseudogradients through W3_init (eq. errh) equal the true
    gate/up gradients under the same conditions (W3_init = W3 at the
    diagnostic's single step).
The model itself is pinned by autograd against central finite differences,
causality, explicit attention loops and the grouped-head equivalence, and
the output error's loss against the model's own cross-entropy.
"""
import math

import numpy as np
import pytest
import torch

from oracle import transformer as OT
from paper_2608_14563_amd import inputs as I


def _model(name):
    m = I.MODELS[name]
    return m, I.model_head(m), [I.model_layer(m, l) for l in range(m.n_layers)], I.model_tokens(m)


def rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


@pytest.fixture(scope="module", params=["tiny", "tiny-post"])
def model(request):
    return _model(request.param)


def test_last_layer_pseudogradient_is_the_true_gradient(model):
    m, head, layers, ids = model
    r = OT.diagnostic(m, head, layers, ids, full_mlp=True)
    # the clamp is a deliberate deviation from the true VJP: make sure it is idle here
    assert r["oe"]["rho"].min() > m.min_rms
    if m.layout == "post":
        assert min(float(np.sqrt((o.detach().numpy() ** 2).mean(1)).min()) for o in r["fw"]["mlp_out"]) > m.min_rms
    last = m.n_layers - 1
    assert rel(r["D3"][last], r["true"]["dW3"][last]) < 1e-12
    assert rel(r["D1"][last], r["true"]["dW1"][last]) < 1e-12
    assert rel(r["D2"][last], r["true"]["dW2"][last]) < 1e-12
    assert rel(r["g_tilde"] / ids[:, 1:].size, r["true"]["dR"][last]) < 1e-12
    assert abs(r["cos_w3"][last] - 1.0) < 1e-12 and abs(r["cos_out"][last] - 1.0) < 1e-12
    # the pin is not vacuous: the first layer's residual is far from zero
    assert r["cos_w3"][0] < 0.9 and r["cos_out"][0] < 0.9
    assert all(abs(c) <= 1.0 + 1e-12 for c in r["cos_w3"] + r["cos_out"] + r["cos_w1"] + r["cos_w2"])


def _identity_after(m, layers, ell):
    out = [dict(w) for w in layers]
    for l in range(ell + 1, m.n_layers):
        if m.layout == "pre":
            out[l]["wo"] = np.zeros_like(out[l]["wo"])
            out[l]["w3"] = np.zeros_like(out[l]["w3"])
        else:
            out[l]["n1"] = np.zeros_like(out[l]["n1"])
            out[l]["n2"] = np.zeros_like(out[l]["n2"])
    return out


@pytest.mark.parametrize("ell", [0, 1])
def test_identity_later_layers_give_the_true_gradient(model, ell):
    m, head, layers, ids = model
    lay = _identity_after(m, layers, ell)
    r = OT.diagnostic(m, head, lay, ids, full_mlp=True, min_rms=0.0)
    assert rel(r["D3"][ell], r["true"]["dW3"][ell]) < 1e-11
    assert rel(r["D1"][ell], r["true"]["dW1"][ell]) < 1e-11
    assert rel(r["D2"][ell], r["true"]["dW2"][ell]) < 1e-11
    assert abs(r["cos_out"][ell] - 1.0) < 1e-12
    # every later residual carries the same gradient
    for l in range(ell, m.n_layers):
        assert rel(r["true"]["dR"][l], r["true"]["dR"][-1]) < 1e-12


def test_post_layout_needs_the_composition():
    """Without the post-FFN VJP the last layer's W3 signal is not the true
    gradient (the composition is a real term, not a no-op)."""
    m, head, layers, ids = _model("tiny-post")
    r = OT.diagnostic(m, head, layers, ids)
    last = m.n_layers - 1
    from oracle import fpo_oracle as O
    T = ids[:, 1:].size
    plain = O.pseudograd(r["g_tilde"], r["fw"]["a"][last].detach().numpy(), 1.0 / T)
    assert O.cosine(plain, r["true"]["dW3"][last])[3] < 0.99
    assert abs(r["cos_w3"][last] - 1.0) < 1e-12


def test_output_error_loss_matches_the_model(model):
    m, head, layers, ids = model
    r = OT.diagnostic(m, head, layers, ids)
    assert abs(float(np.mean(r["oe"]["loss"])) - r["loss"]) < 1e-12 * max(1.0, abs(r["loss"]))
    lse = torch.logsumexp(r["fw"]["logits"].detach(), dim=1).numpy()
    assert np.max(np.abs(r["oe"]["lse"] - lse)) < 1e-10


def test_autograd_matches_finite_differences():
    m, head, layers, ids = _model("tiny")
    tg = OT.true_gradients(OT.forward(m, head, layers, ids, ("w3", "w1", "w2")), full_mlp=True)
    h = 1e-5
    for name, l, (i, j) in (("w3", 0, (3, 17)), ("w3", 2, (100, 5)), ("w1", 1, (7, 60))):
        lp = [dict(w) for w in layers]
        lm = [dict(w) for w in layers]
        lp[l][name] = layers[l][name].astype(np.float64).copy()
        lm[l][name] = layers[l][name].astype(np.float64).copy()
        lp[l][name][i, j] += h
        lm[l][name][i, j] -= h
        fd = (float(OT.forward(m, head, lp, ids, ())["loss"]) - float(OT.forward(m, head, lm, ids, ())["loss"])) / (2 * h)
        ag = tg["dW3" if name == "w3" else "dW1"][l][i, j]
        assert abs(fd - ag) < 1e-7 * max(1.0, abs(ag)) + 1e-9, (name, l, fd, ag)


def test_causal_mask():
    m, head, layers, ids = _model("tiny")
    a = OT.forward(m, head, layers, ids, ())["logits"].detach().numpy()
    ids2 = ids.copy()
    s0 = 20
    ids2[0, s0 + 1:] = (ids2[0, s0 + 1:] + 7) % m.V  # change inputs from position s0 + 1 on
    b = OT.forward(m, head, layers, ids2, ())["logits"].detach().numpy()
    S = m.seq
    assert np.array_equal(a[:s0 + 1], b[:s0 + 1])  # sequence 0, positions <= s0
    assert not np.allclose(a[s0 + 1:S], b[s0 + 1:S])
    assert np.array_equal(a[S:], b[S:])  # sequence 1 untouched


def test_attention_matches_explicit_loops():
    rng = np.random.default_rng(5)
    B, S, H, KV, hd = 2, 5, 4, 2, 3
    d = H * hd
    z = rng.standard_normal((B, S, d))
    w = {"wq": rng.standard_normal((H * hd, d)), "wk": rng.standard_normal((KV * hd, d)),
         "wv": rng.standard_normal((KV * hd, d)), "wo": rng.standard_normal((d, H * hd))}
    got = OT.attention(torch.from_numpy(z), {k: torch.from_numpy(v) for k, v in w.items()}, H, KV).numpy()
    want = np.zeros((B, S, d))
    for b in range(B):
        for t in range(S):
            o = np.zeros(H * hd)
            for h in range(H):
                kvh = h // (H // KV)
                q = w["wq"][h * hd:(h + 1) * hd] @ z[b, t]
                sc = [float(q @ (w["wk"][kvh * hd:(kvh + 1) * hd] @ z[b, s])) / math.sqrt(hd) for s in range(t + 1)]
                mx = max(sc)
                p = [math.exp(x - mx) for x in sc]
                tot = sum(p)
                for s in range(t + 1):
                    o[h * hd:(h + 1) * hd] += p[s] / tot * (w["wv"][kvh * hd:(kvh + 1) * hd] @ z[b, s])
            want[b, t] = w["wo"] @ o
    assert np.max(np.abs(got - want)) < 1e-12


def test_grouped_heads_equal_repeated_full_heads():
    """Grouped key/value heads equal full multi-head attention whose key/value
    weights repeat each group's head for every query head of the group."""
    m, head, layers, ids = _model("tiny")
    grp = m.n_heads // m.n_kv_heads
    hd = m.head_dim
    full = []
    for w in layers:
        w2 = dict(w)
        for k in ("wk", "wv"):
            blocks = [w[k][j * hd:(j + 1) * hd] for j in range(m.n_kv_heads)]
            w2[k] = np.concatenate([b for b in blocks for _ in range(grp)], axis=0)
        full.append(w2)
    mf = m.shrink(n_kv_heads=m.n_heads)
    a = OT.forward(m, head, layers, ids, ())["logits"].detach().numpy()
    b = OT.forward(mf, head, full, ids, ())["logits"].detach().numpy()
    assert np.max(np.abs(a - b)) < 1e-11
