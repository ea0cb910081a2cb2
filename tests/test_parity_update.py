"""GPU parity of fpo_apply_update (relative clip + SGD-momentum / AdamW on
fp32 masters) and of fpo_cosine against the fp64 oracle."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_14563_amd import _lib as L_
from paper_2608_14563_amd import api
from paper_2608_14563_amd import inputs as I
from tests._util import assert_close, bf16_rne_bits, dev_tensor, ulp_diff_f32

pytestmark = pytest.mark.gpu


def make(shapes, seed, gscale):
    r = np.random.default_rng(seed)
    W = [(0.02 * r.standard_normal(s)).astype(np.float32) for s in shapes]
    G = [[(gscale * r.standard_normal(s)).astype(np.float32) for s in shapes] for _ in range(3)]
    return W, G


@pytest.mark.parametrize("kind", ["sgd", "adamw", "sgd-plain"])
@pytest.mark.parametrize("clip,gscale", [(0.01, 1e-2), (0.01, 1e-5), (0.0, 1e-3), (1.0, 1e-3)])
def test_three_steps(dev, kind, clip, gscale):
    """Three optimizer steps against the oracle. sgd-plain: momentum 0 with
    no state buffer (the oracle's SGD-momentum with beta = 0)."""
    shapes = [(256, 688), (64, 100), (8, 4)]
    W, Gs = make(shapes, 7, gscale)
    n = len(shapes)
    tW = [torch.from_numpy(w.copy()).to(dev) for w in W]
    plain = kind == "sgd-plain"
    s1 = None if plain else [torch.zeros_like(w) for w in tW]
    s2 = [torch.zeros_like(w) for w in tW] if kind == "adamw" else None
    lp = [torch.empty(w.shape, dtype=torch.bfloat16, device=dev) for w in tW]
    Wsq = torch.tensor([float((w.astype(np.float64) ** 2).sum()) for w in W], dtype=torch.float64, device=dev)
    clipv = torch.empty(n, dtype=torch.float32, device=dev)
    # oracle state (fp64), fed the same gradients
    oW = [w.astype(np.float64) for w in W]
    ob = [np.zeros(s) for s in shapes]
    om = [np.zeros(s) for s in shapes]
    ov = [np.zeros(s) for s in shapes]
    lr = 1e-3 if kind == "adamw" else 1e-2
    mom = 0.0 if plain else 0.9
    for step in range(1, 4):
        G = Gs[step - 1]
        tg = [torch.from_numpy(g).to(dev) for g in G]
        gsq = torch.tensor([float((g.astype(np.float64) ** 2).sum()) for g in G], dtype=torch.float64, device=dev)
        Wprev = [w.cpu().numpy().copy() for w in tW]
        opt = api.OptConfig(kind=1 if kind == "adamw" else 0, lr=lr, momentum=mom, clip_frac=clip, step=step)
        api.fpo_apply_update(opt, tg, gsq, tW, s1, Wsq, W_lp=lp, state2=s2, clip_scale=clipv)
        torch.cuda.synchronize()
        for m in range(n):
            wsq_in = float((Wprev[m].astype(np.float64) ** 2).sum())
            s = O.clip_scale(float(gsq[m]), wsq_in, clip)
            assert abs(float(clipv[m]) - s) <= 1e-5 * s
            Gh = s * G[m].astype(np.float64)
            if kind != "adamw":
                oW[m], ob[m] = O.sgd_momentum(oW[m], ob[m], Gh, lr, mom, step)
                if plain:  # the step used b = fp32(s) * G, no state
                    b = (np.float32(clipv[m].item()) * G[m]).astype(np.float32).astype(np.float64)
                    assert_close("step", b, ob[m], "f32")
                else:
                    assert_close("momentum", s1[m].cpu().numpy(), ob[m], "f32")
                    b = s1[m].cpu().numpy().astype(np.float64)
                expect = (Wprev[m].astype(np.float64) - np.float64(np.float32(lr)) * b).astype(np.float32)
            else:
                oW[m], om[m], ov[m] = O.adamw(oW[m], om[m], ov[m], Gh, lr, step)
                assert_close("exp_avg", s1[m].cpu().numpy(), om[m], "f32")
                assert_close("exp_avg_sq", s2[m].cpu().numpy(), ov[m], "f32")
                mg = s1[m].cpu().numpy().astype(np.float64)
                vg = s2[m].cpu().numpy().astype(np.float64)
                f32 = lambda v: np.float64(np.float32(v))
                decay = f32(1.0 - lr * 0.01)
                ib1 = f32(1.0 / (1 - 0.9 ** step))
                isb2 = f32(1.0 / np.sqrt(1 - 0.999 ** step))
                expect = (Wprev[m].astype(np.float64) * decay
                          - f32(lr) * (mg * ib1) / (np.sqrt(vg) * isb2 + f32(1e-8))).astype(np.float32)
            Wg = tW[m].cpu().numpy()
            if kind != "adamw":
                assert ulp_diff_f32(Wg, expect).max() <= 1
            else:
                # the AdamW step is ~lr per element, not small against W: allow
                # 2 ulp of W' plus float32 rounding of the step itself
                step_mag = np.abs(expect.astype(np.float64) - Wprev[m].astype(np.float64))
                tol = 2 * np.spacing(np.abs(expect)).astype(np.float64) + 4 * 2.0 ** -23 * step_mag
                assert np.all(np.abs(Wg.astype(np.float64) - expect.astype(np.float64)) <= tol)
            # the master moved as the oracle says, to its own precision
            assert np.max(np.abs(Wg - oW[m])) <= 1e-6 * max(1.0, np.max(np.abs(oW[m])))
            assert np.array_equal(lp[m].view(torch.int16).cpu().numpy().view(np.uint16), bf16_rne_bits(Wg))
            assert abs(float(Wsq[m]) - float((Wg.astype(np.float64) ** 2).sum())) <= 1e-6 * float(Wsq[m])


@pytest.mark.parametrize("kind", ["sgd", "adamw", "sgd-plain"])
@pytest.mark.parametrize("clip,gscale", [(0.01, 1e-1), (0.01, 1e-5), (0.0, 1e-3)])
def test_three_steps_clip_update(dev, kind, clip, gscale):
    """Clip-the-update reading (FPO_CLIP_UPDATE), three steps against the
    oracle's *_update_clip: unclipped optimizer state, the factor applied to
    the step, W' = W + s * delta within fp32 rounding, ||W' - W|| <= clip ||W||."""
    shapes = [(256, 688), (64, 100), (8, 4)]
    W, Gs = make(shapes, 9, gscale)
    n = len(shapes)
    tW = [torch.from_numpy(w.copy()).to(dev) for w in W]
    plain = kind == "sgd-plain"
    adam = kind == "adamw"
    s1 = None if plain else [torch.zeros_like(w) for w in tW]
    s2 = [torch.zeros_like(w) for w in tW] if adam else None
    lp = [torch.empty(w.shape, dtype=torch.bfloat16, device=dev) for w in tW]
    Wsq = torch.tensor([float((w.astype(np.float64) ** 2).sum()) for w in W], dtype=torch.float64, device=dev)
    clipv = torch.empty(n, dtype=torch.float32, device=dev)
    oW = [w.astype(np.float64) for w in W]
    ob = [np.zeros(s) for s in shapes]
    ov = [np.zeros(s) for s in shapes]
    lr = 1e-3 if adam else 1e-2
    mom = 0.0 if plain else 0.9
    active = False
    for step in range(1, 4):
        G = Gs[step - 1]
        tg = [torch.from_numpy(g).to(dev) for g in G]
        gsq = torch.tensor([float((g.astype(np.float64) ** 2).sum()) for g in G], dtype=torch.float64, device=dev)
        Wprev = [w.cpu().numpy().copy() for w in tW]
        opt = api.OptConfig(kind=1 if adam else 0, lr=lr, momentum=mom, clip_frac=clip, step=step,
                            clip_target=L_.FPO_CLIP_UPDATE)
        api.fpo_apply_update(opt, tg, gsq, tW, s1, Wsq, W_lp=lp, state2=s2, clip_scale=clipv)
        torch.cuda.synchronize()
        for m in range(n):
            # the oracle continues from the GPU's weights so that both clip the same step
            Wp = Wprev[m].astype(np.float64)
            if adam:
                oW[m], ob[m], ov[m], s = O.adamw_update_clip(Wp, ob[m], ov[m], G[m], lr, step, frac=clip)
                assert_close("exp_avg", s1[m].cpu().numpy(), ob[m], "f32")
                assert_close("exp_avg_sq", s2[m].cpu().numpy(), ov[m], "f32")
            else:
                oW[m], ob[m], s = O.sgd_momentum_update_clip(Wp, ob[m], G[m], lr, mom, step, frac=clip)
                if not plain:
                    assert_close("momentum", s1[m].cpu().numpy(), ob[m], "f32")
            assert abs(float(clipv[m]) - s) <= 1e-5 * s, (m, step, float(clipv[m]), s)
            active = active or s < 1.0
            Wg = tW[m].cpu().numpy().astype(np.float64)
            # W' from the GPU's own new state and factor, in float64: the step is
            # exact up to fp32 rounding of W' and of the step itself
            f32 = lambda v: np.float64(np.float32(v))  # noqa: E731
            sg = float(clipv[m])
            if adam:
                mg = s1[m].cpu().numpy().astype(np.float64)
                vg = s2[m].cpu().numpy().astype(np.float64)
                ib1 = f32(1.0 / (1 - 0.9 ** step))
                isb2 = f32(1.0 / np.sqrt(1 - 0.999 ** step))
                delta = -f32(lr * 0.01) * Wp - f32(lr) * (mg * ib1) / (np.sqrt(vg) * isb2 + f32(1e-8))
            else:
                bg = G[m].astype(np.float64) if plain else s1[m].cpu().numpy().astype(np.float64)
                delta = -f32(lr) * bg
            expect = Wp + sg * delta
            tol = 2 * np.spacing(np.abs(expect).astype(np.float32)).astype(np.float64) + 4 * 2.0 ** -23 * np.abs(sg * delta)
            assert np.all(np.abs(Wg - expect) <= tol), (m, step)
            # and the master moved as the oracle says, to its own precision
            assert np.max(np.abs(Wg - oW[m])) <= 1e-6 * max(1.0, np.max(np.abs(oW[m])))
            if clip > 0:
                assert np.linalg.norm(Wg - Wp) <= clip * np.linalg.norm(Wp) * (1 + 1e-4)
            assert np.array_equal(lp[m].view(torch.int16).cpu().numpy().view(np.uint16),
                                  bf16_rne_bits(Wg.astype(np.float32)))
            assert abs(float(Wsq[m]) - float((Wg ** 2).sum())) <= 1e-6 * float(Wsq[m])
    # AdamW's step is ~lr per element whatever the gradient's scale
    assert active == (clip > 0 and (adam or gscale > 1e-2))


def test_clip_edge_cases(dev):
    W = torch.full((4, 4), 0.5, dtype=torch.float32, device=dev)
    z = torch.zeros(4, 4, dtype=torch.float32, device=dev)
    s1 = torch.zeros(4, 4, dtype=torch.float32, device=dev)
    Wsq = torch.tensor([4.0], dtype=torch.float64, device=dev)
    cs = torch.empty(1, dtype=torch.float32, device=dev)
    api.fpo_apply_update(api.OptConfig(lr=1.0, clip_frac=0.01), [z], torch.zeros(1, dtype=torch.float64, device=dev),
                         [W], [s1], Wsq, clip_scale=cs, lp_dtype=torch.float32)
    torch.cuda.synchronize()
    assert float(cs[0]) == 1.0 and torch.all(W == 0.5)
    assert not torch.isnan(W).any()


@pytest.mark.parametrize("target", [0, 1], ids=["clip-grad", "clip-update"])
@pytest.mark.parametrize("kind", [L_.FPO_OPT_SGD, L_.FPO_OPT_ADAMW], ids=["sgd", "adamw"])
def test_clip_at_zero_weights(dev, kind, target):
    """The relative clip of a zero matrix: 0.01 ||W|| = 0 bounds the step to
    zero (the oracle's s = 0), so a nonzero gradient moves nothing and leaves
    no optimizer state behind (both clip targets)."""
    W = torch.zeros(4, 8, dtype=torch.float32, device=dev)
    G = torch.linspace(-1.0, 1.0, 32, dtype=torch.float32, device=dev).reshape(4, 8)
    gsq = torch.tensor([float((G.double() ** 2).sum())], dtype=torch.float64, device=dev)
    s1 = torch.zeros_like(W)
    s2 = torch.zeros_like(W) if kind == L_.FPO_OPT_ADAMW else None
    Wsq = torch.zeros(1, dtype=torch.float64, device=dev)
    cs = torch.full((1,), -1.0, dtype=torch.float32, device=dev)
    api.fpo_apply_update(api.OptConfig(kind=kind, lr=1e-2, clip_frac=0.01, clip_target=target), [G], gsq, [W],
                         [s1], Wsq, state2=[s2] if s2 is not None else None, clip_scale=cs,
                         lp_dtype=torch.float32)
    torch.cuda.synchronize()
    assert O.clip_scale(float(gsq[0]), 0.0, 0.01) == 0.0
    assert float(cs[0]) == 0.0
    assert torch.all(W == 0) and float(Wsq[0]) == 0.0
    if target == L_.FPO_CLIP_GRADIENT:  # the clipped gradient (zero) enters the state
        assert torch.all(s1 == 0)


@pytest.mark.parametrize("bdtype", ["f32", "bf16"])
def test_cosine(dev, bdtype):
    r = np.random.default_rng(3)
    A = [r.standard_normal((300, 100)).astype(np.float32) for _ in range(3)] + [np.zeros((8, 8), np.float32)]
    B = [a + 0.5 * r.standard_normal(a.shape).astype(np.float32) for a in A]
    B[1] = -A[1]
    Bs = [b if bdtype == "f32" else I.bf16_bits(b) for b in B]
    tA = [torch.from_numpy(a).to(dev) for a in A]
    tB = [dev_tensor(b, dev) for b in Bs]
    n = len(A)
    dot, sa, sb = (torch.empty(n, dtype=torch.float64, device=dev) for _ in range(3))
    cs = torch.empty(n, dtype=torch.float32, device=dev)
    api.fpo_cosine(tA, tB, dot=dot, sumsq_A=sa, sumsq_B=sb, cos=cs)
    torch.cuda.synchronize()
    for m in range(n):
        d0, na, nb, c0 = O.cosine(A[m], Bs[m])
        if na == 0:
            assert float(cs[m]) == 0.0
            continue
        assert_close("dot", float(dot[m]), d0, "f32")
        assert_close("sa", float(sa[m]), na, "f32")
        assert_close("sb", float(sb[m]), nb, "f32")
        assert abs(float(cs[m]) - c0) <= 1e-6
    if bdtype == "f32":
        assert abs(float(cs[1]) + 1.0) <= 1e-6
    # norms-only mode
    api.fpo_cosine(tA, None, sumsq_A=sa)
    torch.cuda.synchronize()
    assert_close("sa", float(sa[0]), O.cosine(A[0], A[0])[1], "f32")


@pytest.mark.parametrize("target", [0, 1], ids=["clip-grad", "clip-update"])
@pytest.mark.parametrize("kind", ["sgd", "adamw", "sgd-plain"])
@pytest.mark.parametrize("T,d,d_ff,L,clip,pffn", [(256, 256, 512, 2, 0.01, False), (300, 264, 1000, 3, 0.01, False),
                                                  (200, 512, 768, 3, 1e-5, False), (300, 264, 1000, 3, 0.01, True),
                                                  (200, 1032, 1288, 3, 0.01, False)])
def test_fused_update_matches_separate_calls(dev, kind, T, d, d_ff, L, clip, pffn, target):
    """The W3 pseudogradient with the optimizer fused (bf16: one launch per
    layer carrying that layer's outer products and the previous layer's update)
    is bit-identical to the pseudogradient followed by fpo_apply_update, over two
    steps (momentum / moments carried), including a ragged shape, an active
    clip (clip_frac 1e-5), and matrices of more update blocks than the GPU has
    compute units (the overlapped update then visits its blocks grid-stride)."""
    c = I.CONFIGS[1].shrink(T=T, d=d, d_ff=d_ff, L=L)
    g = dev_tensor(I.synthetic_signal(c), dev)
    kw = {}
    if pffn:  # per-layer post-FFN composition on both paths
        g32 = torch.from_numpy(I.normal(c.cid, I.T_G, 7, T * d, std=0.02).reshape(T, d)).to(dev)
        pfs = [I.post_ffn(c, l) for l in range(L)]
        kw = dict(post_ffn=api.PostFfn(g32, [dev_tensor(m, dev) for m, _ in pfs], [dev_tensor(x, dev) for _, x in pfs]))
    acts = [dev_tensor(I.activation(c, l), dev) for l in range(L)]
    W0 = [torch.from_numpy(I.master_weight(c, l)).to(dev) for l in range(L)]
    adam = kind == "adamw"
    plain = kind == "sgd-plain"

    def fresh():
        W = [w.clone() for w in W0]
        return dict(W=W, s1=None if plain else [torch.zeros_like(w) for w in W],
                    s2=[torch.zeros_like(w) for w in W] if adam else None,
                    lp=[torch.empty(w.shape, dtype=torch.bfloat16, device=dev) for w in W],
                    Wsq=torch.tensor([float((w.double() ** 2).sum()) for w in W], dtype=torch.float64, device=dev),
                    dW=[torch.empty(d, d_ff, dtype=torch.float32, device=dev) for _ in range(L)],
                    ss=torch.empty(L, dtype=torch.float64, device=dev),
                    cs=torch.empty(L, dtype=torch.float32, device=dev))

    sep, fus = fresh(), fresh()
    for step in (1, 2):
        opt = api.OptConfig(kind=L_.FPO_OPT_ADAMW if adam else L_.FPO_OPT_SGD, lr=1e-2, clip_frac=clip, step=step,
                            momentum=0.0 if plain else 0.9, clip_target=target)
        api.fpo_pseudograd(g, acts, dW3=sep["dW"], sumsq=sep["ss"], **kw)
        api.fpo_apply_update(opt, sep["dW"], sep["ss"], sep["W"], sep["s1"], sep["Wsq"], W_lp=sep["lp"],
                             state2=sep["s2"], clip_scale=sep["cs"])
        api.fpo_pseudograd(g, acts, dW3=fus["dW"], sumsq=fus["ss"], opt=opt, W_master=fus["W"], W_lp=fus["lp"],
                           state1=fus["s1"], state2=fus["s2"], W_sumsq=fus["Wsq"], clip_scale=fus["cs"], **kw)
        torch.cuda.synchronize()
        for key in ("W", "lp", "dW") + (("s2",) if adam else ()) + (() if plain else ("s1",)):
            for a, b in zip(sep[key], fus[key]):
                assert torch.equal(a, b), (key, step)
        for key in ("Wsq", "ss", "cs"):
            assert torch.equal(sep[key], fus[key]), (key, step)
    if clip < 1e-4:
        assert float(fus["cs"].max()) < 1.0  # the clip was active


@pytest.mark.parametrize("target", [0, 1], ids=["clip-grad", "clip-update"])
@pytest.mark.parametrize("kind", ["sgd", "adamw"])
@pytest.mark.parametrize("T,d,d_ff,L,clip", [(256, 256, 512, 2, 0.01), (300, 264, 1000, 3, 0.01),
                                             (200, 1032, 1288, 2, 1e-5)])
def test_fused_full_mlp_update_matches_separate_calls(dev, kind, T, d, d_ff, L, clip, target):
    """Full-MLP pseudogradient with the optimizer fused (bf16, gradient clip:
    each matrix's update released on the side stream once its outer products
    are done, beside the W1/W2 signal and outer-product launches that follow)
    is bit-identical to the pseudogradient followed by fpo_apply_update over
    the 3 L matrices (W3, W1, W2), over two steps; whole tiles, a ragged shape,
    and matrices of more update blocks than compute units with an active clip."""
    c = I.CONFIGS[1].shrink(T=T, d=d, d_ff=d_ff, L=L)
    g = dev_tensor(I.synthetic_signal(c), dev)
    caches = [I.mlp_cache(c, l) for l in range(L)]
    extras = [I.full_mlp_extra(c, l) for l in range(L)]
    acts = [dev_tensor(cc[2], dev) for cc in caches]
    W0 = [torch.from_numpy(I.master_weight(c, l)).to(dev) for l in range(L)]
    W0 += [torch.from_numpy(e[1]).to(dev) for e in extras] + [torch.from_numpy(e[2]).to(dev) for e in extras]
    fkw = dict(W3_init=[w.to(torch.bfloat16) for w in W0[:L]], gate=[dev_tensor(cc[0], dev) for cc in caches],
               up=[dev_tensor(cc[1], dev) for cc in caches], x_in=[dev_tensor(e[0], dev) for e in extras])
    adam = kind == "adamw"
    n = 3 * L

    def fresh():
        W = [w.clone() for w in W0]
        return dict(W=W, s1=[torch.zeros_like(w) for w in W], s2=[torch.zeros_like(w) for w in W] if adam else None,
                    lp=[torch.empty(w.shape, dtype=torch.bfloat16, device=dev) for w in W],
                    Wsq=torch.tensor([float((w.double() ** 2).sum()) for w in W], dtype=torch.float64, device=dev),
                    dW3=[torch.empty(d, d_ff, dtype=torch.float32, device=dev) for _ in range(L)],
                    dW1=[torch.empty(d_ff, d, dtype=torch.float32, device=dev) for _ in range(L)],
                    dW2=[torch.empty(d_ff, d, dtype=torch.float32, device=dev) for _ in range(L)],
                    ss=torch.empty(n, dtype=torch.float64, device=dev),
                    cs=torch.empty(n, dtype=torch.float32, device=dev))

    sep, fus = fresh(), fresh()
    for step in (1, 2):
        opt = api.OptConfig(kind=L_.FPO_OPT_ADAMW if adam else L_.FPO_OPT_SGD, lr=1e-2, clip_frac=clip, step=step,
                            momentum=0.9, clip_target=target)
        api.fpo_pseudograd(g, acts, dW3=sep["dW3"], dW1=sep["dW1"], dW2=sep["dW2"], sumsq=sep["ss"], **fkw)
        api.fpo_apply_update(opt, sep["dW3"] + sep["dW1"] + sep["dW2"], sep["ss"], sep["W"], sep["s1"], sep["Wsq"],
                             W_lp=sep["lp"], state2=sep["s2"], clip_scale=sep["cs"])
        api.fpo_pseudograd(g, acts, dW3=fus["dW3"], dW1=fus["dW1"], dW2=fus["dW2"], sumsq=fus["ss"], opt=opt,
                           W_master=fus["W"], W_lp=fus["lp"], state1=fus["s1"], state2=fus["s2"],
                           W_sumsq=fus["Wsq"], clip_scale=fus["cs"], **fkw)
        torch.cuda.synchronize()
        for key in ("W", "lp", "s1", "dW3", "dW1", "dW2") + (("s2",) if adam else ()):
            for i, (a, b) in enumerate(zip(sep[key], fus[key])):
                assert torch.equal(a, b), (key, i, step)
        for key in ("Wsq", "ss", "cs"):
            assert torch.equal(sep[key], fus[key]), (key, step)
    if clip < 1e-4:
        assert float(fus["cs"].max()) < 1.0  # the clip was active


@pytest.mark.parametrize("target", [0, 1], ids=["clip-grad", "clip-update"])
@pytest.mark.parametrize("kind", ["sgd", "adamw", "sgd-plain"])
@pytest.mark.parametrize("T,d,d_ff,L,clip,pffn", [(300, 264, 1000, 3, 0.01, False), (200, 1032, 1288, 3, 1e-5, False),
                                                  (300, 264, 1000, 2, 0.01, True)])
def test_fused_update_with_bf16_staged_pseudogradient(dev, kind, T, d, d_ff, L, clip, pffn, target):
    """FPO_MODE_GRAD_BF16: the fused path stages each layer's pseudogradient
    rounded to bf16 (RNE). Over two steps it is bit-identical to the separate
    calls fed the same rounded pseudogradient (the fp32 pseudogradient rounded
    by torch) and the staged call's norms; those norms are the squared norms of
    the rounded values."""
    c = I.CONFIGS[1].shrink(T=T, d=d, d_ff=d_ff, L=L)
    g = dev_tensor(I.synthetic_signal(c), dev)
    kw = {}
    if pffn:
        g32 = torch.from_numpy(I.normal(c.cid, I.T_G, 7, T * d, std=0.02).reshape(T, d)).to(dev)
        pfs = [I.post_ffn(c, l) for l in range(L)]
        kw = dict(post_ffn=api.PostFfn(g32, [dev_tensor(m, dev) for m, _ in pfs], [dev_tensor(x, dev) for _, x in pfs]))
    acts = [dev_tensor(I.activation(c, l), dev) for l in range(L)]
    W0 = [torch.from_numpy(I.master_weight(c, l)).to(dev) for l in range(L)]
    adam = kind == "adamw"
    plain = kind == "sgd-plain"

    def fresh():
        W = [w.clone() for w in W0]
        return dict(W=W, s1=None if plain else [torch.zeros_like(w) for w in W],
                    s2=[torch.zeros_like(w) for w in W] if adam else None,
                    lp=[torch.empty(w.shape, dtype=torch.bfloat16, device=dev) for w in W],
                    Wsq=torch.tensor([float((w.double() ** 2).sum()) for w in W], dtype=torch.float64, device=dev),
                    ss=torch.empty(L, dtype=torch.float64, device=dev),
                    cs=torch.empty(L, dtype=torch.float32, device=dev))

    sep, fus = fresh(), fresh()
    dW = [torch.empty(d, d_ff, dtype=torch.float32, device=dev) for _ in range(L)]
    for step in (1, 2):
        opt = api.OptConfig(kind=L_.FPO_OPT_ADAMW if adam else L_.FPO_OPT_SGD, lr=1e-2, clip_frac=clip, step=step,
                            momentum=0.0 if plain else 0.9, clip_target=target)
        api.fpo_pseudograd(g, acts, dW3=None, sumsq=fus["ss"], opt=opt, W_master=fus["W"], W_lp=fus["lp"],
                           state1=fus["s1"], state2=fus["s2"], W_sumsq=fus["Wsq"], clip_scale=fus["cs"],
                           grad_bf16=True, **kw)
        api.fpo_pseudograd(g, acts, dW3=dW, sumsq=sep["ss"], **kw)
        dWr = [x.to(torch.bfloat16).float() for x in dW]
        torch.cuda.synchronize()
        for l in range(L):
            n2 = float((dWr[l].double() ** 2).sum())
            assert abs(float(fus["ss"][l]) - n2) <= 1e-6 * n2, (l, step)
        api.fpo_apply_update(opt, dWr, fus["ss"], sep["W"], sep["s1"], sep["Wsq"], W_lp=sep["lp"],
                             state2=sep["s2"], clip_scale=sep["cs"])
        torch.cuda.synchronize()
        for key in ("W", "lp") + (("s2",) if adam else ()) + (() if plain else ("s1",)):
            for a, b in zip(sep[key], fus[key]):
                assert torch.equal(a, b), (key, step)
        for key in ("Wsq", "cs"):
            assert torch.equal(sep[key], fus[key]), (key, step)
    if clip < 1e-4:
        assert float(fus["cs"].max()) < 1.0
