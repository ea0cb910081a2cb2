"""GPU parity of fpo_pseudograd against the fp64 oracle: per-layer outer
products dW3 = (1/T) g~^T a, their squared norms, the fused diagnostic cosine
terms, and the full-MLP W1/W2 signals through W3_init."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_14563_amd import _lib as L_
from paper_2608_14563_amd import api
from paper_2608_14563_amd import inputs as I
from tests._util import assert_close, bf16_rne_bits, dev_tensor, host64, ulp_diff_f32

pytestmark = pytest.mark.gpu


def signal(c, std=0.02):
    return I.synthetic_signal(c, std=std)


def run_w3(c, g, acts, dev, refs=None, store=True):
    T, d = g.shape
    tg = dev_tensor(g, dev)
    ta = [dev_tensor(a, dev) for a in acts]
    dW = [torch.empty(d, c.d_ff, dtype=torch.float32, device=dev) for _ in acts] if store else None
    ss = torch.full((len(acts),), -1.0, dtype=torch.float64, device=dev)
    kw = {}
    if refs is not None:
        kw = dict(ref=[dev_tensor(r, dev) for r in refs], ref_dot=torch.empty(len(acts), dtype=torch.float64, device=dev),
                  ref_sumsq=torch.empty(len(acts), dtype=torch.float64, device=dev),
                  ref_cos=torch.full((len(acts),), -7.0, dtype=torch.float32, device=dev))
    api.fpo_pseudograd(tg, ta, dW3=dW, sumsq=ss, **kw)
    torch.cuda.synchronize()
    out = dict(sumsq=ss.cpu().numpy())
    if dW is not None:
        out["dW"] = [w.cpu().numpy().astype(np.float64) for w in dW]
    if refs is not None:
        out["dot"] = kw["ref_dot"].cpu().numpy()
        out["refsq"] = kw["ref_sumsq"].cpu().numpy()
        out["cos"] = kw["ref_cos"].cpu().numpy()
    return out


# (1, 256, 256, 512, 2) and (1, 512, 512, 768, 3): whole tiles (copy form without bounds)
@pytest.mark.parametrize("cid,T,d,d_ff,L", [(0, 128, 256, 688, 2), (0, 300, 264, 520, 3), (1, 300, 264, 520, 2),
                                            (1, 1000, 512, 1032, 2), (1, 1, 256, 512, 1), (3, 333, 256, 1000, 2),
                                            (1, 256, 256, 512, 2), (1, 512, 512, 768, 3)])
def test_w3_outer_products(dev, cid, T, d, d_ff, L):
    c = I.CONFIGS[cid].shrink(T=T, d=d, d_ff=d_ff, L=L)
    g = signal(c)
    acts = [I.activation(c, l) for l in range(L)]
    got = run_w3(c, g, acts, dev)
    for l in range(L):
        D = O.pseudograd(g, acts[l])
        assert_close(f"dW[{l}]", got["dW"][l], D, c.dtype)
        assert_close(f"sumsq[{l}]", got["sumsq"][l], float((D * D).sum()), c.dtype)
        # the reported norm is the norm of the stored matrix
        assert abs(got["sumsq"][l] - float((got["dW"][l] ** 2).sum())) <= 1e-5 * got["sumsq"][l]


@pytest.mark.parametrize("cid", [0, 4])
def test_fused_diagnostic_cosine(dev, cid):
    c = I.CONFIGS[cid].shrink(T=256, d=256, d_ff=512, L=3)
    g = signal(c)
    acts = [I.activation(c, l) for l in range(3)]
    refs = []
    for l in range(3):
        D = O.pseudograd(g, acts[l])
        sigma = np.sqrt(3.0) * np.linalg.norm(D) / np.sqrt(D.size)
        refs.append((D + sigma * I.ref_noise(c, l)).astype(np.float32))
    with_store = run_w3(c, g, acts, dev, refs=refs)
    fused = run_w3(c, g, acts, dev, refs=refs, store=False)
    for l in range(3):
        D = O.pseudograd(g, acts[l])
        dot, na, nb, cs = O.cosine(D, refs[l])
        for out in (with_store, fused):
            assert_close("dot", out["dot"][l], dot, c.dtype)
            assert_close("refsq", out["refsq"][l], nb, "f32")
            assert_close("sumsq", out["sumsq"][l], na, c.dtype)
            cg = out["dot"][l] / np.sqrt(out["sumsq"][l] * out["refsq"][l])
            assert abs(cg - cs) <= 1e-3
            assert abs(cs - 0.5) < 0.05
            # the library's own cosine: the same float64 sums, rounded once to float32
            assert abs(float(out["cos"][l]) - cg) <= 1e-6 * abs(cg) + 1e-7
            assert abs(float(out["cos"][l]) - cs) <= 1e-3
        assert np.array_equal(with_store["dot"], fused["dot"])


@pytest.mark.parametrize("cid,T,d,d_ff,L", [(0, 128, 256, 688, 2), (1, 200, 256, 520, 2), (1, 256, 256, 512, 2)])
def test_full_mlp(dev, cid, T, d, d_ff, L):
    c = I.CONFIGS[cid].shrink(T=T, d=d, d_ff=d_ff, L=L)
    g = signal(c)
    caches = [I.mlp_cache(c, l) for l in range(L)]
    extras = [I.full_mlp_extra(c, l) for l in range(L)]
    W3i = [I.to_storage(I.master_weight(c, l), c.dtype) for l in range(L)]
    tg = dev_tensor(g, dev)
    dW3 = [torch.empty(d, d_ff, dtype=torch.float32, device=dev) for _ in range(L)]
    dW1 = [torch.empty(d_ff, d, dtype=torch.float32, device=dev) for _ in range(L)]
    dW2 = [torch.empty(d_ff, d, dtype=torch.float32, device=dev) for _ in range(L)]
    ss = torch.empty(3 * L, dtype=torch.float64, device=dev)
    api.fpo_pseudograd(tg, [dev_tensor(cc[2], dev) for cc in caches], dW3=dW3, sumsq=ss,
                       W3_init=[dev_tensor(w, dev) for w in W3i], gate=[dev_tensor(cc[0], dev) for cc in caches],
                       up=[dev_tensor(cc[1], dev) for cc in caches], x_in=[dev_tensor(e[0], dev) for e in extras],
                       dW1=dW1, dW2=dW2)
    torch.cuda.synchronize()
    s = ss.cpu().numpy()
    for l in range(L):
        q, u, a = caches[l]
        D1, D2 = O.full_mlp_grads(g, W3i[l], q, u, extras[l][0])
        D3 = O.pseudograd(g, a)
        assert_close("dW3", host64(dW3[l]), D3, c.dtype)
        assert_close("dW1", host64(dW1[l]), D1, c.dtype)
        assert_close("dW2", host64(dW2[l]), D2, c.dtype)
        assert_close("sumsq W1", s[L + l], float((D1 ** 2).sum()), c.dtype)
        assert_close("sumsq W2", s[2 * L + l], float((D2 ** 2).sum()), c.dtype)


@pytest.mark.slow
@pytest.mark.parametrize("cid,L", [(1, 8), (3, 3)], ids=["olmo2-7b-8-layers", "falcon3-7b-3-layers"])
def test_full_size_full_mlp(dev, cid, L):
    """Full-MLP mode (eq. errh) at the 7-8B shapes: OLMo-2 with all 8 target
    layers, Falcon3 (d_ff 23040, the widest operand bands of the error GEMM
    and its transposed dq / du stores) with 3. Per layer, 66 sampled rows of
    dW1 and dW2 (all d columns; at Falcon3 shapes half of them outlier
    channels) against oracle.full_mlp_grads on those d_ff columns of W3_init,
    q and u, sampled columns of dW3 against oracle.pseudograd, and for the
    first and last layer the reported squared norms against the oracle's
    full matrices."""
    c = I.CONFIGS[cid].shrink(L=L)
    g = signal(c)
    caches = [I.mlp_cache(c, l) for l in range(L)]
    extras = [I.full_mlp_extra(c, l) for l in range(L)]
    W3i = [I.to_storage(I.master_weight(c, l), c.dtype) for l in range(L)]
    dW3 = [torch.empty(c.d, c.d_ff, dtype=torch.float32, device=dev) for _ in range(L)]
    dW1 = [torch.empty(c.d_ff, c.d, dtype=torch.float32, device=dev) for _ in range(L)]
    dW2 = [torch.empty(c.d_ff, c.d, dtype=torch.float32, device=dev) for _ in range(L)]
    ss = torch.empty(3 * L, dtype=torch.float64, device=dev)
    print(f"[pg] full-size full-MLP config {cid} L={L}", flush=True)
    api.fpo_pseudograd(dev_tensor(g, dev), [dev_tensor(cc[2], dev) for cc in caches], dW3=dW3, sumsq=ss,
                       W3_init=[dev_tensor(w, dev) for w in W3i], gate=[dev_tensor(cc[0], dev) for cc in caches],
                       up=[dev_tensor(cc[1], dev) for cc in caches], x_in=[dev_tensor(e[0], dev) for e in extras],
                       dW1=dW1, dW2=dW2)
    torch.cuda.synchronize()
    gf = I.storage_to_f64(g)
    r = np.random.default_rng(500 + cid)
    for l in range(L):
        q, u, a = caches[l]
        x_in = extras[l][0]
        rows = [r.integers(0, c.d_ff, 64), [0, c.d_ff - 1]]
        if c.outliers:
            rows.append(I.outlier_channels(c, l)[:64])
        ii = np.concatenate(rows)
        D1s, D2s = O.full_mlp_grads(gf, W3i[l][:, ii], q[:, ii], u[:, ii], x_in)
        assert_close(f"dW1[{l}] rows", dW1[l][ii].cpu().numpy().astype(np.float64), D1s, "bf16")
        assert_close(f"dW2[{l}] rows", dW2[l][ii].cpu().numpy().astype(np.float64), D2s, "bf16")
        jj = np.concatenate([r.integers(0, c.d_ff, 64), [c.d_ff - 1, 0]])
        D3s = O.pseudograd(gf, a[:, jj])
        assert_close(f"dW3[{l}] columns", dW3[l][:, jj].cpu().numpy().astype(np.float64), D3s, "bf16")
        if l in (0, L - 1):
            D1, D2 = O.full_mlp_grads(gf, W3i[l], q, u, x_in)
            assert_close(f"sumsq W1[{l}]", float(ss[L + l]), float(np.sum(D1 * D1)), "bf16")
            assert_close(f"sumsq W2[{l}]", float(ss[2 * L + l]), float(np.sum(D2 * D2)), "bf16")
            del D1, D2


def test_deterministic(dev):
    c = I.CONFIGS[1].shrink(T=700, d=512, d_ff=1024, L=2)
    g = signal(c)
    acts = [I.activation(c, l) for l in range(2)]
    a = run_w3(c, g, acts, dev)
    b = run_w3(c, g, acts, dev)
    assert np.array_equal(a["sumsq"], b["sumsq"])
    for x, y in zip(a["dW"], b["dW"]):
        assert np.array_equal(x, y)


def oracle_layer(gf, act):
    """The oracle's pseudogradient of one layer at full size (float64 on the
    host: 2 T d d_ff flops through BLAS) and its squared Frobenius norm."""
    D = O.pseudograd(gf, act)
    return D, float(np.sum(D * D))


@pytest.mark.slow
@pytest.mark.parametrize("cid", [1, 2, 3])
def test_full_size_w3(dev, cid):
    """Full workload shapes: every layer's whole dW against oracle.pseudograd
    and its reported squared norm against the oracle's."""
    c = I.CONFIGS[cid]
    g = signal(c)
    tg = dev_tensor(g, dev)
    acts = [I.activation(c, l) for l in range(c.L)]
    ta = [dev_tensor(a, dev) for a in acts]
    dW = [torch.empty(c.d, c.d_ff, dtype=torch.float32, device=dev) for _ in range(c.L)]
    ss = torch.empty(c.L, dtype=torch.float64, device=dev)
    print(f"[pg] full-size W3 config {cid}", flush=True)
    api.fpo_pseudograd(tg, ta, dW3=dW, sumsq=ss)
    torch.cuda.synchronize()
    gf = I.storage_to_f64(g)
    for l in range(c.L):
        D, n2 = oracle_layer(gf, acts[l])
        assert_close(f"dW[{l}]", host64(dW[l]), D, "bf16")
        assert_close(f"sumsq[{l}]", float(ss[l]), n2, "bf16")
        del D


@pytest.mark.slow
@pytest.mark.parametrize("cid,stage", [(1, False), (2, False), (3, False), (1, True), (2, True), (3, True)])
def test_full_size_fused_update(dev, cid, stage):
    """The benchmark's launch configuration at full size: pseudogradient with
    the SGD-momentum step overlapped (first step), its pseudogradient returned
    in fp32 or staged in bf16 (FPO_MODE_GRAD_BF16). For every layer: the
    reported ||dW||^2 against the oracle's ||D||^2, the clip factor against
    the oracle's clip of D, the whole momentum buffer against the oracle's
    clipped pseudogradient s * D, W' within one ulp of fp32(W - lr * b) from
    the GPU's momentum and its bf16 copy exactly RNE of W'."""
    c = I.CONFIGS[cid]
    g = signal(c)
    acts = [I.activation(c, l) for l in range(c.L)]
    Wh = [I.master_weight(c, l) for l in range(c.L)]
    tg = dev_tensor(g, dev)
    ta = [dev_tensor(a, dev) for a in acts]
    W = [torch.from_numpy(w).to(dev) for w in Wh]
    wsq = np.array([float((w.astype(np.float64) ** 2).sum()) for w in Wh])
    Wsq = torch.tensor(wsq, dtype=torch.float64, device=dev)
    s1 = [torch.zeros_like(w) for w in W]
    lp = [torch.empty(w.shape, dtype=torch.bfloat16, device=dev) for w in W]
    dW = [torch.empty(c.d, c.d_ff, dtype=torch.float32, device=dev) for _ in range(c.L)]
    ss = torch.empty(c.L, dtype=torch.float64, device=dev)
    cs = torch.empty(c.L, dtype=torch.float32, device=dev)
    opt = api.OptConfig(lr=c.lr, clip_frac=c.clip_frac, step=1)
    print(f"[pg] full-size fused update config {cid} staged={stage}", flush=True)
    api.fpo_pseudograd(tg, ta, dW3=None if stage else dW, sumsq=ss, opt=opt, W_master=W, W_lp=lp, state1=s1,
                       W_sumsq=Wsq, clip_scale=cs, grad_bf16=stage)
    torch.cuda.synchronize()
    gf = I.storage_to_f64(g)
    active = 0
    for l in range(c.L):
        D, n2 = oracle_layer(gf, acts[l])
        assert_close(f"sumsq[{l}]", float(ss[l]), n2, "bf16")
        assert abs(float(ss[l]) - n2) <= 1e-4 * n2, (l, float(ss[l]), n2)
        s = O.clip_scale(n2, wsq[l], c.clip_frac)
        active += s < 1.0
        assert abs(float(cs[l]) - s) <= 1e-4 * s, (l, float(cs[l]), s)
        m = s1[l].cpu().numpy()
        assert_close(f"momentum[{l}]", m.astype(np.float64), s * D, "bf16")
        if not stage:
            assert_close(f"dW[{l}]", host64(dW[l]), D, "bf16")
        del D
        w_new = W[l].cpu().numpy()
        # the kernel's single-rounding fma(-lr, b, W): the product of two floats is
        # exact in float64, so W - lr b there is within one float64 rounding
        w_exp = (Wh[l].astype(np.float64) - np.float64(np.float32(c.lr)) * m.astype(np.float64)).astype(np.float32)
        assert np.all(ulp_diff_f32(w_new, w_exp) <= 1), l
        lpv = lp[l].view(torch.int16).cpu().numpy().view(np.uint16)
        assert np.array_equal(lpv, bf16_rne_bits(w_new)), l
    # the workload's clip is active on the OLMo-2 and Falcon3 shapes (||D|| / ||W|| ~ 1.3% and 2.1%)
    if cid in (1, 3):
        assert active == c.L, active
    # ||W'||^2 reported for the next step's clip
    for l in (0, c.L - 1):
        wn = W[l].double()
        assert abs(float(Wsq[l]) - float((wn * wn).sum())) <= 1e-9 * float(Wsq[l])


@pytest.mark.slow
@pytest.mark.parametrize("cid", [1, 3])
def test_full_size_fused_adamw(dev, cid):
    """AdamW in the benchmark's launch configuration (--optimizer adamw): the
    bf16-staged pseudogradient, the step overlapped with the next layer's
    outer products, first step. Per layer: the reported ||dW||^2 and the clip
    factor against the oracle's, both moments in full against the oracle's
    AdamW on its clipped pseudogradient s * D; W' (sampled) against the
    kernel's float32 formula applied to the GPU's own moments (a few ulp: the
    step ~ lr sign(D) makes the oracle's W' sensitive to near-zero D); the
    bf16 copy exactly RNE of W'; the reported ||W'||^2."""
    c = I.CONFIGS[cid]
    g = signal(c)
    acts = [I.activation(c, l) for l in range(c.L)]
    Wh = [I.master_weight(c, l) for l in range(c.L)]
    W = [torch.from_numpy(w).to(dev) for w in Wh]
    wsq = np.array([float((w.astype(np.float64) ** 2).sum()) for w in Wh])
    Wsq = torch.tensor(wsq, dtype=torch.float64, device=dev)
    m1 = [torch.zeros_like(w) for w in W]
    m2 = [torch.zeros_like(w) for w in W]
    lp = [torch.empty(w.shape, dtype=torch.bfloat16, device=dev) for w in W]
    ss = torch.empty(c.L, dtype=torch.float64, device=dev)
    cs = torch.empty(c.L, dtype=torch.float32, device=dev)
    opt = api.OptConfig(kind=L_.FPO_OPT_ADAMW, lr=c.lr, clip_frac=c.clip_frac, step=1)
    print(f"[pg] full-size AdamW config {cid}", flush=True)
    api.fpo_pseudograd(dev_tensor(g, dev), [dev_tensor(a, dev) for a in acts], dW3=None, sumsq=ss, opt=opt,
                       W_master=W, W_lp=lp, state1=m1, state2=m2, W_sumsq=Wsq, clip_scale=cs, grad_bf16=True)
    torch.cuda.synchronize()
    gf = I.storage_to_f64(g)
    f32 = lambda v: np.float64(np.float32(v))  # noqa: E731
    r = np.random.default_rng(200 + cid)
    for l in range(c.L):
        Df, n2 = oracle_layer(gf, acts[l])
        assert abs(float(ss[l]) - n2) <= 1e-4 * n2, (l, float(ss[l]), n2)
        s = O.clip_scale(n2, wsq[l], c.clip_frac)
        assert abs(float(cs[l]) - s) <= 1e-4 * s, (l, float(cs[l]), s)
        _, om_f, ov_f = O.adamw(Wh[l], 0.0, 0.0, s * Df, opt.lr, 1, opt.beta1, opt.beta2, opt.adam_eps,
                                opt.weight_decay)
        del Df
        assert_close(f"exp_avg[{l}]", m1[l].cpu().numpy().astype(np.float64), om_f, "bf16")
        assert_close(f"exp_avg_sq[{l}]", m2[l].cpu().numpy().astype(np.float64), ov_f, "bf16")
        del om_f, ov_f
        ii = np.concatenate([r.integers(0, c.d, 64), [0, c.d - 1]])
        jj = np.concatenate([r.integers(0, c.d_ff, 64), [c.d_ff - 1, 0]])
        w0 = Wh[l][ii, jj].astype(np.float64)
        mg = m1[l][ii, jj].cpu().numpy().astype(np.float64)
        vg = m2[l][ii, jj].cpu().numpy().astype(np.float64)
        step = f32(opt.lr) * (mg * f32(1.0 / (1.0 - opt.beta1))) / (
            np.sqrt(vg) * f32(1.0 / np.sqrt(1.0 - opt.beta2)) + f32(opt.adam_eps))
        expect = w0 * f32(1.0 - opt.lr * opt.weight_decay) - step
        wg = W[l][ii, jj].cpu().numpy()
        tol = 2 * np.spacing(np.abs(expect).astype(np.float32)).astype(np.float64) + 8 * 2.0 ** -23 * np.abs(step)
        assert np.all(np.abs(wg.astype(np.float64) - expect) <= tol), l
        lpv = lp[l][ii, jj].view(torch.int16).cpu().numpy().view(np.uint16)
        assert np.array_equal(lpv, bf16_rne_bits(wg)), l
    for l in (0, c.L - 1):
        wn = W[l].double()
        assert abs(float(Wsq[l]) - float((wn * wn).sum())) <= 1e-9 * float(Wsq[l])


@pytest.mark.slow
@pytest.mark.parametrize("lr", [None, 2.0], ids=["workload-lr", "lr2-clip-active"])
def test_full_size_fused_update_clip(dev, lr):
    """The clip-the-update reading at full size (--clip-target update, OLMo-2
    shapes, bf16-staged pseudogradient): SGD-momentum state advances on the
    unclipped pseudogradient (the whole buffer against the oracle's D), the
    applied step -lr b is scaled by s = min(1, 0.01 ||W|| / ||lr b||), checked
    against the oracle's clip-the-update step on its own D, and W' equals
    W + s (-lr b) from the GPU's state within fp32 rounding. At the
    workload's lr (1e-4) the bound is idle (s = 1); lr = 2 makes it bite on
    every layer."""
    c = I.CONFIGS[1]
    g = signal(c)
    acts = [I.activation(c, l) for l in range(c.L)]
    Wh = [I.master_weight(c, l) for l in range(c.L)]
    W = [torch.from_numpy(w).to(dev) for w in Wh]
    wsq = np.array([float((w.astype(np.float64) ** 2).sum()) for w in Wh])
    Wsq = torch.tensor(wsq, dtype=torch.float64, device=dev)
    b1 = [torch.zeros_like(w) for w in W]
    lp = [torch.empty(w.shape, dtype=torch.bfloat16, device=dev) for w in W]
    ss = torch.empty(c.L, dtype=torch.float64, device=dev)
    cs = torch.empty(c.L, dtype=torch.float32, device=dev)
    lr = c.lr if lr is None else lr
    opt = api.OptConfig(lr=lr, clip_frac=c.clip_frac, step=1, clip_target=L_.FPO_CLIP_UPDATE)
    print(f"[pg] full-size clip-the-update lr={lr}", flush=True)
    api.fpo_pseudograd(dev_tensor(g, dev), [dev_tensor(a, dev) for a in acts], dW3=None, sumsq=ss, opt=opt,
                       W_master=W, W_lp=lp, state1=b1, W_sumsq=Wsq, clip_scale=cs, grad_bf16=True)
    torch.cuda.synchronize()
    gf = I.storage_to_f64(g)
    f32 = lambda v: np.float64(np.float32(v))  # noqa: E731
    r = np.random.default_rng(300)
    for l in range(c.L):
        Df, _ = oracle_layer(gf, acts[l])
        _, ob, s = O.sgd_momentum_update_clip(Wh[l], None, Df, lr, 0.9, step=1, frac=c.clip_frac)
        del Df
        assert abs(float(cs[l]) - s) <= 1e-4 * s, (l, float(cs[l]), s)
        assert (s < 1.0) == (lr > 1.0), (l, s)
        assert_close(f"momentum[{l}]", b1[l].cpu().numpy().astype(np.float64), ob, "bf16")  # unclipped state
        del ob
        ii = np.concatenate([r.integers(0, c.d, 64), [0, c.d - 1]])
        jj = np.concatenate([r.integers(0, c.d_ff, 64), [c.d_ff - 1, 0]])
        bg = b1[l][ii, jj].cpu().numpy().astype(np.float64)
        w0 = Wh[l][ii, jj].astype(np.float64)
        delta = -f32(lr) * bg
        expect = w0 + float(cs[l]) * delta
        wg = W[l][ii, jj].cpu().numpy()
        tol = 2 * np.spacing(np.abs(expect).astype(np.float32)).astype(np.float64) + 4 * 2.0 ** -23 * np.abs(delta)
        assert np.all(np.abs(wg.astype(np.float64) - expect) <= tol), l
        lpv = lp[l][ii, jj].view(torch.int16).cpu().numpy().view(np.uint16)
        assert np.array_equal(lpv, bf16_rne_bits(wg)), l
        # the whole applied step respects the bound
        dW = W[l].double() - torch.from_numpy(Wh[l]).to(dev).double()
        assert float(torch.linalg.norm(dW)) <= c.clip_frac * np.sqrt(wsq[l]) * (1 + 1e-4)


@pytest.mark.slow
def test_full_size_diagnostic_rank1_reference(dev):
    """Diagnostic workload at full size (T = 8192, Qwen3-8B shapes, 36 layers):
    the fused cosine terms against a rank-1 reference R = u v^T, for which
    <D_l, R> = (1/T) sum_t (u . g~_t)(a_lt . v) and ||R||^2 = |u|^2 |v|^2 are
    exact closed forms at any size; sampled dW entries of every layer. Layers
    cycle through four seeded activations (the kernels see 36 matrices; the
    host generates four)."""
    c = I.CONFIGS[4]
    nd = 4
    g = signal(c)
    distinct = [I.activation(c, l) for l in range(nd)]
    tg = dev_tensor(g, dev)
    td = [dev_tensor(a, dev) for a in distinct]
    ta = [td[l % nd] for l in range(c.L)]
    u, v = I.rank1_reference(c)
    R = torch.outer(torch.from_numpy(u).to(dev), torch.from_numpy(v).to(dev)).contiguous()
    dW = [torch.empty(c.d, c.d_ff, dtype=torch.float32, device=dev) for _ in range(c.L)]
    ss = torch.empty(c.L, dtype=torch.float64, device=dev)
    dot = torch.empty(c.L, dtype=torch.float64, device=dev)
    rsq = torch.empty(c.L, dtype=torch.float64, device=dev)
    cosl = torch.empty(c.L, dtype=torch.float32, device=dev)
    api.fpo_pseudograd(tg, ta, dW3=dW, sumsq=ss, ref=[R] * c.L, ref_dot=dot, ref_sumsq=rsq, ref_cos=cosl)
    torch.cuda.synchronize()
    gf = I.storage_to_f64(g)
    ug = gf @ u.astype(np.float64)                      # u . g~_t
    Rf = R.double()
    rsq_exact = float((Rf * Rf).sum())                  # of the fp32-rounded R
    assert abs(float(rsq_exact) - float(np.dot(u, u)) * float(np.dot(v, v))) <= 1e-5 * rsq_exact
    r = np.random.default_rng(4)
    for k in range(nd):
        af = I.storage_to_f64(distinct[k])
        dot_exact = float(ug @ (af @ v.astype(np.float64))) / c.T
        ii = np.concatenate([r.integers(0, c.d, 64), [0, c.d - 1]])
        jj = np.concatenate([r.integers(0, c.d_ff, 64), [c.d_ff - 1, 0]])
        D = np.einsum("ti,ti->i", gf[:, ii], af[:, jj]) / c.T
        for l in range(k, c.L, nd):
            assert_close(f"dot[{l}]", float(dot[l]), dot_exact, "bf16")
            assert abs(float(rsq[l]) - rsq_exact) <= 1e-6 * rsq_exact
            assert_close(f"dW[{l}] samples", dW[l][ii, jj].cpu().numpy().astype(np.float64), D, "bf16")
            # the reported norm is that of the stored matrix (layers of one activation agree exactly)
            assert float(ss[l]) == float(ss[k])
            cg = float(dot[l]) / np.sqrt(float(ss[l]) * float(rsq[l]))
            assert abs(float(cosl[l]) - cg) <= 1e-6 * abs(cg) + 1e-7
        del af


def pffn_case(c, L):
    """fp32 g~ [T, d] and each layer's (mlp_out, gamma_pffn) storage arrays."""
    g32 = I.normal(c.cid, I.T_G, 7, c.T * c.d, std=0.02).reshape(c.T, c.d)
    return g32, [I.post_ffn(c, l) for l in range(L)]


def run_pffn(c, g32, pf, acts, dev, extra=None, **kw):
    tg = torch.from_numpy(g32).to(dev)
    mo = [dev_tensor(m, dev) for m, _ in pf]
    gm = [dev_tensor(g, dev) for _, g in pf]
    ta = [dev_tensor(a, dev) for a in acts]
    dW = [torch.empty(c.d, c.d_ff, dtype=torch.float32, device=dev) for _ in acts]
    ss = torch.empty(len(acts) * (3 if extra else 1), dtype=torch.float64, device=dev)
    args = dict(dW3=dW, sumsq=ss, post_ffn=api.PostFfn(tg, mo, gm, c.eps, c.min_rms), **kw)
    if extra is not None:
        args.update(extra(dev))
    api.fpo_pseudograd(None, ta, **args)
    torch.cuda.synchronize()
    return dW, ss, args


@pytest.mark.parametrize("cid,T,d,d_ff,L", [(0, 128, 256, 688, 2), (0, 300, 264, 520, 3), (1, 300, 264, 520, 2),
                                            (1, 1000, 512, 1032, 2)])
def test_post_ffn_w3(dev, cid, T, d, d_ff, L):
    """Post-feedforward RMSNorm composition (per-layer left operands, 1% of
    tokens below the min-RMS floor) against the oracle."""
    c = I.CONFIGS[cid].shrink(T=T, d=d, d_ff=d_ff, L=L)
    g32, pf = pffn_case(c, L)
    acts = [I.activation(c, l) for l in range(L)]
    dW, ss, _ = run_pffn(c, g32, pf, acts, dev)
    for l in range(L):
        gl = O.post_ffn_signal(g32, pf[l][0], pf[l][1], eps=c.eps, min_rms=c.min_rms)
        D = O.pseudograd(gl, acts[l])
        assert_close(f"dW[{l}] (post-FFN)", host64(dW[l]), D, c.dtype)
        assert_close(f"sumsq[{l}]", float(ss[l]), float((D * D).sum()), c.dtype)
        # the composition matters here: skipping it is far outside the tolerance
        assert np.linalg.norm(O.pseudograd(g32, acts[l]) - D) > 0.2 * np.linalg.norm(D)


@pytest.mark.parametrize("cid,T,d,d_ff,L", [(0, 128, 256, 688, 2), (1, 200, 256, 520, 2)])
def test_post_ffn_full_mlp(dev, cid, T, d, d_ff, L):
    c = I.CONFIGS[cid].shrink(T=T, d=d, d_ff=d_ff, L=L)
    g32, pf = pffn_case(c, L)
    caches = [I.mlp_cache(c, l) for l in range(L)]
    extras = [I.full_mlp_extra(c, l) for l in range(L)]
    W3i = [I.master_weight(c, l) for l in range(L)]
    store = {}

    def extra(dev):
        op = dev_tensor(caches[0][2], dev).dtype
        store["dW1"] = [torch.empty(c.d_ff, c.d, dtype=torch.float32, device=dev) for _ in range(L)]
        store["dW2"] = [torch.empty(c.d_ff, c.d, dtype=torch.float32, device=dev) for _ in range(L)]
        return dict(W3_init=[dev_tensor(I.to_storage(w, c.dtype), dev) for w in W3i],
                    gate=[dev_tensor(q, dev) for q, _, _ in caches], up=[dev_tensor(u, dev) for _, u, _ in caches],
                    x_in=[dev_tensor(e[0], dev) for e in extras], dW1=store["dW1"], dW2=store["dW2"])

    dW3, ss, _ = run_pffn(c, g32, pf, [a for _, _, a in caches], dev, extra=extra)
    for l in range(L):
        gl = O.post_ffn_signal(g32, pf[l][0], pf[l][1], eps=c.eps, min_rms=c.min_rms)
        q, u, a = caches[l]
        D1, D2 = O.full_mlp_grads(gl, I.to_storage(W3i[l], c.dtype), q, u, extras[l][0])
        assert_close("dW3", host64(dW3[l]), O.pseudograd(gl, a), c.dtype)
        assert_close("dW1", host64(store["dW1"][l]), D1, c.dtype)
        assert_close("dW2", host64(store["dW2"][l]), D2, c.dtype)
        assert_close("sumsq W1", float(ss[L + l]), float((D1 ** 2).sum()), c.dtype)


def run_chain(c, g32, acts, dev, pf=None, pre=None, extra=None, **kw):
    """fpo_pseudograd with the post-FFN (pf) and / or pre-MLP (pre) composition."""
    tg = torch.from_numpy(g32).to(dev)
    ta = [dev_tensor(a, dev) for a in acts]
    dW = [torch.empty(c.d, c.d_ff, dtype=torch.float32, device=dev) for _ in acts]
    ss = torch.empty(len(acts) * (3 if extra else 1), dtype=torch.float64, device=dev)
    args = dict(dW3=dW, sumsq=ss, **kw)
    if pf is not None:
        args["post_ffn"] = api.PostFfn(tg, [dev_tensor(m, dev) for m, _ in pf], [dev_tensor(g, dev) for _, g in pf],
                                       c.eps, c.min_rms)
    if pre is not None:
        args["pre_mlp"] = api.PreMlp(tg, [dev_tensor(x, dev) for x, _ in pre], [dev_tensor(g, dev) for _, g in pre],
                                     c.eps, c.min_rms)
    if extra is not None:
        args.update(extra(dev))
    api.fpo_pseudograd(None, ta, **args)
    torch.cuda.synchronize()
    return dW, ss, args


@pytest.mark.parametrize("post", [False, True], ids=["pre-MLP", "post-FFN+pre-MLP"])
@pytest.mark.parametrize("cid,T,d,d_ff,L", [(0, 128, 256, 688, 2), (0, 300, 264, 520, 3), (1, 300, 264, 520, 2),
                                            (1, 1000, 512, 1032, 2)])
def test_pre_mlp_w3(dev, cid, T, d, d_ff, L, post):
    """Pre-MLP RMSNorm composition (Qwen3 layout; with the post-FFN one first,
    the Gemma 3 layout): each layer's left operand is oracle.layer_signal of
    the fp32 g~, 1% of tokens below the min-RMS floor in each norm."""
    c = I.CONFIGS[cid].shrink(T=T, d=d, d_ff=d_ff, L=L)
    g32, pf = pffn_case(c, L)
    pre = [I.pre_mlp(c, l) for l in range(L)]
    acts = [I.activation(c, l) for l in range(L)]
    dW, ss, _ = run_chain(c, g32, acts, dev, pf=pf if post else None, pre=pre)
    for l in range(L):
        gl = O.layer_signal(g32, pf[l][0] if post else None, pf[l][1] if post else None, pre[l][0], pre[l][1],
                            eps=c.eps, min_rms=c.min_rms)
        D = O.pseudograd(gl, acts[l])
        assert_close(f"dW[{l}] (pre-MLP)", host64(dW[l]), D, c.dtype)
        assert_close(f"sumsq[{l}]", float(ss[l]), float((D * D).sum()), c.dtype)
        # the composition matters: skipping the pre-MLP VJP is far outside the tolerance
        g0 = O.layer_signal(g32, pf[l][0] if post else None, pf[l][1] if post else None, eps=c.eps,
                            min_rms=c.min_rms)
        assert np.linalg.norm(O.pseudograd(g0, acts[l]) - D) > 0.2 * np.linalg.norm(D)


@pytest.mark.parametrize("cid,T,d,d_ff,L", [(0, 128, 256, 688, 2), (1, 200, 256, 520, 2)])
def test_pre_mlp_full_mlp(dev, cid, T, d, d_ff, L):
    """Full-MLP mode with both norms composed: W1 / W2 through W3_init take
    the composed signal too."""
    c = I.CONFIGS[cid].shrink(T=T, d=d, d_ff=d_ff, L=L)
    g32, pf = pffn_case(c, L)
    pre = [I.pre_mlp(c, l) for l in range(L)]
    caches = [I.mlp_cache(c, l) for l in range(L)]
    extras = [I.full_mlp_extra(c, l) for l in range(L)]
    W3i = [I.to_storage(I.master_weight(c, l), c.dtype) for l in range(L)]
    store = {}

    def extra(dev):
        store["dW1"] = [torch.empty(c.d_ff, c.d, dtype=torch.float32, device=dev) for _ in range(L)]
        store["dW2"] = [torch.empty(c.d_ff, c.d, dtype=torch.float32, device=dev) for _ in range(L)]
        return dict(W3_init=[dev_tensor(w, dev) for w in W3i], gate=[dev_tensor(q, dev) for q, _, _ in caches],
                    up=[dev_tensor(u, dev) for _, u, _ in caches], x_in=[dev_tensor(e[0], dev) for e in extras],
                    dW1=store["dW1"], dW2=store["dW2"])

    dW3, ss, _ = run_chain(c, g32, [a for _, _, a in caches], dev, pf=pf, pre=pre, extra=extra)
    for l in range(L):
        gl = O.layer_signal(g32, pf[l][0], pf[l][1], pre[l][0], pre[l][1], eps=c.eps, min_rms=c.min_rms)
        q, u, a = caches[l]
        D1, D2 = O.full_mlp_grads(gl, W3i[l], q, u, extras[l][0])
        assert_close("dW3", host64(dW3[l]), O.pseudograd(gl, a), c.dtype)
        assert_close("dW1", host64(store["dW1"][l]), D1, c.dtype)
        assert_close("dW2", host64(store["dW2"][l]), D2, c.dtype)
        assert_close("sumsq W2", float(ss[2 * L + l]), float((D2 ** 2).sum()), c.dtype)


@pytest.mark.slow
def test_full_size_pre_mlp_fused_update(dev):
    """Qwen3-8B shapes (a pre-MLP-norm family) at full size with the pre-MLP
    composition and the overlapped SGD-momentum step: the composed signal
    against oracle.layer_signal in full, sampled columns of every layer's
    momentum against the oracle's clipped s * D (s from the oracle's norm of
    those layers' full D for the first and last layer)."""
    c = I.CONFIGS[2]
    g32 = I.normal(c.cid, I.T_G, 7, c.T * c.d, std=0.02).reshape(c.T, c.d)
    pre = [I.pre_mlp(c, l) for l in range(c.L)]
    acts = [I.activation(c, l) for l in range(c.L)]
    Wh = [I.master_weight(c, l) for l in range(c.L)]
    W = [torch.from_numpy(w).to(dev) for w in Wh]
    wsq = np.array([float((w.astype(np.float64) ** 2).sum()) for w in Wh])
    s1 = [torch.zeros_like(w) for w in W]
    cs = torch.empty(c.L, dtype=torch.float32, device=dev)
    print("[pg] full-size pre-MLP fused update (Qwen3-8B shapes)", flush=True)
    dW, ss, _ = run_chain(c, g32, acts, dev, pre=pre,
                          opt=api.OptConfig(lr=c.lr, clip_frac=c.clip_frac, step=1), W_master=W,
                          W_lp=[torch.empty(w.shape, dtype=torch.bfloat16, device=dev) for w in W], state1=s1,
                          W_sumsq=torch.tensor(wsq, dtype=torch.float64, device=dev), clip_scale=cs)
    r = np.random.default_rng(8)
    for l in range(c.L):
        gl = O.layer_signal(g32, pre_in=pre[l][0], gamma_pre=pre[l][1], eps=c.eps, min_rms=c.min_rms)
        jj = np.concatenate([r.integers(0, c.d_ff, 96), [c.d_ff - 1, 0]])
        Ds = O.pseudograd(gl, acts[l][:, jj])
        assert_close(f"dW[{l}] columns", dW[l][:, jj].cpu().numpy().astype(np.float64), Ds, "bf16")
        if l in (0, c.L - 1):
            D, n2 = oracle_layer(gl, acts[l])
            s = O.clip_scale(n2, wsq[l], c.clip_frac)
            assert abs(float(cs[l]) - s) <= 1e-3 * s, (l, float(cs[l]), s)
            assert_close(f"momentum[{l}]", s1[l].cpu().numpy().astype(np.float64), s * D, "bf16")
            del D


@pytest.mark.slow
def test_full_size_post_ffn_fused_update(dev):
    """OLMo-2 shapes (the layout with a post-FFN norm) at full size, in the
    benchmark's launch configuration with --post-ffn: the composed signal, the
    outer products and the overlapped SGD-momentum step; sampled entries."""
    c = I.CONFIGS[1]
    g32, pf = pffn_case(c, c.L)
    acts = [I.activation(c, l) for l in range(c.L)]
    Wh = [I.master_weight(c, l) for l in range(c.L)]
    W = [torch.from_numpy(w).to(dev) for w in Wh]
    wsq = np.array([float((w.astype(np.float64) ** 2).sum()) for w in Wh])
    s1 = [torch.zeros_like(w) for w in W]
    cs = torch.empty(c.L, dtype=torch.float32, device=dev)
    dW, ss, _ = run_pffn(c, g32, pf, acts, dev,
                         opt=api.OptConfig(lr=c.lr, clip_frac=c.clip_frac, step=1), W_master=W,
                         W_lp=[torch.empty(w.shape, dtype=torch.bfloat16, device=dev) for w in W], state1=s1,
                         W_sumsq=torch.tensor(wsq, dtype=torch.float64, device=dev), clip_scale=cs)
    r = np.random.default_rng(7)
    for l in range(c.L):
        gl = O.post_ffn_signal(g32, pf[l][0], pf[l][1], eps=c.eps, min_rms=c.min_rms)
        ii = np.concatenate([r.integers(0, c.d, 64), [0, c.d - 1]])
        jj = np.concatenate([r.integers(0, c.d_ff, 64), [c.d_ff - 1, 0]])
        D = np.einsum("ti,ti->i", gl[:, ii], I.storage_to_f64(acts[l][:, jj])) / c.T
        assert_close(f"dW[{l}] samples", dW[l][ii, jj].cpu().numpy().astype(np.float64), D, "bf16")
        s = min(1.0, c.clip_frac * np.sqrt(wsq[l]) / np.sqrt(float(ss[l])))
        assert abs(float(cs[l]) - s) <= 1e-6 * s
        assert_close(f"momentum[{l}] samples", s1[l][ii, jj].cpu().numpy().astype(np.float64), s * D, "bf16")

