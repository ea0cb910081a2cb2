"""The smallest legal shapes (d, d_ff, V = 8; T = 1..3) through every call,
against the oracle: each GEMM is then one partial tile whose K is below one
64-deep stage, and the row kernels see a single 4-element quad pair."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_14563_amd import _lib as L_
from paper_2608_14563_amd import api
from paper_2608_14563_amd import inputs as I
from tests._util import assert_close, dev_tensor, host64
from tests.test_parity_output_error import check_against_oracle, run_gpu, small_case

pytestmark = pytest.mark.gpu

CFG = {"f32": I.CONFIGS[0], "bf16": I.CONFIGS[1]}


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("T,d,V", [(3, 8, 8), (1, 8, 16), (2, 16, 8)])
def test_output_error_min_sizes(dev, dtype, T, d, V):
    print(f"[min] output error {dtype} T={T} d={d} V={V}", flush=True)
    c, x, g, W, y = small_case(CFG[dtype], T, d, V)
    got = run_gpu(x, g, W, y, dtype, dev)
    check_against_oracle(x, g, W, y, dtype, got)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("T,d,d_ff,L", [(3, 8, 8, 1), (2, 16, 24, 3), (1, 8, 16, 2)])
def test_pseudograd_min_sizes(dev, dtype, T, d, d_ff, L):
    """W3 outer products and the full-MLP W1/W2 signals."""
    print(f"[min] pseudograd {dtype} T={T} d={d} d_ff={d_ff} L={L}", flush=True)
    c = CFG[dtype].shrink(T=T, d=d, d_ff=d_ff, L=L)
    g = I.synthetic_signal(c)
    caches = [I.mlp_cache(c, l) for l in range(L)]
    extras = [I.full_mlp_extra(c, l) for l in range(L)]
    W3i = [I.to_storage(I.master_weight(c, l), c.dtype) for l in range(L)]
    f32 = torch.float32
    dW3 = [torch.empty(d, d_ff, dtype=f32, device=dev) for _ in range(L)]
    dW1 = [torch.empty(d_ff, d, dtype=f32, device=dev) for _ in range(L)]
    dW2 = [torch.empty(d_ff, d, dtype=f32, device=dev) for _ in range(L)]
    ss = torch.empty(3 * L, dtype=torch.float64, device=dev)
    api.fpo_pseudograd(dev_tensor(g, dev), [dev_tensor(cc[2], dev) for cc in caches], dW3=dW3, sumsq=ss,
                       W3_init=[dev_tensor(w, dev) for w in W3i], gate=[dev_tensor(cc[0], dev) for cc in caches],
                       up=[dev_tensor(cc[1], dev) for cc in caches], x_in=[dev_tensor(e[0], dev) for e in extras],
                       dW1=dW1, dW2=dW2)
    torch.cuda.synchronize()
    s = ss.cpu().numpy()
    for l in range(L):
        q, u, a = caches[l]
        D3 = O.pseudograd(g, a)
        D1, D2 = O.full_mlp_grads(g, W3i[l], q, u, extras[l][0])
        assert_close("dW3", host64(dW3[l]), D3, c.dtype)
        assert_close("dW1", host64(dW1[l]), D1, c.dtype)
        assert_close("dW2", host64(dW2[l]), D2, c.dtype)
        assert_close("sumsq W3", s[l], float((D3 ** 2).sum()), c.dtype)
        assert_close("sumsq W1", s[L + l], float((D1 ** 2).sum()), c.dtype)


@pytest.mark.parametrize("T,d,d_ff,L", [(3, 8, 8, 2), (2, 16, 24, 1)])
def test_post_ffn_min_sizes(dev, T, d, d_ff, L):
    print(f"[min] post-FFN T={T} d={d} d_ff={d_ff} L={L}", flush=True)
    c = I.CONFIGS[1].shrink(T=T, d=d, d_ff=d_ff, L=L)
    g32 = I.normal(c.cid, I.T_G, 7, T * d, std=0.02).reshape(T, d)
    pf = [I.post_ffn(c, l) for l in range(L)]
    acts = [I.activation(c, l) for l in range(L)]
    dW = [torch.empty(d, d_ff, dtype=torch.float32, device=dev) for _ in range(L)]
    ss = torch.empty(L, dtype=torch.float64, device=dev)
    api.fpo_pseudograd(None, [dev_tensor(a, dev) for a in acts], dW3=dW, sumsq=ss,
                       post_ffn=api.PostFfn(torch.from_numpy(g32).to(dev), [dev_tensor(m, dev) for m, _ in pf],
                                            [dev_tensor(x, dev) for _, x in pf], c.eps, c.min_rms))
    torch.cuda.synchronize()
    for l in range(L):
        gl = O.post_ffn_signal(g32, pf[l][0], pf[l][1], eps=c.eps, min_rms=c.min_rms)
        assert_close("dW3", host64(dW[l]), O.pseudograd(gl, acts[l]), c.dtype)


@pytest.mark.parametrize("stage", [False, True])
@pytest.mark.parametrize("target", [0, 1])
def test_fused_update_min_sizes(dev, stage, target):
    """Two layers of 8 x 8 through the fused pseudogradient + SGD-momentum step
    (overlapped path for the gradient clip; bf16-staged or fp32 pseudogradient)
    against the oracle's clipped step."""
    print(f"[min] fused update stage={stage} target={target}", flush=True)
    c = I.CONFIGS[1].shrink(T=3, d=8, d_ff=8, L=2)
    g = I.synthetic_signal(c)
    acts = [I.activation(c, l) for l in range(c.L)]
    Wh = [I.master_weight(c, l) for l in range(c.L)]
    W = [torch.from_numpy(w.copy()).to(dev) for w in Wh]
    s1 = [torch.zeros_like(w) for w in W]
    lp = [torch.empty(w.shape, dtype=torch.bfloat16, device=dev) for w in W]
    wsq = [float((w.astype(np.float64) ** 2).sum()) for w in Wh]
    Wsq = torch.tensor(wsq, dtype=torch.float64, device=dev)
    ss = torch.empty(c.L, dtype=torch.float64, device=dev)
    dW = None if stage else [torch.empty(c.d, c.d_ff, dtype=torch.float32, device=dev) for _ in range(c.L)]
    lr, frac = 1e-2, 1e-3
    api.fpo_pseudograd(dev_tensor(g, dev), [dev_tensor(a, dev) for a in acts], dW3=dW, sumsq=ss, grad_bf16=stage,
                       opt=api.OptConfig(lr=lr, clip_frac=frac, step=1, clip_target=target), W_master=W, W_lp=lp,
                       state1=s1, W_sumsq=Wsq)
    torch.cuda.synchronize()
    for l in range(c.L):
        D = O.pseudograd(g, acts[l])
        if target == L_.FPO_CLIP_GRADIENT:
            s = O.clip_scale(float((D * D).sum()), wsq[l], frac)
            Wo, b = O.sgd_momentum(Wh[l], np.zeros_like(D), s * D, lr, 0.9, step=1)
        else:
            Wo, b, s = O.sgd_momentum_update_clip(Wh[l], np.zeros_like(D), D, lr, 0.9, step=1, frac=frac)
        assert s < 1.0
        assert_close("momentum", host64(s1[l]), b, "bf16")
        assert_close("W step", host64(W[l]) - Wh[l].astype(np.float64), Wo - Wh[l].astype(np.float64), "bf16")


def test_cosine_min_size(dev):
    r = np.random.default_rng(3)
    A = [r.standard_normal(4).astype(np.float32), r.standard_normal(8).astype(np.float32)]
    B = [r.standard_normal(4).astype(np.float32), -A[1]]
    cos = torch.empty(2, dtype=torch.float32, device=dev)
    dot = torch.empty(2, dtype=torch.float64, device=dev)
    api.fpo_cosine([torch.from_numpy(a).to(dev) for a in A], [torch.from_numpy(b).to(dev) for b in B], dot=dot,
                   cos=cos)
    torch.cuda.synchronize()
    for m in range(2):
        d0, _, _, c0 = O.cosine(A[m], B[m])
        assert abs(float(dot[m]) - d0) <= 1e-6 * abs(d0)
        assert abs(float(cos[m]) - c0) <= 1e-6
    assert abs(float(cos[1]) + 1.0) <= 1e-6


def test_binding_checks_shapes(dev):
    """Mismatched buffer shapes are refused by the binding before the library
    sees a pointer (the C ABI cannot check a bare pointer's extent)."""
    T, d, V = 4, 8, 16
    f = dict(device=dev)
    x = torch.zeros(T, d, **f)
    good = dict(gamma=torch.ones(d, **f), W_U=torch.zeros(V, d, **f), targets=torch.zeros(T, dtype=torch.int32, **f))
    with pytest.raises(ValueError, match="g_tilde"):
        api.fpo_output_error(x, good["gamma"], good["W_U"], good["targets"], torch.empty(T, d + 8, **f))
    with pytest.raises(ValueError, match="targets"):
        api.fpo_output_error(x, good["gamma"], good["W_U"], torch.zeros(T - 1, dtype=torch.int32, **f),
                             torch.empty(T, d, **f))
    a = [torch.zeros(T, 16, **f)]
    with pytest.raises(ValueError, match="dW3"):
        api.fpo_pseudograd(torch.zeros(T, d, **f), a, dW3=[torch.empty(16, d, **f)])
    with pytest.raises(ValueError, match="W_master"):
        api.fpo_apply_update(api.OptConfig(), [torch.zeros(64, **f)], torch.zeros(1, dtype=torch.float64, **f),
                             [torch.zeros(32, **f)], [torch.zeros(64, **f)], torch.zeros(1, dtype=torch.float64, **f))
    with pytest.raises(ValueError, match="B\\[0\\]"):
        api.fpo_cosine([torch.zeros(8, **f)], [torch.zeros(12, **f)])
