"""GPU parity of fpo_pseudograd against the fp64 oracle: per-layer outer
products dW3 = (1/T) g~^T a, their squared norms, the fused diagnostic cosine
terms, and the full-MLP W1/W2 signals through W3_init."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_14563_amd import api
from paper_2608_14563_amd import inputs as I
from tests._util import assert_close, dev_tensor, host64

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
                  ref_sumsq=torch.empty(len(acts), dtype=torch.float64, device=dev))
    api.fpo_pseudograd(tg, ta, dW3=dW, sumsq=ss, **kw)
    torch.cuda.synchronize()
    out = dict(sumsq=ss.cpu().numpy())
    if dW is not None:
        out["dW"] = [w.cpu().numpy().astype(np.float64) for w in dW]
    if refs is not None:
        out["dot"] = kw["ref_dot"].cpu().numpy()
        out["refsq"] = kw["ref_sumsq"].cpu().numpy()
    return out


@pytest.mark.parametrize("cid,T,d,d_ff,L", [(0, 128, 256, 688, 2), (0, 300, 264, 520, 3), (1, 300, 264, 520, 2),
                                            (1, 1000, 512, 1032, 2), (1, 1, 256, 512, 1), (3, 333, 256, 1000, 2)])
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
        assert np.array_equal(with_store["dot"], fused["dot"])


@pytest.mark.parametrize("cid,T,d,d_ff,L", [(0, 128, 256, 688, 2), (1, 200, 256, 520, 2)])
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


def test_deterministic(dev):
    c = I.CONFIGS[1].shrink(T=700, d=512, d_ff=1024, L=2)
    g = signal(c)
    acts = [I.activation(c, l) for l in range(2)]
    a = run_w3(c, g, acts, dev)
    b = run_w3(c, g, acts, dev)
    assert np.array_equal(a["sumsq"], b["sumsq"])
    for x, y in zip(a["dW"], b["dW"]):
        assert np.array_equal(x, y)


@pytest.mark.slow
@pytest.mark.parametrize("cid", [1, 2, 3])
def test_full_size_sampled(dev, cid):
    """Full workload shapes: sampled entries of every layer against the oracle,
    and layer 0's squared norm through the Gram identity
    ||G^T A||_F^2 = <G G^T, A A^T> (exact in fp64 at any size)."""
    c = I.CONFIGS[cid]
    g = signal(c)
    acts = [I.activation(c, l) for l in range(c.L)]
    got = run_w3(c, g, acts, dev)
    gf = I.storage_to_f64(g)
    r = np.random.default_rng(cid)
    for l in range(c.L):
        af = I.storage_to_f64(acts[l])
        ii = r.integers(0, c.d, 64)
        jj = r.integers(0, c.d_ff, 64)
        ii = np.concatenate([ii, [0, c.d - 1]])
        jj = np.concatenate([jj, [c.d_ff - 1, 0]])
        ref = np.einsum("ti,ti->i", gf[:, ii], af[:, jj]) / c.T
        assert_close(f"dW[{l}] samples", got["dW"][l][ii, jj], ref, "bf16")
        if l == 0:
            G = gf @ gf.T
            A = af @ af.T
            n2 = float(np.sum(G * A)) / c.T ** 2
            assert_close("sumsq[0] (Gram)", got["sumsq"][0], n2, "bf16")
