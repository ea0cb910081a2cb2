"""A seeded sweep of ragged shapes against the oracle, both dtypes: the output
error (T, d, V and the vocabulary chunk drawn so that every tile dimension has
a partial tail), and the pseudogradient with the fused optimizer step
(SGD-momentum or AdamW, gradient or update clip, fp32 or bf16-staged
pseudogradient, one to four layers). The cases are drawn once from a fixed
seed and sized so that the oracle finishes each in about a second."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_14563_amd import _lib as L_
from paper_2608_14563_amd import api
from paper_2608_14563_amd import inputs as I
from tests._util import assert_close, bf16_rne_bits, dev_tensor
from tests.test_parity_output_error import check_against_oracle, run_gpu, small_case

pytestmark = pytest.mark.gpu

CFG = {"f32": I.CONFIGS[0], "bf16": I.CONFIGS[1]}


def _oe_cases(n=10, seed=2608):
    r = np.random.default_rng(seed)
    out = []
    for k in range(n):
        dtype = ("f32", "bf16")[k % 2]
        T = int(r.integers(1, 700))
        d = 8 * int(r.integers(1, 97))
        V = 8 * int(r.integers(1, 1500))
        chunk = int(r.choice([0, 256 * int(r.integers(1, 24))]))
        out.append((dtype, T, d, V, chunk))
    return out


def _pg_cases(n=12, seed=14563):
    r = np.random.default_rng(seed)
    out = []
    for k in range(n):
        dtype = ("f32", "bf16")[k % 2]
        T = int(r.integers(1, 600))
        d = 8 * int(r.integers(1, 65))
        d_ff = 8 * int(r.integers(1, 150))
        L = int(r.integers(1, 5))
        kind = ("sgd", "adamw")[(k // 2) % 2]
        target = int(r.integers(0, 2))
        stage = dtype == "bf16" and bool(r.integers(0, 2))
        lr = float(r.choice([1e-2, 1.0]))
        out.append((dtype, T, d, d_ff, L, kind, target, stage, lr))
    return out


@pytest.mark.parametrize("dtype,T,d,V,chunk", _oe_cases())
def test_output_error_sweep(dev, dtype, T, d, V, chunk):
    print(f"[sweep] output error {dtype} T={T} d={d} V={V} chunk={chunk}", flush=True)
    c, x, g, W, y = small_case(CFG[dtype], T, d, V)
    got = run_gpu(x, g, W, y, dtype, dev, chunk=chunk)
    check_against_oracle(x, g, W, y, dtype, got)


@pytest.mark.parametrize("dtype,T,d,d_ff,L,kind,target,stage,lr", _pg_cases())
def test_fused_step_sweep(dev, dtype, T, d, d_ff, L, kind, target, stage, lr):
    """First optimizer step. Oracle side: D = (1/T) g~^T a; the clip factor
    from the GPU's reported norm (||dW||, or ||W' - W|| of the unclipped step
    for the update clip); the new state against the oracle's optimizer;
    W' against the kernels' float32 formula on the GPU's own state and factor
    (a few ulp), its low-precision copy exactly W' (bf16: RNE of W')."""
    print(f"[sweep] fused step {dtype} T={T} d={d} d_ff={d_ff} L={L} {kind} target={target} "
          f"stage={stage} lr={lr}", flush=True)
    c = CFG[dtype].shrink(T=T, d=d, d_ff=d_ff, L=L)
    adam = kind == "adamw"
    g = I.synthetic_signal(c)
    acts = [I.activation(c, l) for l in range(L)]
    Wh = [I.master_weight(c, l) for l in range(L)]
    W = [torch.from_numpy(w.copy()).to(dev) for w in Wh]
    wsq = [float((w.astype(np.float64) ** 2).sum()) for w in Wh]
    Wsq = torch.tensor(wsq, dtype=torch.float64, device=dev)
    s1 = [torch.zeros_like(w) for w in W]
    s2 = [torch.zeros_like(w) for w in W] if adam else None
    lpt = torch.bfloat16 if dtype == "bf16" else torch.float32  # the copy takes the operand dtype
    lp = [torch.empty(w.shape, dtype=lpt, device=dev) for w in W]
    ss = torch.empty(L, dtype=torch.float64, device=dev)
    cs = torch.empty(L, dtype=torch.float32, device=dev)
    dW = None if stage else [torch.empty(d, d_ff, dtype=torch.float32, device=dev) for _ in range(L)]
    frac = 0.01
    opt = api.OptConfig(kind=L_.FPO_OPT_ADAMW if adam else L_.FPO_OPT_SGD, lr=lr, clip_frac=frac, step=1,
                        clip_target=target)
    api.fpo_pseudograd(dev_tensor(g, dev), [dev_tensor(a, dev) for a in acts], dW3=dW, sumsq=ss, grad_bf16=stage,
                       opt=opt, W_master=W, W_lp=lp, state1=s1, state2=s2, W_sumsq=Wsq, clip_scale=cs)
    torch.cuda.synchronize()
    f32 = lambda v: np.float64(np.float32(v))  # noqa: E731
    for l in range(L):
        D = O.pseudograd(g, acts[l])
        assert_close(f"sumsq[{l}]", float(ss[l]), float((D * D).sum()), c.dtype)
        if dW is not None:
            assert_close(f"dW[{l}]", dW[l].cpu().numpy().astype(np.float64), D, c.dtype)
        w0 = Wh[l].astype(np.float64)
        m = s1[l].cpu().numpy().astype(np.float64)
        sg = float(cs[l])
        if target == L_.FPO_CLIP_GRADIENT:
            s = O.clip_scale(float(ss[l]), wsq[l], frac)
            G = s * D
        else:
            G = D
        if adam:
            _, om, ov = O.adamw(w0, 0.0, 0.0, G, lr, 1, opt.beta1, opt.beta2, opt.adam_eps, opt.weight_decay)
            v = s2[l].cpu().numpy().astype(np.float64)
            assert_close(f"exp_avg[{l}]", m, om, c.dtype)
            assert_close(f"exp_avg_sq[{l}]", v, ov, c.dtype)
            step = f32(lr) * (m * f32(1.0 / (1.0 - opt.beta1))) / (
                np.sqrt(v) * f32(1.0 / np.sqrt(1.0 - opt.beta2)) + f32(opt.adam_eps))
            if target == L_.FPO_CLIP_GRADIENT:
                expect = w0 * f32(1.0 - lr * opt.weight_decay) - step
                tol_step = step
            else:
                delta = -f32(lr * opt.weight_decay) * w0 - step
                s = O.clip_scale(float(np.sum(delta * delta)), wsq[l], frac)
                expect = w0 + sg * delta
                tol_step = np.abs(sg * delta)
        else:
            assert_close(f"momentum[{l}]", m, G, c.dtype)
            delta = -f32(lr) * m
            if target == L_.FPO_CLIP_UPDATE:
                s = O.clip_scale(float(np.sum(delta * delta)), wsq[l], frac)
                expect = w0 + sg * delta
            else:
                expect = w0 + delta
            tol_step = np.abs(delta)
        assert abs(sg - s) <= 1e-5 * max(s, 1e-30), (l, sg, s)
        wg = W[l].cpu().numpy()
        tol = 2 * np.spacing(np.abs(expect).astype(np.float32)).astype(np.float64) + 8 * 2.0 ** -23 * np.abs(tol_step)
        assert np.all(np.abs(wg.astype(np.float64) - expect) <= tol), l
        if dtype == "bf16":
            assert np.array_equal(lp[l].view(torch.int16).cpu().numpy().view(np.uint16), bf16_rne_bits(wg)), l
        else:
            assert np.array_equal(lp[l].cpu().numpy(), wg), l
        assert abs(float(Wsq[l]) - float((wg.astype(np.float64) ** 2).sum())) <= 1e-6 * float(Wsq[l])
