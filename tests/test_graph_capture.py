"""The hot-path calls are capturable into a HIP graph (torch.cuda.CUDAGraph):
they allocate nothing, never synchronise the host and use no memset; the
overlapped optimizer path's side stream joins the capture through its events.
One SGD-momentum step (output error + pseudogradient with the fused update,
bf16-staged) captured at step 3 is replayed three times, with eager work and
synchronisations between replays, and every replay is bit-identical to the
same step run eagerly from the same state. The optimizer scalars (step
number, hence the first-step and AdamW bias terms) are fixed at capture."""
import numpy as np
import pytest
import torch

from paper_2608_14563_amd import api
from paper_2608_14563_amd import inputs as I
from tests._util import dev_tensor

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("variant", ["sgd", "sgd-post-ffn", "adamw", "sgd-clip-update", "adamw-clip-update"])
def test_step_graph_replays_match_eager(dev, variant):
    """Overlapped path (gradient clip: SGD-momentum, with the post-FFN
    composition, AdamW) and the two-pass clip-the-update path."""
    post_ffn = variant == "sgd-post-ffn"
    adam = variant.startswith("adamw")
    target = 1 if variant.endswith("clip-update") else 0
    c = I.CONFIGS[1].shrink(T=300, d=520, d_ff=1288, V=4104, L=3)
    x, gam, WU, y = (dev_tensor(a, dev) for a in (I.hidden(c), I.gain(c), I.unembedding(c), I.targets(c)))
    acts = [dev_tensor(I.activation(c, l), dev) for l in range(c.L)]
    W0 = [torch.from_numpy(I.master_weight(c, l)).to(dev) for l in range(c.L)]
    pf = [I.post_ffn(c, l) for l in range(c.L)] if post_ffn else None

    def state():
        W = [w.clone() for w in W0]
        s = dict(W=W, s1=[torch.zeros_like(w) for w in W], s2=[torch.zeros_like(w) for w in W] if adam else None,
                 lp=[torch.empty(w.shape, dtype=torch.bfloat16, device=dev) for w in W],
                 Wsq=torch.tensor([float((w.double() ** 2).sum()) for w in W], dtype=torch.float64, device=dev),
                 ss=torch.empty(c.L, dtype=torch.float64, device=dev),
                 g=torch.empty(c.T, c.d, device=dev), glp=torch.empty(c.T, c.d, dtype=torch.bfloat16, device=dev),
                 ws_oe=api.workspace(api.fpo_output_error_workspace(c.T, c.d, c.V, torch.bfloat16), dev),
                 ws_pg=api.workspace(api.fpo_pseudograd_workspace(c.T, c.d, c.d_ff, c.L, torch.bfloat16,
                                                                  post_ffn=post_ffn, grad_bf16=True), dev))
        if post_ffn:
            s["pf"] = api.PostFfn(s["g"], [dev_tensor(m, dev) for m, _ in pf], [dev_tensor(gm, dev) for _, gm in pf])
        return s

    def step(s, k):
        api.fpo_output_error(x, gam, WU, y, s["g"], s["glp"], ws=s["ws_oe"])
        api.fpo_pseudograd(None if post_ffn else s["glp"], acts, dW3=None, sumsq=s["ss"], grad_bf16=True,
                           ws=s["ws_pg"], post_ffn=s.get("pf"),
                           opt=api.OptConfig(kind=1 if adam else 0, lr=1e-3 if adam else 1e-2, clip_frac=0.01,
                                             step=k, clip_target=target),
                           W_master=s["W"], W_lp=s["lp"], state1=s["s1"], state2=s["s2"], W_sumsq=s["Wsq"])

    eager, graphed = state(), state()
    for k in (1, 2):
        step(eager, k)
        step(graphed, k)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=torch.cuda.Stream()):
        step(graphed, 3)  # recorded, not run
    torch.cuda.synchronize()
    for k in (3, 4, 5):
        # the graph keeps step 3's scalars (AdamW's bias correction depends on
        # the step number; SGD-momentum's only on whether it is the first)
        step(eager, 3 if adam else k)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        x.add_(0)  # the program's own eager work between replays
        for key in ("W", "s1", "lp") + (("s2",) if adam else ()):
            for a, b in zip(eager[key], graphed[key]):
                assert torch.equal(a, b), (key, k)
        for key in ("Wsq", "ss", "g", "glp"):
            assert torch.equal(eager[key], graphed[key]), (key, k)


def test_full_mlp_step_graph_replays_match_eager(dev):
    """The full-MLP step with the overlapped optimizer (each of the 3 L
    matrices' norm and update released on the side stream after its outer
    products) replays from a graph bit-identically to eager execution."""
    c = I.CONFIGS[1].shrink(T=256, d=256, d_ff=512, V=4104, L=2)
    x, gam, WU, y = (dev_tensor(a, dev) for a in (I.hidden(c), I.gain(c), I.unembedding(c), I.targets(c)))
    caches = [I.mlp_cache(c, l) for l in range(c.L)]
    extras = [I.full_mlp_extra(c, l) for l in range(c.L)]
    acts = [dev_tensor(cc[2], dev) for cc in caches]
    W0 = [torch.from_numpy(I.master_weight(c, l)).to(dev) for l in range(c.L)]
    W0 += [torch.from_numpy(e[1]).to(dev) for e in extras] + [torch.from_numpy(e[2]).to(dev) for e in extras]
    fkw = dict(W3_init=[w.to(torch.bfloat16) for w in W0[:c.L]], gate=[dev_tensor(cc[0], dev) for cc in caches],
               up=[dev_tensor(cc[1], dev) for cc in caches], x_in=[dev_tensor(e[0], dev) for e in extras])
    n = 3 * c.L

    def state():
        W = [w.clone() for w in W0]
        return dict(W=W, s1=[torch.zeros_like(w) for w in W],
                    lp=[torch.empty(w.shape, dtype=torch.bfloat16, device=dev) for w in W],
                    Wsq=torch.tensor([float((w.double() ** 2).sum()) for w in W], dtype=torch.float64, device=dev),
                    ss=torch.empty(n, dtype=torch.float64, device=dev),
                    dW3=[torch.empty(c.d, c.d_ff, device=dev) for _ in range(c.L)],
                    dW1=[torch.empty(c.d_ff, c.d, device=dev) for _ in range(c.L)],
                    dW2=[torch.empty(c.d_ff, c.d, device=dev) for _ in range(c.L)],
                    g=torch.empty(c.T, c.d, device=dev), glp=torch.empty(c.T, c.d, dtype=torch.bfloat16, device=dev),
                    ws_oe=api.workspace(api.fpo_output_error_workspace(c.T, c.d, c.V, torch.bfloat16), dev),
                    ws_pg=api.workspace(api.fpo_pseudograd_workspace(c.T, c.d, c.d_ff, c.L, torch.bfloat16,
                                                                     full_mlp=True), dev))

    def step(s, k):
        api.fpo_output_error(x, gam, WU, y, s["g"], s["glp"], ws=s["ws_oe"])
        api.fpo_pseudograd(s["glp"], acts, dW3=s["dW3"], dW1=s["dW1"], dW2=s["dW2"], sumsq=s["ss"], ws=s["ws_pg"],
                           opt=api.OptConfig(kind=0, lr=1e-2, clip_frac=0.01, step=k),
                           W_master=s["W"], W_lp=s["lp"], state1=s["s1"], W_sumsq=s["Wsq"], **fkw)

    eager, graphed = state(), state()
    for k in (1, 2):
        step(eager, k)
        step(graphed, k)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=torch.cuda.Stream()):
        step(graphed, 3)  # recorded, not run
    torch.cuda.synchronize()
    for k in (3, 4, 5):
        step(eager, k)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        x.add_(0)  # the program's own eager work between replays
        for key in ("W", "s1", "lp", "dW3", "dW1", "dW2"):
            for i, (a, b) in enumerate(zip(eager[key], graphed[key])):
                assert torch.equal(a, b), (key, i, k)
        for key in ("Wsq", "ss", "g", "glp"):
            assert torch.equal(eager[key], graphed[key]), (key, k)
