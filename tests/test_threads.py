"""Concurrent callers: two host threads, each on its own stream with its own
buffers, run the overlapped pseudogradient + SGD-momentum step three times,
either with the library's shared side stream (enqueue serialised by its lock)
or each with a side stream and events of its own (fpo_overlap); each thread's
results must equal the same steps run alone on one stream."""
import threading

import pytest
import torch

from paper_2608_14563_amd import api
from paper_2608_14563_amd import inputs as I
from tests._util import dev_tensor

pytestmark = pytest.mark.gpu


def _case(c, dev, seed_layer):
    acts = [dev_tensor(I.activation(c, seed_layer + l), dev) for l in range(c.L)]
    W = [torch.from_numpy(I.master_weight(c, seed_layer + l)).to(dev) for l in range(c.L)]
    return dict(g=dev_tensor(I.synthetic_signal(c), dev), a=acts, W=W, s1=[torch.zeros_like(w) for w in W],
                lp=[torch.empty(w.shape, dtype=torch.bfloat16, device=dev) for w in W],
                Wsq=torch.tensor([float((w.double() ** 2).sum()) for w in W], dtype=torch.float64, device=dev),
                ss=torch.empty(c.L, dtype=torch.float64, device=dev),
                ws=api.workspace(api.fpo_pseudograd_workspace(c.T, c.d, c.d_ff, c.L, torch.bfloat16, grad_bf16=True),
                                 dev))


def _steps(s, n=3, overlap=None):
    for k in range(1, n + 1):
        api.fpo_pseudograd(s["g"], s["a"], dW3=None, sumsq=s["ss"], grad_bf16=True, ws=s["ws"],
                           opt=api.OptConfig(lr=1e-2, clip_frac=0.01, step=k), W_master=s["W"], W_lp=s["lp"],
                           state1=s["s1"], W_sumsq=s["Wsq"], overlap=overlap)


@pytest.mark.parametrize("own_side_stream", [False, True], ids=["library-side-stream", "caller-side-streams"])
def test_two_threads_two_streams(dev, own_side_stream):
    c = I.CONFIGS[1].shrink(T=256, d=520, d_ff=1288, L=3)
    ref = [_case(c, dev, 0), _case(c, dev, 3)]
    for s in ref:
        _steps(s)
    torch.cuda.synchronize()
    got = [_case(c, dev, 0), _case(c, dev, 3)]
    errors = []

    def run(s):
        try:
            st = torch.cuda.Stream()
            ov = api.Overlap(dev) if own_side_stream else None
            with torch.cuda.stream(st):
                _steps(s, overlap=ov)
            st.synchronize()
        except Exception as e:  # pragma: no cover - reported below
            errors.append(e)

    th = [threading.Thread(target=run, args=(s,)) for s in got]
    for t in th:
        t.start()
    for t in th:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for r, g in zip(ref, got):
        for key in ("W", "s1", "lp"):
            for a, b in zip(r[key], g[key]):
                assert torch.equal(a, b), key
        assert torch.equal(r["Wsq"], g["Wsq"]) and torch.equal(r["ss"], g["ss"])
