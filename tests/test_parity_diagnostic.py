"""End-to-end layer-viability diagnostic on a random-init transformer
(Sec. 2.2 eq. cosine): the product harness (model forward with cache and
autograd gradient in float32 PyTorch on the GPU, FPO side in libfpo) against
the float64 oracle pipeline (oracle/transformer.py) on the same seeded
weights and tokens.

Tolerances. The two sides run the model body in different precisions
(float32 on the GPU, float64 in the oracle); on these models the float32
forward and autograd differ from float64 by at most 7e-6 relative Frobenius
(measured on the CPU), so float32-operand quantities are held to 5e-5 and
cosines to 1e-4. With bfloat16 operands (the cache rounded to bf16) the
bound is the 2e-2 relative Frobenius of the bf16 path and 1e-2 on cosines.
At full size the checks are properties that hold at any size: the last
layer's pseudogradient is its true gradient, so is an earlier layer's once
the later blocks are identity maps, and the output error's mean loss is the
model's loss.
"""
import functools

import numpy as np
import pytest
import torch

from oracle import transformer as OT
from paper_2608_14563_amd import diagnostic as D
from paper_2608_14563_amd import inputs as I

pytestmark = pytest.mark.gpu

OPS = {"f32": torch.float32, "bf16": torch.bfloat16}
TOL = {"f32": (5e-5, 1e-4), "bf16": (2e-2, 1e-2)}
# mean per-token loss of the output error against the model's float64 loss:
# float32 logits, or logits from bf16-rounded operands (about 2^-9 relative
# error per operand, averaged over d products and T tokens)
LOSS_TOL = {"f32": 1e-5, "bf16": 2e-3}


@functools.lru_cache(maxsize=None)
def _weights(name):
    m = I.MODELS[name]
    return m, I.model_head(m), [I.model_layer(m, l) for l in range(m.n_layers)], I.model_tokens(m)


@functools.lru_cache(maxsize=None)
def _oracle(name, full):
    m, head, layers, ids = _weights(name)
    return OT.diagnostic(m, head, layers, ids, full_mlp=full)


def rel(a, b):
    a = a.double().cpu().numpy() if isinstance(a, torch.Tensor) else np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def cosv(a, b):
    a = a.double().cpu().numpy().ravel()
    b = np.asarray(b, np.float64).ravel()
    return float(a @ b / np.sqrt((a @ a) * (b @ b)))


@pytest.mark.parametrize("full", [False, True], ids=["w3", "full_mlp"])
@pytest.mark.parametrize("op", ["f32", "bf16"])
@pytest.mark.parametrize("name", ["tiny", "tiny-post", "small", "small-post"])
def test_diagnostic_matches_oracle(dev, name, op, full):
    print(f"[diag] {name} {op} full={full}", flush=True)
    m, head, layers, ids = _weights(name)
    ref = _oracle(name, full)
    model = D.Transformer.from_arrays(m, head, layers, dev)
    res = D.run(model, torch.from_numpy(ids.astype(np.int64)).to(dev), op=OPS[op], full_mlp=full, keep=True)
    torch.cuda.synchronize()
    tr, tc = TOL[op]
    L = m.n_layers
    assert rel(res["g_tilde"], ref["g_tilde"]) < tr
    assert cosv(res["g_tilde"], ref["g_tilde"]) > 0.9999
    assert abs(float(res["loss_tok"].double().mean()) - ref["loss"]) < LOSS_TOL[op] * abs(ref["loss"])
    assert abs(res["loss"] - ref["loss"]) < 1e-5 * abs(ref["loss"])
    for l in range(L):
        D3 = ref["D3"][l]
        assert abs(res["sumsq_D"][l] / float((D3 * D3).sum()) - 1.0) < 2 * tr, l
        R = ref["true"]["dW3"][l]
        assert abs(res["sumsq_R"][l] / float((R * R).sum()) - 1.0) < 1e-4, l
        assert abs(res["cos_w3"][l] - ref["cos_w3"][l]) < tc, (l, res["cos_w3"][l], ref["cos_w3"][l])
        assert abs(res["cos_out"][l] - ref["cos_out"][l]) < tc, (l, res["cos_out"][l], ref["cos_out"][l])
        assert rel(res["true"]["dW3"][l], R) < 5e-5
        if full:
            assert rel(res["D1"][l], ref["D1"][l]) < tr, l
            assert rel(res["D2"][l], ref["D2"][l]) < tr, l
            assert abs(res["cos_w1"][l] - ref["cos_w1"][l]) < tc, l
            assert abs(res["cos_w2"][l] - ref["cos_w2"][l]) < tc, l
    assert abs(res["cos_w3"][-1] - 1.0) < tc
    assert abs(D.summary(res["cos_w3"]) - ref["summary_w3"]) < tc


def _identity_after(model, ell):
    for l in range(ell + 1, model.m.n_layers):
        w = model.layers[l]
        if model.m.layout == "pre":
            w["wo"].zero_()
            w["w3"].zero_()
        else:
            w["n1"].zero_()
            w["n2"].zero_()
    model._op_cache.clear()


@pytest.mark.slow
@pytest.mark.parametrize("name", ["qwen3-8b", "olmo2-7b"])
def test_full_size_properties(dev, name):
    """The diagnostic workload at full size (16 sequences of 512 tokens, every
    layer scored), bf16 operands as in the benchmark: the last layer scores 1,
    an earlier layer scores 1 once the later blocks are identity maps, every
    cosine lies in [-1, 1], and the output error's loss is the model's."""
    m = I.MODELS[name]
    print(f"[diag] full size {name}: T={m.T} L={m.n_layers}", flush=True)
    torch.manual_seed(0)
    model = D.Transformer.seeded_on_device(m, dev)
    ids = torch.from_numpy(I.model_tokens(m).astype(np.int64)).to(dev)
    res = D.run(model, ids, op=torch.bfloat16, min_rms=0.0)
    torch.cuda.synchronize()
    c3, co = res["cos_w3"], res["cos_out"]
    print(f"[diag] cos_w3 {np.round(c3, 3).tolist()}", flush=True)
    assert np.all(np.abs(c3) <= 1.0 + 1e-6) and np.all(np.abs(co) <= 1.0 + 1e-6)
    assert c3[-1] > 0.999 and co[-1] > 0.999
    assert abs(float(res["loss_tok"].double().mean()) - res["loss"]) < 1e-3 * res["loss"]
    ell = m.n_layers - 4
    _identity_after(model, ell)
    res2 = D.run(model, ids, op=torch.bfloat16, min_rms=0.0)
    torch.cuda.synchronize()
    assert res2["cos_w3"][ell] > 0.999 and res2["cos_out"][ell] > 0.999
    del model, res, res2
    torch.cuda.empty_cache()
