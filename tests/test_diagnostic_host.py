"""Host-side checks of the end-to-end diagnostic harness: the product's
float32 model forward with cache and its autograd gradient (PyTorch, here on
the CPU) against the float64 oracle model on the same seeded weights, and the
model-level summary. The FPO side itself needs the GPU (test_parity_diagnostic)."""
import numpy as np
import pytest
import torch

from oracle import transformer as OT
from paper_2608_14563_amd import diagnostic as D
from paper_2608_14563_amd import inputs as I


def rel(a, b):
    a = a.detach().double().numpy() if isinstance(a, torch.Tensor) else np.asarray(a, np.float64)
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


@pytest.mark.parametrize("name", ["tiny", "tiny-post"])
def test_forward_cache_and_true_gradient_match_the_oracle(name):
    m = I.MODELS[name]
    head, layers, ids = I.model_head(m), [I.model_layer(m, l) for l in range(m.n_layers)], I.model_tokens(m)
    fw = OT.forward(m, head, layers, ids, ("w3", "w1", "w2"))
    tg_ref = OT.true_gradients(fw, full_mlp=True)
    model = D.Transformer.from_arrays(m, head, layers, "cpu")
    c = D.forward_with_cache(model, torch.from_numpy(ids.astype(np.int64)), torch.float32, full_mlp=True)
    assert abs(float(c.loss.detach()) - float(fw["loss"].detach())) < 1e-5
    assert np.array_equal(c.targets.numpy(), fw["targets"].numpy())
    assert rel(c.h_final, fw["h_final"].detach().numpy()) < 5e-5
    for l in range(m.n_layers):
        for k in ("a", "x_in", "q", "u") + (("mlp_out",) if m.layout == "post" else ()):
            assert rel(getattr(c, k)[l], fw[k][l].detach().numpy()) < 5e-5, (k, l)
    tg = D.true_gradients(c)
    for k in ("dW3", "dR", "dW1", "dW2"):
        for l in range(m.n_layers):
            assert rel(tg[k][l], tg_ref[k][l]) < 5e-5, (k, l)


def test_cache_in_bf16_is_the_rounded_float32_cache():
    m = I.MODELS["tiny"]
    model = D.Transformer.seeded(m, "cpu")
    ids = torch.from_numpy(I.model_tokens(m).astype(np.int64))
    c32 = D.forward_with_cache(model, ids, torch.float32)
    c16 = D.forward_with_cache(model, ids, torch.bfloat16)
    assert c16.a[0].dtype == torch.bfloat16
    assert torch.equal(c16.a[1], c32.a[1].to(torch.bfloat16))
    assert torch.equal(c16.h_final, c32.h_final.to(torch.bfloat16))


def test_summary_is_the_last_quarter_mean():
    assert D.summary([0.1] * 27 + [0.5] * 9) == pytest.approx(0.5)
    assert D.summary([0.2, 0.4, 0.6]) == pytest.approx(0.6)
    assert D.summary(list(range(32))) == pytest.approx(np.mean(range(24, 32)))
