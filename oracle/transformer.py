"""Plain float64 CPU model of the end-to-end layer-viability diagnostic
(Sec. 2.1 eq. decomp, Sec. 2.2 eq. cosine): a decoder-only SwiGLU transformer's
forward pass with cache, its true gradient by autograd, and the
output-projected pseudogradient of every layer formed by the FPO oracle
(fpo_oracle.output_error, pseudograd, post_ffn_signal, full_mlp_grads,
cosine).

TEST INFRASTRUCTURE ONLY. Only tests/, the smoke check and the benchmark's
CPU-baseline leg may import or call this module. It shares no code with the
product path; weights and token ids come from the seeded inputs module.

The model (the body under diagnosis; the method itself only reads its cache):
  x_0 = E[ids]
  "pre" layout  (Llama, Qwen3, Falcon3): x += Attn(n1(x));  z = n2(x);  r = x + MLP(z)
  "post" layout (OLMo-2):                x += n1(Attn(x));  z = x;      r = x + n2(MLP(z))
  MLP(z) = W3 (SiLU(q) * u) with gate q = W1 z and up u = W2 z
  Attn: causal multi-head attention, query head h reading key/value head
        h // (H / KV), scores scaled by 1/sqrt(head_dim), no positional code
  logits = final_norm(r_{L-1}) W_U^T; loss = mean over the T tokens of the
  next-token cross-entropy.
n(.) is RMSNorm with gain, eps inside the root and no clamp (the clamp belongs
to the pseudogradient's VJP, App. E, not to the model).

Per layer l the diagnostic reports (readings listed in the design notes):
  cos_w3  = cos(dW3 pseudogradient, true dL/dW3)           (eq. cosine, Sec. 2.2)
  cos_out = cos(g~, true dL/dr_l), flattened over [T, d]   (the "output" cosine
            the paper tabulates beside the W3 cosine, Sec. 2.3)
  cos_w1, cos_w2 (full-MLP mode): the gate/up pseudogradients through
            W3_init = the layer's current W3 (eq. errh) against autograd.
In the "post" layout the W3 (and W1/W2) signal is post_ffn_signal(g~) for the
layer (Sec. 3.2 post-feedforward composition).
"""
from __future__ import annotations

import math

import numpy as np
import torch

from . import fpo_oracle as O

def _t(a) -> torch.Tensor:
    return torch.from_numpy(np.asarray(a, dtype=np.float64))


def rmsnorm(x: torch.Tensor, g: torch.Tensor, eps: float) -> torch.Tensor:
    return g * x / torch.sqrt(torch.mean(x * x, dim=-1, keepdim=True) + eps)


def attention(z: torch.Tensor, w: dict, n_heads: int, n_kv: int) -> torch.Tensor:
    """Causal grouped-key/value attention of z [B, S, d]."""
    B, S, _ = z.shape
    hd = w["wq"].shape[0] // n_heads
    q = (z @ w["wq"].T).reshape(B, S, n_heads, hd).transpose(1, 2)
    k = (z @ w["wk"].T).reshape(B, S, n_kv, hd).transpose(1, 2)
    v = (z @ w["wv"].T).reshape(B, S, n_kv, hd).transpose(1, 2)
    grp = n_heads // n_kv
    k = k.repeat_interleave(grp, dim=1)
    v = v.repeat_interleave(grp, dim=1)
    s = (q @ k.transpose(-1, -2)) / math.sqrt(hd)
    mask = torch.ones(S, S, dtype=torch.bool).triu(1)
    s = s.masked_fill(mask, float("-inf"))
    p = torch.softmax(s, dim=-1)
    o = (p @ v).transpose(1, 2).reshape(B, S, n_heads * hd)
    return o @ w["wo"].T


def forward(m, head: dict, layers: list, ids: np.ndarray, grad_names=("w3",)):
    """Run the model on ids [batch, seq + 1] (inputs ids[:, :-1], targets
    ids[:, 1:]). Weights listed in grad_names require grad. Returns a dict:
      loss (scalar tensor), logits [T, V], targets [T] (int64),
      h_final [T, d] (final-norm input), W (per-layer float64 weight dicts),
      per layer (lists of [T, .] tensors, token order b * seq + s):
      r (residual after the block), a (SiLU(q) * u), mlp_out, x_in (the
      MLP input z), q (gate pre-activation), u (up value)."""
    B, S = ids.shape[0], ids.shape[1] - 1
    T = B * S
    inp = torch.from_numpy(ids[:, :-1].astype(np.int64))
    tgt = torch.from_numpy(ids[:, 1:].astype(np.int64)).reshape(T)
    E = _t(head["embed"])
    x = E[inp]
    W, rs, acts, outs, xins, qs, us = [], [], [], [], [], [], []
    for lw in layers:
        w = {k: _t(v) for k, v in lw.items()}
        for k in grad_names:
            w[k].requires_grad_(True)
        W.append(w)
        if m.layout == "pre":
            x = x + attention(rmsnorm(x, w["n1"], m.eps), w, m.n_heads, m.n_kv_heads)
            z = rmsnorm(x, w["n2"], m.eps)
        else:
            x = x + rmsnorm(attention(x, w, m.n_heads, m.n_kv_heads), w["n1"], m.eps)
            z = x
        q = z @ w["w1"].T
        u = z @ w["w2"].T
        a = torch.nn.functional.silu(q) * u
        mo = a @ w["w3"].T
        r = (x + (mo if m.layout == "pre" else rmsnorm(mo, w["n2"], m.eps))).reshape(T, -1)
        x = r.reshape(B, S, -1)  # the rest of the model reads r, so dL/dr is defined
        rs.append(r)
        acts.append(a.reshape(T, -1))
        outs.append(mo.reshape(T, -1))
        xins.append(z.reshape(T, -1))
        qs.append(q.reshape(T, -1))
        us.append(u.reshape(T, -1))
    h = x.reshape(T, -1)
    logits = rmsnorm(h, _t(head["final_norm"]), m.eps) @ _t(head["W_U"]).T
    loss = torch.nn.functional.cross_entropy(logits, tgt, reduction="mean")
    return {"loss": loss, "logits": logits, "targets": tgt, "h_final": h, "W": W, "r": rs, "a": acts,
            "mlp_out": outs, "x_in": xins, "q": qs, "u": us}


def true_gradients(fw: dict, full_mlp: bool = False) -> dict:
    """Autograd gradients of the mean loss: dW3 [d, d_ff] per layer, dR [T, d]
    per layer (the residual after the block), and dW1, dW2 [d_ff, d] in
    full-MLP mode."""
    L = len(fw["W"])
    wrt = [w["w3"] for w in fw["W"]] + list(fw["r"])
    if full_mlp:
        wrt += [w["w1"] for w in fw["W"]] + [w["w2"] for w in fw["W"]]
    gr = torch.autograd.grad(fw["loss"], wrt, allow_unused=True)
    out = {"dW3": [g.detach().numpy() for g in gr[:L]]}
    out["dR"] = [g.detach().numpy() for g in gr[L:2 * L]]
    if full_mlp:
        out["dW1"] = [g.detach().numpy() for g in gr[2 * L:3 * L]]
        out["dW2"] = [g.detach().numpy() for g in gr[3 * L:4 * L]]
    return out


def diagnostic(m, head: dict, layers: list, ids: np.ndarray, min_rms: float | None = None,
               full_mlp: bool = False) -> dict:
    """The end-to-end diagnostic in float64. Returns per-layer lists cos_w3,
    cos_out (and cos_w1, cos_w2), the model summaries (mean over the last
    quarter of layers, Sec. 2.3), and the intermediates: loss, g_tilde,
    output_error's dict, pseudogradients D3 (D1, D2), true gradients, the
    forward cache."""
    min_rms = m.min_rms if min_rms is None else min_rms
    fw = forward(m, head, layers, ids, ("w3", "w1", "w2") if full_mlp else ("w3",))
    tg = true_gradients(fw, full_mlp)
    T = fw["h_final"].shape[0]
    det = lambda t: t.detach().numpy()  # noqa: E731
    oe = O.output_error(det(fw["h_final"]), np.asarray(head["final_norm"], np.float64),
                        np.asarray(head["W_U"], np.float64), fw["targets"].numpy(), eps=m.eps, min_rms=min_rms)
    g = oe["g_tilde"]
    res = {"loss": float(fw["loss"].detach()), "oe": oe, "g_tilde": g, "true": tg, "fw": fw,
           "cos_w3": [], "cos_out": [], "D3": [], "signal": []}
    if full_mlp:
        res.update(cos_w1=[], cos_w2=[], D1=[], D2=[])
    for l, lw in enumerate(layers):
        sig = g if m.layout == "pre" else O.post_ffn_signal(g, det(fw["mlp_out"][l]), lw["n2"], m.eps, min_rms)
        D3 = O.pseudograd(sig, det(fw["a"][l]), 1.0 / T)
        res["signal"].append(sig)
        res["D3"].append(D3)
        res["cos_w3"].append(O.cosine(D3, tg["dW3"][l])[3])
        res["cos_out"].append(O.cosine(g, tg["dR"][l])[3])
        if full_mlp:
            D1, D2 = O.full_mlp_grads(sig, lw["w3"], det(fw["q"][l]), det(fw["u"][l]), det(fw["x_in"][l]), 1.0 / T)
            res["D1"].append(D1)
            res["D2"].append(D2)
            res["cos_w1"].append(O.cosine(D1, tg["dW1"][l])[3])
            res["cos_w2"].append(O.cosine(D2, tg["dW2"][l])[3])
    res["summary_w3"] = O.layer_summary(res["cos_w3"])
    res["summary_out"] = O.layer_summary(res["cos_out"])
    return res
