"""End-to-end layer-viability diagnostic (Sec. 2.2 eq. cosine, Sec. 2.3) on a
decoder-only SwiGLU transformer.

The model under diagnosis runs in PyTorch on the GPU in float32: its forward
pass with cache and its true gradient by autograd (the gradient the
pseudogradient is compared with; the method itself never builds one). Every
step of the FPO side runs in libfpo:
  fpo_output_error  error over the full vocabulary, projection through W_U,
                    clamped final-norm VJP -> g~ (Sec. 3.1 steps 2-4)
  fpo_pseudograd    each layer's W3 pseudogradient (1/T) g_l^T a_l reduced
                    against the autograd dL/dW3_l without being stored
                    (<D, R>, ||D||^2, ||R||^2); g_l = g~, or its post-FFN
                    composition in the OLMo-2 layout; in full-MLP mode the
                    W1/W2 pseudogradients through W3_init = W3 (eq. errh)
  fpo_cosine        the output cosine cos(g~, dL/dr_l) per layer, and the
                    W1/W2 cosines in full-MLP mode.
The per-layer W3 cosine is <D, R> / sqrt(||D||^2 ||R||^2) of the library's
float64 reductions.

Model (the same definition the float64 reference uses; layouts per
architecture, Sec. 3.2):
  x_0 = E[ids]
  "pre":  x += Attn(n1(x)); z = n2(x); r = x + MLP(z)
  "post": x += n1(Attn(x)); z = x;     r = x + n2(MLP(z))
  MLP(z) = W3 (SiLU(W1 z) * (W2 z)); causal attention with grouped key/value
  heads (query head h reads key/value head h // (H / KV)), 1/sqrt(head_dim)
  scaling, no positional code; logits = final_norm(r_{L-1}) W_U^T; loss =
  mean next-token cross-entropy over the T tokens.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Optional

import numpy as np
import torch

from . import api
from . import inputs as I


def _rmsnorm(x: torch.Tensor, g: torch.Tensor, eps: float) -> torch.Tensor:
    return x * torch.rsqrt((x * x).mean(dim=-1, keepdim=True) + eps) * g


class Transformer:
    """Weights of a ModelConfig on one device (float32)."""

    def __init__(self, m: I.ModelConfig, head: dict, layers: list):
        self.m = m
        self.head = head
        self.layers = layers
        self._op_cache: dict = {}

    @classmethod
    def from_arrays(cls, m: I.ModelConfig, head: dict, layers: list, device) -> "Transformer":
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)  # noqa: E731
        return cls(m, {k: t(v) for k, v in head.items()}, [{k: t(v) for k, v in w.items()} for w in layers])

    @classmethod
    def seeded(cls, m: I.ModelConfig, device) -> "Transformer":
        """Weights drawn with the host streams of the inputs module, layer by
        layer (host memory stays at one layer)."""
        t = lambda a: torch.from_numpy(a).to(device)  # noqa: E731
        head = {k: t(v) for k, v in I.model_head(m).items()}
        return cls(m, head, [{k: t(v) for k, v in I.model_layer(m, l).items()} for l in range(m.n_layers)])

    @classmethod
    def seeded_on_device(cls, m: I.ModelConfig, device, seed: int = 0) -> "Transformer":
        """Same distributions drawn on the device (I.model_weights_device):
        for 7-8B shapes, whose host draws would take minutes."""
        head, layers = I.model_weights_device(m, device, seed)
        return cls(m, head, layers)

    def operand(self, name: str, layer: Optional[int], dtype: torch.dtype) -> torch.Tensor:
        """A weight rounded to the FPO operand dtype, kept for reuse."""
        key = (name, layer, dtype)
        if key not in self._op_cache:
            src = self.head[name] if layer is None else self.layers[layer][name]
            self._op_cache[key] = src.to(dtype).contiguous()
        return self._op_cache[key]


def _attention(z: torch.Tensor, w: dict, H: int, KV: int) -> torch.Tensor:
    B, S, d = z.shape
    hd = w["wq"].shape[0] // H
    q = (z @ w["wq"].T).view(B, S, H, hd).transpose(1, 2)
    k = (z @ w["wk"].T).view(B, S, KV, hd).transpose(1, 2)
    v = (z @ w["wv"].T).view(B, S, KV, hd).transpose(1, 2)
    if KV != H:
        k = k.repeat_interleave(H // KV, dim=1)
        v = v.repeat_interleave(H // KV, dim=1)
    s = torch.matmul(q, k.transpose(-1, -2).contiguous()) * (1.0 / math.sqrt(hd))
    causal = torch.ones(S, S, dtype=torch.bool, device=z.device).triu(1)
    p = torch.softmax(s.masked_fill(causal, float("-inf")), dim=-1)
    o = torch.matmul(p, v.contiguous()).transpose(1, 2).reshape(B, S, H * hd)
    return o @ w["wo"].T


@dataclass
class Cache:
    """What the forward pass keeps for the FPO side, in the operand dtype:
    h_final [T, d]; per layer a [T, d_ff]; mlp_out [T, d] ("post" layout);
    gate q, up u [T, d_ff] and x_in [T, d] (full-MLP mode). targets int32 [T].
    The float32 graph tensors (r, W3/W1/W2 leaves) are kept for autograd."""
    targets: torch.Tensor
    h_final: torch.Tensor
    a: list
    mlp_out: list = field(default_factory=list)
    q: list = field(default_factory=list)
    u: list = field(default_factory=list)
    x_in: list = field(default_factory=list)
    loss: Optional[torch.Tensor] = None
    r: list = field(default_factory=list)
    leaves: dict = field(default_factory=dict)


def forward_with_cache(model: Transformer, ids: torch.Tensor, op: torch.dtype, full_mlp: bool = False) -> Cache:
    """ids int64 [batch, seq + 1] on the device. W3 (and W1, W2 in full-MLP
    mode) are autograd leaves; each block's residual output r_l is kept."""
    m = model.m
    B, S = ids.shape[0], ids.shape[1] - 1
    T = B * S
    inp, tgt = ids[:, :-1], ids[:, 1:].reshape(T)
    x = model.head["embed"][inp]
    names = ("w3", "w1", "w2") if full_mlp else ("w3",)
    leaves = {n: [] for n in names}
    c = Cache(targets=tgt.to(torch.int32).contiguous(), h_final=None, a=[])
    for w in model.layers:
        lw = dict(w)
        for n in names:
            lw[n] = w[n].detach().requires_grad_(True)
            leaves[n].append(lw[n])
        if m.layout == "pre":
            x = x + _attention(_rmsnorm(x, lw["n1"], m.eps), lw, m.n_heads, m.n_kv_heads)
            z = _rmsnorm(x, lw["n2"], m.eps)
        else:
            x = x + _rmsnorm(_attention(x, lw, m.n_heads, m.n_kv_heads), lw["n1"], m.eps)
            z = x
        q = z @ lw["w1"].T
        u = z @ lw["w2"].T
        a = torch.nn.functional.silu(q) * u
        mo = a @ lw["w3"].T
        r = (x + (mo if m.layout == "pre" else _rmsnorm(mo, lw["n2"], m.eps))).view(T, -1)
        x = r.view(B, S, -1)
        c.r.append(r)
        c.a.append(a.detach().reshape(T, -1).to(op).contiguous())
        if m.layout == "post":
            c.mlp_out.append(mo.detach().reshape(T, -1).to(op).contiguous())
        if full_mlp:
            c.q.append(q.detach().reshape(T, -1).to(op).contiguous())
            c.u.append(u.detach().reshape(T, -1).to(op).contiguous())
            c.x_in.append(z.detach().reshape(T, -1).to(op).contiguous())
    h = x.view(T, -1)
    c.h_final = h.detach().to(op).contiguous()
    logits = _rmsnorm(h, model.head["final_norm"], m.eps) @ model.head["W_U"].T
    c.loss = torch.nn.functional.cross_entropy(logits, tgt, reduction="mean")
    c.leaves = leaves
    return c


def true_gradients(c: Cache) -> dict:
    """Autograd gradients of the mean loss (float32): dW3 [d, d_ff], dR [T, d]
    per layer, and dW1, dW2 [d_ff, d] when the cache has W1/W2 leaves. Frees
    the graph."""
    L = len(c.r)
    wrt = list(c.leaves["w3"]) + list(c.r)
    full = "w1" in c.leaves
    if full:
        wrt += list(c.leaves["w1"]) + list(c.leaves["w2"])
    gr = torch.autograd.grad(c.loss, wrt)
    out = {"dW3": [g.contiguous() for g in gr[:L]], "dR": [g.contiguous() for g in gr[L:2 * L]]}
    if full:
        out["dW1"] = [g.contiguous() for g in gr[2 * L:3 * L]]
        out["dW2"] = [g.contiguous() for g in gr[3 * L:4 * L]]
    c.r, c.leaves = [], {}
    return out


def fpo_launch(model: Transformer, c: Cache, tg: dict, op: torch.dtype, min_rms: Optional[float] = None) -> dict:
    """Enqueue the FPO half of the diagnostic (all in libfpo) on the current
    stream; returns its device outputs: g~ (float32), per-token loss, the
    float64 reductions dot / sumsq (||D||^2, then W1 and W2 in full-MLP mode)
    / rsq, the output cosines, and in full-MLP mode D1, D2 and their
    cosines."""
    m = model.m
    min_rms = m.min_rms if min_rms is None else min_rms
    dev = c.h_final.device
    T, d = c.h_final.shape
    L = len(c.a)
    full = "dW1" in tg
    g = torch.empty(T, d, dtype=torch.float32, device=dev)
    glp = torch.empty(T, d, dtype=op, device=dev) if (op != torch.float32 and m.layout == "pre") else None
    loss = torch.empty(T, dtype=torch.float32, device=dev)
    api.fpo_output_error(c.h_final, model.operand("final_norm", None, op), model.operand("W_U", None, op),
                         c.targets, g, glp, loss=loss, eps=m.eps, min_rms=min_rms)
    sig = None
    post = None
    if m.layout == "pre":
        sig = glp if glp is not None else g
    else:
        post = api.PostFfn(g, c.mlp_out, [model.operand("n2", l, op) for l in range(L)], m.eps, min_rms)
    out = {"g_tilde": g, "loss_tok": loss,
           "sumsq": torch.empty(3 * L if full else L, dtype=torch.float64, device=dev),
           "dot": torch.empty(L, dtype=torch.float64, device=dev),
           "rsq": torch.empty(L, dtype=torch.float64, device=dev),
           "cos_w3": torch.empty(L, dtype=torch.float32, device=dev),
           "cos_out": torch.empty(L, dtype=torch.float32, device=dev)}
    kw = {}
    if full:
        d_ff = c.a[0].shape[1]
        kw = dict(W3_init=[model.operand("w3", l, op) for l in range(L)], gate=c.q, up=c.u, x_in=c.x_in,
                  dW1=[torch.empty(d_ff, d, dtype=torch.float32, device=dev) for _ in range(L)],
                  dW2=[torch.empty(d_ff, d, dtype=torch.float32, device=dev) for _ in range(L)])
    api.fpo_pseudograd(sig, c.a, dW3=None, sumsq=out["sumsq"], ref=tg["dW3"], ref_dot=out["dot"],
                       ref_sumsq=out["rsq"], ref_cos=out["cos_w3"], scale=1.0 / T, post_ffn=post, **kw)
    api.fpo_cosine([g] * L, tg["dR"], cos=out["cos_out"])
    if full:
        out["D1"], out["D2"] = kw["dW1"], kw["dW2"]
        for name, D, R in (("cos_w1", kw["dW1"], tg["dW1"]), ("cos_w2", kw["dW2"], tg["dW2"])):
            out[name] = torch.empty(L, dtype=torch.float32, device=dev)
            api.fpo_cosine(D, R, cos=out[name])
    return out


def fpo_finish(out: dict, keep: bool = False) -> dict:
    """Copy fpo_launch's per-layer results to the host (synchronizes): the
    library's cosines cos_w3, cos_out (cos_w1, cos_w2) as float64 arrays, the
    reductions dot, sumsq_D, sumsq_R, and the device per-token loss; with
    keep=True also g~ (and D1, D2)."""
    L = out["dot"].numel()
    dot_h, ss_h, rsq_h = out["dot"].cpu().numpy(), out["sumsq"].cpu().numpy()[:L], out["rsq"].cpu().numpy()
    res = {"cos_w3": out["cos_w3"].double().cpu().numpy(),
           "cos_out": out["cos_out"].double().cpu().numpy(), "dot": dot_h, "sumsq_D": ss_h, "sumsq_R": rsq_h,
           "loss_tok": out["loss_tok"]}
    for k in ("cos_w1", "cos_w2"):
        if k in out:
            res[k] = out[k].double().cpu().numpy()
    if keep:
        res["g_tilde"] = out["g_tilde"]
        for k in ("D1", "D2"):
            if k in out:
                res[k] = out[k]
    return res


def summary(cos_per_layer) -> float:
    """Model-level summary: mean cosine over the last quarter of the layers
    (at least one), Sec. 2.3."""
    c = list(cos_per_layer)
    k = max(1, int(round(len(c) / 4)))
    return float(np.mean(c[-k:]))


def run(model: Transformer, ids: torch.Tensor, op: torch.dtype = torch.bfloat16, full_mlp: bool = False,
        min_rms: Optional[float] = None, keep: bool = False) -> dict:
    """Forward with cache, true gradient, FPO side. Returns fpo_finish's dict
    plus the model loss and the two summaries."""
    c = forward_with_cache(model, ids, op, full_mlp)
    tg = true_gradients(c)
    res = fpo_finish(fpo_launch(model, c, tg, op, min_rms), keep)
    res["loss"] = float(c.loss.detach())
    res["summary_w3"] = summary(res["cos_w3"])
    res["summary_out"] = summary(res["cos_out"])
    if keep:
        res["true"] = tg
        res["cache"] = c
    return res
