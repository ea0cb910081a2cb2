"""Seeded synthetic inputs for the FPO hot path.

This module only draws random numbers and rounds them to the storage dtype.
It holds none of the method's arithmetic (no softmax, no projection, no norm
VJP, no outer products, no optimizer): the GPU path and the CPU oracle both
receive exactly the arrays produced here, and nothing else is shared between
them.

Workloads (shapes follow the models the paper adapts, Sec. 4 "Models and target
layers"; the last quarter of layers is the paper's model-level summary window,
Sec. 2.3):

  id  name           dtype  d     d_ff   V       T     L   targets
  0   tiny-fp32      f32    256   688    4096    128   2   uniform
  1   olmo2-7b       bf16   4096  11008  100352  2048  8   Zipf(1.1)
  2   qwen3-8b       bf16   4096  12288  151936  4096  9   Zipf(1.1)
  3   falcon3-7b     bf16   3072  23040  131072  4096  7   Zipf(1.1), 1% outlier channels x20
  4   qwen3-8b-diag  bf16   4096  12288  151936  8192  36  Zipf(1.1), reference-gradient noise

Distributions: final-norm input x ~ N(0,1); RMSNorm gain 1 + N(0, 0.1^2);
W_U ~ N(0, 0.02^2); cached MLP activation a = SiLU(q) * u with q, u ~ N(0,1)
(q and u are also the gate / up values the full-MLP mode differentiates
through); down-projection masters ~ N(0, 0.02^2).

Every tensor is drawn from its own counter-addressed stream:
SeedSequence(entropy=260814563, spawn_key=(cfg, tensor, layer, block)), in
blocks of 2**20 elements, so any block can be regenerated on its own and the
result does not depend on the number of threads used to draw it.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, replace

import numpy as np

ENTROPY = 260814563
BLOCK = 1 << 20

# tensor ids inside the spawn key
T_X, T_GAMMA, T_WU, T_TARGETS, T_Q, T_U, T_W, T_OUTLIER, T_REFNOISE, T_XIN, T_W1, T_W2, T_G, T_STATE, T_MISC, T_REF1, \
    T_PFFN, T_MODEL, T_PRE = range(19)


@dataclass(frozen=True)
class Config:
    cid: int
    name: str
    dtype: str          # "f32" or "bf16": storage / operand dtype of the inputs
    d: int
    d_ff: int
    V: int
    T: int
    L: int
    zipf: bool
    outliers: bool
    diag: bool = False
    eps: float = 1e-6
    min_rms: float = 0.5
    lr: float = 1e-4
    clip_frac: float = 0.01

    def shrink(self, **kw) -> "Config":
        return replace(self, **kw)


CONFIGS = {
    0: Config(0, "tiny-fp32", "f32", 256, 688, 4096, 128, 2, zipf=False, outliers=False),
    1: Config(1, "olmo2-7b", "bf16", 4096, 11008, 100352, 2048, 8, zipf=True, outliers=False),
    2: Config(2, "qwen3-8b", "bf16", 4096, 12288, 151936, 4096, 9, zipf=True, outliers=False),
    3: Config(3, "falcon3-7b", "bf16", 3072, 23040, 131072, 4096, 7, zipf=True, outliers=True),
    4: Config(4, "qwen3-8b-diag", "bf16", 4096, 12288, 151936, 8192, 36, zipf=True, outliers=False, diag=True),
}

_POOL_WORKERS = max(1, min(16, len(os.sched_getaffinity(0))))


def _rng(cfg: int, tensor: int, layer: int, block: int) -> np.random.Generator:
    ss = np.random.SeedSequence(entropy=ENTROPY, spawn_key=(cfg, tensor, layer, block))
    return np.random.Generator(np.random.PCG64(ss))


def normal(cfg: int, tensor: int, layer: int, n: int, std: float = 1.0, mean: float = 0.0) -> np.ndarray:
    """n float32 draws of N(mean, std^2) from the (cfg, tensor, layer) stream."""
    out = np.empty(n, dtype=np.float32)
    nblk = (n + BLOCK - 1) // BLOCK

    def fill(b):
        lo, hi = b * BLOCK, min(n, (b + 1) * BLOCK)
        _rng(cfg, tensor, layer, b).standard_normal(hi - lo, dtype=np.float32, out=out[lo:hi])
        if std != 1.0:
            out[lo:hi] *= np.float32(std)
        if mean != 0.0:
            out[lo:hi] += np.float32(mean)

    if nblk == 1:
        fill(0)
    else:
        with ThreadPoolExecutor(_POOL_WORKERS) as ex:
            list(ex.map(fill, range(nblk)))
    return out


def uniform01(cfg: int, tensor: int, layer: int, n: int) -> np.ndarray:
    return _rng(cfg, tensor, layer, 0).random(n)


# ---------------------------------------------------------------- rounding
def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even.
    Inputs here are finite (no NaN handling needed)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """Return the storage array: float32 as is, or bf16 bit patterns (uint16)."""
    if dtype == "f32":
        return np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "bf16":
        return bf16_bits(x)
    raise ValueError(dtype)


def storage_to_f64(s: np.ndarray) -> np.ndarray:
    """Exact upcast of a storage array to float64."""
    if s.dtype == np.uint16:
        return bf16_to_f32(s).astype(np.float64)
    return s.astype(np.float64)


# ---------------------------------------------------------------- targets
def zipf_cdf(V: int, s: float = 1.1) -> np.ndarray:
    """CDF of the bounded Zipf law P(k) ~ k^-s, k = 1..V (token id = k-1)."""
    w = np.arange(1, V + 1, dtype=np.float64) ** (-s)
    c = np.cumsum(w)
    return c / c[-1]


def targets(cfg: Config, T: int | None = None) -> np.ndarray:
    T = cfg.T if T is None else T
    u = uniform01(cfg.cid, T_TARGETS, 0, T)
    if cfg.zipf:
        t = np.searchsorted(zipf_cdf(cfg.V), u, side="right")
    else:
        t = np.floor(u * cfg.V).astype(np.int64)
    return np.minimum(t, cfg.V - 1).astype(np.int32)


# ---------------------------------------------------------------- tensors
def hidden(cfg: Config) -> np.ndarray:
    """Cached final-norm input x [T, d] (storage dtype)."""
    return to_storage(normal(cfg.cid, T_X, 0, cfg.T * cfg.d).reshape(cfg.T, cfg.d), cfg.dtype)


def gain(cfg: Config) -> np.ndarray:
    """Final RMSNorm gain [d] = 1 + N(0, 0.1^2) (storage dtype)."""
    return to_storage(normal(cfg.cid, T_GAMMA, 0, cfg.d, std=0.1, mean=1.0), cfg.dtype)


def unembedding(cfg: Config) -> np.ndarray:
    """W_U [V, d] ~ N(0, 0.02^2) (storage dtype)."""
    return to_storage(normal(cfg.cid, T_WU, 0, cfg.V * cfg.d, std=0.02).reshape(cfg.V, cfg.d), cfg.dtype)


def _silu32(q: np.ndarray) -> np.ndarray:
    # forward-pass activation used only to synthesise the cached MLP input
    return q / (np.float32(1.0) + np.exp(-q))


def outlier_channels(cfg: Config, layer: int) -> np.ndarray:
    k = int(round(0.01 * cfg.d_ff))
    return _rng(cfg.cid, T_OUTLIER, layer, 0).choice(cfg.d_ff, size=k, replace=False)


def mlp_cache(cfg: Config, layer: int):
    """(q, u, a) for one target layer, each [T, d_ff] in storage dtype.

    q, u ~ N(0,1) are rounded to storage first; a = SiLU(q) * u is formed in
    float32 from the rounded values (with the outlier channels scaled x20 when
    the workload asks for them) and then rounded to storage."""
    n = cfg.T * cfg.d_ff
    q = to_storage(normal(cfg.cid, T_Q, layer, n).reshape(cfg.T, cfg.d_ff), cfg.dtype)
    u = to_storage(normal(cfg.cid, T_U, layer, n).reshape(cfg.T, cfg.d_ff), cfg.dtype)
    if cfg.dtype == "bf16":
        qf, uf = bf16_to_f32(q), bf16_to_f32(u)
    else:
        qf, uf = q, u
    a = _silu32(qf) * uf
    if cfg.outliers:
        a[:, outlier_channels(cfg, layer)] *= np.float32(20.0)
    return q, u, to_storage(a, cfg.dtype)


def activation(cfg: Config, layer: int) -> np.ndarray:
    return mlp_cache(cfg, layer)[2]


def master_weight(cfg: Config, layer: int, tensor: int = T_W, shape=None) -> np.ndarray:
    """fp32 master weight, N(0, 0.02^2). Down-projection W3 is [d, d_ff]."""
    shape = (cfg.d, cfg.d_ff) if shape is None else shape
    return normal(cfg.cid, tensor, layer, int(np.prod(shape)), std=0.02).reshape(shape)


def full_mlp_extra(cfg: Config, layer: int):
    """Inputs of the full-MLP mode for one layer: x_in [T, d] (storage dtype),
    W1 (gate) and W2 (up) masters [d_ff, d] fp32. W3_init is the layer's
    down-projection master, rounded to storage."""
    x_in = to_storage(normal(cfg.cid, T_XIN, layer, cfg.T * cfg.d).reshape(cfg.T, cfg.d), cfg.dtype)
    W1 = master_weight(cfg, layer, T_W1, (cfg.d_ff, cfg.d))
    W2 = master_weight(cfg, layer, T_W2, (cfg.d_ff, cfg.d))
    return x_in, W1, W2


def ref_noise(cfg: Config, layer: int) -> np.ndarray:
    """N(0,1) [d, d_ff] float32 for the diagnostic's reference gradient
    R = D + sigma * N, sigma = sqrt(3) * ||D||_F / sqrt(d * d_ff)."""
    return normal(cfg.cid, T_REFNOISE, layer, cfg.d * cfg.d_ff).reshape(cfg.d, cfg.d_ff)


def post_ffn(cfg: Config, layer: int):
    """Cached MLP output (the post-FFN norm's input) [T, d] and the layer's
    post-FFN gain [d], both in the storage dtype, shaped after the paper's
    OLMo-2 measurements (App. on norm statistics): per-token RMS around a layer
    mean rising from 0.9 (first target layer) to 2.7 (last), log-normal spread
    (sigma 0.3), with 1% of tokens (token 0 included, BOS-like) at RMS 0.09 so
    the min-RMS clamp is active; gain mean rising from 0.25 to 0.39 with a 10%
    per-channel spread."""
    frac = layer / max(1, cfg.L - 1)
    mean_rms = 0.9 + 1.8 * frac
    r = mean_rms * np.exp(0.3 * normal(cfg.cid, T_PFFN, 4 * layer, cfg.T))
    k = max(1, int(round(0.01 * cfg.T)))
    idx = np.unique(np.concatenate([[0], _rng(cfg.cid, T_PFFN, 4 * layer + 1, 0).choice(cfg.T, k, replace=False)]))
    r[idx] = 0.09
    z = normal(cfg.cid, T_PFFN, 4 * layer + 2, cfg.T * cfg.d).reshape(cfg.T, cfg.d)
    out = (z * r[:, None].astype(np.float32)).astype(np.float32)
    gam = ((0.25 + 0.14 * frac) * (1.0 + 0.1 * normal(cfg.cid, T_PFFN, 4 * layer + 3, cfg.d))).astype(np.float32)
    return to_storage(out, cfg.dtype), to_storage(gam, cfg.dtype)


def pre_mlp(cfg: Config, layer: int):
    """Cached pre-MLP norm input (the residual stream entering the layer's MLP
    sub-block) [T, d] and the layer's pre-MLP norm gain [d], storage dtype.
    The paper prints no statistics for this norm; the stand-in follows the
    usual growth of the residual stream with depth: per-token RMS around a
    layer mean rising from 2 (first target layer) to 8 (last), log-normal
    spread (sigma 0.3), with 1% of tokens (token 0 included) at RMS 0.3 so the
    min-RMS clamp is active; gain 1 + N(0, 0.1^2) like the final norm's."""
    frac = layer / max(1, cfg.L - 1)
    mean_rms = 2.0 + 6.0 * frac
    r = mean_rms * np.exp(0.3 * normal(cfg.cid, T_PRE, 4 * layer, cfg.T))
    k = max(1, int(round(0.01 * cfg.T)))
    idx = np.unique(np.concatenate([[0], _rng(cfg.cid, T_PRE, 4 * layer + 1, 0).choice(cfg.T, k, replace=False)]))
    r[idx] = 0.3
    z = normal(cfg.cid, T_PRE, 4 * layer + 2, cfg.T * cfg.d).reshape(cfg.T, cfg.d)
    x = (z * r[:, None].astype(np.float32)).astype(np.float32)
    gam = normal(cfg.cid, T_PRE, 4 * layer + 3, cfg.d, std=0.1, mean=1.0)
    return to_storage(x, cfg.dtype), to_storage(gam, cfg.dtype)


def rank1_reference(cfg: Config, layer: int = 0):
    """u [d], v [d_ff] float32 N(0,1): factors of a rank-1 reference gradient
    R = u v^T, whose inner product with any outer product has a closed form."""
    u = normal(cfg.cid, T_REF1, 2 * layer, cfg.d)
    v = normal(cfg.cid, T_REF1, 2 * layer + 1, cfg.d_ff)
    return u, v


def _device_generator(cfg: Config, tensor: int, layer: int, device):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(((ENTROPY * 64 + cfg.cid) * 64 + tensor) * 4096 + layer)
    return g


def device_activation(cfg: Config, layer: int, device):
    """Cached MLP activation a = SiLU(q) * u [T, d_ff] (bf16) drawn on the
    device from torch's seeded Philox stream of (cfg, layer): q, u ~ N(0,1)
    rounded to bf16 first, as in mlp_cache. For workloads whose activations
    take too long to draw on the host (the diagnostic's 36 x 8192 x 12288);
    the values differ from mlp_cache's (another generator), the distribution
    does not."""
    import torch
    g = _device_generator(cfg, T_Q, layer, device)
    q = torch.randn(cfg.T, cfg.d_ff, generator=g, device=device).to(torch.bfloat16).float()
    u = torch.randn(cfg.T, cfg.d_ff, generator=g, device=device).to(torch.bfloat16).float()
    a = (q / (1.0 + torch.exp(-q)) * u).to(torch.bfloat16)
    del q, u
    return a


def device_noise(cfg: Config, layer: int, shape, device):
    """N(0,1) float32 noise of `shape` drawn on the device (seeded Philox
    stream of (cfg, layer)): the diagnostic reference's noise term."""
    import torch
    return torch.randn(*shape, generator=_device_generator(cfg, T_REFNOISE, layer, device), device=device)


def synthetic_signal(cfg: Config, std: float = 0.02, tensor: int = T_G) -> np.ndarray:
    """A seeded stand-in for the pseudogradient signal g~ [T, d] (storage
    dtype), used to exercise the outer-product call on its own at full size."""
    return to_storage(normal(cfg.cid, tensor, 0, cfg.T * cfg.d, std=std).reshape(cfg.T, cfg.d), cfg.dtype)


# ---------------------------------------------------------------- transformer
# A decoder-only SwiGLU transformer with random weights: the model whose
# forward pass with cache and autograd gradient feed the end-to-end
# layer-viability diagnostic (Sec. 2.1-2.2). Only its weights and token ids are
# drawn here; each side of the comparison runs the model itself.
@dataclass(frozen=True)
class ModelConfig:
    mid: int            # first element of the spawn key (disjoint from Config ids)
    name: str
    V: int
    d: int
    d_ff: int
    n_layers: int
    n_heads: int
    n_kv_heads: int     # grouped key/value heads; n_heads % n_kv_heads == 0
    batch: int          # sequences
    seq: int            # tokens per sequence (T = batch * seq)
    layout: str         # "pre": norms on the block inputs (Llama, Qwen3, Falcon3)
                        # "post": norms on the block outputs (OLMo-2)
    eps: float = 1e-6
    min_rms: float = 0.5
    emb_std: float = 1.0

    @property
    def T(self) -> int:
        return self.batch * self.seq

    @property
    def head_dim(self) -> int:
        return self.d // self.n_heads

    def shrink(self, **kw) -> "ModelConfig":
        return replace(self, **kw)


MODELS = {
    "tiny": ModelConfig(200, "tiny", 512, 128, 344, 4, 4, 2, 2, 48, "pre"),
    "tiny-post": ModelConfig(201, "tiny-post", 512, 128, 344, 4, 4, 2, 2, 48, "post"),
    # several 256-wide tiles with ragged tails in T, d, d_ff and V
    "small": ModelConfig(204, "small", 2000, 384, 1032, 3, 6, 2, 3, 100, "pre"),
    "small-post": ModelConfig(205, "small-post", 2000, 384, 1032, 3, 6, 6, 3, 100, "post"),
    "qwen3-8b": ModelConfig(202, "qwen3-8b", 151936, 4096, 12288, 36, 32, 8, 16, 512, "pre"),
    "olmo2-7b": ModelConfig(203, "olmo2-7b", 100352, 4096, 11008, 32, 32, 32, 16, 512, "post"),
}

# per-layer weight names, shapes (row-major [out, in]) and fan-in; weights are
# N(0, 1/fan_in), norm gains 1 + N(0, 0.1^2)
_LAYER_SHAPES = ("wq", "wk", "wv", "wo", "w1", "w2", "w3")


def layer_shapes(m: ModelConfig) -> dict:
    hq, hkv = m.n_heads * m.head_dim, m.n_kv_heads * m.head_dim
    return {"wq": (hq, m.d), "wk": (hkv, m.d), "wv": (hkv, m.d), "wo": (m.d, hq),
            "w1": (m.d_ff, m.d), "w2": (m.d_ff, m.d), "w3": (m.d, m.d_ff)}


def model_layer(m: ModelConfig, layer: int) -> dict:
    """float32 weights of one block: wq, wk, wv, wo (attention), w1 (gate),
    w2 (up), w3 (down) and the gains n1, n2 of its two norms (before attention
    and the MLP in the "pre" layout, after them in the "post" layout)."""
    out = {}
    for k, name in enumerate(_LAYER_SHAPES):
        shp = layer_shapes(m)[name]
        out[name] = normal(m.mid, T_MODEL, 16 * (layer + 1) + k, shp[0] * shp[1],
                           std=1.0 / np.sqrt(shp[1])).reshape(shp)
    for k, name in enumerate(("n1", "n2")):
        out[name] = normal(m.mid, T_MODEL, 16 * (layer + 1) + 8 + k, m.d, std=0.1, mean=1.0)
    return out


def model_head(m: ModelConfig) -> dict:
    """float32 embedding E [V, d] (N(0, emb_std^2)), final-norm gain [d] and
    unembedding W_U [V, d] (N(0, 1/d))."""
    return {"embed": normal(m.mid, T_MODEL, 0, m.V * m.d, std=m.emb_std).reshape(m.V, m.d),
            "final_norm": normal(m.mid, T_MODEL, 1, m.d, std=0.1, mean=1.0),
            "W_U": normal(m.mid, T_MODEL, 2, m.V * m.d, std=1.0 / np.sqrt(m.d)).reshape(m.V, m.d)}


def model_tokens(m: ModelConfig) -> np.ndarray:
    """int32 token ids [batch, seq + 1], Zipf(1.1) over the vocabulary; inputs
    are ids[:, :-1] and next-token targets ids[:, 1:]."""
    n = m.batch * (m.seq + 1)
    u = uniform01(m.mid, T_MODEL, 3, n)
    t = np.minimum(np.searchsorted(zipf_cdf(m.V), u, side="right"), m.V - 1)
    return t.astype(np.int32).reshape(m.batch, m.seq + 1)


def model_weights_device(m: ModelConfig, device, seed: int = 0):
    """The distributions of model_head / model_layer drawn directly on a GPU
    with torch's seeded Philox generator (a different stream from the host
    draws): for 7-8B shapes, whose host draws would take minutes. Returns
    (head, layers) dicts of float32 device tensors."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(ENTROPY * 1000 + m.mid * 10 + seed)

    def nrm(shape, std, mean=0.0):
        t = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
        if std != 1.0:
            t.mul_(std)
        if mean != 0.0:
            t.add_(mean)
        return t

    head = {"embed": nrm((m.V, m.d), m.emb_std), "final_norm": nrm((m.d,), 0.1, 1.0),
            "W_U": nrm((m.V, m.d), 1.0 / np.sqrt(m.d))}
    layers = []
    for _ in range(m.n_layers):
        w = {name: nrm(shp, 1.0 / np.sqrt(shp[1])) for name, shp in layer_shapes(m).items()}
        w["n1"] = nrm((m.d,), 0.1, 1.0)
        w["n2"] = nrm((m.d,), 0.1, 1.0)
        layers.append(w)
    return head, layers
