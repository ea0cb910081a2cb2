"""Python binding of libfpo: the four calls of include/fpo.h under the same
names, taking torch tensors. Argument marshalling only: every step of the
path runs in the HIP library; torch supplies device memory and the stream.

All tensors must be on the same CUDA (HIP) device and contiguous. The
operand dtype follows h_final / g_tilde_lp: torch.bfloat16 (FPO_BF16) or
torch.float32 (FPO_F32). Work is enqueued on torch's current stream.
"""
from __future__ import annotations

import ctypes as C
from dataclasses import dataclass
from typing import Optional, Sequence

import torch

from . import _lib as L

__all__ = [
    "fpo_abi_version", "fpo_output_error", "fpo_output_error_workspace", "fpo_pseudograd", "PostFfn", "PreMlp",
    "fpo_pseudograd_workspace", "fpo_apply_update", "fpo_apply_update_workspace", "fpo_cosine", "Overlap",
    "fpo_cosine_workspace", "OptConfig", "workspace", "dtype_code",
]


def dtype_code(t: torch.dtype) -> int:
    if t == torch.bfloat16:
        return L.FPO_BF16
    if t == torch.float32:
        return L.FPO_F32
    raise TypeError(f"unsupported dtype {t}")


def _p(t: Optional[torch.Tensor], dtype: Optional[torch.dtype] = None, shape=None, dev=None,
       name: str = "tensor") -> Optional[int]:
    """Device pointer of t after the checks the C ABI cannot make from a bare
    pointer: a contiguous tensor on the (given) GPU, of the given dtype and
    shape (a tuple: exact; an int: at least that many elements)."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ValueError(f"{name}: libfpo takes GPU tensors")
    if dev is not None and t.device != dev:
        raise ValueError(f"{name}: on {t.device}, expected {dev}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: tensors passed to libfpo must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name}: expected a {dtype} tensor, got {t.dtype}")
    if isinstance(shape, tuple) and tuple(t.shape) != shape:
        raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {shape}")
    if isinstance(shape, int) and t.numel() < shape:
        raise ValueError(f"{name}: {t.numel()} elements, at least {shape} needed")
    return t.data_ptr()


F32, F64, I32 = torch.float32, torch.float64, torch.int32


def _stream(dev: torch.device) -> int:
    return torch.cuda.current_stream(dev).cuda_stream


class _Keep:
    """Builds [host] pointer arrays and keeps them alive for one call."""

    def __init__(self):
        self.refs = []

    def arr(self, tensors: Optional[Sequence[Optional[torch.Tensor]]], dtype=None, shape=None, dev=None,
            n: Optional[int] = None, name: str = "tensors"):
        """[host] array of device pointers; n: required length; shape per
        entry (a tuple, or a callable of the index)."""
        if tensors is None:
            return None
        if n is not None and len(tensors) != n:
            raise ValueError(f"{name}: {len(tensors)} entries, expected {n}")
        a = (C.c_void_p * max(1, len(tensors)))()
        for i, t in enumerate(tensors):
            a[i] = _p(t, dtype, shape(i) if callable(shape) else shape, dev, f"{name}[{i}]")
        self.refs.append(a)
        return C.cast(a, L.PP)

    def i64(self, vals):
        a = (C.c_int64 * len(vals))(*vals)
        self.refs.append(a)
        return a


def workspace(nbytes: int, device) -> torch.Tensor:
    """Caller-owned scratch (torch allocations are 256-byte aligned)."""
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def _nbytes(t: torch.Tensor) -> int:
    return t.numel() * t.element_size()


def fpo_abi_version() -> int:
    return L.load().fpo_abi_version()


# --------------------------------------------------------------------- output error
def _oe_desc(T, d, V, dtype, eps, min_rms, vocab_chunk):
    return L.OeDesc(T, d, V, dtype, eps, min_rms, vocab_chunk)


def fpo_output_error_workspace(T: int, d: int, V: int, dtype: torch.dtype, vocab_chunk: int = 0) -> int:
    desc = _oe_desc(T, d, V, dtype_code(dtype), 0.0, 0.0, vocab_chunk)
    return L.load().fpo_output_error_workspace(C.byref(desc))


def fpo_output_error(h_final, gamma, W_U, targets, g_tilde, g_tilde_lp=None, g_pre=None, lse=None,
                     loss=None, argmax=None, bad_targets=None, ws=None, eps=1e-6, min_rms=0.5,
                     vocab_chunk=0):
    T, d = h_final.shape
    V = W_U.shape[0]
    op = h_final.dtype
    dev = h_final.device
    desc = _oe_desc(T, d, V, dtype_code(op), eps, min_rms, vocab_chunk)
    lib = L.load()
    if ws is None:
        ws = workspace(lib.fpo_output_error_workspace(C.byref(desc)), dev)
    L.check(lib.fpo_output_error(
        C.byref(desc), _p(h_final, op, (T, d), dev, "h_final"), _p(gamma, op, (d,), dev, "gamma"),
        _p(W_U, op, (V, d), dev, "W_U"), _p(targets, I32, (T,), dev, "targets"),
        _p(g_tilde, F32, (T, d), dev, "g_tilde"), _p(g_tilde_lp, op, (T, d), dev, "g_tilde_lp"),
        _p(g_pre, F32, (T, d), dev, "g_pre"), _p(lse, F32, (T,), dev, "lse"), _p(loss, F32, (T,), dev, "loss"),
        _p(argmax, I32, (T,), dev, "argmax"), _p(bad_targets, I32, 1, dev, "bad_targets"),
        _p(ws, None, None, dev, "ws"), _nbytes(ws), _stream(dev)))
    return ws


# --------------------------------------------------------------------- optimizer
@dataclass
class OptConfig:
    kind: int = L.FPO_OPT_SGD
    lr: float = 1e-4
    momentum: float = 0.9
    beta1: float = 0.9
    beta2: float = 0.999
    adam_eps: float = 1e-8
    weight_decay: float = 0.01
    clip_frac: float = 0.01
    step: int = 1
    clip_target: int = L.FPO_CLIP_GRADIENT  # or L.FPO_CLIP_UPDATE: bound ||W' - W|| instead of ||dW||

    def c(self) -> L.Opt:
        return L.Opt(self.kind, self.lr, self.momentum, self.beta1, self.beta2, self.adam_eps,
                     self.weight_decay, self.clip_frac, self.step, self.clip_target)


def _upd_bufs(keep: _Keep, W_master, W_lp, state1, state2, W_sumsq, clip_scale, lp_dtype, numels, dev):
    """Update buffers of len(numels) matrices, entry m of numels[m] elements."""
    n = len(numels)
    if W_master is None:
        raise ValueError("W_master is required")
    sh = lambda m: numels[m]  # noqa: E731

    def same(ts, name):
        if ts is not None:
            for m, t in enumerate(ts):
                if t is not None and t.numel() != numels[m]:
                    raise ValueError(f"{name}[{m}]: {t.numel()} elements, expected {numels[m]}")

    for ts, name in ((W_master, "W_master"), (W_lp, "W_lp"), (state1, "state1"), (state2, "state2")):
        same(ts, name)
    return L.UpdateBufs(keep.arr(W_master, F32, sh, dev, n, "W_master"), keep.arr(W_lp, lp_dtype, sh, dev, n, "W_lp"),
                        keep.arr(state1, F32, sh, dev, n, "state1"), keep.arr(state2, F32, sh, dev, n, "state2"),
                        _p(W_sumsq, F64, n, dev, "W_sumsq"), _p(clip_scale, F32, n, dev, "clip_scale"))


# --------------------------------------------------------------------- pseudograd
def _mode(full_mlp: bool, post_ffn: bool, grad_bf16: bool = False, pre_mlp: bool = False) -> int:
    return ((L.FPO_MODE_FULL_MLP if full_mlp else L.FPO_MODE_W3) | (L.FPO_MODE_POST_FFN if post_ffn else 0)
            | (L.FPO_MODE_GRAD_BF16 if grad_bf16 else 0) | (L.FPO_MODE_PRE_MLP if pre_mlp else 0))


def fpo_pseudograd_workspace(T, d, d_ff, Lyr, dtype: torch.dtype, full_mlp=False, post_ffn=False,
                             grad_bf16=False, pre_mlp=False) -> int:
    desc = L.PgDesc(T, d, d_ff, Lyr, dtype_code(dtype), _mode(full_mlp, post_ffn, grad_bf16, pre_mlp), 1.0)
    return L.load().fpo_pseudograd_workspace(C.byref(desc))


@dataclass
class PostFfn:
    """Per-layer post-feedforward RMSNorm composition (fpo_post_ffn): the fp32
    g~ [T, d], each target layer's cached MLP output [T, d] and post-FFN gain
    [d] (operand dtype)."""
    g_tilde: torch.Tensor
    mlp_out: Sequence[torch.Tensor]
    gamma: Sequence[torch.Tensor]
    eps: float = 1e-6
    min_rms: float = 0.5


@dataclass
class PreMlp:
    """Per-layer pre-MLP RMSNorm composition (fpo_pre_mlp): the fp32 g~ [T, d]
    (the same tensor as PostFfn.g_tilde when both are given), each target
    layer's cached pre-MLP norm input [T, d] and gain [d] (operand dtype)."""
    g_tilde: torch.Tensor
    x: Sequence[torch.Tensor]
    gamma: Sequence[torch.Tensor]
    eps: float = 1e-6
    min_rms: float = 0.5


class Overlap:
    """The caller's own side stream and two events for fpo_pseudograd's
    overlapped optimizer path (fpo_overlap): a torch stream at the default
    priority and two torch events (created here by recording them once).
    Keep one per concurrent caller; it holds no device memory."""

    def __init__(self, device=None):
        self.stream = torch.cuda.Stream(device=device)
        self.ready = torch.cuda.Event()
        self.done = torch.cuda.Event()
        self.ready.record(self.stream)
        self.done.record(self.stream)

    def c(self) -> L.Overlap:
        return L.Overlap(self.stream.cuda_stream, self.ready.cuda_event, self.done.cuda_event)


def fpo_pseudograd(g_tilde_lp, a, dW3=None, sumsq=None, ref=None, ref_dot=None, ref_sumsq=None,
                   W3_init=None, gate=None, up=None, x_in=None, dW1=None, dW2=None, scale=None,
                   opt: Optional[OptConfig] = None, W_master=None, W_lp=None, state1=None,
                   state2=None, W_sumsq=None, clip_scale=None, ws=None, post_ffn: Optional[PostFfn] = None,
                   grad_bf16: bool = False, ref_cos=None, overlap: Optional[Overlap] = None,
                   pre_mlp: Optional[PreMlp] = None):
    """g_tilde_lp may be None when post_ffn is given (its left operands are
    then formed per layer from post_ffn.g_tilde). grad_bf16 (FPO_MODE_GRAD_BF16,
    fused update only, dW3 None): the pseudogradient is staged in bf16 in the
    workspace instead of being returned. ref_cos (float32 [L]): the per-layer
    cosine with ref, computed in the library. overlap: the side stream and
    events of the overlapped optimizer path (default: the library's own)."""
    op = a[0].dtype
    dev = a[0].device
    T = a[0].shape[0]
    d = (g_tilde_lp if g_tilde_lp is not None else (post_ffn or pre_mlp).g_tilde).shape[1]
    Lyr = len(a)
    d_ff = a[0].shape[1]
    full = W3_init is not None
    desc = L.PgDesc(T, d, d_ff, Lyr, dtype_code(op),
                    _mode(full, post_ffn is not None, grad_bf16, pre_mlp is not None),
                    (1.0 / T) if scale is None else scale)
    lib = L.load()
    if ws is None:
        ws = workspace(lib.fpo_pseudograd_workspace(C.byref(desc)), dev)
    k = _Keep()
    o = opt.c() if opt is not None else None
    nm = 3 * Lyr if full else Lyr
    numels = [d * d_ff] * nm
    ub = (_upd_bufs(k, W_master, W_lp, state1, state2, W_sumsq, clip_scale, op, numels, dev)
          if opt is not None else None)
    ov = overlap.c() if overlap is not None else None
    pm = None
    if pre_mlp is not None:
        pm = L.PreMlp(_p(pre_mlp.g_tilde, F32, (T, d), dev, "pre_mlp.g_tilde"),
                      k.arr(pre_mlp.x, op, (T, d), dev, Lyr, "pre_mlp.x"),
                      k.arr(pre_mlp.gamma, op, (d,), dev, Lyr, "pre_mlp.gamma"), pre_mlp.eps, pre_mlp.min_rms)
    pf = None
    if post_ffn is not None:
        pf = L.PostFfn(_p(post_ffn.g_tilde, F32, (T, d), dev, "post_ffn.g_tilde"),
                       k.arr(post_ffn.mlp_out, op, (T, d), dev, Lyr, "post_ffn.mlp_out"),
                       k.arr(post_ffn.gamma, op, (d,), dev, Lyr, "post_ffn.gamma"), post_ffn.eps, post_ffn.min_rms)
    L.check(lib.fpo_pseudograd(
        C.byref(desc), _p(g_tilde_lp, op, (T, d), dev, "g_tilde_lp"), k.arr(a, op, (T, d_ff), dev, Lyr, "a"),
        k.arr(W3_init, op, (d, d_ff), dev, Lyr, "W3_init"), k.arr(gate, op, (T, d_ff), dev, Lyr, "gate"),
        k.arr(up, op, (T, d_ff), dev, Lyr, "up"), k.arr(x_in, op, (T, d), dev, Lyr, "x_in"),
        k.arr(dW3, F32, (d, d_ff), dev, Lyr, "dW3"), k.arr(dW1, F32, (d_ff, d), dev, Lyr, "dW1"),
        k.arr(dW2, F32, (d_ff, d), dev, Lyr, "dW2"), _p(sumsq, F64, nm, dev, "sumsq"),
        k.arr(ref, F32, (d, d_ff), dev, Lyr, "ref"), _p(ref_dot, F64, Lyr, dev, "ref_dot"),
        _p(ref_sumsq, F64, Lyr, dev, "ref_sumsq"), _p(ref_cos, F32, Lyr, dev, "ref_cos"),
        C.byref(pf) if pf is not None else None, C.byref(pm) if pm is not None else None,
        C.byref(o) if o is not None else None, C.byref(ub) if ub is not None else None,
        C.byref(ov) if ov is not None else None, _p(ws, None, None, dev, "ws"), _nbytes(ws), _stream(dev)))
    return ws


# --------------------------------------------------------------------- update
def fpo_apply_update_workspace(numels: Sequence[int]) -> int:
    k = _Keep()
    return L.load().fpo_apply_update_workspace(len(numels), k.i64(list(numels)))


def fpo_apply_update(opt: OptConfig, grad, grad_sumsq, W_master, state1, W_sumsq, W_lp=None,
                     state2=None, clip_scale=None, lp_dtype: torch.dtype = torch.bfloat16, ws=None):
    n = len(grad)
    k = _Keep()
    numels = [g.numel() for g in grad]
    numel = k.i64(numels)
    dev = grad[0].device
    lib = L.load()
    if ws is None:
        ws = workspace(lib.fpo_apply_update_workspace(n, numel), dev)
    o = opt.c()
    ub = _upd_bufs(k, W_master, W_lp, state1, state2, W_sumsq, clip_scale, lp_dtype, numels, dev)
    L.check(lib.fpo_apply_update(C.byref(o), n, numel, k.arr(grad, F32, None, dev, n, "grad"),
                                 _p(grad_sumsq, F64, n, dev, "grad_sumsq"), C.byref(ub), dtype_code(lp_dtype),
                                 _p(ws, None, None, dev, "ws"), _nbytes(ws), _stream(dev)))
    return ws


# --------------------------------------------------------------------- cosine
def fpo_cosine_workspace(numels: Sequence[int]) -> int:
    k = _Keep()
    return L.load().fpo_cosine_workspace(len(numels), k.i64(list(numels)))


def fpo_cosine(A, B=None, dot=None, sumsq_A=None, sumsq_B=None, cos=None, ws=None):
    n = len(A)
    k = _Keep()
    numel = k.i64([t.numel() for t in A])
    lib = L.load()
    if ws is None:
        ws = workspace(lib.fpo_cosine_workspace(n, numel), A[0].device)
    bdt = B[0].dtype if B is not None else F32
    dt = dtype_code(bdt)
    dev = A[0].device
    if B is not None:
        if len(B) != n:
            raise ValueError(f"B: {len(B)} entries, expected {n}")
        for m in range(n):
            if B[m].numel() != A[m].numel():
                raise ValueError(f"B[{m}]: {B[m].numel()} elements, A[{m}] has {A[m].numel()}")
    L.check(lib.fpo_cosine(n, numel, k.arr(A, F32, None, dev, n, "A"), k.arr(B, bdt, None, dev, n, "B"), dt,
                           _p(dot, F64, n, dev, "dot"), _p(sumsq_A, F64, n, dev, "sumsq_A"),
                           _p(sumsq_B, F64, n, dev, "sumsq_B"), _p(cos, F32, n, dev, "cos"),
                           _p(ws, None, None, dev, "ws"), _nbytes(ws), _stream(dev)))
    return ws
