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
    "fpo_abi_version", "fpo_output_error", "fpo_output_error_workspace", "fpo_pseudograd", "PostFfn",
    "fpo_pseudograd_workspace", "fpo_apply_update", "fpo_apply_update_workspace", "fpo_cosine",
    "fpo_cosine_workspace", "OptConfig", "workspace", "dtype_code",
]


def dtype_code(t: torch.dtype) -> int:
    if t == torch.bfloat16:
        return L.FPO_BF16
    if t == torch.float32:
        return L.FPO_F32
    raise TypeError(f"unsupported dtype {t}")


def _p(t: Optional[torch.Tensor], dtype: Optional[torch.dtype] = None) -> Optional[int]:
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to libfpo must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"expected a {dtype} tensor, got {t.dtype}")
    return t.data_ptr()


F32, F64, I32 = torch.float32, torch.float64, torch.int32


def _stream(dev: torch.device) -> int:
    return torch.cuda.current_stream(dev).cuda_stream


class _Keep:
    """Builds [host] pointer arrays and keeps them alive for one call."""

    def __init__(self):
        self.refs = []

    def arr(self, tensors: Optional[Sequence[Optional[torch.Tensor]]], dtype=None):
        if tensors is None:
            return None
        a = (C.c_void_p * max(1, len(tensors)))()
        for i, t in enumerate(tensors):
            a[i] = _p(t, dtype)
        self.refs.append(a)
        return C.cast(a, L.PP)

    def i64(self, vals):
        a = (C.c_int64 * len(vals))(*vals)
        self.refs.append(a)
        return a


def workspace(nbytes: int, device) -> torch.Tensor:
    """Caller-owned scratch (torch allocations are 256-byte aligned)."""
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


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
    desc = _oe_desc(T, d, V, dtype_code(op), eps, min_rms, vocab_chunk)
    lib = L.load()
    if ws is None:
        ws = workspace(lib.fpo_output_error_workspace(C.byref(desc)), h_final.device)
    L.check(lib.fpo_output_error(
        C.byref(desc), _p(h_final), _p(gamma, op), _p(W_U, op), _p(targets, I32), _p(g_tilde, F32),
        _p(g_tilde_lp, op), _p(g_pre, F32), _p(lse, F32), _p(loss, F32), _p(argmax, I32),
        _p(bad_targets, I32), _p(ws), ws.numel(),
        _stream(h_final.device)))
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


def _upd_bufs(keep: _Keep, W_master, W_lp, state1, state2, W_sumsq, clip_scale, lp_dtype):
    return L.UpdateBufs(keep.arr(W_master, F32), keep.arr(W_lp, lp_dtype), keep.arr(state1, F32),
                        keep.arr(state2, F32), _p(W_sumsq, F64), _p(clip_scale, F32))


# --------------------------------------------------------------------- pseudograd
def _mode(full_mlp: bool, post_ffn: bool, grad_bf16: bool = False) -> int:
    return ((L.FPO_MODE_FULL_MLP if full_mlp else L.FPO_MODE_W3) | (L.FPO_MODE_POST_FFN if post_ffn else 0)
            | (L.FPO_MODE_GRAD_BF16 if grad_bf16 else 0))


def fpo_pseudograd_workspace(T, d, d_ff, Lyr, dtype: torch.dtype, full_mlp=False, post_ffn=False,
                             grad_bf16=False) -> int:
    desc = L.PgDesc(T, d, d_ff, Lyr, dtype_code(dtype), _mode(full_mlp, post_ffn, grad_bf16), 1.0)
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


def fpo_pseudograd(g_tilde_lp, a, dW3=None, sumsq=None, ref=None, ref_dot=None, ref_sumsq=None,
                   W3_init=None, gate=None, up=None, x_in=None, dW1=None, dW2=None, scale=None,
                   opt: Optional[OptConfig] = None, W_master=None, W_lp=None, state1=None,
                   state2=None, W_sumsq=None, clip_scale=None, ws=None, post_ffn: Optional[PostFfn] = None,
                   grad_bf16: bool = False):
    """g_tilde_lp may be None when post_ffn is given (its left operands are
    then formed per layer from post_ffn.g_tilde). grad_bf16 (FPO_MODE_GRAD_BF16,
    fused update only, dW3 None): the pseudogradient is staged in bf16 in the
    workspace instead of being returned."""
    op = a[0].dtype
    dev = a[0].device
    T = a[0].shape[0]
    d = (g_tilde_lp if g_tilde_lp is not None else post_ffn.g_tilde).shape[1]
    Lyr = len(a)
    d_ff = a[0].shape[1]
    full = W3_init is not None
    desc = L.PgDesc(T, d, d_ff, Lyr, dtype_code(op), _mode(full, post_ffn is not None, grad_bf16),
                    (1.0 / T) if scale is None else scale)
    lib = L.load()
    if ws is None:
        ws = workspace(lib.fpo_pseudograd_workspace(C.byref(desc)), dev)
    k = _Keep()
    o = opt.c() if opt is not None else None
    ub = _upd_bufs(k, W_master, W_lp, state1, state2, W_sumsq, clip_scale, op) if opt is not None else None
    pf = None
    if post_ffn is not None:
        pf = L.PostFfn(_p(post_ffn.g_tilde, F32), k.arr(post_ffn.mlp_out, op), k.arr(post_ffn.gamma, op),
                       post_ffn.eps, post_ffn.min_rms)
    L.check(lib.fpo_pseudograd(
        C.byref(desc), _p(g_tilde_lp, op), k.arr(a, op), k.arr(W3_init, op), k.arr(gate, op), k.arr(up, op),
        k.arr(x_in, op), k.arr(dW3, F32), k.arr(dW1, F32), k.arr(dW2, F32), _p(sumsq, F64),
        k.arr(ref, F32), _p(ref_dot, F64), _p(ref_sumsq, F64), C.byref(pf) if pf is not None else None,
        C.byref(o) if o is not None else None, C.byref(ub) if ub is not None else None,
        _p(ws), ws.numel(), _stream(dev)))
    return ws


# --------------------------------------------------------------------- update
def fpo_apply_update_workspace(numels: Sequence[int]) -> int:
    k = _Keep()
    return L.load().fpo_apply_update_workspace(len(numels), k.i64(list(numels)))


def fpo_apply_update(opt: OptConfig, grad, grad_sumsq, W_master, state1, W_sumsq, W_lp=None,
                     state2=None, clip_scale=None, lp_dtype: torch.dtype = torch.bfloat16, ws=None):
    n = len(grad)
    k = _Keep()
    numel = k.i64([g.numel() for g in grad])
    lib = L.load()
    if ws is None:
        ws = workspace(lib.fpo_apply_update_workspace(n, numel), grad[0].device)
    o = opt.c()
    ub = _upd_bufs(k, W_master, W_lp, state1, state2, W_sumsq, clip_scale, lp_dtype)
    L.check(lib.fpo_apply_update(C.byref(o), n, numel, k.arr(grad, F32), _p(grad_sumsq, F64), C.byref(ub),
                                 dtype_code(lp_dtype), _p(ws), ws.numel(), _stream(grad[0].device)))
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
    L.check(lib.fpo_cosine(n, numel, k.arr(A, F32), k.arr(B, bdt), dt, _p(dot, F64), _p(sumsq_A, F64),
                           _p(sumsq_B, F64), _p(cos, F32), _p(ws), ws.numel(), _stream(A[0].device)))
    return ws
