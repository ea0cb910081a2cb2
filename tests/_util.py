"""Helpers shared by the GPU parity tests: moving storage arrays to the device
and the comparison metrics of the parity contract."""
import math

import numpy as np
import torch


def dev_tensor(a: np.ndarray, device) -> torch.Tensor:
    """Storage array (float32, bf16 bits as uint16, int32) -> device tensor."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(a).to(device)


def host64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64) if t.dtype == torch.bfloat16 \
        else t.detach().cpu().numpy().astype(np.float64)


def rel_fro(x, ref) -> float:
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    n = np.linalg.norm(ref)
    return float(np.linalg.norm(x - ref) / (n if n > 0 else 1.0))


def cosine(x, ref) -> float:
    x = np.asarray(x, dtype=np.float64).ravel()
    ref = np.asarray(ref, dtype=np.float64).ravel()
    nx, nr = np.linalg.norm(x), np.linalg.norm(ref)
    if nx == 0 and nr == 0:
        return 1.0
    return float(x @ ref / (nx * nr))


TOL = {"f32": 1e-5, "bf16": 2e-2}
COS_MIN = 0.9999


def assert_close(name, x, ref, dtype):
    e = rel_fro(x, ref)
    c = cosine(x, ref)
    assert e <= TOL[dtype], f"{name}: rel Frobenius error {e:.3e} > {TOL[dtype]:.0e}"
    assert c >= COS_MIN, f"{name}: cosine {c:.6f} < {COS_MIN}"
    return e


def bf16_rne_bits(x32: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def ulp_diff_f32(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """|a - b| in units of float32 ulps (same sign assumed for nonzero)."""
    ia = np.ascontiguousarray(a, dtype=np.float32).view(np.int32).astype(np.int64)
    ib = np.ascontiguousarray(b, dtype=np.float32).view(np.int32).astype(np.int64)
    ia = np.where(ia < 0, -(ia & 0x7FFFFFFF), ia)
    ib = np.where(ib < 0, -(ib & 0x7FFFFFFF), ib)
    return np.abs(ia - ib)
