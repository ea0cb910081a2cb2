"""ctypes declaration of the libfpo C ABI (include/fpo.h).

Loads paper_2608_14563_amd/libfpo.so from the package directory and raises if
it is missing: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfpo.so")

FPO_OK, FPO_ERR_NULL, FPO_ERR_SHAPE, FPO_ERR_DTYPE, FPO_ERR_ARG, FPO_ERR_WORKSPACE, FPO_ERR_UNSUPPORTED, FPO_ERR_HIP = range(8)
FPO_F32, FPO_BF16 = 0, 1
FPO_MODE_W3, FPO_MODE_FULL_MLP, FPO_MODE_POST_FFN, FPO_MODE_GRAD_BF16, FPO_MODE_PRE_MLP = 0, 1, 2, 4, 8  # bit flags
FPO_OPT_SGD, FPO_OPT_ADAMW = 0, 1
FPO_CLIP_GRADIENT, FPO_CLIP_UPDATE = 0, 1

STATUS_NAMES = {0: "FPO_OK", 1: "FPO_ERR_NULL", 2: "FPO_ERR_SHAPE", 3: "FPO_ERR_DTYPE", 4: "FPO_ERR_ARG",
                5: "FPO_ERR_WORKSPACE", 6: "FPO_ERR_UNSUPPORTED", 7: "FPO_ERR_HIP"}

EXPORTS = (
    "fpo_abi_version", "fpo_last_error", "fpo_output_error_workspace", "fpo_output_error",
    "fpo_pseudograd_workspace", "fpo_pseudograd", "fpo_apply_update_workspace", "fpo_apply_update",
    "fpo_cosine_workspace", "fpo_cosine", "fpo_apply_update_noalloc",
)
NOALLOC_SCRATCH_BYTES = 8 << 20  # FPO_NOALLOC_SCRATCH_BYTES


class OeDesc(C.Structure):
    _fields_ = [("T", C.c_int64), ("d", C.c_int64), ("V", C.c_int64), ("dtype", C.c_int32),
                ("eps", C.c_float), ("min_rms", C.c_float), ("vocab_chunk", C.c_int64)]


class PgDesc(C.Structure):
    _fields_ = [("T", C.c_int64), ("d", C.c_int64), ("d_ff", C.c_int64), ("L", C.c_int64),
                ("dtype", C.c_int32), ("mode", C.c_int32), ("scale", C.c_float)]


class Opt(C.Structure):
    _fields_ = [("kind", C.c_int32), ("lr", C.c_double), ("momentum", C.c_double), ("beta1", C.c_double),
                ("beta2", C.c_double), ("adam_eps", C.c_double), ("weight_decay", C.c_double),
                ("clip_frac", C.c_double), ("step", C.c_int64), ("clip_target", C.c_int32)]


class UpdateBufs(C.Structure):
    _fields_ = [("W_master", C.POINTER(C.c_void_p)), ("W_lp", C.POINTER(C.c_void_p)),
                ("state1", C.POINTER(C.c_void_p)), ("state2", C.POINTER(C.c_void_p)),
                ("W_sumsq", C.c_void_p), ("clip_scale", C.c_void_p)]


class PostFfn(C.Structure):
    _fields_ = [("g_tilde", C.c_void_p), ("mlp_out", C.POINTER(C.c_void_p)), ("gamma", C.POINTER(C.c_void_p)),
                ("eps", C.c_float), ("min_rms", C.c_float)]


class PreMlp(C.Structure):
    _fields_ = [("g_tilde", C.c_void_p), ("x", C.POINTER(C.c_void_p)), ("gamma", C.POINTER(C.c_void_p)),
                ("eps", C.c_float), ("min_rms", C.c_float)]


class Overlap(C.Structure):
    _fields_ = [("side_stream", C.c_void_p), ("ready_event", C.c_void_p), ("done_event", C.c_void_p)]


ABI_VERSION = 7
PP = C.POINTER(C.c_void_p)
VP = C.c_void_p
_lib = None


class FpoError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def load() -> C.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is not built; run `python -m paper_2608_14563_amd.build` "
            "(or __graft_entry__.build()). There is no fallback path.")
    lib = C.CDLL(LIB_PATH)
    lib.fpo_abi_version.restype = C.c_int
    lib.fpo_abi_version.argtypes = []
    if lib.fpo_abi_version() != ABI_VERSION:
        raise RuntimeError(f"{LIB_PATH} has ABI version {lib.fpo_abi_version()}, this binding expects "
                           f"{ABI_VERSION}: rebuild the library")
    lib.fpo_last_error.restype = C.c_char_p
    lib.fpo_last_error.argtypes = []
    lib.fpo_output_error_workspace.restype = C.c_size_t
    lib.fpo_output_error_workspace.argtypes = [C.POINTER(OeDesc)]
    lib.fpo_output_error.restype = C.c_int
    lib.fpo_output_error.argtypes = [C.POINTER(OeDesc), VP, VP, VP, VP, VP, VP, VP, VP, VP, VP, VP,
                                     VP, C.c_size_t, VP]
    lib.fpo_pseudograd_workspace.restype = C.c_size_t
    lib.fpo_pseudograd_workspace.argtypes = [C.POINTER(PgDesc)]
    lib.fpo_pseudograd.restype = C.c_int
    lib.fpo_pseudograd.argtypes = [C.POINTER(PgDesc), VP, PP, PP, PP, PP, PP, PP, PP, PP, VP, PP, VP,
                                   VP, VP, C.POINTER(PostFfn), C.POINTER(PreMlp), C.POINTER(Opt),
                                   C.POINTER(UpdateBufs), C.POINTER(Overlap), VP, C.c_size_t, VP]
    lib.fpo_apply_update_workspace.restype = C.c_size_t
    lib.fpo_apply_update_workspace.argtypes = [C.c_int64, C.POINTER(C.c_int64)]
    lib.fpo_apply_update.restype = C.c_int
    lib.fpo_apply_update.argtypes = [C.POINTER(Opt), C.c_int64, C.POINTER(C.c_int64), PP, VP,
                                     C.POINTER(UpdateBufs), C.c_int32, VP, C.c_size_t, VP]
    lib.fpo_apply_update_noalloc.restype = C.c_int
    lib.fpo_apply_update_noalloc.argtypes = [C.POINTER(Opt), C.c_int64, C.POINTER(C.c_int64), PP, VP,
                                             C.POINTER(UpdateBufs), C.c_int32, VP]
    lib.fpo_cosine_workspace.restype = C.c_size_t
    lib.fpo_cosine_workspace.argtypes = [C.c_int64, C.POINTER(C.c_int64)]
    lib.fpo_cosine.restype = C.c_int
    lib.fpo_cosine.argtypes = [C.c_int64, C.POINTER(C.c_int64), PP, PP, C.c_int32, VP, VP, VP, VP, VP,
                               C.c_size_t, VP]
    _lib = lib
    return lib


def check(status: int) -> None:
    if status != FPO_OK:
        raise FpoError(status, load().fpo_last_error().decode())
