"""ctypes declarations for libcaddtree.so (the C ABI in include/caddtree.h)."""

from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcaddtree.so")

OK, E_INVALID, E_UNSUPPORTED, E_COST, E_WORKSPACE, E_HIP = range(6)
DTYPES = {"f32": 0, "bf16": 1}
MASKS = {"none": 0, "u8": 1, "bits": 2}
ALLOW_NONCONVEX = 1
FIXED_BUDGET = 2
MAX_L, MAX_K, MAX_CAP, MAX_CTX = 32, 16, 4096, 64
NOALLOC_SCRATCH_BYTES = 8 << 20


class CaddtreeError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"caddtree status {status}: {message}")
        self.status = status


class Config(ctypes.Structure):
    _fields_ = [
        ("L", ctypes.c_int32),
        ("V", ctypes.c_int64),
        ("K", ctypes.c_int32),
        ("budget_cap", ctypes.c_int32),
        ("dtype", ctypes.c_int),
        ("mask", ctypes.c_int),
        ("flags", ctypes.c_uint32),
        ("t_draft", ctypes.c_double),
        ("t_verify_host", ctypes.POINTER(ctypes.c_double)),
        ("n_ctx", ctypes.c_int32),
        ("ctx_grid_host", ctypes.POINTER(ctypes.c_int64)),
    ]


class Outputs(ctypes.Structure):
    _fields_ = [(name, ctypes.c_void_p) for name in (
        "token_ids", "parent", "depth", "path_prob", "n_star", "phi", "theta",
        "mask", "pos_ids", "topk_ids", "topk_logit", "topk_lq", "lse")]


EXPORTS = [
    "caddtree_plan_create", "caddtree_plan_destroy", "caddtree_workspace_bytes", "caddtree_build",
    "caddtree_build_noalloc",
    "caddtree_reduce_topk", "caddtree_expand", "caddtree_emit", "caddtree_accept", "caddtree_fit_cost", "caddtree_status_string",
    "caddtree_last_error",
]


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build the HIP library first (python -m paper_2606_01813_amd._build)")
    # PyTorch-ROCm ships its own HIP runtime under the same soname (libamdhip64.so.7).  Importing
    # torch first makes this library bind to that runtime, so the tensors' memory and streams and
    # the kernels share one runtime; in the other order torch would later find no GPU.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(path)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    lib.caddtree_plan_create.argtypes = [ctypes.POINTER(Config), ctypes.POINTER(vp)]
    lib.caddtree_plan_create.restype = ctypes.c_int
    lib.caddtree_plan_destroy.argtypes = [vp]
    lib.caddtree_plan_destroy.restype = None
    lib.caddtree_workspace_bytes.argtypes = [vp, i64]
    lib.caddtree_workspace_bytes.restype = sz
    lib.caddtree_build.argtypes = [vp, vp, i64, i64, i32, vp, ctypes.POINTER(Outputs), vp, sz, vp]
    lib.caddtree_build.restype = ctypes.c_int
    lib.caddtree_build_noalloc.argtypes = [vp, vp, i64, i64, i32, vp, ctypes.POINTER(Outputs), vp]
    lib.caddtree_build_noalloc.restype = ctypes.c_int
    lib.caddtree_reduce_topk.argtypes = [vp, vp, i64, i64, vp, vp, vp, vp, vp]
    lib.caddtree_reduce_topk.restype = ctypes.c_int
    lib.caddtree_expand.argtypes = [vp, vp, vp, vp, i64, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.caddtree_expand.restype = ctypes.c_int
    lib.caddtree_emit.argtypes = [vp, vp, vp, vp, i64, i32, vp, vp, vp]
    lib.caddtree_emit.restype = ctypes.c_int
    lib.caddtree_accept.argtypes = [vp, vp, vp, vp, i64, vp, vp, i32, vp, vp, vp, vp, vp, vp]
    lib.caddtree_accept.restype = ctypes.c_int
    lib.caddtree_fit_cost.argtypes = [vp, vp, i64, vp, i32, vp]
    lib.caddtree_fit_cost.restype = ctypes.c_int
    lib.caddtree_status_string.argtypes = [ctypes.c_int]
    lib.caddtree_status_string.restype = ctypes.c_char_p
    lib.caddtree_last_error.argtypes = []
    lib.caddtree_last_error.restype = ctypes.c_char_p
    return lib


_LIB = None


def lib() -> ctypes.CDLL:
    global _LIB
    if _LIB is None:
        _LIB = load()
    return _LIB


def check(status: int) -> None:
    if status != OK:
        msg = lib().caddtree_last_error().decode(errors="replace")
        name = lib().caddtree_status_string(status).decode()
        raise CaddtreeError(status, f"{name}: {msg}")
