"""CaDDTree draft-tree construction on MI355X (gfx950): Python binding.

A thin marshalling layer over libcaddtree.so (include/caddtree.h): it turns
torch tensors into device pointers and the current torch stream into the HIP
stream, and calls the library.  Every step of the hot path runs in the HIP
kernels; there is no fallback.  Importing works without a GPU (the library
loads on first use); calls need the built library and a gfx950 device.

    plan = Plan(L=16, V=151936, K=8, cap=512, t_draft=1.0, t_verify=table,
                dtype="bf16", mask="u8")
    out = plan.new_outputs(B)                 # torch tensors on the current device
    ws = plan.new_workspace(B)
    plan.build(logits, out, workspace=ws)      # logits: [B, L, >=V] bf16 tensor

Context-aware cost (Sec. 4.6): pass ``t_verify`` as [J, cap + 1] tables with
``ctx_grid`` (J increasing context lengths) and give ``ctx_len`` (int64 [B],
on the device) to ``build`` / ``expand``.  ``fixed_budget=True`` selects the
fixed-budget (DDTree) construction: the top ``cap`` nodes, no stop rule.
"""

from __future__ import annotations

import ctypes
import dataclasses
from typing import Optional

import numpy as np

from . import _lib
from ._lib import CaddtreeError, MAX_CAP, MAX_CTX, MAX_K, MAX_L

__all__ = ["Plan", "TreeOutputs", "CaddtreeError", "fit_cost", "MAX_L", "MAX_K", "MAX_CAP", "MAX_CTX"]


def _torch():
    import torch
    return torch


def _ptr(t) -> Optional[int]:
    return None if t is None else int(t.data_ptr())


def _stream(stream, device) -> int:
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream)


def _on_device(t, device: int) -> bool:
    return bool(t.is_cuda) and t.device.index == device


def _check(name: str, t, dtype, dims, B: int, device: int, required: bool = True) -> None:
    """Raises unless ``t`` is a contiguous tensor of ``dtype`` on cuda:``device`` shaped [>= B, *dims]."""
    torch = _torch()
    if t is None:
        if required:
            raise ValueError(f"{name} is required")
        return
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor, got {type(t).__name__}")
    if not _on_device(t, device):
        raise ValueError(f"{name} must be on cuda:{device} (the plan's device), got {t.device}")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.dim() != 1 + len(dims) or t.shape[0] < B or tuple(t.shape[1:]) != tuple(dims):
        raise ValueError(f"{name} must have shape [>= {B}{''.join(', ' + str(d) for d in dims)}], "
                         f"got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def fit_cost(x, y, cap: Optional[int] = None):
    """Convex non-decreasing least-squares fit of a cost profile (host, ``caddtree_fit_cost``).

    Returns the fitted values at ``x``, and with ``cap`` also the cost table C_v(0 .. cap)."""
    xs = np.ascontiguousarray(np.asarray(x, dtype=np.float64))
    ys = np.ascontiguousarray(np.asarray(y, dtype=np.float64))
    if xs.ndim != 1 or xs.shape != ys.shape:
        raise ValueError("x and y must be 1-d arrays of equal length")
    fit = np.empty_like(xs)
    table = None if cap is None else np.empty(int(cap) + 1, dtype=np.float64)
    dp = lambda a: None if a is None else a.ctypes.data
    _lib.check(_lib.lib().caddtree_fit_cost(dp(xs), dp(ys), int(xs.shape[0]), dp(fit),
                                            -1 if cap is None else int(cap), dp(table)))
    return fit if cap is None else (fit, table)


@dataclasses.dataclass
class TreeOutputs:
    """Device tensors written by Plan.build (see caddtree_outputs_t)."""
    token_ids: object
    parent: object
    depth: object
    path_prob: object
    n_star: object
    phi: object
    theta: object
    mask: object = None
    pos_ids: object = None
    topk_ids: object = None
    topk_logit: object = None
    topk_lq: object = None
    lse: object = None

    def as_struct(self) -> _lib.Outputs:
        s = _lib.Outputs()
        for f in _lib.Outputs._fields_:
            setattr(s, f[0], _ptr(getattr(self, f[0])))
        return s


class Plan:
    """An immutable CaDDTree plan (shape limits, dtype, mask format, cost model)."""

    def __init__(self, L: int, V: int, K: int, cap: int, t_draft: float, t_verify,
                 dtype: str = "bf16", mask: str = "u8", allow_nonconvex: bool = False,
                 ctx_grid=None, fixed_budget: bool = False):
        self.L, self.V, self.K, self.cap = int(L), int(V), int(K), int(cap)
        self.dtype, self.mask = dtype, mask
        if dtype not in _lib.DTYPES:
            raise ValueError(f"dtype must be one of {sorted(_lib.DTYPES)}")
        if mask not in _lib.MASKS:
            raise ValueError(f"mask must be one of {sorted(_lib.MASKS)}")
        tv = np.asarray(t_verify, dtype=np.float64)
        if ctx_grid is None:
            if tv.ndim != 1 or tv.shape[0] < self.cap + 1:
                raise ValueError(f"t_verify needs cap + 1 = {self.cap + 1} values")
            tv = np.ascontiguousarray(tv[: self.cap + 1])
            grid = np.zeros(1, dtype=np.int64)
            n_ctx = 1
        else:
            grid = np.ascontiguousarray(np.asarray(ctx_grid, dtype=np.int64))
            n_ctx = int(grid.shape[0])
            if tv.ndim != 2 or tv.shape[0] != n_ctx or tv.shape[1] < self.cap + 1:
                raise ValueError(f"t_verify needs [len(ctx_grid), cap + 1] = [{n_ctx}, {self.cap + 1}] values")
            tv = np.ascontiguousarray(tv[:, : self.cap + 1])
        self._tv, self._grid, self.n_ctx = tv, grid, n_ctx
        self.fixed_budget = bool(fixed_budget)
        flags = (_lib.ALLOW_NONCONVEX if allow_nonconvex else 0) | (_lib.FIXED_BUDGET if fixed_budget else 0)
        cfg = _lib.Config(self.L, self.V, self.K, self.cap, _lib.DTYPES[dtype], _lib.MASKS[mask],
                          flags, float(t_draft), tv.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                          n_ctx, grid.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)))
        self._lib = _lib.lib()
        h = ctypes.c_void_p()
        _lib.check(self._lib.caddtree_plan_create(ctypes.byref(cfg), ctypes.byref(h)))
        self._h = h
        self.device = _torch().cuda.current_device()   # the library binds the plan to this device

    # ------------------------------------------------------------ lifetime
    def close(self) -> None:
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            self._lib.caddtree_plan_destroy(h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    # ------------------------------------------------------------ allocation helpers
    def workspace_bytes(self, B: int) -> int:
        return int(self._lib.caddtree_workspace_bytes(self._h, int(B)))

    def new_workspace(self, B: int, device=None):
        torch = _torch()
        n = max(self.workspace_bytes(B), 1)
        return torch.empty(n, dtype=torch.uint8, device=device or "cuda")

    def new_outputs(self, B: int, device=None, topk: bool = False) -> TreeOutputs:
        torch = _torch()
        dev = device or "cuda"
        cap = max(self.cap, 1)
        i32 = dict(dtype=torch.int32, device=dev)
        f32 = dict(dtype=torch.float32, device=dev)
        mask = None
        if self.mask == "u8":
            mask = torch.zeros((B, cap, cap), dtype=torch.uint8, device=dev)
        elif self.mask == "bits":
            mask = torch.zeros((B, cap, (cap + 31) // 32), dtype=torch.int32, device=dev)
        out = TreeOutputs(
            token_ids=torch.full((B, cap), -1, **i32), parent=torch.full((B, cap), -2, **i32),
            depth=torch.zeros((B, cap), **i32), path_prob=torch.zeros((B, cap), **f32),
            n_star=torch.full((B,), -1, **i32), phi=torch.zeros((B,), **f32), theta=torch.zeros((B,), **f32),
            mask=mask, pos_ids=torch.zeros((B, cap), **i32))
        if topk:
            out.topk_ids = torch.empty((B, self.L, self.K), **i32)
            out.topk_logit = torch.empty((B, self.L, self.K), **f32)
            out.topk_lq = torch.empty((B, self.L, self.K), **f32)
            out.lse = torch.empty((B, self.L), dtype=torch.float64, device=dev)
        return out

    # ------------------------------------------------------------ calls
    # ------------------------------------------------------------ argument checks (before any C call)
    def _logits(self, logits):
        torch = _torch()
        want = torch.bfloat16 if self.dtype == "bf16" else torch.float32
        if not isinstance(logits, torch.Tensor):
            raise TypeError(f"logits must be a torch tensor, got {type(logits).__name__}")
        if not _on_device(logits, self.device):
            raise ValueError(f"logits must be on cuda:{self.device} (the plan's device), got {logits.device}")
        if logits.dtype != want:
            raise TypeError(f"logits must be {want}, got {logits.dtype}")
        if logits.dim() != 3 or logits.shape[1] != self.L or logits.shape[2] < self.V:
            raise ValueError(f"logits must be [B, {self.L}, >= {self.V}], got {tuple(logits.shape)}")
        B, L = int(logits.shape[0]), int(logits.shape[1])
        # row (b, i) must sit at (b * L + i) * row_stride; strides of size-1 dims are free
        if L > 1:
            rs = int(logits.stride(1))
            ok = B == 1 or int(logits.stride(0)) == rs * L
        else:
            rs = int(logits.stride(0)) if B > 1 else int(logits.shape[2])
            ok = True
        if logits.shape[2] > 1 and logits.stride(2) != 1:
            ok = False
        if not ok or rs < self.V:
            raise ValueError("logits rows must be evenly strided: [B, L, >=V] with a unit last stride")
        return B, rs

    def _ctx(self, ctx_len, B: int) -> Optional[int]:
        if ctx_len is None:
            return None
        torch = _torch()
        _check("ctx_len", ctx_len, torch.int64, (), B, self.device)
        if ctx_len.shape[0] != B:
            raise ValueError(f"ctx_len must have shape ({B},), got {tuple(ctx_len.shape)}")
        return _ptr(ctx_len)

    def _topk(self, B: int, ids, logit, lse, lq=None, required: bool = True) -> None:
        torch = _torch()
        _check("topk_ids", ids, torch.int32, (self.L, self.K), B, self.device, required)
        _check("topk_logit", logit, torch.float32, (self.L, self.K), B, self.device, required)
        _check("lse", lse, torch.float64, (self.L,), B, self.device, required)
        _check("topk_lq", lq, torch.float32, (self.L, self.K), B, self.device, required=False)

    def _tree(self, B: int, out: "TreeOutputs", emit: bool = False) -> None:
        torch = _torch()
        cap = max(self.cap, 1)
        _check("parent", out.parent, torch.int32, (cap,), B, self.device)
        _check("n_star", out.n_star, torch.int32, (), B, self.device)
        _check("depth", out.depth, torch.int32, (cap,), B, self.device, required=not emit or out.pos_ids is not None)
        if not emit:
            _check("token_ids", out.token_ids, torch.int32, (cap,), B, self.device)
            _check("path_prob", out.path_prob, torch.float32, (cap,), B, self.device, required=False)
            _check("phi", out.phi, torch.float32, (), B, self.device, required=False)
            _check("theta", out.theta, torch.float32, (), B, self.device, required=False)
        else:
            _check("pos_ids", out.pos_ids, torch.int32, (cap,), B, self.device, required=False)
            if self.mask == "u8":
                _check("mask", out.mask, torch.uint8, (cap, cap), B, self.device, required=False)
            elif self.mask == "bits" and out.mask is not None:
                if out.mask.dtype not in (torch.int32, getattr(torch, "uint32", torch.int32)):
                    raise TypeError(f"mask must be int32 or uint32 words, got {out.mask.dtype}")
                _check("mask", out.mask, out.mask.dtype, (cap, (cap + 31) // 32), B, self.device)

    def _workspace(self, B: int, workspace, out: "TreeOutputs"):
        torch = _torch()
        if workspace is None:
            return None, 0
        if not isinstance(workspace, torch.Tensor) or not _on_device(workspace, self.device) \
                or not workspace.is_contiguous():
            raise ValueError(f"workspace must be a contiguous tensor on cuda:{self.device}")
        return _ptr(workspace), workspace.numel() * workspace.element_size()

    def build(self, logits, out: TreeOutputs, pos_offset: int = 0, workspace=None, stream=None,
              ctx_len=None) -> None:
        B, stride = self._logits(logits)
        self._tree(B, out)
        self._tree(B, out, emit=True)
        self._topk(B, out.topk_ids, out.topk_logit, out.lse, out.topk_lq, required=False)
        ws_ptr, ws_bytes = self._workspace(B, workspace, out)
        ctx = self._ctx(ctx_len, B)
        st = out.as_struct()
        _lib.check(self._lib.caddtree_build(self._h, _ptr(logits), B, stride, int(pos_offset),
                                            ctx, ctypes.byref(st), ws_ptr, ws_bytes,
                                            _stream(stream, logits.device)))

    def build_noalloc(self, logits, out: TreeOutputs, pos_offset: int = 0, stream=None, ctx_len=None) -> None:
        """``build`` without a workspace (``caddtree_build_noalloc``): the top-K table not asked for in
        ``out`` lives in the library's own device array, shared by every such call on the GPU, so calls
        that overlap in time on one GPU race."""
        B, stride = self._logits(logits)
        self._tree(B, out)
        self._tree(B, out, emit=True)
        self._topk(B, out.topk_ids, out.topk_logit, out.lse, out.topk_lq, required=False)
        ctx = self._ctx(ctx_len, B)
        st = out.as_struct()
        _lib.check(self._lib.caddtree_build_noalloc(self._h, _ptr(logits), B, stride, int(pos_offset), ctx,
                                                    ctypes.byref(st), _stream(stream, logits.device)))

    def reduce_topk(self, logits, topk_ids, topk_logit, lse, topk_lq=None, stream=None) -> None:
        B, stride = self._logits(logits)
        self._topk(B, topk_ids, topk_logit, lse, topk_lq)
        _lib.check(self._lib.caddtree_reduce_topk(self._h, _ptr(logits), B, stride, _ptr(topk_ids),
                                                  _ptr(topk_logit), _ptr(topk_lq), _ptr(lse),
                                                  _stream(stream, logits.device)))

    def expand(self, topk_ids, topk_logit, lse, out: TreeOutputs, stream=None, ctx_len=None) -> None:
        self._topk(0, topk_ids, topk_logit, lse)
        B = int(topk_ids.shape[0])
        self._topk(B, topk_ids, topk_logit, lse)
        self._tree(B, out)
        ctx = self._ctx(ctx_len, B)
        _lib.check(self._lib.caddtree_expand(self._h, _ptr(topk_ids), _ptr(topk_logit), _ptr(lse), B,
                                             ctx, _ptr(out.token_ids), _ptr(out.parent), _ptr(out.depth),
                                             _ptr(out.path_prob), _ptr(out.n_star), _ptr(out.phi),
                                             _ptr(out.theta), _stream(stream, topk_ids.device)))

    def accept(self, topk: TreeOutputs, tree: TreeOutputs, u, accept_len, round_cost=None, ctx_len=None,
               stream=None) -> None:
        """Synthetic acceptance of ``tree`` (built from the top-K table in ``topk``) against target paths
        drawn from the uniforms ``u`` (float64 [B, L]); writes ``accept_len`` (int32 [B]) and optionally
        ``round_cost`` (float64 [B], this plan's C_d + C_v(n*))."""
        torch = _torch()
        if not isinstance(tree.token_ids, torch.Tensor) or tree.token_ids.dim() != 2:
            raise ValueError("tree.token_ids must be a [B, tree_stride] tensor")
        _check("token_ids", tree.token_ids, torch.int32, tree.token_ids.shape[1:], 0, self.device)
        B, stride = int(tree.token_ids.shape[0]), int(tree.token_ids.shape[1])
        _check("parent", tree.parent, torch.int32, (stride,), B, self.device)
        _check("n_star", tree.n_star, torch.int32, (), B, self.device)
        self._topk(B, topk.topk_ids, topk.topk_logit, topk.lse)
        _check("u", u, torch.float64, (self.L,), B, self.device)
        if u.shape[0] != B:
            raise ValueError(f"u must be a contiguous float64 tensor of shape ({B}, {self.L})")
        _check("accept_len", accept_len, torch.int32, (), B, self.device)
        _check("round_cost", round_cost, torch.float64, (), B, self.device, required=False)
        ctx = self._ctx(ctx_len, B) if round_cost is not None else None
        _lib.check(self._lib.caddtree_accept(self._h, _ptr(topk.topk_ids), _ptr(topk.topk_logit), _ptr(topk.lse),
                                             B, _ptr(tree.token_ids), _ptr(tree.parent),
                                             stride, _ptr(tree.n_star), _ptr(u),
                                             ctx, _ptr(accept_len), _ptr(round_cost),
                                             _stream(stream, u.device)))

    def emit(self, out: TreeOutputs, pos_offset: int = 0, stream=None) -> None:
        _check("parent", out.parent, _torch().int32, (max(self.cap, 1),), 0, self.device)
        B = int(out.parent.shape[0])
        self._tree(B, out, emit=True)
        _lib.check(self._lib.caddtree_emit(self._h, _ptr(out.parent), _ptr(out.depth), _ptr(out.n_star), B,
                                           int(pos_offset), _ptr(out.mask), _ptr(out.pos_ids),
                                           _stream(stream, out.parent.device)))
