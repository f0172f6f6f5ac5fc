"""Training-side gather-scatter (Section 3.2, Eq. 6-7) and the router's
straight-through estimator (Appendix B) as autograd functions over libtlf.

Argument marshalling only: the active set, the gather, the scatter, their
gradients and the estimator all run in libtlf's HIP kernels, on the current
torch stream.  The shared block between gather and scatter is the caller's.

    p = plan(depth, batch, seq_len, loop)     # loop i's active rows
    x = gather(h, p)                          # [p.count, d], Eq. 6
    h = scatter(h, block(x), p)               # Eq. 7 (scatter_ writes into h)
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass

import torch

from . import tlf


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _check(status: int, where: str):
    if status != tlf.OK:
        raise tlf.TlfError(status, where)


def _rows_tensor(h: torch.Tensor, name: str):
    if h.dtype != torch.float32 or h.dim() != 2 or not h.is_cuda or not h.is_contiguous():
        raise ValueError(f"{name}: expected a contiguous float32 [rows, d] CUDA tensor")


@dataclass
class LoopPlan:
    """Active set of one loop: compact index -> row (`index`), row -> compact
    index or -1 (`slot`), each sequence's start in the compact tensor plus the
    total (`offsets`), the count on the device (`count_dev`) and on the host."""
    loop: int
    rows: int
    index: torch.Tensor
    slot: torch.Tensor
    offsets: torch.Tensor
    count_dev: torch.Tensor
    count: int


def plan_workspace(batch: int, seq_len: int, device="cuda") -> torch.Tensor:
    """Scratch for the multi-workgroup planner (one int32 count per chunk of rows)."""
    return torch.empty(max(tlf.gs_plan_ws_bytes(batch * seq_len), 4), dtype=torch.uint8, device=device)


def plan(depth: torch.Tensor, batch: int, seq_len: int, loop: int, workspace: torch.Tensor = None) -> LoopPlan:
    """Active rows of loop `loop`; reads the count back to the host (one
    synchronisation), since the compact tensor's size must be known there.
    With a `workspace` (plan_workspace) the multi-workgroup planner runs,
    otherwise the single-workgroup one; both give the same plan."""
    if depth.dtype != torch.int32 or not depth.is_cuda or not depth.is_contiguous():
        raise ValueError("depth: expected a contiguous int32 CUDA tensor")
    rows = batch * seq_len
    if depth.numel() != rows:
        raise ValueError(f"depth holds {depth.numel()} entries, batch * seq_len = {rows}")
    dev = depth.device
    index = torch.empty(max(rows, 1), dtype=torch.int32, device=dev)
    slot = torch.empty(max(rows, 1), dtype=torch.int32, device=dev)
    offsets = torch.empty(batch + 1, dtype=torch.int32, device=dev)
    count = torch.empty(1, dtype=torch.int32, device=dev)
    if workspace is None:
        _check(tlf.load().tlf_gs_plan(_ptr(depth), batch, seq_len, loop, _ptr(index), _ptr(slot), _ptr(offsets),
                                      _ptr(count), _stream()), "tlf_gs_plan")
    else:
        if workspace.dtype != torch.uint8 or not workspace.is_cuda or not workspace.is_contiguous():
            raise ValueError("workspace: expected a contiguous uint8 CUDA tensor (plan_workspace)")
        _check(tlf.load().tlf_gs_plan_ws(_ptr(depth), batch, seq_len, loop, _ptr(index), _ptr(slot),
                                         _ptr(offsets), _ptr(count), _ptr(workspace), workspace.numel(),
                                         _stream()), "tlf_gs_plan_ws")
    n = int(count.item())
    return LoopPlan(loop, rows, index[:n], slot[:rows], offsets, count, n)


def gather_raw(h: torch.Tensor, p: LoopPlan, out: torch.Tensor = None) -> torch.Tensor:
    _rows_tensor(h, "h")
    d = h.shape[1]
    if out is None:
        out = torch.empty((p.count, d), dtype=h.dtype, device=h.device)
    _check(tlf.load().tlf_gs_gather(_ptr(h), _ptr(p.index), _ptr(p.count_dev), p.count, d, _ptr(out), _stream()),
           "tlf_gs_gather")
    return out


def scatter_raw(h_prev: torch.Tensor, y: torch.Tensor, p: LoopPlan, out: torch.Tensor = None) -> torch.Tensor:
    """Eq. 7 into `out` (a new tensor by default; `out is h_prev` updates in place)."""
    _rows_tensor(h_prev, "h_prev")
    _rows_tensor(y, "y")
    if h_prev.shape[0] != p.rows or y.shape != (p.count, h_prev.shape[1]):
        raise ValueError(f"scatter: h_prev {tuple(h_prev.shape)}, y {tuple(y.shape)}, plan rows {p.rows} "
                         f"count {p.count}")
    if out is None:
        out = torch.empty_like(h_prev)
    # with no active row y is empty (no address) and never read: pass h_prev's
    yp = _ptr(y) if y.numel() else _ptr(h_prev)
    _check(tlf.load().tlf_gs_scatter(_ptr(h_prev), yp, _ptr(p.slot), p.rows, h_prev.shape[1], _ptr(out),
                                     _stream()), "tlf_gs_scatter")
    return out


class _Gather(torch.autograd.Function):
    @staticmethod
    def forward(ctx, h, p):
        ctx.p = p
        ctx.shape = h.shape
        return gather_raw(h.contiguous(), p)

    @staticmethod
    def backward(ctx, g):
        dh = torch.zeros(ctx.shape, dtype=g.dtype, device=g.device)
        scatter_raw(dh, g.contiguous(), ctx.p, out=dh)
        return dh, None


class _Scatter(torch.autograd.Function):
    @staticmethod
    def forward(ctx, h_prev, y, p):
        ctx.p = p
        return scatter_raw(h_prev.contiguous(), y.contiguous(), p)

    @staticmethod
    def backward(ctx, g):
        g = g.contiguous()
        return g, gather_raw(g, ctx.p), None


class _ScatterInPlace(torch.autograd.Function):
    """Eq. 7 written into h_prev: neither gradient needs the previous state
    (the block's backward uses its own compact input), so the rows that no
    loop touches need not be copied."""
    @staticmethod
    def forward(ctx, h_prev, y, p):
        ctx.p = p
        scatter_raw(h_prev, y.contiguous(), p, out=h_prev)
        ctx.mark_dirty(h_prev)
        return h_prev

    @staticmethod
    def backward(ctx, g):
        g = g.contiguous()
        return g, gather_raw(g, ctx.p), None


class _Ste(torch.autograd.Function):
    @staticmethod
    def forward(ctx, score, depth):
        ctx.save_for_backward(score, depth)
        value = torch.empty(depth.shape, dtype=torch.float32, device=depth.device)
        _check(tlf.load().tlf_ste(_ptr(depth), None, None, depth.numel(), _ptr(value), None, _stream()), "tlf_ste")
        return value

    @staticmethod
    def backward(ctx, g):
        score, depth = ctx.saved_tensors
        g = g.contiguous().float()
        ds = torch.empty_like(score)
        _check(tlf.load().tlf_ste(None, _ptr(score), _ptr(g), score.numel(), None, _ptr(ds), _stream()), "tlf_ste")
        return ds, None


def gather(h: torch.Tensor, p: LoopPlan) -> torch.Tensor:
    """Eq. 6 with its gradient (the compact gradient added into the rows)."""
    return _Gather.apply(h, p)


def scatter(h_prev: torch.Tensor, y: torch.Tensor, p: LoopPlan) -> torch.Tensor:
    """Eq. 7 with its gradient (identity to h_prev, gathered rows to y)."""
    return _Scatter.apply(h_prev, y, p)


def scatter_(h_prev: torch.Tensor, y: torch.Tensor, p: LoopPlan) -> torch.Tensor:
    """Eq. 7 in place on h_prev (which must be contiguous and not a leaf that
    requires grad); same gradients as `scatter`, traffic only on active rows."""
    return _ScatterInPlace.apply(h_prev, y, p)


def ste(score: torch.Tensor, depth: torch.Tensor) -> torch.Tensor:
    """Appendix B: value `depth`, gradient sigma'(score) to `score`."""
    if score.dtype != torch.float32 or depth.dtype != torch.int32 or score.shape != depth.shape:
        raise ValueError("ste: float32 score and int32 depth of one shape expected")
    return _Ste.apply(score.contiguous(), depth.contiguous())
