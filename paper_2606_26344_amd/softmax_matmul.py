"""Python binding of the Softmax+MatMul entry points of libgmlp.so
(include/softmax_matmul.h).

Argument marshalling only: the exponentials, row sums, matmul and divide run
in the library's HIP kernels.  Names mirror the C entry points:

    softmax_matmul(x, y)    -> softmax_matmul / softmax_matmul_ws
    exp_rows(x)             -> softmax_matmul_exp_rows   (P = exp(x - rowmax), s)
    divide(p, s, y)         -> softmax_matmul_divide_ws  ((p y) / s, row by row)
    describe(M, K, N)       -> softmax_matmul_describe
    workspace_size(M, K, N) -> softmax_matmul_workspace_size

Tensors are ``torch.bfloat16``, contiguous, on one HIP device: x [M, K],
y [K, N]; the result is z = softmax(x) y [M, N], softmax along each row.
"""
from __future__ import annotations

import ctypes
from typing import Optional

import torch

from .gmlp import _PATHS, Workspace, _check, _empty, _expect, _parse_plan, _ptr, _stream, library


def workspace_size(M: int, K: int, N: int) -> int:
    return int(library().softmax_matmul_workspace_size(M, K, N))


def make_workspace(M: int, K: int, N: int, device=None, stream=None) -> Workspace:
    """A zeroed workspace that fits softmax_matmul(x [M, K], y [K, N])."""
    n = workspace_size(M, K, N)
    if n == 0:
        raise ValueError("invalid shape M=%d K=%d N=%d" % (M, K, N))
    return Workspace(M, N, K, device=device, stream=stream, nbytes=n)


def describe(M: int, K: int, N: int, path: str = "auto") -> list:
    """The kernels softmax_matmul() enqueues: (name, grid, block, k_splits)."""
    buf = ctypes.create_string_buffer(1024)
    _check(library().softmax_matmul_describe(M, K, N, _PATHS[path], buf, len(buf)))
    return _parse_plan(buf)


def softmax_matmul(x: torch.Tensor, y: torch.Tensor, out: Optional[torch.Tensor] = None,
                   path: str = "auto", workspace: Optional[Workspace] = None,
                   stream=None) -> torch.Tensor:
    """z = softmax(x) y on the current HIP stream (softmax along rows of x)."""
    if x.dim() != 2 or y.dim() != 2:
        raise ValueError("x and y must be 2-D")
    M, K = x.shape
    N = y.shape[1]
    dev = x.device
    _expect(x, "x", (M, K), dev)
    _expect(y, "y", (K, N), dev)
    if out is None:
        out = _empty((M, N), torch.bfloat16, dev, stream)
    _expect(out, "out", (M, N), dev)
    st = _stream(stream)
    if workspace is None and path == "auto":
        _check(library().softmax_matmul(_ptr(x), _ptr(y), _ptr(out), M, K, N, st))
        return out
    if workspace is None:
        workspace = make_workspace(M, K, N, device=dev, stream=stream)
    _check(library().softmax_matmul_ws(_ptr(x), _ptr(y), _ptr(out), M, K, N, _PATHS[path],
                                       _ptr(workspace.buffer), workspace.nbytes, st))
    return out


def exp_rows(x: torch.Tensor, p: Optional[torch.Tensor] = None, s: Optional[torch.Tensor] = None,
             stream=None):
    """The exp/row-sum half: p = bf16(exp(x - rowmax)) [M, K], s = row sums
    of the unrounded exponentials [M] (float32).  Returns (p, s)."""
    M, K = x.shape
    dev = x.device
    _expect(x, "x", (M, K), dev)
    if p is None:
        p = _empty((M, K), torch.bfloat16, dev, stream)
    _expect(p, "p", (M, K), dev)
    if s is None:
        s = _empty((M,), torch.float32, dev, stream)
    if s.dtype != torch.float32 or s.shape != (M,) or not s.is_contiguous() or s.device != dev:
        raise ValueError("s must be a contiguous float32 tensor of shape (%d,) on %s" % (M, dev))
    _check(library().softmax_matmul_exp_rows(_ptr(x), _ptr(p), _ptr(s), M, K, _stream(stream)))
    return p, s


def divide(p: torch.Tensor, s: torch.Tensor, y: torch.Tensor, out: Optional[torch.Tensor] = None,
           path: str = "auto", workspace: Optional[Workspace] = None, stream=None) -> torch.Tensor:
    """The matmul-then-divide half: z = bf16((p y) / s) row by row."""
    M, K = p.shape
    N = y.shape[1]
    dev = p.device
    _expect(p, "p", (M, K), dev)
    _expect(y, "y", (K, N), dev)
    if s.dtype != torch.float32 or s.shape != (M,) or not s.is_contiguous() or s.device != dev:
        raise ValueError("s must be a contiguous float32 tensor of shape (%d,) on %s" % (M, dev))
    if out is None:
        out = _empty((M, N), torch.bfloat16, dev, stream)
    _expect(out, "out", (M, N), dev)
    if workspace is None:
        workspace = make_workspace(M, K, N, device=dev, stream=stream)
    _check(library().softmax_matmul_divide_ws(_ptr(p), _ptr(s), _ptr(y), _ptr(out), M, K, N,
                                              _PATHS[path], _ptr(workspace.buffer),
                                              workspace.nbytes, _stream(stream)))
    return out
