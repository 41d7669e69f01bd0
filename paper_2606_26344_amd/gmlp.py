"""Python binding of libgmlp.so (the C ABI declared in include/gmlp.h; the
Softmax+MatMul entry points of include/softmax_matmul.h are bound in
``softmax_matmul.py`` on the same library).

Argument marshalling only: every step of the Gated MLP runs in the library's
HIP kernels.  PyTorch supplies device memory and the current HIP stream.  The
names mirror the C entry points:

    forward(x, wg, wu, wd)   -> gmlp_forward / gmlp_forward_ex / gmlp_forward_variant
    gate_up(x, wg, wu)       -> gmlp_gate_up / gmlp_gate_up_ws / gmlp_gate_up_variant
    down(h, wd)              -> gmlp_down / gmlp_down_ws

forward() and gate_up() also take the members of the Gated MLP family:
activation "silu" (default), "swish" (g * sigmoid(beta g)) or "sigmoid"
(GLU), and rmsnorm=True (RMSNorm of X in front, epsilon eps).

Tensors are ``torch.bfloat16``, contiguous, on one HIP device, with shapes
x [T, D], wg [D, F], wu [D, F], wd [F, D].  Loading fails loudly if the
library has not been built (``python -m paper_2606_26344_amd.build``).
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIBRARY = os.path.join(HERE, "libgmlp.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "gmlp.h")
HEADERS = [HEADER, os.path.join(os.path.dirname(HERE), "include", "softmax_matmul.h")]

PATH_AUTO, PATH_GEMV, PATH_MFMA, PATH_FUSED, PATH_FUSED_MFMA = 0, 1, 2, 3, 4
_PATHS = {"auto": PATH_AUTO, "gemv": PATH_GEMV, "mfma": PATH_MFMA, "fused": PATH_FUSED,
          "fused_mfma": PATH_FUSED_MFMA}
ACT_SILU, ACT_SWISH, ACT_SIGMOID = 0, 1, 2
ACTIVATIONS = {"silu": ACT_SILU, "swish": ACT_SWISH, "sigmoid": ACT_SIGMOID}

_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_SZ = ctypes.c_size_t
_F = ctypes.c_float
_INT = ctypes.c_int

_SIGNATURES = {
    "gmlp_version": ([], ctypes.c_int),
    "gmlp_status_string": ([ctypes.c_int], ctypes.c_char_p),
    "gmlp_last_error": ([], ctypes.c_char_p),
    "gmlp_validate": ([_I64, _I64, _I64, _P, _P, _P, _P, _P], ctypes.c_int),
    "gmlp_describe": ([_I64, _I64, _I64, ctypes.c_int, ctypes.c_char_p, _SZ], ctypes.c_int),
    "gmlp_workspace_size": ([_I64, _I64, _I64], _SZ),
    "gmlp_workspace_init": ([_P, _SZ, _P], ctypes.c_int),
    "gmlp_workspace_status": ([_P, _SZ, _P, ctypes.POINTER(ctypes.c_uint32)], ctypes.c_int),
    "gmlp_test_fused_spin_limit": ([ctypes.c_uint32], ctypes.c_uint32),
    "gmlp_forward": ([_P, _P, _P, _P, _P, _I64, _I64, _I64, _P], ctypes.c_int),
    "gmlp_forward_ws": ([_P, _P, _P, _P, _P, _I64, _I64, _I64, _P, _SZ, _P], ctypes.c_int),
    "gmlp_forward_noalloc": ([_P, _P, _P, _P, _P, _I64, _I64, _I64, _P], ctypes.c_int),
    "gmlp_forward_ex": ([_P, _P, _P, _P, _P, _I64, _I64, _I64, ctypes.c_int, _P, _SZ, _P],
                        ctypes.c_int),
    "gmlp_forward_variant": ([_P, _P, _P, _P, _P, _I64, _I64, _I64, _INT, _F, _INT, _F, _INT, _P,
                              _SZ, _P], _INT),
    "gmlp_gate_up_variant": ([_P, _P, _P, _P, _I64, _I64, _I64, _INT, _F, _INT, _F, _INT, _P, _SZ,
                              _P], _INT),
    "gmlp_gate_up": ([_P, _P, _P, _P, _I64, _I64, _I64, _P], ctypes.c_int),
    "gmlp_down": ([_P, _P, _P, _I64, _I64, _I64, _P], ctypes.c_int),
    "gmlp_gate_up_ws": ([_P, _P, _P, _P, _I64, _I64, _I64, ctypes.c_int, _P, _SZ, _P],
                        ctypes.c_int),
    "gmlp_down_ws": ([_P, _P, _P, _I64, _I64, _I64, ctypes.c_int, _P, _SZ, _P], ctypes.c_int),
    "softmax_matmul_workspace_size": ([_I64, _I64, _I64], _SZ),
    "softmax_matmul_describe": ([_I64, _I64, _I64, _INT, ctypes.c_char_p, _SZ], _INT),
    "softmax_matmul_ws": ([_P, _P, _P, _I64, _I64, _I64, _INT, _P, _SZ, _P], _INT),
    "softmax_matmul": ([_P, _P, _P, _I64, _I64, _I64, _P], _INT),
    "softmax_matmul_exp_rows": ([_P, _P, _P, _I64, _I64, _P], _INT),
    "softmax_matmul_divide_ws": ([_P, _P, _P, _P, _I64, _I64, _I64, _INT, _P, _SZ, _P], _INT),
}

_lib = None


class GmlpError(RuntimeError):
    def __init__(self, code: int, detail: str):
        self.code = code
        super().__init__("%s: %s" % (status_string(code), detail))


def library() -> ctypes.CDLL:
    """The loaded libgmlp.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIBRARY):
            raise RuntimeError("libgmlp.so is not built: run `python -m paper_2606_26344_amd.build`")
        lib = ctypes.CDLL(LIBRARY)
        for name, (args, res) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.argtypes = args
            fn.restype = res
        _lib = lib
    return _lib


def header_functions() -> list:
    """Names of the functions include/gmlp.h and include/softmax_matmul.h
    declare."""
    names = set()
    for path in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(path).read(), flags=re.S)
        names.update(re.findall(r"\b((?:gmlp|softmax_matmul)(?:_[a-z_0-9]+)?)\s*\(", text))
    return sorted(names)


def version() -> int:
    return library().gmlp_version()


def status_string(code: int) -> str:
    return library().gmlp_status_string(code).decode()


def last_error() -> str:
    return library().gmlp_last_error().decode()


def _check(rc: int) -> None:
    if rc != 0:
        raise GmlpError(rc, last_error())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _empty(shape, dtype, device, stream=None) -> torch.Tensor:
    """torch.empty on the stream the library will use the memory on.  The
    caching allocator hands a freed block to the next allocation on the
    stream it was allocated on without waiting for other streams, so memory
    that a call's kernels use on `stream` must be allocated on `stream`:
    allocated on the current stream instead, it could be given out again
    there while the kernels still write to it."""
    if stream is None:
        return torch.empty(shape, dtype=dtype, device=device)
    with torch.cuda.stream(stream):
        return torch.empty(shape, dtype=dtype, device=device)


def _expect(t: torch.Tensor, name: str, shape, device) -> None:
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.dtype != torch.bfloat16:
        raise TypeError("%s must be torch.bfloat16, got %s" % (name, t.dtype))
    if t.device.type != "cuda" or (device is not None and t.device != device):
        raise ValueError("%s must be on the HIP device %s, got %s" % (name, device, t.device))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if tuple(t.shape) != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))


def describe(T: int, D: int, F: int, path: str = "auto") -> list:
    """The kernels forward() enqueues for this shape: a list of
    (name, grid, block, k_splits), in launch order."""
    buf = ctypes.create_string_buffer(1024)
    _check(library().gmlp_describe(T, D, F, _PATHS[path], buf, len(buf)))
    return _parse_plan(buf)


def _parse_plan(buf) -> list:
    out = []
    for line in buf.value.decode().splitlines():
        name, rest = line.rsplit(" grid=", 1)
        grid, block, splits = (int(f.split("=")[1]) for f in ("grid=" + rest).split())
        out.append((name, grid, block, splits))
    return out


def workspace_size(T: int, D: int, F: int) -> int:
    return int(library().gmlp_workspace_size(T, D, F))


class Workspace:
    """A caller-owned workspace for forward(), zeroed once at creation
    (``nbytes`` overrides the size gmlp_workspace_size gives)."""

    def __init__(self, T: int, D: int, F: int, device=None, stream=None, nbytes: int = 0):
        n = nbytes or workspace_size(T, D, F)
        if n == 0:
            raise ValueError("invalid shape T=%d D=%d F=%d" % (T, D, F))
        # 256 bytes of slack so the buffer can be 256-byte aligned.  Allocated
        # on the stream the calls will run on (see _empty).
        self.storage = _empty(n + 256, torch.uint8, device or "cuda", stream)
        off = (-self.storage.data_ptr()) % 256
        self.buffer = self.storage[off:off + n]
        self.nbytes = n
        _check(library().gmlp_workspace_init(_ptr(self.buffer), n, _stream(stream)))

    def fits(self, T: int, D: int, F: int) -> bool:
        return workspace_size(T, D, F) <= self.nbytes

    def fused_giveups(self, stream=None) -> int:
        """gmlp_workspace_status: read and clear the count of fused-kernel
        down blocks whose bounded wait gave up (their strips of Y are NaN)."""
        n = ctypes.c_uint32(0)
        _check(library().gmlp_workspace_status(_ptr(self.buffer), self.nbytes, _stream(stream),
                                               ctypes.byref(n)))
        return int(n.value)


def fused_spin_limit(limit: int) -> int:
    """gmlp_test_fused_spin_limit (test hook): polls before a fused-kernel
    down block gives up, for the calls that follow; returns the previous."""
    return int(library().gmlp_test_fused_spin_limit(limit))


def _variant(activation: str, beta: float, rmsnorm: bool, eps: float):
    if activation not in ACTIVATIONS:
        raise ValueError("activation must be one of %s" % sorted(ACTIVATIONS))
    return ACTIVATIONS[activation], float(beta), int(bool(rmsnorm)), float(eps)


def forward(x: torch.Tensor, wg: torch.Tensor, wu: torch.Tensor, wd: torch.Tensor,
            out: Optional[torch.Tensor] = None, path: str = "auto",
            workspace: Optional[Workspace] = None, stream=None, activation: str = "silu",
            beta: float = 1.0, rmsnorm: bool = False, eps: float = 1e-6) -> torch.Tensor:
    """Y = (act(xn wg) * (xn wu)) wd on the current HIP stream, act = silu by
    default, xn = x or, with ``rmsnorm``, x / sqrt(mean(x^2) + eps) per row."""
    if x.dim() != 2 or wg.dim() != 2:
        raise ValueError("x and wg must be 2-D")
    T, D = x.shape
    F = wg.shape[1]
    dev = x.device
    _expect(x, "x", (T, D), dev)
    _expect(wg, "wg", (D, F), dev)
    _expect(wu, "wu", (D, F), dev)
    _expect(wd, "wd", (F, D), dev)
    if out is None:
        out = _empty((T, D), torch.bfloat16, dev, stream)
    _expect(out, "out", (T, D), dev)
    lib = library()
    st = _stream(stream)
    plain = activation == "silu" and not rmsnorm
    if workspace is None and path == "auto" and plain:
        _check(lib.gmlp_forward(_ptr(x), _ptr(wg), _ptr(wu), _ptr(wd), _ptr(out), T, D, F, st))
        return out
    if workspace is None:
        workspace = Workspace(T, D, F, device=dev, stream=stream)
    if plain:
        _check(lib.gmlp_forward_ex(_ptr(x), _ptr(wg), _ptr(wu), _ptr(wd), _ptr(out), T, D, F,
                                   _PATHS[path], _ptr(workspace.buffer), workspace.nbytes, st))
    else:
        _check(lib.gmlp_forward_variant(_ptr(x), _ptr(wg), _ptr(wu), _ptr(wd), _ptr(out), T, D, F,
                                        *_variant(activation, beta, rmsnorm, eps), _PATHS[path],
                                        _ptr(workspace.buffer), workspace.nbytes, st))
    return out


def forward_noalloc(x: torch.Tensor, wg: torch.Tensor, wu: torch.Tensor, wd: torch.Tensor,
                    out: torch.Tensor, stream=None) -> torch.Tensor:
    """gmlp_forward_noalloc: Y = (silu(x wg) * (x wu)) wd into the caller's
    ``out``, with the library's static per-device scratch array as workspace
    (no allocation; calls that overlap on one device race on that array)."""
    T, D = x.shape
    F = wg.shape[1]
    dev = x.device
    for t, name, shape in ((x, "x", (T, D)), (wg, "wg", (D, F)), (wu, "wu", (D, F)),
                           (wd, "wd", (F, D)), (out, "out", (T, D))):
        _expect(t, name, shape, dev)
    _check(library().gmlp_forward_noalloc(_ptr(x), _ptr(wg), _ptr(wu), _ptr(wd), _ptr(out), T, D, F,
                                          _stream(stream)))
    return out


def gate_up(x: torch.Tensor, wg: torch.Tensor, wu: torch.Tensor,
            out: Optional[torch.Tensor] = None, path: str = "auto",
            workspace: Optional[Workspace] = None, stream=None, activation: str = "silu",
            beta: float = 1.0, rmsnorm: bool = False, eps: float = 1e-6) -> torch.Tensor:
    """H = bf16(act(xn wg) * (xn wu)), H [T, F] (see forward for the options)."""
    T, D = x.shape
    F = wg.shape[1]
    dev = x.device
    _expect(x, "x", (T, D), dev)
    _expect(wg, "wg", (D, F), dev)
    _expect(wu, "wu", (D, F), dev)
    if out is None:
        out = _empty((T, F), torch.bfloat16, dev, stream)
    _expect(out, "out", (T, F), dev)
    plain = activation == "silu" and not rmsnorm
    if workspace is None and path == "auto" and plain:
        _check(library().gmlp_gate_up(_ptr(x), _ptr(wg), _ptr(wu), _ptr(out), T, D, F,
                                      _stream(stream)))
        return out
    if workspace is None:
        workspace = Workspace(T, D, F, device=dev, stream=stream)
    if plain:
        _check(library().gmlp_gate_up_ws(_ptr(x), _ptr(wg), _ptr(wu), _ptr(out), T, D, F,
                                         _PATHS[path], _ptr(workspace.buffer), workspace.nbytes,
                                         _stream(stream)))
    else:
        _check(library().gmlp_gate_up_variant(_ptr(x), _ptr(wg), _ptr(wu), _ptr(out), T, D, F,
                                              *_variant(activation, beta, rmsnorm, eps),
                                              _PATHS[path], _ptr(workspace.buffer),
                                              workspace.nbytes, _stream(stream)))
    return out


def down(h: torch.Tensor, wd: torch.Tensor, out: Optional[torch.Tensor] = None,
         path: str = "auto", workspace: Optional[Workspace] = None, stream=None) -> torch.Tensor:
    """Y = bf16(h wd), h [T, F], wd [F, D]."""
    T, F = h.shape
    D = wd.shape[1]
    dev = h.device
    _expect(h, "h", (T, F), dev)
    _expect(wd, "wd", (F, D), dev)
    if out is None:
        out = _empty((T, D), torch.bfloat16, dev, stream)
    _expect(out, "out", (T, D), dev)
    if workspace is None and path == "auto":
        _check(library().gmlp_down(_ptr(h), _ptr(wd), _ptr(out), T, F, D, _stream(stream)))
        return out
    if workspace is None:
        workspace = Workspace(T, D, F, device=dev, stream=stream)
    _check(library().gmlp_down_ws(_ptr(h), _ptr(wd), _ptr(out), T, F, D, _PATHS[path],
                                  _ptr(workspace.buffer), workspace.nbytes, _stream(stream)))
    return out


def from_bf16_bits(bits, device="cuda") -> torch.Tensor:
    """A bfloat16 device tensor holding the given uint16 bit patterns (numpy)."""
    import numpy as np

    arr = np.ascontiguousarray(bits, dtype=np.uint16)
    return torch.from_numpy(arr.view(np.int16)).view(torch.bfloat16).to(device)


def to_bf16_bits(t: torch.Tensor):
    """uint16 numpy array of a bfloat16 tensor's bit patterns."""
    import numpy as np

    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
