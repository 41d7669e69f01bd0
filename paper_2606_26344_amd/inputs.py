"""Seeded synthetic inputs for the SiLU Gated MLP and Softmax+MatMul workloads.

This module only draws and encodes inputs; it holds none of the Gated MLP's
arithmetic, so that the HIP path and the CPU oracle can both be fed the same
bytes from it without sharing any of the method's code.  It needs numpy only.

Recipe (the paper times kernels on random inputs because their run time
depends only on tensor shapes, Section 6.1):
  * ``numpy.random.default_rng(seed)``, ``standard_normal(dtype=float32)``,
    drawn in row blocks in the fixed order X, Wg, Wu, Wd;
  * X ~ N(0, 1); Wg, Wu ~ N(0, 1/D) and Wd ~ N(0, 1/F) (variance 1/fan_in,
    i.e. the float32 draws scaled by 1/sqrt(fan_in));
  * optionally every row of X rescaled to unit RMS in float32 (no epsilon),
    the shape of activations that leave an RMSNorm;
  * every value rounded once to bf16, round-to-nearest-even.
Arrays are returned as ``uint16`` bf16 bit patterns, row-major:
X [T, D], Wg [D, F], Wu [D, F], Wd [F, D].

Softmax+MatMul (Z = softmax(X) Y): the same generator, drawn in the order
X, Y; logits X ~ N(0, s^2) with s = ``logit_scale`` (1 by default), Y ~ N(0, 1);
X [M, K], Y [K, N].
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Dict

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    T: int
    D: int
    F: int
    unit_rms_rows: bool = False
    seed: int = 0
    description: str = ""


# The five shapes this library is measured and checked on.
WORKLOADS: Dict[str, Workload] = {
    w.name: w
    for w in (
        Workload("tiny", 16, 256, 512, description="T=16, D=256, F=512"),
        Workload("decode", 1, 4096, 14336,
                 description="decode, memory-bound: T=1, D=4096, F=14336"),
        Workload("small_batch", 128, 4096, 14336,
                 description="small-batch decode: T=128, D=4096, F=14336"),
        Workload("prefill", 4096, 4096, 14336, unit_rms_rows=True,
                 description="prefill, compute-bound: T=4096, D=4096, F=14336, "
                             "X rows at unit RMS"),
        Workload("large_prefill", 2048, 8192, 28672,
                 description="large-model prefill: T=2048, D=8192, F=28672"),
    )
}


@dataclass(frozen=True)
class SoftmaxMatmulWorkload:
    name: str
    M: int
    K: int
    N: int
    logit_scale: float = 1.0
    seed: int = 0
    description: str = ""


# The paper sweeps every dimension of Softmax+MatMul over 2K, 4K and 8K
# (table tab:multi-op-eval, Section 6.3); the largest point is the benchmark
# shape, the tiny one is for full checks against the oracle.
SOFTMAX_MATMUL_WORKLOADS: Dict[str, SoftmaxMatmulWorkload] = {
    w.name: w
    for w in (
        SoftmaxMatmulWorkload("softmax_matmul_tiny", 16, 256, 512,
                              description="Softmax+MatMul: M=16, K=256, N=512"),
        SoftmaxMatmulWorkload("softmax_matmul", 8192, 8192, 8192,
                              description="Softmax+MatMul: M=8192, K=8192, N=8192"),
    )
}


def f32_to_bf16_bits(a, out=None, scratch=None) -> np.ndarray:
    """Round float32 values to bf16 (round-to-nearest-even); return bit patterns.

    NaN stays NaN (quiet, sign kept); values past the bf16 range round to
    +-inf; subnormals round like any other value (no flush to zero).
    ``out`` (uint16) and ``scratch`` (uint32), of a's size, may be given to
    avoid allocations.
    """
    a = np.ascontiguousarray(np.asarray(a, dtype=np.float32))
    u = a.view(np.uint32)
    r = scratch.reshape(a.shape) if scratch is not None else np.empty(a.shape, np.uint32)
    # u + 0x7FFF + lsb(u >> 16), then keep the high half.  In uint32 this can
    # only wrap for NaN bit patterns, which are replaced below.
    np.right_shift(u, np.uint32(16), out=r)
    r &= np.uint32(1)
    r += u
    r += np.uint32(0x7FFF)
    r >>= np.uint32(16)
    if out is None:
        out = np.empty(a.shape, np.uint16)
    np.copyto(out, r, casting="unsafe")
    nan = np.isnan(a)
    if nan.any():
        out[nan] = (u[nan] >> np.uint32(16)).astype(np.uint16) | np.uint16(0x0040)
    return out


def bf16_bits_to_f32(bits) -> np.ndarray:
    """Exact decode of bf16 bit patterns to float32."""
    b = np.ascontiguousarray(np.asarray(bits, dtype=np.uint16))
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


_BLOCK_ELEMS = 1 << 22  # draw at most this many values at a time


class _Scratch:
    def __init__(self):
        self.f = np.empty(_BLOCK_ELEMS, np.float32)
        self.u = np.empty(_BLOCK_ELEMS, np.uint32)


def _draw_bf16(rng: np.random.Generator, rows: int, cols: int, scale: float,
               unit_rms_rows: bool = False, scratch: _Scratch = None) -> np.ndarray:
    out = np.empty((rows, cols), dtype=np.uint16)
    scratch = scratch or _Scratch()
    step = max(1, _BLOCK_ELEMS // max(cols, 1))
    s = np.float32(scale)
    for r0 in range(0, rows, step):
        r1 = min(rows, r0 + step)
        n = (r1 - r0) * cols
        if n <= _BLOCK_ELEMS:
            blk = scratch.f[:n].reshape(r1 - r0, cols)
            rng.standard_normal(dtype=np.float32, out=blk)
            tmp = scratch.u[:n]
        else:  # a single row longer than a block
            blk = rng.standard_normal(size=(r1 - r0, cols), dtype=np.float32)
            tmp = None
        if unit_rms_rows:
            rms = np.sqrt(np.mean(blk * blk, axis=1, dtype=np.float32), dtype=np.float32)
            blk /= rms[:, None]
        elif scale != 1.0:
            blk *= s
        f32_to_bf16_bits(blk, out=out[r0:r1], scratch=tmp)
    return out


def generate(T: int, D: int, F: int, seed: int = 0, unit_rms_rows: bool = False):
    """Draw X, Wg, Wu, Wd (bf16 bit patterns) for one Gated MLP problem."""
    rng = np.random.default_rng(seed)
    scratch = _Scratch()
    X = _draw_bf16(rng, T, D, 1.0, unit_rms_rows, scratch)
    Wg = _draw_bf16(rng, D, F, 1.0 / math.sqrt(D), scratch=scratch)
    Wu = _draw_bf16(rng, D, F, 1.0 / math.sqrt(D), scratch=scratch)
    Wd = _draw_bf16(rng, F, D, 1.0 / math.sqrt(F), scratch=scratch)
    return X, Wg, Wu, Wd


def generate_softmax_matmul(M: int, K: int, N: int, seed: int = 0, logit_scale: float = 1.0):
    """Draw X [M, K] (logits, N(0, logit_scale^2)) and Y [K, N] (N(0, 1)) as
    bf16 bit patterns for one Softmax+MatMul problem."""
    rng = np.random.default_rng(seed)
    scratch = _Scratch()
    X = _draw_bf16(rng, M, K, logit_scale, scratch=scratch)
    Y = _draw_bf16(rng, K, N, 1.0, scratch=scratch)
    return X, Y


def generate_workload(name: str, T: int = None, seed: int = None):
    """Inputs of a named workload (optionally with a different T or seed)."""
    w = WORKLOADS[name]
    return generate(w.T if T is None else T, w.D, w.F,
                    w.seed if seed is None else seed, w.unit_rms_rows)


def sample_rows(T: int, n: int = 256, seed: int = 1234) -> np.ndarray:
    """Rows to check when checking every row is too slow.

    Covers rows 0, 1, T/2 and T-1, every residue modulo 32 and, as far as n
    allows, every 256-row block; the rest are drawn uniformly.  Sorted, unique.
    """
    if T <= n:
        return np.arange(T, dtype=np.int64)
    rng = np.random.default_rng(seed)
    picks = {0, 1, T // 2, T - 1}
    for res in range(32):
        base = int(rng.integers(0, max(1, (T - res + 31) // 32)))
        r = res + 32 * base
        if r < T:
            picks.add(r)
    for blk in range(0, T, 256):
        if len(picks) >= n:
            break
        picks.add(min(T - 1, blk + int(rng.integers(0, 256))))
    while len(picks) < n:
        picks.add(int(rng.integers(0, T)))
    return np.array(sorted(picks)[:n], dtype=np.int64)
