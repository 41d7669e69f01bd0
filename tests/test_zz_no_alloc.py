"""gmlp_forward_noalloc: the entry point for callers that cannot allocate.

It runs the kernels of gmlp_forward with the library's static per-device
scratch array as workspace, so its Y must equal gmlp_forward's bit for bit
(and be within the oracle's tolerance |Y - Y_ref| <= 1e-2 (|Y_ref| + rms)).
Two calls in a row, the second on a smaller shape, check that the array's
leftover contents from one call do not leak into the next.  The size check
runs on the host before any HIP call, so it is tested without a GPU.
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_2606_26344_amd import gmlp
from paper_2606_26344_amd import inputs as I

TOL = 1e-2
A = 0x10000000  # fake, aligned, far-apart addresses: rejected calls never dereference them
GB = 1 << 30


def _check(got_bits, ref, what):
    got = I.bf16_bits_to_f32(got_bits).astype(np.float64)
    bound = TOL * (np.abs(ref) + np.sqrt(np.mean(ref ** 2)))
    ratio = float(np.max(np.abs(got - ref) / bound))
    print("%s max err/bound = %.3f" % (what, ratio), flush=True)
    assert np.all(np.abs(got - ref) <= bound), what


def test_noalloc_rejects_shapes_past_its_scratch():
    lib = gmlp.library()
    T, D, F = 4096, 4096, 14336  # needs ~112 MiB of workspace
    assert gmlp.workspace_size(T, D, F) > lib_limit()
    rc = lib.gmlp_forward_noalloc(A, A + GB, A + 2 * GB, A + 3 * GB, A + 4 * GB, T, D, F, None)
    assert rc == 2, gmlp.last_error()
    assert "noalloc" in gmlp.last_error()
    # Invalid arguments are rejected as by gmlp_forward.
    assert lib.gmlp_forward_noalloc(None, A + GB, A + 2 * GB, A + 3 * GB, A + 4 * GB, 4, 256, 512,
                                    None) == 1
    # No rows: nothing to do, nothing launched.
    assert lib.gmlp_forward_noalloc(None, A + GB, A + 2 * GB, A + 3 * GB, None, 0, 256, 512, None) == 0


def lib_limit():
    import re

    text = open(gmlp.HEADER).read()
    m = re.search(r"#define GMLP_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", text)
    return int(m.group(1)) << int(m.group(2))


@pytest.mark.gpu
def test_noalloc_equals_allocating_entry_on_two_calls(orc):
    assert torch.cuda.is_available(), "GPU test needs a HIP device"
    # First a T = 128 call (MFMA path with split-K partial sums), then a
    # smaller one on the GEMV path (T = 3) and a small MFMA one (T = 20).
    for T, D, F in [(128, 4096, 14336), (3, 1032, 2056), (20, 264, 520)]:
        print("noalloc T=%d D=%d F=%d" % (T, D, F), flush=True)
        assert gmlp.workspace_size(T, D, F) <= lib_limit()
        X, Wg, Wu, Wd = I.generate(T, D, F, seed=300 + T)
        args = [gmlp.from_bf16_bits(a) for a in (X, Wg, Wu, Wd)]
        ref = gmlp.forward(*args)  # gmlp_forward, the allocating entry point
        y = torch.full((T, D), float("nan"), dtype=torch.bfloat16, device="cuda")
        gmlp.forward_noalloc(*args, out=y)
        torch.cuda.synchronize()
        got = gmlp.to_bf16_bits(y)
        assert np.array_equal(got, gmlp.to_bf16_bits(ref)), "T=%d: differs from gmlp_forward" % T
        rows = I.sample_rows(T, 16)
        _check(got[rows], orc.gated_mlp_rows(X, Wg, Wu, Wd, rows=rows), "noalloc T=%d" % T)


@pytest.mark.gpu
def test_noalloc_repeated_calls_on_a_side_stream(orc):
    # The counters of the shared array stay at zero between calls: calls
    # ordered on one (non-default) stream give the same bits each time.
    T, D, F = 48, 1032, 2056
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=77)
    args = [gmlp.from_bf16_bits(a) for a in (X, Wg, Wu, Wd)]
    s = torch.cuda.Stream()
    outs = [torch.empty((T, D), dtype=torch.bfloat16, device="cuda") for _ in range(3)]
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for y in outs:
            gmlp.forward_noalloc(*args, out=y, stream=s)
    s.synchronize()
    first = gmlp.to_bf16_bits(outs[0])
    for y in outs[1:]:
        assert np.array_equal(gmlp.to_bf16_bits(y), first)
    _check(first, orc.gated_mlp_rows(X, Wg, Wu, Wd), "noalloc side stream")
