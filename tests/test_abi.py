"""Host-side checks of the C ABI (no GPU): the library loads, exports every
function include/gmlp.h declares, and rejects bad arguments before touching
any device (validation runs first and makes no HIP call)."""
import ctypes

import pytest

from paper_2606_26344_amd import gmlp
from paper_2606_26344_amd import softmax_matmul as smm

A = 0x10000000  # fake, 256-byte aligned addresses: validation never dereferences
MB = 1 << 20


@pytest.fixture(scope="module")
def lib():
    return gmlp.library()


def test_every_declared_symbol_is_exported(lib):
    names = gmlp.header_functions()
    assert len(names) >= 11
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(gmlp._SIGNATURES)


def test_version_and_status_strings(lib):
    assert gmlp.version() == 100
    assert gmlp.status_string(0) == "GMLP_OK"
    assert gmlp.status_string(1) == "GMLP_ERR_INVALID_ARG"
    assert gmlp.status_string(2) == "GMLP_ERR_UNSUPPORTED"
    assert gmlp.status_string(3) == "GMLP_ERR_HIP"
    assert gmlp.status_string(4) == "GMLP_ERR_NO_MEMORY"
    assert gmlp.status_string(99) == "GMLP_ERR_UNKNOWN"


def _validate(lib, T, D, F, X=A, Wg=A + 64 * MB, Wu=A + 128 * MB, Wd=A + 192 * MB, Y=A + 256 * MB):
    return lib.gmlp_validate(T, D, F, X, Wg, Wu, Wd, Y)


def test_validate_accepts_good_arguments(lib):
    assert _validate(lib, 16, 256, 512) == 0
    assert gmlp.last_error() == ""
    assert _validate(lib, 0, 8, 8, X=None, Y=None) == 0  # no rows: X, Y may be NULL


@pytest.mark.parametrize("T,D,F,code", [
    (-1, 256, 512, 1), (4, 0, 512, 1), (4, 256, 0, 1), (4, -8, 512, 1),
    (4, 260, 512, 2), (4, 256, 516, 2), (4, 1 << 23, 8, 2), (1 << 31, 8, 8, 2),
])
def test_validate_rejects_bad_shapes(lib, T, D, F, code):
    assert _validate(lib, T, D, F) == code
    assert gmlp.last_error() != ""


@pytest.mark.parametrize("which", ["X", "Wg", "Wu", "Wd", "Y"])
def test_validate_rejects_null_and_misaligned(lib, which):
    assert _validate(lib, 4, 256, 512, **{which: None}) == 1
    assert _validate(lib, 4, 256, 512, **{which: A + 8}) == 2
    assert which in gmlp.last_error()


def test_validate_rejects_aliasing_output(lib):
    assert _validate(lib, 4, 256, 512, Y=A) == 1  # Y on top of X
    assert _validate(lib, 4, 256, 512, Y=A + 64 * MB + 1024) == 1  # inside Wg
    assert "overlap" in gmlp.last_error()


def test_workspace_size(lib):
    # T = 0 is a valid shape (a call launches nothing); sizing it must not
    # divide by the empty token-tile count.
    assert gmlp.workspace_size(0, 256, 512) > 0
    assert smm.workspace_size(0, 256, 512) > 0
    assert gmlp.workspace_size(16, 256, 512) > 0
    assert gmlp.workspace_size(4096, 4096, 14336) >= 4096 * 14336 * 2  # holds H
    assert gmlp.workspace_size(1, 4096, 14336) > 0
    assert gmlp.workspace_size(-1, 256, 512) == 0
    assert gmlp.workspace_size(4, 260, 512) == 0


def test_zero_tokens_is_a_no_op(lib):
    assert lib.gmlp_forward(None, A, A + 64 * MB, A + 128 * MB, None, 0, 256, 512, None) == 0
    assert lib.gmlp_forward_ex(None, A, A + 64 * MB, A + 128 * MB, None, 0, 256, 512, 0,
                               None, 0, None) == 0


def test_forward_ex_checks_path_and_workspace_before_launching(lib):
    args = (A, A + 64 * MB, A + 128 * MB, A + 192 * MB, A + 256 * MB, 16, 256, 512)
    n = gmlp.workspace_size(16, 256, 512)
    assert lib.gmlp_forward_ex(*args, 7, A + 300 * MB, n, None) == 1  # unknown path
    assert lib.gmlp_forward_ex(*args, gmlp.PATH_GEMV, A + 300 * MB, n, None) == 2  # T > 8
    assert lib.gmlp_forward_ex(*args, 0, None, n, None) == 1  # no workspace
    assert lib.gmlp_forward_ex(*args, 0, A + 300 * MB + 16, n, None) == 2  # misaligned
    assert lib.gmlp_forward_ex(*args, 0, A + 300 * MB, n - 1, None) == 4  # too small
    assert lib.gmlp_workspace_init(None, 1024, None) == 1


def test_helpers_validate_too(lib):
    assert lib.gmlp_gate_up(A, A + 64 * MB, A + 128 * MB, None, 4, 256, 512, None) == 1
    assert lib.gmlp_gate_up(A, A + 64 * MB, A + 128 * MB, A, 4, 256, 512, None) == 1  # H on X
    assert lib.gmlp_down(A, A + 64 * MB, None, 4, 512, 256, None) == 1
    assert lib.gmlp_down(A, A + 64 * MB, A + 8, 4, 512, 256, None) == 2


def test_describe_names_the_kernels_of_each_path(lib):
    gemv = gmlp.describe(1, 4096, 14336)
    assert [k[0] for k in gemv] == ["gemv_splitk_kernel<1, 2, 0, false>",
                                    "gemv_splitk_kernel<1, 1, 1, false>"]
    for name, grid, block, splits in gemv:
        assert block == 512 and 128 < grid <= 256 and splits > 1  # 8-wave blocks up to 2 tokens
    big = gmlp.describe(4096, 4096, 14336)
    assert [k[0].split("<")[0] for k in big] == ["gemm_mfma_kernel", "gemm_mfma_kernel"]
    # <shape, epilogue, split-K, streamed weights>: prefill has neither.
    assert big[0][0].endswith(", 0, false, false>") and big[1][0].endswith(", 1, false, false>")
    # One token tile (T = 128): split-K, and weights read once, so streamed;
    # gate/up as pairs of one-weight blocks (epilogue 2) over the whole of K.
    mid = gmlp.describe(128, 4096, 14336)
    assert mid[0][0].endswith(", 2, true, true>") and mid[1][0].endswith(", 1, true, true>")
    assert mid[0][0].startswith("gemm_mfma_kernel<GemmShape<1,") and mid[0][1] == 224 and mid[0][3] == 2
    # Up to 64 tokens the dual-B tiles split over K.
    assert gmlp.describe(64, 4096, 14336)[0][0].endswith(", 0, true, true>")
    # Up to 32, 64 and 96 tokens: one tile of 32, 64 or 96 tokens (streamed).
    for T, bn in [(9, 32), (32, 32), (33, 64), (64, 64), (65, 96), (96, 96), (97, 128)]:
        for name, *_ in gmlp.describe(T, 4096, 14336):
            wm, wn, tm, tn = [int(v) for v in name.split("<")[2].split(",")[1:5]]
            assert wn * tn * 32 == bn and name.endswith(", true, true>"), (T, name)
    # Two token tiles re-read each weight tile: not streamed.
    assert all(k[0].endswith(", false>") for k in gmlp.describe(256, 4096, 14336))
    assert gmlp.describe(0, 256, 512) == []


def test_describe_rejects_bad_arguments(lib):
    buf = ctypes.create_string_buffer(64)
    assert lib.gmlp_describe(4, 260, 512, 0, buf, 64) == 2
    assert lib.gmlp_describe(9, 256, 512, 1, buf, 64) == 2  # GEMV needs T <= 8
    assert lib.gmlp_describe(4, 256, 512, 5, buf, 64) == 1  # unknown path
    assert lib.gmlp_describe(65, 256, 512, 4, buf, 64) == 2  # fused MFMA needs T <= 64
    assert lib.gmlp_describe(4, 256, 512, 0, None, 64) == 1
    assert lib.gmlp_describe(4, 256, 512, 0, buf, 8) == 0 and len(buf.value) == 7  # truncated


@pytest.mark.parametrize("T", [1, 2, 3, 5, 8])
@pytest.mark.parametrize("D,F", [(4096, 14336), (8192, 28672), (264, 520), (4104, 2056), (8, 8)])
def test_gemv_plan_covers_k_with_at_most_one_round_of_blocks(lib, T, D, F):
    for step, ((name, grid, block, splits), (M, K)) in enumerate(zip(gmlp.describe(T, D, F, "gemv"),
                                                                     [(F, D), (D, F)])):
        # 8-wave blocks up to 2 tokens; gate/up strips of 512 columns there.
        width = 512 if T <= 2 and step == 0 else 256
        strips = -(-M // width)
        assert grid == strips * splits and block == (512 if T <= 2 else 256)
        assert splits <= K // 8 + 1
        assert grid <= max(512, strips)


def test_variant_entry_points_validate_before_launching(lib):
    n = gmlp.workspace_size(4, 256, 512)
    base = (A, A + 64 * MB, A + 128 * MB, A + 192 * MB, A + 256 * MB, 4, 256, 512)
    fwd = lambda act, beta, rms, eps: lib.gmlp_forward_variant(*base, act, beta, rms, eps, 0,
                                                                A + 300 * MB, n, None)
    assert fwd(3, 1.0, 0, 0.0) == 1 and "activation" in gmlp.last_error()
    assert fwd(-1, 1.0, 0, 0.0) == 1
    assert fwd(1, float("nan"), 0, 0.0) == 1 and "beta" in gmlp.last_error()
    assert fwd(1, float("inf"), 0, 0.0) == 1
    assert fwd(0, 1.0, 2, 0.0) == 1 and "rmsnorm" in gmlp.last_error()
    assert fwd(0, 1.0, 1, -1e-6) == 1 and "eps" in gmlp.last_error()
    assert fwd(0, 1.0, 1, float("nan")) == 1
    gu = lambda act: lib.gmlp_gate_up_variant(A, A + 64 * MB, A + 128 * MB, A + 192 * MB, 4, 256, 512,
                                              act, 1.0, 0, 0.0, 0, A + 300 * MB, n, None)
    assert gu(7) == 1
    # Shape and workspace errors come first, as for gmlp_forward_ex.
    assert lib.gmlp_forward_variant(A, A + 64 * MB, A + 128 * MB, A + 192 * MB, A + 256 * MB, 4, 260,
                                    512, 0, 1.0, 0, 0.0, 0, A + 300 * MB, n, None) == 2
    assert lib.gmlp_forward_variant(*base, 2, 1.0, 1, 1e-5, 0, A + 300 * MB, n - 256, None) == 4
    with pytest.raises(ValueError):
        gmlp._variant("relu", 1.0, False, 0.0)


# ---- Softmax+MatMul (include/softmax_matmul.h) --------------------------------


def test_softmax_matmul_describe_names_the_kernels(lib):
    big = smm.describe(8192, 8192, 8192)
    assert big[0] == ("softmax_exp_rows_kernel<16>", 2048, 256, 1)
    assert big[1][0].startswith("gemm_mfma_kernel<GemmShape<1,") and big[1][0].endswith(", 1, false, false>")
    small = smm.describe(3, 4096, 1032)
    assert small[0] == ("softmax_exp_rows_kernel<8>", 1, 256, 1)
    assert small[1][0] == "gemv_splitk_kernel<3, 1, 1, false>"
    assert smm.describe(3, 4096, 1032, "mfma")[1][0].endswith(", 1, true, true>")
    # Chunks per lane: the smallest power of two with 512 columns each that
    # covers K, at most 16 (longer rows are streamed).
    for K, r in [(8, 1), (512, 1), (520, 2), (1024, 2), (2048, 4), (4104, 16), (8192, 16),
                 (16392, 16)]:
        assert smm.describe(1, K, 64)[0][0] == "softmax_exp_rows_kernel<%d>" % r, K
    assert smm.describe(0, 64, 64) == []


def test_softmax_matmul_rejects_bad_arguments(lib):
    buf = ctypes.create_string_buffer(256)
    assert lib.softmax_matmul_describe(4, 260, 512, 0, buf, 256) == 2  # K % 8
    assert lib.softmax_matmul_describe(4, 256, 36, 0, buf, 256) == 2   # N % 8
    assert lib.softmax_matmul_describe(-1, 256, 512, 0, buf, 256) == 1
    assert lib.softmax_matmul_describe(9, 256, 512, 1, buf, 256) == 2  # GEMV needs M <= 8
    assert lib.softmax_matmul_workspace_size(4, 260, 512) == 0
    assert lib.softmax_matmul_workspace_size(4, 256, 0) == 0
    n = smm.workspace_size(4, 256, 512)
    assert n >= 4 * 256 * 2 + 4 * 4
    X, Y, Z, W = A, A + 64 * MB, A + 128 * MB, A + 192 * MB
    call = lambda *a: lib.softmax_matmul_ws(*a)
    assert call(None, Y, Z, 4, 256, 512, 0, W, n, None) == 1
    assert call(X, Y, None, 4, 256, 512, 0, W, n, None) == 1
    assert call(X + 8, Y, Z, 4, 256, 512, 0, W, n, None) == 2   # misaligned
    assert call(X, Y, X, 4, 256, 512, 0, W, n, None) == 1       # Z on X
    assert call(X, Y, Y + 64, 4, 256, 512, 0, W, n, None) == 1  # Z on Y
    assert call(X, Y, Z, 4, 256, 512, 0, W, n - 256, None) == 4  # workspace too small
    assert call(X, Y, Z, 4, 256, 512, 0, W + 16, n, None) == 2  # workspace misaligned
    assert call(X, Y, Z, 4, 256, 512, 0, None, n, None) == 1
    assert call(X, Y, W + 256, 4, 256, 512, 0, W, n, None) == 1  # Z inside the workspace
    assert call(X, Y, Z, 4, 256, 512, 5, W, n, None) == 1        # unknown path
    assert call(None, Y, None, 0, 256, 512, 0, None, 0, None) == 0  # M == 0: nothing to do
    assert lib.softmax_matmul(X, Y, X, 4, 256, 512, None) == 1


def test_softmax_matmul_halves_validate_before_launching(lib):
    X, P, S, Y, Z, W = A, A + 64 * MB, A + 128 * MB, A + 160 * MB, A + 192 * MB, A + 256 * MB
    n = smm.workspace_size(4, 256, 512)
    assert lib.softmax_matmul_exp_rows(X, P, None, 4, 256, None) == 1
    assert lib.softmax_matmul_exp_rows(X, P, S + 2, 4, 256, None) == 2
    assert lib.softmax_matmul_exp_rows(X, X + 512, S, 4, 256, None) == 1  # P on X
    assert lib.softmax_matmul_exp_rows(X, P, P + 16, 4, 256, None) == 1    # s on P
    assert lib.softmax_matmul_exp_rows(X, P, S, 4, 260, None) == 2
    assert lib.softmax_matmul_exp_rows(None, None, None, 0, 256, None) == 0
    div = lambda *a: lib.softmax_matmul_divide_ws(*a)
    assert div(P, None, Y, Z, 4, 256, 512, 0, W, n, None) == 1
    assert div(P, S, Y, S, 4, 256, 512, 0, W, n, None) == 1   # Z on s
    assert div(P, S, Y, Z, 4, 256, 512, 0, W, n - 256, None) == 4
    assert div(P, S, Y, Z, 9, 256, 512, 1, W, n, None) == 2   # GEMV needs M <= 8


def test_fused_path_plan_and_validation(lib):
    fused = gmlp.describe(1, 4096, 14336, "fused")
    gemv = gmlp.describe(1, 4096, 14336, "gemv")
    assert len(fused) == 1 and fused[0][0] == "gemv_fused_kernel<1, false>"
    # One block per item of either step: the gate/up items first.
    assert fused[0][1] == sum(g[1] for g in gemv) and fused[0][2] == gemv[0][2] == 512
    assert fused[0][3] == gemv[0][3]
    for T in range(1, 9):
        (name, grid, block, splits), = gmlp.describe(T, 264, 520, "fused")
        assert name == "gemv_fused_kernel<%d, false>" % T
        assert grid == sum(g[1] for g in gmlp.describe(T, 264, 520, "gemv"))
    buf = ctypes.create_string_buffer(64)
    assert lib.gmlp_describe(9, 256, 512, 3, buf, 64) == 2  # fused needs T <= 8
    n = gmlp.workspace_size(4, 256, 512)
    args = (A, A + 64 * MB, A + 128 * MB, A + 192 * MB, A + 256 * MB, 9, 256, 512)
    assert lib.gmlp_forward_ex(*args, 3, A + 300 * MB, n, None) == 2
    # The single-step entry points and Softmax+MatMul have no fused form.
    assert lib.gmlp_gate_up_ws(A, A + 64 * MB, A + 128 * MB, A + 192 * MB, 4, 256, 512, 3,
                               A + 300 * MB, n, None) == 2
    assert lib.gmlp_down_ws(A, A + 64 * MB, A + 128 * MB, 4, 512, 256, 3, A + 300 * MB, n,
                            None) == 2
    m = smm.workspace_size(4, 256, 512)
    assert lib.softmax_matmul_ws(A, A + 64 * MB, A + 128 * MB, 4, 256, 512, 3, A + 192 * MB, m,
                                 None) == 2
    assert "fused" in gmlp.last_error()


def test_last_error_is_kept_per_thread(lib):
    # Two host threads fail validation for different reasons at the same
    # time; each reads back its own detail (ctypes drops the GIL in calls).
    import threading

    start = threading.Barrier(2)
    seen = {}

    def worker(key, T, D, code, needle):
        start.wait()
        bad = 0
        for _ in range(500):
            rc = lib.gmlp_validate(T, D, 512, A, A + 64 * MB, A + 128 * MB, A + 192 * MB, A + 256 * MB)
            if rc != code or needle not in gmlp.last_error():
                bad += 1
        seen[key] = bad

    threads = [threading.Thread(target=worker, args=("shape", -1, 256, 1, "invalid shape")),
               threading.Thread(target=worker, args=("align", 4, 12, 2, "multiples of 8"))]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert seen == {"shape": 0, "align": 0}
    assert lib.gmlp_validate(4, 256, 512, A, A + 64 * MB, A + 128 * MB, A + 192 * MB, A + 256 * MB) == 0
