"""Randomised host-side checks of the kernel plans (no GPU): for shapes drawn
over the supported range, gmlp_describe and softmax_matmul_describe give
plans whose grids cover the problem, whose split-K splits cover the
contracted axis, and whose workspace fits, and every entry point rejects
what it must before touching a device."""
import ctypes

import pytest
from hypothesis import given, settings, strategies as st

from paper_2606_26344_amd import gmlp
from paper_2606_26344_amd import softmax_matmul as smm

dims = st.integers(min_value=1, max_value=4096).map(lambda v: 8 * v)  # multiples of 8, up to 32768
tokens = st.one_of(st.integers(min_value=1, max_value=8), st.integers(min_value=9, max_value=20000))


def _cdiv(a, b):
    return -(-a // b)


def _tile(name):
    # GemmShape<NW, WM, WN, TM, TN, STAGES, BK> -> (columns per weight, tokens per tile)
    args = [int(v) for v in name.split("GemmShape<")[1].split(">")[0].split(",")]
    nw, wm, wn, tm, tn = args[:5]
    return wm * tm * 32, wn * tn * 32


def _flags(name):
    # gemm_mfma_kernel<GemmShape<...>, epilogue, split-K, streamed weights>
    epi, split_k, streamed = [f.strip() for f in name[:-1].split(">, ")[1].split(",")]
    return int(epi), split_k == "true", streamed == "true"


def _steps(plan):
    """The plan's lines grouped by step (gate/up, then down): a GEMM step may
    be followed by the split-K launch of its tail tiles."""
    steps = []
    for line in plan:
        name = line[0]
        if name.startswith("gemv"):
            step = 0 if name.split(",")[1].strip() == "2" else 1
        else:
            step = {0: 0, 1: 1, 2: 0}[_flags(name)[0]]  # epilogue 2: the paired gate/up blocks
        if steps and steps[-1][0] == step:
            steps[-1][1].append(line)
        else:
            steps.append((step, [line]))
    return steps


def _check_step(step, lines, M, K, T):
    """One step's launches cover its M x T outputs over K."""
    for name, grid, block, splits in lines:
        assert grid >= 1 and splits >= 1 and block in (256, 512)
    name, grid, block, splits = lines[0]
    if name.startswith("gemv"):
        # The automatic path takes the GEMV kernels up to 5 tokens.
        assert len(lines) == 1
        assert T <= 5 and name.startswith("gemv_splitk_kernel<%d," % T)
        # Up to 2 tokens: 8-wave blocks; the gate/up step reads 1 KB row
        # segments (512-column strips), the down step 512 bytes (256).
        # Above, 4-wave blocks of 256-column strips.
        assert block == (512 if T <= 2 else 256)
        strips = _cdiv(M, 512 if T <= 2 and step == 0 else 256)
        assert grid == strips * splits
        assert splits <= _cdiv(K, 16)  # each split holds at least one 16-row batch
        return
    assert T > 5
    bmw, bn = _tile(name)
    tiles = _cdiv(M, bmw) * _cdiv(T, bn)
    assert len(lines) == 1
    if splits > 1 and grid != tiles * splits:
        # A tail: whole rounds of 256 tiles, one block each over all of K,
        # then, in the same launch, a partial round of at most half the chip
        # split 2 to 8 ways over K.
        assert _tile(name) in ((128, 256), (256, 256)) and _flags(name)[1]
        whole, tail = tiles // 256 * 256, tiles % 256
        assert whole >= 256 and 0 < tail <= 128 and 2 <= splits <= 8
        assert grid == whole + tail * splits and tail * splits <= 256
        return
    # Every tile is computed by exactly one block, or by one block per split.
    assert grid == tiles * splits
    for name_i, grid_i, _, splits_i in lines:
        assert _tile(name_i) == (bmw, bn) and grid_i % splits_i == 0
        _, split_k, streamed = _flags(name_i)
        # Weights take the streaming cache policy exactly when one token
        # tile reads each of them once.
        assert streamed == (_cdiv(T, bn) == 1)
        if splits_i > 1:
            assert split_k
            assert splits_i * 4 * bmw * bn * 2 * (grid_i // splits_i) <= 2 ** 31  # partials addressable
        if _flags(name_i)[0] == 2:
            # A G and a U block per column tile of one token tile, where
            # the dual-B plan would split K in two or run two 128-token
            # tiles: 65 to 192 tokens.
            assert step == 0 and splits_i == 2 and 65 <= T <= 192 and _cdiv(T, bn) == 1
            assert 96 < grid_i // 2 <= 128  # two-way split of more than 3/4 of a round


def _gate_up_lines(T, D, F):
    return _steps(gmlp.describe(T, D, F))[0][1]


SPLITS = [(T, 4096, 14336, split) for T, split in [(512, False), (513, True), (520, True), (640, True), (704, False),
                                                   (768, False), (1088, True), (1600, True), (1800, False), (2048, False),
                                                   (2112, False), (2340, True), (2880, True)]]
SPLITS += [(T, 8192, 28672, split) for T, split in [(800, False), (1100, True), (1600, True), (2048, False)]]


@pytest.mark.parametrize("T,D,F,split", SPLITS)
def test_gate_up_token_split(T, D, F, split):
    """The gate/up step runs on a token split where the last token tile of
    the 256-token tiles holds at most 128 tokens and the fitted round cost
    of the split plan is lower (the cases measured); the down step keeps
    one plan over all T rows."""
    (_, gu), (_, dn) = _steps(gmlp.describe(T, D, F))
    r = T % 256
    if split:
        assert gu == _gate_up_lines(T - r, D, F) + _gate_up_lines(r, D, F)
    else:
        assert gu[0][0].startswith("gemm_mfma_kernel<GemmShape<2, 4, 2, 1, 4, 2, 64>")
        assert all(_tile(line[0]) == (128, 256) for line in gu)
    assert dn == _steps(gmlp.describe(T, D, F))[1][1]


@settings(max_examples=300, deadline=None)
@given(T=tokens, D=dims, F=dims)
def test_gated_mlp_plan_covers_the_problem(T, D, F):
    plan = gmlp.describe(T, D, F)
    steps = _steps(plan)
    assert [s for s, _ in steps] == [0, 1]
    (_, gu), (_, dn) = steps
    # A token split of the gate/up step: the whole 256-token tiles of the
    # first T - r rows, then the last r <= 128 rows planned on their own,
    # from 513 tokens.
    r = T % 256
    split = 0 < r <= 128 and T > 512 and gu == _gate_up_lines(T - r, D, F) + _gate_up_lines(r, D, F)
    if split:
        head = _gate_up_lines(T - r, D, F)
        assert head[0][0].startswith("gemm_mfma_kernel<GemmShape<2, 4, 2, 1, 4, 2, 64>")
        _check_step(0, head, F, D, T - r)
        _check_step(0, gu[len(head):], F, D, r)
    else:
        _check_step(0, gu, F, D, T)
    _check_step(1, dn, D, F, T)
    ws = gmlp.workspace_size(T, D, F)
    assert ws >= T * F * 2  # holds H
    assert ws % 256 == 0


@pytest.mark.parametrize("T", [256, 257, 300, 320, 383, 384, 385])
@pytest.mark.parametrize("D, F", [(4096, 14336), (8192, 28672), (8200, 16384), (1024, 4096), (2048, 14336)])
def test_192_token_tiles_from_257_to_384_tokens(T, D, F):
    """257 to 384 tokens run as two 192-token tiles: the gate/up step where
    its tiles fill between 3/4 of a round and one round of 256 blocks, the
    down step only where it has 64 to 128 tiles (two or more splits fill a
    round), and at the model dimensions; each weight is then read by both
    token tiles, so neither step streams it."""
    (_, gu), (_, dn) = _steps(gmlp.describe(T, D, F))
    in_range = 256 < T <= 384
    gu_tiles = _cdiv(F, 128) * _cdiv(T, 192)
    dn_tiles = _cdiv(D, 128) * _cdiv(T, 192)
    assert (_tile(gu[0][0]) == (128, 192)) == (in_range and 192 <= gu_tiles <= 256)
    if _tile(dn[0][0]) == (128, 192):
        assert 128 < T <= 192 or (in_range and 64 <= dn_tiles <= 128)
    if in_range and (D, F) in ((4096, 14336), (8192, 28672)):
        assert _tile(dn[0][0]) == (128, 192)
    for name, _, _, _ in gu + dn:
        if _tile(name) == (128, 192) and in_range:
            assert not _flags(name)[2]


@settings(max_examples=100, deadline=None)
@given(T=st.integers(min_value=1, max_value=8), D=dims, F=dims)
def test_fused_plan_is_the_gemv_items(T, D, F):
    (name, grid, block, splits), = gmlp.describe(T, D, F, "fused")
    gemv = gmlp.describe(T, D, F, "gemv")
    assert name == "gemv_fused_kernel<%d, false>" % T
    assert grid == sum(g[1] for g in gemv) and splits == gemv[0][3]


@settings(max_examples=200, deadline=None)
@given(M=tokens, K=dims, N=dims)
def test_softmax_matmul_plan(M, K, N):
    plan = smm.describe(M, K, N)
    assert plan[0][0].startswith("softmax_exp_rows_kernel<")
    assert plan[0][1] == _cdiv(M, 4) and plan[0][2] == 256
    r = int(plan[0][0].split("<")[1].rstrip(">"))
    assert r in (1, 2, 4, 8, 16)
    assert r == 16 or 512 * r >= K  # the row fits in registers unless streamed
    mm = plan[1:]
    if mm[0][0].startswith("gemm"):
        # The matmul's launch (with a tail or not) covers its tiles once.
        _check_step(1, mm, N, K, M)
    else:
        assert len(mm) == 1 and M <= 8
    assert smm.workspace_size(M, K, N) >= M * K * 2 + M * 4


@settings(max_examples=100, deadline=None)
@given(T=st.integers(min_value=0, max_value=20000), D=dims, F=dims)
def test_workspace_holds_h_for_any_token_count(T, D, F):
    # Including T = 0 (nothing to launch; sized as for one token).
    assert gmlp.workspace_size(T, D, F) >= max(T, 1) * F * 2
    assert smm.workspace_size(T, D, F) >= max(T, 1) * D * 2


@settings(max_examples=200, deadline=None)
@given(T=st.integers(min_value=-5, max_value=100), D=st.integers(min_value=-8, max_value=600),
       F=st.integers(min_value=-8, max_value=600))
def test_validation_agrees_with_workspace_size(T, D, F):
    A = 0x10000000
    rc = gmlp.library().gmlp_validate(T, D, F, A, A + (1 << 26), A + (2 << 26), A + (3 << 26),
                                      A + (4 << 26))
    ok_shape = T >= 0 and D > 0 and F > 0 and D % 8 == 0 and F % 8 == 0
    assert (rc == 0) == ok_shape
    assert (gmlp.workspace_size(T, D, F) > 0) == ok_shape
