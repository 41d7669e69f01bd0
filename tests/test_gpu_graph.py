"""The workspace entry points under HIP graph capture.

gmlp_forward_ex, gmlp_forward_variant and softmax_matmul_ws allocate
nothing, issue no memset and leave every arrival counter and ready word of
the workspace at zero, so a call can be captured once and replayed.  Each
replay here follows some eager work on the same stream and must give the
eager result bit for bit.
"""
import numpy as np
import pytest
import torch

from paper_2606_26344_amd import gmlp
from paper_2606_26344_amd import inputs as I
from paper_2606_26344_amd import softmax_matmul as smm

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    gmlp.library()


CASES = [(1, 1032, 2056, "auto", {}), (4, 1032, 2056, "fused", {}), (3, 264, 520, "gemv",
         dict(activation="swish", beta=1.702, rmsnorm=True, eps=1e-6)),
         (200, 1032, 2056, "auto", {}), (16, 264, 520, "mfma", dict(rmsnorm=True, eps=1e-5)),
         (48, 1032, 2056, "auto", dict(activation="sigmoid")), (7, 264, 520, "auto", {})]


@pytest.mark.parametrize("T,D,F,path,variant", CASES, ids=["T%d-%s-%d" % (c[0], c[3], i) for i, c in enumerate(CASES)])
def test_gated_mlp_graph_replays_match_eager(T, D, F, path, variant):
    print("graph T=%d D=%d F=%d path=%s %s" % (T, D, F, path, variant), flush=True)
    X, Wg, Wu, Wd = I.generate(T, D, F, seed=T + D)
    x, wg, wu, wd = (gmlp.from_bf16_bits(a) for a in (X, Wg, Wu, Wd))
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        ws = gmlp.Workspace(T, D, F, stream=stream)
        y = torch.empty((T, D), dtype=torch.bfloat16, device="cuda")
        gmlp.forward(x, wg, wu, wd, out=y, path=path, workspace=ws, **variant)
    torch.cuda.synchronize()
    eager = gmlp.to_bf16_bits(y)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        gmlp.forward(x, wg, wu, wd, out=y, path=path, workspace=ws, **variant)
    for i in range(4):
        # Eager work on the same stream between replays: the same call on
        # other inputs, then clearing the output.
        with torch.cuda.stream(stream):
            gmlp.forward(x * (i + 2), wg, wu, wd, out=y, path=path, workspace=ws, **variant)
            y.zero_()
            graph.replay()  # on the same stream, after that work
        torch.cuda.synchronize()
        assert np.array_equal(gmlp.to_bf16_bits(y), eager), "replay %d differs" % i


def test_softmax_matmul_graph_replays_match_eager():
    X, Y = I.generate_softmax_matmul(64, 2056, 520, seed=3)
    x, yw = gmlp.from_bf16_bits(X), gmlp.from_bf16_bits(Y)
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        ws = smm.make_workspace(64, 2056, 520, stream=stream)
        z = torch.empty((64, 520), dtype=torch.bfloat16, device="cuda")
        smm.softmax_matmul(x, yw, out=z, workspace=ws)
    torch.cuda.synchronize()
    eager = gmlp.to_bf16_bits(z)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        smm.softmax_matmul(x, yw, out=z, workspace=ws)
    for i in range(4):
        with torch.cuda.stream(stream):
            smm.softmax_matmul(x * 0.5, yw, out=z, workspace=ws)
            z.zero_()
            graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(gmlp.to_bf16_bits(z), eager), "replay %d differs" % i
