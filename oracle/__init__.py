"""CPU fp64 oracles for the Gated MLP and its variants, and for Softmax+MatMul
(test infrastructure only).

Only the test-suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP path.
"""
from .oracle import (  # noqa: F401
    Oracle,
    default_oracle,
    gated_mlp_rows,
    silu,
)
from .softmax_matmul import SoftmaxMatmulOracle, softmax_matmul_rows  # noqa: F401
from .brute import (  # noqa: F401
    brute_gate,
    brute_gated_mlp,
    brute_sigmoid,
    brute_silu,
    brute_softmax_matmul,
)


def build() -> None:
    """Compile both oracle libraries with gcc."""
    from . import oracle as _gmlp, softmax_matmul as _smm

    _gmlp.build()
    _smm.build()
