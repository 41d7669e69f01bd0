"""CPU fp64 oracle for the Gated MLP and its variants (test infrastructure only).

Only the test-suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP path.
"""
from .oracle import (  # noqa: F401
    Oracle,
    build,
    default_oracle,
    gated_mlp_rows,
    silu,
)
from .brute import brute_gate, brute_gated_mlp, brute_sigmoid, brute_silu  # noqa: F401
