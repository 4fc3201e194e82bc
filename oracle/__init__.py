"""CPU oracle of the SlimWise batched-decode MoE layer (test infrastructure).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this package.  It shares no code with the HIP library.
"""
from .oracle import (  # noqa: F401
    CFLAGS,
    build,
    dispatch,
    forward,
    forward_f64,
    layer,
    lib_path,
    prune_compact,
    route,
    routing_mass,
    shared_expert,
)
