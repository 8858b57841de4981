"""MI355X (gfx950) batched dynamic updates of proximity-graph ANN indexes
(GrAND: Vamana with GrANDRobustPrune and a CAGRA-style fixed-degree
variant).  The work runs in the HIP library libgrand.so; this package holds
its sources (csrc/), its build script and a thin ctypes binding."""
from .grand import GrandError, GrandIndex, Params, Reader, load_library, params_from_config  # noqa: F401
