"""fp64 CPU oracle of the Deja Vu decode hot path.

TEST INFRASTRUCTURE ONLY: imported by tests/, by the package smoke check and by the
benchmark's CPU-baseline leg. The HIP library and its binding never import it, and
it imports nothing from them.
"""
from . import dejavu  # noqa: F401
