"""fp64 CPU oracle (test infrastructure only: imported by the tests, the smoke check and
the bench's CPU-baseline leg, never by the GPU library or its binding)."""
from .crown64 import *  # noqa: F401,F403
