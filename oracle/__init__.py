"""fp64 CPU oracle for Radar's decode path (test infrastructure only: tests,
the smoke check and the benchmark's CPU-baseline leg use it; the HIP library
never does)."""
from .radar_oracle import *  # noqa: F401,F403
