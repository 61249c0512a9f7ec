"""CPU oracle of the decode hot path (float64 numpy). TEST INFRASTRUCTURE ONLY:
imported by tests, the smoke check and the benchmark's CPU-baseline leg, never
by the product path."""
from .ods_oracle import *  # noqa: F401,F403
from . import ods_oracle
