"""fp64 CPU oracle of the LaCT fast-weight path. Test infrastructure only:
imported by tests, the smoke check and the benchmark's CPU-baseline leg."""
from .lact_oracle import *  # noqa: F401,F403
