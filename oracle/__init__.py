"""CPU oracle for the RingAda stage path.  Test infrastructure only: imported
by tests/, by the smoke check and by the benchmark's CPU-baseline leg, never by
the product package."""
from .ringada_oracle import *  # noqa: F401,F403
