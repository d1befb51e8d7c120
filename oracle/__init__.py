"""CPU oracle of the eviction path: test infrastructure only (tests/, the smoke check and
the CPU-baseline leg of bench.py may use it; the product path never does)."""
from .taskpress_oracle import *  # noqa: F401,F403
