"""CPU oracle for the K-seed DiT denoise step (test infrastructure only).

Plain, slow, float64 numpy definitions of every step on the hot path. Only the
test suite, the smoke check and the CPU-baseline leg of the benchmark may
import it; the product library never does, and this package imports nothing
from the product library.
"""
from .dit_oracle import *  # noqa: F401,F403
