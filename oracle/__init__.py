"""CPU oracle for GrowPage's decode-step hot path (test infrastructure only).

Plain, slow, fp64 NumPy written from the paper's definitions.  Only the test
suite, the package smoke check and the benchmark's CPU-baseline leg may import
it; the library and its Python binding never do.
"""
from .growpage_oracle import *  # noqa: F401,F403
