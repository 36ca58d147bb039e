"""Oracle (test infrastructure): a plain float64 CPU reference of the LSA hot path.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import this package.
"""
from .lsa_oracle import *  # noqa: F401,F403
from .lsa_oracle import IndexParams  # noqa: F401
