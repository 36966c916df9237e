"""CPU oracle for two-level sparse decode attention.

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.
"""
from .tls_oracle import *  # noqa: F401,F403
from . import tls_oracle  # noqa: F401
