"""CPU oracle for the attribution hot path (test infrastructure).

This package is test infrastructure only.  The product library never imports,
links or calls it; only the tests, the smoke check and the bench's CPU
baseline leg do.  See ``attr_oracle`` for the functions and their citations.
"""
from .attr_oracle import *  # noqa: F401,F403
