"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and the bench.

This package only draws random numbers and lays them out; it holds none of
the attribution method's arithmetic (no projection, normalisation,
preconditioning or scoring).  Both the CPU oracle and the HIP path receive
the arrays produced here.
"""
from .gen import *  # noqa: F401,F403
