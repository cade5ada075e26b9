"""Seeded synthetic workloads shared by the tests, the smoke check and the
benchmark. Input generation only: no part of the matrix product or of the
planner lives here, so the oracle and the GPU path can both use it.
"""
from .gen import *  # noqa: F401,F403
