"""Seeded synthetic point clouds shaped like the paper's four workload families.

This package is the only code shared by the CPU oracle side and the HIP side
of the tests: it produces inputs (positions, features, batch ids, conv
weights) and holds none of the lattice arithmetic.
"""
from .clouds import CONFIGS, Workload, make_workload

__all__ = ["CONFIGS", "Workload", "make_workload"]
