"""Seeded synthetic inputs (clouds, features, weights) and pipeline
descriptions shared by the oracle tests and the GPU path.  Holds none of the
lattice method's arithmetic."""
from . import rng, generators, configs  # noqa: F401
