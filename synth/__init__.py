"""Seeded synthetic inputs (data rows, queries, encoder weights) shared by the
oracle tests and the GPU path.  Holds no arithmetic of the search method."""
from .philox import philox4x32_10  # noqa: F401
from . import generators, configs  # noqa: F401
