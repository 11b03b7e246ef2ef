"""Seeded synthetic inputs (graphs, features, weights) shared by the CPU
oracle and the GPU path.  Holds none of the layer's arithmetic."""
from . import configs, graphs, tensors  # noqa: F401
