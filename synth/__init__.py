"""Seeded synthetic inputs shared by the product path's tests/bench and the oracle.

This package holds no arithmetic of the clustering method: it only draws points
(Gaussian mixtures shaped like embedding collections), initial-centroid indices,
random rotations and the named workload configurations.
"""
from .mixture import (CONFIGS, MixtureSpec, config, for_each_chunk, init_indices, make_chunk, make_points,
                      random_rotation)

__all__ = ["MixtureSpec", "CONFIGS", "make_points", "make_chunk", "for_each_chunk", "init_indices", "config",
           "random_rotation"]
