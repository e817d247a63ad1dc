"""Seeded synthetic inputs shared by the product path's tests/bench and the oracle.

This package holds no arithmetic of the clustering method: it only draws points
(Gaussian mixtures shaped like embedding collections), initial-centroid indices
and the named workload configurations.
"""
from .mixture import MixtureSpec, CONFIGS, make_points, make_chunk, init_indices, config

__all__ = ["MixtureSpec", "CONFIGS", "make_points", "make_chunk", "init_indices", "config"]
