"""Lloyd k-means on compressed vectors for AMD MI355X (gfx950).

Python face of libkmq.so, the HIP library whose C ABI is declared in
``include/kmq.h``: quantize (bfloat16, SQ8, LVQ4, 1-bit, RabitQ), PCA statistics and
projection, and the Lloyd steps (assign, update, fit) on fp32, bfloat16, SQ8, LVQ4,
1-bit, RabitQ and hybrid points, with dimension pruning for fp32 and SQ8 points, and
hierarchical k-means built from them.
"""
from ._kmq import (  # noqa: F401
    KM_BF16, KM_EMPTY_KEEP, KM_EMPTY_SPLIT, KM_F32, KM_HYBRID, KM_LVQ4, KM_RABITQ, KM_SIGN1, KM_SQ8, KmFitStats,
    KmHierParams, KmPrune, KmqError, Points, kmeans_assign, kmeans_assign_noalloc, kmeans_assign_pruned, kmeans_cost, kmeans_fine, kmeans_fit,
    kmeans_fit_hier, kmeans_fit_pruned, kmeans_update, lib, pca_fit_cov, pca_project,
    points_bf16, points_f32, points_hybrid, points_lvq4, points_rabitq, points_sign1, points_sq8, quantize_bf16,
    quantize_lvq4, quantize_sign1, quantize_sq8, rabitq_encode, release)
