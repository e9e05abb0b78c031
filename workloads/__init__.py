"""Seeded synthetic workloads for the SS-Conv hot path.

This package only describes layer shapes and draws random inputs (voxelised
surfaces, features, coefficients, upstream gradients).  It holds none of the
convolution's arithmetic, so both the CPU oracle and the GPU library can take
their inputs from it without sharing any method code.
"""
from .configs import CONFIGS, LayerSpec, WorkloadSpec, get_config  # noqa: F401
from .gen import (  # noqa: F401
    make_workload,
    make_features,
    make_coeffs,
    make_grad,
    make_motion,
    make_point_cloud,
    make_query_points,
    round_bf16,
    shuffle_rows,
)
