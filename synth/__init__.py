"""Seeded synthetic inputs for the propagate path.

This module generates graphs and features only: it holds none of the
method's arithmetic (no degrees, normalisation or aggregation). Both the
oracle-side checks and the HIP-side runs draw their inputs from here.
"""
from .graphs import (  # noqa: F401
    CONFIG_NAMES,
    chung_lu_pairs,
    config1_sparse_uniform,
    config2_power_law,
    config3_minibatch,
    config4_knn_clouds,
    config5_large_power_law,
    erdos_renyi,
    make_config,
    graded_in_degree,
    random_coo,
    rng_for,
    star_graph,
    symmetrize,
    uniform_pairs,
    with_self_loops,
)
