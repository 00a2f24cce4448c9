"""Seeded synthetic inputs for the TSID template-fit path.

This module generates data only.  It holds none of the method's arithmetic:
no residuals, gradients, updates, losses, template maps or bucket orders.
Both the HIP path (through its Python binding) and the CPU oracle consume
what it returns, so neither side can feed the other.

Every workload stands in for a dataset of the paper (Section 6.1) or for a
shape named in the benchmark configurations; none reproduces dataset records.
All randomness comes from numpy's Philox counter-based generator keyed by
(config seed, purpose), so each purpose (latent factors, row/column
popularity, values, hold-out, template, initial factors) draws an
independent stream and a change in one never shifts another.
"""
from .generate import (  # noqa: F401
    Problem,
    PURPOSE,
    make_rng,
    holdout_mask,
    init_factors,
    tiny,
    mid,
    rating,
    scientific_template,
    billion_template,
    random_case,
    dense_lowrank_case,
    similarity_graph,
    CONFIGS,
    make,
    make_cached,
)
from .stream import Phase, omega_outside_template  # noqa: F401,E402
