"""Seeded synthetic workloads for the AtSpeed verify path.

This package only draws inputs: item catalogs, user histories, prompts and
random-init weights.  It holds none of the method's arithmetic, so both the
CPU oracle and the GPU path may use it.
"""
from .workloads import (  # noqa: F401
    ModelDims, Workload, WORKLOADS, get_workload, make_catalog, make_prefixes,
    make_weights, philox_key, item_token, seed_streams,
)
