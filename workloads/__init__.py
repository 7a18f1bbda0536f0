"""Seeded synthetic workloads for the SAME Gibbs sampler.

This package only makes inputs: network structures, true and initial CPTs,
forward-sampled data, missing-data masks and initial replica states.  It holds
none of the sampler's arithmetic and is shared by the oracle tests, the GPU
parity tests, ``bench.py`` and the smoke check, which all receive the same
arrays from it.
"""
from .synth import (  # noqa: F401
    CONFIGS,
    Network,
    Workload,
    cpt_layout,
    holdout,
    koller,
    make_network,
    make_workload,
    sampler_seed,
)
