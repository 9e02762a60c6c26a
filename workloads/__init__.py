"""Seeded synthetic inputs shared by the tests, the bench and the smoke run.

This package holds only input recipes (random draws, length rescaling and
index layout). It contains none of the reduction arithmetic, so both the CPU
oracle side and the GPU side of a parity test can consume the same arrays.
"""
from .generators import (  # noqa: F401
    CONFIGS,
    lr_rescale,
    index_from_lengths,
    lengths_from_index,
    values_uniform,
    values_normal,
    make_config,
    config_lengths,
    random_problem,
    random_gather_problem,
)
