"""Seeded synthetic inputs and workload shapes.

This package only draws random numbers and names shapes.  It holds none of
the method's arithmetic (no rotation, no quantization, no products), so the
oracle and the HIP path can both be fed from it without sharing any of the
computation they are compared on.
"""
from .generators import (  # noqa: F401
    rng_for,
    gaussian,
    outlier_channels,
    with_outliers,
    random_orthogonal,
    log_uniform,
)
from . import configs  # noqa: F401
