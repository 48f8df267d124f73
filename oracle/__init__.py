"""CPU oracle for the conv2d forward primitive (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg import
this package.  It shares no code with the GPU library.
"""
from .oracle import (OracleError, conv2d, conv2d_points, normalised_errors, output_dims,
                     max_threads, load)

__all__ = ["OracleError", "conv2d", "conv2d_points", "normalised_errors", "output_dims",
           "max_threads", "load"]
