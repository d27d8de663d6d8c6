"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke run.

This package draws random numbers and nothing else: it holds none of the
boosting method's arithmetic (no binning, no histograms, no gains, no
boosting).  Both the CPU oracle and the GPU library receive the arrays it
produces as plain inputs.
"""
from .generators import (  # noqa: F401
    CONFIGS,
    ConfigSpec,
    make_training_set,
    make_apply_chunk,
    apply_chunks,
    random_forest,
    random_binned,
    digest,
)
