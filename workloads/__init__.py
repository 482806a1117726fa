"""Seeded synthetic inputs for the similarity join (shared by the tests, the
oracle checks and the benchmark).

This package only draws and encodes numbers. It computes no inner products,
distances or thresholds tests: those belong to the oracle on one side and to
the GPU library on the other, which share nothing but these inputs.
"""
from .gen import (  # noqa: F401
    Workload,
    CONFIGS,
    NAMES,
    make_config,
    random_case,
    encode,
    bf16_bits_from_f32,
    DTYPES,
    ESIZE,
    to_torch,
    LshParams,
    lsh_params,
)
