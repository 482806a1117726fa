"""Oracle for the similarity join -- TEST INFRASTRUCTURE ONLY.

Only the tests, the package smoke check and the benchmark's CPU-baseline leg
may import this package.  The GPU library and its Python binding never do.
"""
from .oracle import (  # noqa: F401
    build,
    decode,
    join,
    count,
    scores,
    max_threads,
    lsh_keys,
    lsh_join,
    round_to,
    normalize,
    hamming,
    hamming_join,
    JoinResult,
)
from . import jl  # noqa: F401,E402
