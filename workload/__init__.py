"""Seeded synthetic decode-step inputs shared by the tests, the benchmark and
the oracle's callers.  This package builds inputs only: it holds none of the
attention arithmetic (no softmax, no CDF, no sampling, no gather)."""

from .gen import (  # noqa: F401
    CONFIGS,
    Workload,
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    make_workload,
)
