"""Seeded synthetic inputs for the coded matrix-multiplication workloads.

This package holds random draws, dtype rounding, workload shapes and the
choice among seeded generators by their decode conditioning only; it contains
none of the coded method's arithmetic (no encode, product or decode).  Both the oracle and the GPU
path take their inputs from here.
"""
from .inputs import (  # noqa: F401
    STREAM_A, STREAM_X, STREAM_P, STREAM_RUNTIME, STREAM_NOISE, STREAM_WSTAR,
    STREAM_PT, STREAM_SETS, ROW_CHUNK, generator, gaussian, gaussian_rows, integers,
    bf16_round, bf16_bits, bf16_from_bits, parity_matrix, integer_parity_matrix,
    worst_decode_condition, conditioned_parity_matrix, exact_parity_sets,
)
from .workloads import WORKLOADS, Workload, gd_codes  # noqa: F401
