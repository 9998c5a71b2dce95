"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This package draws model weights and row tables; it holds none of the
operator's arithmetic (no dequantisation, normalisation, attention or
decoding).  Everything it returns is plain data: numpy / torch arrays in the
library's weight layout and CSR row tables.
"""
from .workloads import (  # noqa: F401
    SHAPES,
    ModelShape,
    QMat,
    Layer,
    Weights,
    Workload,
    make_weights,
    make_workload,
    quantize_int4_g32,
    quantize_fp8_e4m3,
    WORKLOADS,
    Automaton,
    option_trie,
    automaton_of_options,
    automaton_of_list,
    automaton_of_record,
    KIND_AUTOMATON,
    parity_rows,
)
