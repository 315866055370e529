"""Seeded synthetic workloads shared by the oracle, the tests and the benchmark.

This package holds model shapes, workload definitions and seeded random
generators only. It contains none of the decoder's arithmetic: the oracle
(``oracle/``) and the HIP engine (``paper_2502_15524_amd``) each implement the
computation on their own and meet only here, at their inputs.
"""
from .configs import ModelCfg, Workload, MODELS, WORKLOADS, workload  # noqa: F401
from .gen import (  # noqa: F401
    TENSOR_IDS, weight_f32, gains, tokens, ragged_lengths, to_bf16_bits,
    bf16_bits_to_f32, round_to_bf16, hidden_input,
)
