"""Plain CPU oracle for the pipeline-stage engine. TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package. The engine (``paper_2502_15524_amd``) never imports it,
links it or calls it, and the two share no code: the oracle is a plain,
slow, float32 (or float64) numpy transcription of the decoder's definition,
written to be checked by eye against the paper and against the pins in
``tests/test_oracle_pins.py``.

Parity status of each function is listed in its docstring; everything here is
pinned by brute force, closed forms, invariants or paper-printed sizes, except
the behaviour of the paper's trained models, which is unavailable ("parity
unpinned" for real-model numerics).
"""
from .llama import (  # noqa: F401
    rms_norm, rope_angles, apply_rope, attention_probs, attention, silu,
    swiglu, SyntheticWeights, Stage, greedy_generate, full_forward,
    argmax_lowest, param_count, image_bytes_16bit, boundary_bytes_per_token,
)
from . import kvblob  # noqa: F401
