"""CPU oracle of the speculative-sampling verification step (test infrastructure only).

Importable only from the tests, the smoke check and the benchmark's CPU
baseline; it shares no code with the library.
"""
from .spec_oracle import (  # noqa: F401
    SENTINEL,
    OracleResult,
    acceptance_ratio,
    first_rejection,
    inverse_cdf,
    logits_as_float64,
    max_norm,
    sigmoid,
    sigmoid_approximation,
    softmax,
    verify,
    verify_ragged,
)
