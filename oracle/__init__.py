"""Plain CPU oracle for the GASLoC gossip round: test infrastructure only.

Importable by the tests, the smoke check and the benchmark's CPU-baseline leg.
The GPU library (paper_2606_11081_amd) never imports it.
"""
from .oracle import (  # noqa: F401
    PARAM_BF16,
    PARAM_NATIVE,
    Oracle,
    OracleHParams,
    TOPOLOGY_CODES,
    adamw_scalars,
    bf16_bits_to_f32,
    bounded_draws,
    csr_to_dense,
    f32_to_bf16_bits,
    lib,
    lr_schedule,
    round_state,
    shuffled_identity,
    skip_exchanges,
    splitmix64_stream,
    topology_csr,
)
