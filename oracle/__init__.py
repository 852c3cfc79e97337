"""CPU oracle for the cached MAR transformer step (test infrastructure).

Plain, slow, fp64 numpy code that states what the method computes.  Only the
tests, the smoke check and the benchmark's CPU-baseline leg may import it;
the product path never does, and this package imports nothing from the
product.
"""
from .mar_oracle import (  # noqa: F401
    MarOracle,
    attention,
    block_rows,
    cfg_reuse,
    cfg_store,
    cosine_scores,
    gelu,
    guided,
    layer_norm,
    linear,
    select_least_similar,
    select_most_similar,
    storage_round,
    value_rows,
)
