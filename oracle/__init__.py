"""CPU fp64 oracle of the tile-filtered attention forward pass.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py``; the product path never calls it.
"""

from .attention import (
    RULES,
    QTileResult,
    RuleRun,
    bf16_to_f64,
    dense_attention,
    diagonal_first_order,
    filter_q_tile,
    lambda_from_recall,
    log_threshold_blasst,
    rule_attention,
)

__all__ = [
    "RULES",
    "QTileResult",
    "RuleRun",
    "bf16_to_f64",
    "dense_attention",
    "diagonal_first_order",
    "filter_q_tile",
    "lambda_from_recall",
    "log_threshold_blasst",
    "rule_attention",
]
