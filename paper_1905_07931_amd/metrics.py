"""Host-side bookkeeping figures of a compressed network.

The compression rate (Section 4.1, comparison of the training algorithms) is
the share of zero weights among all learnable weights; the layer-wise
compression tables (Table A1 and the tables after it) print it as a
percentage with two decimals beside the reduction factor total / nnz, shown
rounded down to a whole number.
"""
from __future__ import annotations

import math

__all__ = ["compression_rate", "compression_label"]


def compression_rate(nnz: int, total: int) -> tuple[float, float]:
    """(rate, factor): rate = zero weights / all weights = 1 - nnz / total, and
    factor = total / nnz (inf for an empty layer)."""
    if total <= 0 or nnz < 0 or nnz > total:
        raise ValueError("need 0 <= nnz <= total and total > 0")
    return 1.0 - nnz / total, (math.inf if nnz == 0 else total / nnz)


def compression_label(nnz: int, total: int) -> str:
    """The tables' form, e.g. '97.16% (35x)'."""
    rate, factor = compression_rate(nnz, total)
    fx = "inf" if math.isinf(factor) else str(math.floor(factor))
    return f"{100.0 * rate:.2f}% ({fx}x)"
