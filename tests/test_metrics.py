"""The compression-rate bookkeeping against the figures Table A1 prints."""
import math
import os

import pytest

from paper_1905_07931_amd import synth
from paper_1905_07931_amd.metrics import compression_label, compression_rate

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "table_a1_compression.txt")


def _rows():
    with open(GOLDEN) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                method, layer, nnz, total, pct, fx = line.split()
                yield method, layer, int(nnz), int(total), pct, int(fx)


def test_table_a1_rows():
    rows = list(_rows())
    assert len(rows) == 10
    for method, layer, nnz, total, pct, fx in rows:
        assert compression_label(nnz, total) == f"{pct}% ({fx}x)", (method, layer)


def test_table_a1_totals_are_the_layer_sums():
    rows = list(_rows())
    for method in ("SpC", "SpC(Retrain)"):
        layers = [r for r in rows if r[0] == method and r[1] != "total"]
        tot = [r for r in rows if r[0] == method and r[1] == "total"][0]
        assert sum(r[2] for r in layers) == tot[2] and sum(r[3] for r in layers) == tot[3]


def test_synthetic_lenet5_has_the_retrained_counts():
    # the inference workload's layers carry Table A1's SpC(Retrain) nonzeros
    assert sum(synth.LENET5_NNZ.values()) == 12217
    assert compression_label(12217, 430500) == "97.16% (35x)"


def test_edges():
    assert compression_rate(0, 10) == (1.0, math.inf)
    assert compression_rate(10, 10) == (0.0, 1.0)
    assert compression_label(0, 10) == "100.00% (infx)"
    for bad in [(-1, 10), (11, 10), (0, 0)]:
        with pytest.raises(ValueError):
            compression_rate(*bad)
