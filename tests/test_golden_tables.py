"""Pin of the work counters and the throughput metric against the paper's Table 2.

Table 2 reports a sparse method's attention TFLOPs as the kept fraction of the
dense FLOPs over its time, i.e. dense TFLOPs x speedup x (1 - sparsity): every
SPADE row satisfies it to print rounding. The oracle's counters must give that
same quantity: on an unpadded grid, kept FLOPs = (1 - block sparsity) x the
dense 4 N^2 d H, so kept-FLOP throughput follows the table's convention.
"""
import os

import numpy as np
import pytest

from oracle import spade_oracle as O

HERE = os.path.dirname(os.path.abspath(__file__))


def _rows():
    rows = []
    for line in open(os.path.join(HERE, "golden", "table2_attention_tflops.txt")):
        if line.strip() and not line.startswith("#"):
            name, dense, sparse, speedup, spars = line.split()
            rows.append((name, float(dense), float(sparse), float(speedup), float(spars) / 100))
    return rows


@pytest.mark.parametrize("row", _rows(), ids=lambda r: r[0])
def test_table2_tflops_are_kept_flops_over_time(row):
    _, dense, sparse, speedup, s = row
    # each factor is printed to 3-4 significant figures: agreement within 0.5%
    implied = dense * speedup * (1 - s)
    assert abs(implied - sparse) <= 0.005 * sparse, (implied, sparse)


@pytest.mark.parametrize("s", [0.8521, 0.8232, 0.5])
def test_kept_flops_fraction_is_one_minus_block_sparsity(s):
    g = O.Geometry(4, 8, 8, 2, 4, 4)            # divisible: every block has BS tokens
    B, H, d = 1, 3, 16
    rng = np.random.default_rng(7)
    total = B * H * g.NB * g.NB
    keep = max(1, int(round((1 - s) * total)))
    flat = np.zeros(total, bool)
    flat[rng.choice(total, keep, replace=False)] = True
    mask = flat.reshape(B, H, g.NB, g.NB)
    counts = mask.sum(-1).astype(np.int32)
    indices = np.full((B, H, g.NB, g.NB), -1, np.int32)
    for idx in np.ndindex(B, H, g.NB):
        js = np.flatnonzero(mask[idx])
        indices[idx][: js.size] = js
    kept = O.kept_flops(counts, indices, g, d)
    dense = 4.0 * g.N ** 2 * d * H * B
    assert kept == pytest.approx((1 - O.block_sparsity(counts, g.NB)) * dense, rel=1e-15)
    assert O.block_sparsity(counts, g.NB) == pytest.approx(1 - keep / total, rel=1e-15)
