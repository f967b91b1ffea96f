"""Pins for the oracle's head-wise blocking choice (§3.2, Eq. (3)) and the block-shape sweep.

The normalised Aggregation Score is bounded by Cauchy-Schwarz (|sum of n unit
vectors|^2 <= n^2), reaches 1 exactly when every block's vectors are parallel,
and a field that is constant on the tiles of one candidate must make that
candidate win. The sweep reduces to dense attention when every block is kept.
"""
import numpy as np
import pytest

from oracle import spade_oracle as O

GRID = (4, 8, 12)
CANDS = [(2, 4, 4), (4, 2, 6), (1, 8, 3)]


def _tile_constant_field(rng, grid, shape, d, offset=3.0):
    """[N, d] field equal to one random vector (plus a common offset) on each tile."""
    g = O.Geometry(*grid, *shape)
    vals = rng.standard_normal((g.NB, d)) + offset
    nT, nH, nW = g.grid
    t, y, x = np.meshgrid(np.arange(grid[0]), np.arange(grid[1]), np.arange(grid[2]),
                          indexing="ij")
    blk = ((t // shape[0]) * nH + y // shape[1]) * nW + x // shape[2]
    return vals[blk.reshape(-1)]


def test_normalised_as_is_bounded_by_one():
    rng = np.random.default_rng(0)
    for shape in CANDS:
        g = O.Geometry(*GRID, *shape)
        X = rng.standard_normal((2, 3, g.N, 8)) + rng.standard_normal(8)
        raw, norm = O.aggregation_score(O.block_sics(O.reorder(X, g), g), g)
        assert np.all(norm > 0) and np.all(norm <= 1 + 1e-12)
        assert np.all(raw >= norm)     # the divisor sum_b n_b^2 >= 1


def test_tile_constant_field_scores_one_on_its_own_tiling():
    rng = np.random.default_rng(1)
    for shape in CANDS:
        F = _tile_constant_field(rng, GRID, shape, 8)[None, None]
        for other in CANDS:
            g = O.Geometry(*GRID, *other)
            _, norm = O.aggregation_score(O.block_sics(O.reorder(F, g), g), g)
            if other == shape:
                assert abs(norm[0, 0] - 1.0) < 1e-12
            else:
                assert norm[0, 0] < 1.0 - 1e-6


def test_ragged_tiles_score_one_too():
    """Normalising by sum n_b^2 (not NB * BS^2) keeps partial edge blocks at 1."""
    grid, shape = (5, 7, 9), (2, 3, 4)
    F = _tile_constant_field(np.random.default_rng(2), grid, shape, 4)[None, None]
    g = O.Geometry(*grid, *shape)
    raw, norm = O.aggregation_score(O.block_sics(O.reorder(F, g), g), g)
    assert abs(norm[0, 0] - 1.0) < 1e-12
    _, n_valid = O.block_tables(g)
    assert abs(raw[0, 0] - float((n_valid ** 2).sum())) < 1e-9


def test_each_head_picks_the_tiling_its_field_follows():
    rng = np.random.default_rng(3)
    d = 8
    heads = [_tile_constant_field(rng, GRID, CANDS[c], d) for c in (2, 0, 1, 0)]
    Q = np.stack(heads)[None]
    K = np.stack([_tile_constant_field(rng, GRID, CANDS[c], d) for c in (2, 0, 1, 0)])[None]
    as_qk = np.stack([O.scheme_scores(Q, K, O.Geometry(*GRID, *s)) for s in CANDS])
    choice, best = O.choose_schemes(as_qk)
    assert choice.tolist() == [2, 0, 1, 0]
    assert np.allclose(best, 2.0, atol=1e-12)       # AS(Q) = AS(K) = 1
    assert O.head_groups(choice, 3) == [[1, 3], [2], [0]]


def test_choice_table_by_hand():
    # [C=3, B=2, H=4]; head means: h0 (1, 3, 2) -> 1; h1 (5, 5, 4) tie -> 0;
    # h2 (0, 0, 0.5) -> 2; h3 (-1, -2, -1) tie of 0 and 2 -> 0
    as_qk = np.array([
        [[1, 5, 0, -1], [1, 5, 0, -1]],
        [[2, 4, 0, -3], [4, 6, 0, -1]],
        [[2, 4, 1, -1], [2, 4, 0, -1]],
    ], dtype=np.float64)
    choice, best = O.choose_schemes(as_qk)
    assert choice.tolist() == [1, 0, 2, 0]
    assert best.tolist() == [3.0, 5.0, 0.5, -1.0]
    assert O.head_groups(choice, 4) == [[1, 3], [0], [2], []]


@pytest.mark.parametrize("s,NB,k", [(0.85, 360, 54), (0.85, 480, 72), (0.70, 360, 108),
                                    (0.95, 480, 24), (0.95, 10, 1), (0.999, 10, 1), (0.0, 7, 7)])
def test_sweep_topk_values(s, NB, k):
    assert O.sweep_topk(s, NB) == k


def test_sweep_keeping_every_block_is_dense_attention():
    rng = np.random.default_rng(4)
    B, H, d = 1, 3, 8
    N = GRID[0] * GRID[1] * GRID[2]
    Q, K, V = (rng.standard_normal((B, H, N, d)) for _ in range(3))
    r = O.spade_sweep_attention(Q, K, V, GRID, CANDS, sparsity=0.0)
    ref = O.dense_attention(Q, K, V, 1.0 / np.sqrt(d))
    np.testing.assert_allclose(r["O"], ref, rtol=0, atol=1e-12)
    assert sorted(h for grp in r["groups"] for h in grp) == list(range(H))


def test_sweep_outputs_land_in_their_heads():
    """Tile-aligned heads choose different schemes; every head's output is that
    head's own single-scheme result, in its own slot."""
    rng = np.random.default_rng(5)
    d, picks = 8, (1, 0, 2)
    Q = np.stack([_tile_constant_field(rng, GRID, CANDS[c], d) for c in picks])[None]
    K = np.stack([_tile_constant_field(rng, GRID, CANDS[c], d) for c in picks])[None]
    V = rng.standard_normal(Q.shape)
    r = O.spade_sweep_attention(Q, K, V, GRID, CANDS, sparsity=0.5)
    assert r["choice"].tolist() == list(picks)
    for h, c in enumerate(picks):
        g = O.Geometry(*GRID, *CANDS[c])
        one = O.spade_attention(Q[:, h:h + 1], K[:, h:h + 1], V[:, h:h + 1], g, "topk",
                                topk=O.sweep_topk(0.5, g.NB))
        np.testing.assert_allclose(r["O"][:, h:h + 1], one["O"], rtol=0, atol=1e-13)
        kept = r["per_group"][c]["counts"]
        assert np.all(kept == O.sweep_topk(0.5, g.NB))
