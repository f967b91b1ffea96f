"""Pins for the oracle's Summarizer (mean, §3.1) and SICS / Aggregation Score (§3.2, Eq. (3)-(5), Alg. 1)."""
import math

import numpy as np
import pytest

from oracle import spade_oracle as O


@pytest.mark.parametrize("g", [O.Geometry(4, 8, 8, 2, 4, 4), O.Geometry(5, 7, 9, 2, 3, 4)], ids=str)
def test_means_match_direct_tile_slices(g):
    """Block means equal the means of the 3D tile slices of the raster tensor."""
    rng = np.random.default_rng(2)
    d = 6
    X = rng.standard_normal((1, 2, g.N, d))
    got = O.block_means(O.reorder(X, g), g)
    grid = X.reshape(1, 2, g.T, g.Hs, g.Ws, d)
    nT, nH, nW = g.grid
    b = 0
    for tb in range(nT):
        for hb in range(nH):
            for wb in range(nW):
                tile = grid[:, :, tb * g.bt:(tb + 1) * g.bt, hb * g.bh:(hb + 1) * g.bh,
                            wb * g.bw:(wb + 1) * g.bw, :]
                ref = tile.reshape(1, 2, -1, d).mean(axis=2)
                np.testing.assert_allclose(got[:, :, b], ref, rtol=0, atol=1e-14)
                b += 1


def test_mean_of_constant_is_constant():
    g = O.Geometry(5, 7, 9, 2, 3, 4)
    X = np.full((1, 1, g.N, 4), 0.375)
    assert np.all(O.block_means(O.reorder(X, g), g) == 0.375)


def _rand_block(rng, n, d):
    return rng.standard_normal((n, d)) + rng.standard_normal(d)  # correlated rows


@pytest.mark.parametrize("n,d", [(1, 4), (2, 3), (7, 16), (32, 64), (45, 8)])
def test_three_sics_forms_agree(n, d):
    Q = _rand_block(np.random.default_rng(n * 100 + d), n, d)
    a, b, c = O.sics_pairwise(Q), O.sics_prefix(Q), O.sics_closed(Q)
    assert abs(a - c) <= 1e-9 * max(1.0, abs(a))
    assert abs(b - c) <= 1e-9 * max(1.0, abs(a))
    assert -1e-12 <= c <= n * n + 1e-9


def test_sics_special_cases():
    rng = np.random.default_rng(3)
    v = rng.standard_normal(8)
    par = np.outer(rng.uniform(0.5, 2.0, 10), v)          # parallel rows -> n^2
    assert math.isclose(O.sics_closed(par), 100.0, rel_tol=1e-12)
    pm = np.stack([v, -2 * v, 3 * v, -0.5 * v])             # +/- pairs cancel -> 0
    assert abs(O.sics_closed(pm)) < 1e-12 and abs(O.sics_prefix(pm)) < 1e-12
    orth = np.linalg.qr(rng.standard_normal((8, 8)))[0][:5] * rng.uniform(0.1, 9, (5, 1))
    assert math.isclose(O.sics_pairwise(orth), 5.0, rel_tol=1e-12)  # orthogonal -> n
    assert math.isclose(O.sics_prefix(orth), 5.0, rel_tol=1e-12)


def test_sics_is_invariant_to_positive_row_scaling():
    rng = np.random.default_rng(4)
    Q = _rand_block(rng, 12, 10)
    s = rng.uniform(0.01, 100, (12, 1))
    assert math.isclose(O.sics_closed(Q), O.sics_closed(Q * s), rel_tol=1e-12)


def test_block_sics_and_aggregation_score():
    g = O.Geometry(4, 8, 8, 2, 4, 4)
    rng = np.random.default_rng(5)
    X = rng.standard_normal((1, 2, g.N, 16))
    Xb = O.reorder(X, g)
    s1 = O.block_sics(Xb, g, "closed")
    s2 = O.block_sics(Xb, g, "pairwise")
    np.testing.assert_allclose(s1, s2, rtol=1e-9)
    raw, norm = O.aggregation_score(s1, g)
    np.testing.assert_allclose(raw, s1.sum(-1), rtol=0)
    np.testing.assert_allclose(norm, raw / (g.NB * g.BS ** 2), rtol=1e-15)
    # a perfectly coherent head (every token the same direction) scores 1
    Xc = np.broadcast_to(rng.standard_normal(16), (1, 1, g.N, 16)) * rng.uniform(1, 2, (1, 1, g.N, 1))
    _, nc = O.aggregation_score(O.block_sics(O.reorder(Xc, g), g), g)
    assert math.isclose(float(nc[0, 0]), 1.0, rel_tol=1e-12)
