"""Pins for the oracle's full mask composition (§3.1 vDiT-SSR, §3.3).

The max/min Summarizer is checked against direct slices of the token grid.
The DSA estimators are pinned to what they are built to be: DSA is the largest
<q~, k> over the box spanned by the key block (a bound every key of the block
respects, reached at a corner of the box), DSA2 bounds every logit of the block
pair, and both reduce to the exact logit for one-token blocks. The intra filter,
the window and the sink are checked against closed forms and hand tables, and
the composition against its OR semantics and the dense limit.
"""
import itertools

import numpy as np
import pytest

from oracle import spade_oracle as O

G_RAGGED = O.Geometry(5, 7, 9, 2, 3, 4)


def _qk(g, d=6, B=1, H=2, seed=0, offset=0.0):
    rng = np.random.default_rng(seed)
    Q = rng.standard_normal((B, H, g.N, d)) + offset
    K = rng.standard_normal((B, H, g.N, d)) - offset
    return Q, K


def _tile_slices(g):
    """(block index, (t0, t1), (y0, y1), (x0, x1)) of every block, T-major."""
    nT, nH, nW = g.grid
    b = 0
    for tb in range(nT):
        for hb in range(nH):
            for wb in range(nW):
                yield (b, (tb * g.bt, min((tb + 1) * g.bt, g.T)),
                       (hb * g.bh, min((hb + 1) * g.bh, g.Hs)),
                       (wb * g.bw, min((wb + 1) * g.bw, g.Ws)))
                b += 1


@pytest.mark.parametrize("g", [G_RAGGED, O.Geometry(4, 8, 8, 2, 4, 4)])
def test_maxmin_match_direct_tile_slices(g):
    X, _ = _qk(g, d=5, H=3)
    mx, mn = O.block_maxmin(O.reorder(X, g), g)
    grid = X.reshape(X.shape[0], X.shape[1], g.T, g.Hs, g.Ws, X.shape[-1])
    for b, (t0, t1), (y0, y1), (x0, x1) in _tile_slices(g):
        tile = grid[:, :, t0:t1, y0:y1, x0:x1, :]
        assert np.array_equal(mx[:, :, b], tile.max(axis=(2, 3, 4)))
        assert np.array_equal(mn[:, :, b], tile.min(axis=(2, 3, 4)))


def _block_rows(X, g):
    """Per block, its real token rows [.., n_b, d] (via the tile slices)."""
    grid = X.reshape(X.shape[0], X.shape[1], g.T, g.Hs, g.Ws, X.shape[-1])
    out = {}
    for b, (t0, t1), (y0, y1), (x0, x1) in _tile_slices(g):
        tile = grid[:, :, t0:t1, y0:y1, x0:x1, :]
        out[b] = tile.reshape(X.shape[0], X.shape[1], -1, X.shape[-1])
    return out


def test_dsa_bounds_every_key_and_is_reached_at_a_corner():
    g = G_RAGGED
    Q, K = _qk(g, seed=1)
    scale = 0.37
    (qmax, qmin), (kmax, kmin) = O.block_maxmin(O.reorder(Q, g), g), O.block_maxmin(O.reorder(K, g), g)
    s = O.dsa_scores(qmax, qmin, kmax, kmin, scale)
    krows = _block_rows(K, g)
    qt = (qmax + qmin) / 2
    for h in range(Q.shape[1]):
        for i in range(g.NB):
            for j in range(g.NB):
                a = qt[0, h, i]
                true_max = (krows[j][0, h] @ a).max() * scale
                assert s[0, h, i, j] >= true_max - 1e-12
                corner = np.where(a >= 0, kmax[0, h, j], kmin[0, h, j])
                assert abs(s[0, h, i, j] - (corner @ a) * scale) < 1e-12


def test_dsa_is_centre_plus_radius_contraction():
    """max(a x, a y) = a (x + y)/2 + |a| |x - y|/2 channel by channel, so DSA is
    <q~, k_c> + <|q~|, k_r> with the key box's centre and half width."""
    g = G_RAGGED
    Q, K = _qk(g, seed=2)
    (qmax, qmin), (kmax, kmin) = O.block_maxmin(O.reorder(Q, g), g), O.block_maxmin(O.reorder(K, g), g)
    qt = (qmax + qmin) / 2
    kc, kr = (kmax + kmin) / 2, (kmax - kmin) / 2
    ref = (qt @ np.swapaxes(kc, -1, -2) + np.abs(qt) @ np.swapaxes(kr, -1, -2)) * 0.5
    np.testing.assert_allclose(O.dsa_scores(qmax, qmin, kmax, kmin, 0.5), ref, rtol=0, atol=1e-12)


def test_dsa2_bounds_every_logit_of_the_pair():
    g = G_RAGGED
    Q, K = _qk(g, seed=3, offset=0.4)
    scale = 0.25
    (qmax, qmin), (kmax, kmin) = O.block_maxmin(O.reorder(Q, g), g), O.block_maxmin(O.reorder(K, g), g)
    s2 = O.dsa2_scores(qmax, qmin, kmax, kmin, scale)
    s1 = O.dsa_scores(qmax, qmin, kmax, kmin, scale)
    qrows, krows = _block_rows(Q, g), _block_rows(K, g)
    for h in range(Q.shape[1]):
        for i in range(g.NB):
            for j in range(g.NB):
                true_max = (qrows[i][0, h] @ krows[j][0, h].T).max() * scale
                assert s2[0, h, i, j] >= true_max - 1e-12
                assert s2[0, h, i, j] >= s1[0, h, i, j] - 1e-12   # q~ lies in the query box


def test_one_token_blocks_give_exact_logits():
    g = O.Geometry(2, 3, 4, 1, 1, 1)
    Q, K = _qk(g, seed=4)
    Qb, Kb = O.reorder(Q, g), O.reorder(K, g)
    (qmax, qmin), (kmax, kmin) = O.block_maxmin(Qb, g), O.block_maxmin(Kb, g)
    exact = (Q @ np.swapaxes(K, -1, -2)) * 0.3
    for est in (O.dsa_scores, O.dsa2_scores):
        np.testing.assert_allclose(est(qmax, qmin, kmax, kmin, 0.3), exact, rtol=0, atol=1e-12)
    mean = O.block_scores(O.block_means(Qb, g), O.block_means(Kb, g), 0.3)
    np.testing.assert_allclose(mean, exact, rtol=0, atol=1e-12)


def test_coherence_range_and_parallel_blocks():
    g = G_RAGGED
    Q, _ = _qk(g, seed=5)
    c = O.block_coherence(O.block_sics(O.reorder(Q, g), g), g)
    _, n_valid = O.block_tables(g)
    assert np.all(c <= 1 + 1e-12) and np.all(c >= 0)
    # every block's rows parallel (one direction per block, any positive lengths)
    rng = np.random.default_rng(6)
    dirs = rng.standard_normal((g.NB, 6))
    slot_token, _ = O.block_tables(g)
    P = np.zeros((1, 1, g.N, 6))
    for p, t in enumerate(slot_token):
        if t >= 0:
            P[0, 0, t] = dirs[p // g.BS] * rng.uniform(0.5, 2.0)
    c1 = O.block_coherence(O.block_sics(O.reorder(P, g), g), g)
    np.testing.assert_allclose(c1, 1.0, rtol=0, atol=1e-12)


def test_intra_threshold_marks_exactly_the_noisy_blocks():
    g = O.Geometry(4, 8, 8, 2, 4, 4)
    rng = np.random.default_rng(7)
    d = 16
    slot_token, _ = O.block_tables(g)
    noisy = {1, 5}
    X = np.zeros((1, 1, g.N, d))
    base = rng.standard_normal((g.NB, d))
    for p, t in enumerate(slot_token):
        b = p // g.BS
        X[0, 0, t] = rng.standard_normal(d) if b in noisy else base[b] + 0.01 * rng.standard_normal(d)
    sics = O.block_sics(O.reorder(X, g), g)
    marks = O.intra_marks(sics, g, "threshold", theta=0.5)
    assert set(np.nonzero(marks[0, 0])[0].tolist()) == noisy


def test_intra_topk_table_by_hand():
    g = O.Geometry(1, 2, 4, 1, 1, 1)  # 8 one-token blocks: n_b = 1, coherence = SICS
    sics = np.array([[[0.9, 0.2, 0.5, 0.2, 1.0, 0.1, 0.7, 0.5]]])
    m = O.intra_marks(sics, g, "topk", k=3)
    assert np.nonzero(m[0, 0])[0].tolist() == [1, 3, 5]           # 0.1, then the 0.2 tie
    m = O.intra_marks(sics, g, "topk", k=4)
    assert np.nonzero(m[0, 0])[0].tolist() == [1, 2, 3, 5]        # 0.5 tie: lower index 2
    assert O.intra_marks(sics, g, "topk", k=100)[0, 0].all()
    assert not O.intra_marks(sics, g, "topk", k=0)[0, 0].any()
    assert np.nonzero(O.intra_marks(sics, g, "threshold", theta=0.5)[0, 0])[0].tolist() == [1, 3, 5]


@pytest.mark.parametrize("w", [(0, 0, 0), (1, 1, 1), (0, 1, 2), (2, 0, 1), (5, 5, 5)])
def test_window_row_counts_closed_form(w):
    g = G_RAGGED
    m = O.window_mask(g, w)
    nT, nH, nW = g.grid
    for b, (tb, hb, wb) in enumerate(itertools.product(range(nT), range(nH), range(nW))):
        n = 1
        for c, r, size in ((tb, w[0], nT), (hb, w[1], nH), (wb, w[2], nW)):
            n *= min(c + r, size - 1) - max(c - r, 0) + 1
        assert m[b].sum() == n
    assert np.array_equal(m, m.T)
    if w == (0, 0, 0):
        assert np.array_equal(m, np.eye(g.NB, dtype=bool))
    assert not O.window_mask(g, (-1, 2, 2)).any()


def test_sink_blocks_by_token_count():
    g = G_RAGGED                      # grid 5x7x9, blocks 2x3x4 -> block grid 3x3x3
    nT, nH, nW = g.grid
    coords = O.block_coords(g)
    assert not O.sink_blocks(g, 0).any()
    assert np.nonzero(O.sink_blocks(g, 1))[0].tolist() == [0]
    assert np.nonzero(O.sink_blocks(g, 5))[0].tolist() == [0, 1]     # x = 0..4 spans wb 0, 1
    row0 = O.sink_blocks(g, g.Ws)     # first row of frame 0: every wb of (tb, hb) = (0, 0)
    assert np.array_equal(row0, (coords[:, 0] == 0) & (coords[:, 1] == 0))
    frame0 = O.sink_blocks(g, g.Hs * g.Ws)
    assert np.array_equal(frame0, coords[:, 0] == 0)
    assert O.sink_blocks(g, g.N).all()


def test_composition_is_the_or_of_its_parts():
    g = G_RAGGED
    Q, K = _qk(g, seed=8, offset=0.3)
    base = O.MaskSpec(estimator="dsa", mode="topk", topk=3)
    r0 = O.composed_selection(Q, K, g, base)
    assert np.array_equal(r0["counts"], r0["inter_counts"])        # nothing else switched on
    spec = O.MaskSpec(estimator="dsa", mode="topk", topk=3, intra="topk", intra_topk=2,
                      window=(0, 1, 0), sink=10)
    r = O.composed_selection(Q, K, g, spec)
    inter = O.block_mask(r["inter_counts"], r["inter_indices"])
    win = O.window_mask(g, (0, 1, 0))
    snk = O.sink_blocks(g, 10)
    m = r["mask"]
    assert np.array_equal(inter, O.block_mask(r0["counts"], r0["indices"]))
    for (b, h, i, j) in np.ndindex(*m.shape):
        want = (inter[b, h, i, j] or r["intra_q"][b, h, i] or r["intra_k"][b, h, j]
                or win[i, j] or snk[j])
        assert m[b, h, i, j] == want
    assert np.array_equal(O.block_mask(r["counts"], r["indices"]), m)
    assert np.all(r["intra_q"].sum(-1) == 2) and np.all(r["intra_k"].sum(-1) == 2)


def test_window_covering_the_grid_gives_dense_attention():
    g = G_RAGGED
    rng = np.random.default_rng(9)
    Q, K, V = (rng.standard_normal((1, 2, g.N, 8)) for _ in range(3))
    spec = O.MaskSpec(estimator="dsa2", mode="topk", topk=1, window=(9, 9, 9))
    r = O.spade_attention_composed(Q, K, V, g, spec)
    np.testing.assert_allclose(r["O"], O.dense_attention(Q, K, V, 1 / np.sqrt(8)), rtol=0, atol=1e-12)


def test_per_head_budgets():
    g = G_RAGGED
    Q, K = _qk(g, seed=10, H=3)
    same = O.composed_selection(Q, K, g, O.MaskSpec(mode="topk", topk=4))
    per = O.composed_selection(Q, K, g, O.MaskSpec(mode="topk", topk=99, topk_per_head=(4, 4, 4)))
    assert np.array_equal(same["counts"], per["counts"])
    assert np.array_equal(same["indices"], per["indices"])
    r = O.composed_selection(Q, K, g, O.MaskSpec(mode="topp", tau=0.5, tau_per_head=(1.0, 0.5, 0.2)))
    assert np.all(r["counts"][:, 0] == g.NB)                     # tau = 1 keeps every block
    ref = O.composed_selection(Q, K, g, O.MaskSpec(mode="topp", tau=0.2))
    assert np.array_equal(r["counts"][:, 2], ref["counts"][:, 2])
    k_heads = O.composed_selection(Q, K, g, O.MaskSpec(mode="topk", topk_per_head=(1, 5, 27)))
    assert np.all(k_heads["counts"][:, 0] == 1) and np.all(k_heads["counts"][:, 1] == 5)
    assert np.all(k_heads["counts"][:, 2] == g.NB)
