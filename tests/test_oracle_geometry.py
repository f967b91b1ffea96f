"""Pins for the oracle's blocking (paper §3.1 blocking schemes, Fig. 3) and layout restore (§3.3).

Each check compares the oracle against something other than itself: an
independent counting enumeration, the numpy reshape/transpose form that a
divisible grid reduces to, and permutation invariants.
"""
import numpy as np
import pytest

from oracle import spade_oracle as O

GEOMS = [
    O.Geometry(4, 8, 8, 2, 4, 4),       # tiny workload
    O.Geometry(5, 7, 9, 2, 3, 4),       # ragged on every axis
    O.Geometry(21, 30, 52, 3, 6, 8),    # Wan-2.1-1.3B 480p shape: Ws ragged
    O.Geometry(3, 3, 3, 4, 4, 4),       # one block larger than the grid
    O.Geometry(1, 1, 1, 1, 1, 1),       # single token
]


@pytest.mark.parametrize("g", GEOMS, ids=str)
def test_reorder_is_a_permutation_with_zero_padding(g):
    slot_token, n_valid = O.block_tables(g)
    valid = slot_token >= 0
    assert np.array_equal(np.sort(slot_token[valid]), np.arange(g.N))
    assert n_valid.sum() == g.N and (n_valid >= 1).all() and (n_valid <= g.BS).all()
    # valid slots first in every block
    for b in range(g.NB):
        blk = valid[b * g.BS:(b + 1) * g.BS]
        assert blk[: n_valid[b]].all() and not blk[n_valid[b]:].any()
    rng = np.random.default_rng(0)
    X = rng.standard_normal((1, 2, g.N, 3))
    Xb = O.reorder(X, g)
    assert Xb.shape == (1, 2, g.NB * g.BS, 3)
    assert np.all(Xb[..., ~valid, :] == 0)
    assert np.array_equal(O.inverse_reorder(Xb, g), X)  # bitwise


def _counting_positions(g):
    """Independent enumeration: block from integer division, slot by counting
    the block's tokens that precede this one in (dt, dy, dx) raster order."""
    nT, nH, nW = g.grid
    pos = np.empty(g.N, dtype=np.int64)
    coords = [(t, y, x) for t in range(g.T) for y in range(g.Hs) for x in range(g.Ws)]
    for n, (t, y, x) in enumerate(coords):
        tb, hb, wb = t // g.bt, y // g.bh, x // g.bw
        blk = (tb * nH + hb) * nW + wb
        key = (t - tb * g.bt, y - hb * g.bh, x - wb * g.bw)
        slot = sum(1 for (t2, y2, x2) in coords
                   if (t2 // g.bt, y2 // g.bh, x2 // g.bw) == (tb, hb, wb)
                   and (t2 - tb * g.bt, y2 - hb * g.bh, x2 - wb * g.bw) < key)
        pos[n] = blk * g.BS + slot
    return pos


@pytest.mark.parametrize("g", [GEOMS[0], GEOMS[1], GEOMS[3], O.Geometry(6, 5, 7, 4, 2, 3)], ids=str)
def test_positions_match_independent_enumeration(g):
    assert np.array_equal(O.token_position(g), _counting_positions(g))


# Fig. 3's example schemes (order T, H, W): spatial (1,8,8), temporal (16,1,4),
# mixed (2,4,8). On a divisible grid blocking is a plain reshape + transpose.
@pytest.mark.parametrize("blk", [(1, 8, 8), (16, 1, 4), (2, 4, 8)])
def test_paper_schemes_reduce_to_reshape_transpose(blk):
    T, Hs, Ws, d = 16, 16, 16, 5
    bt, bh, bw = blk
    g = O.Geometry(T, Hs, Ws, bt, bh, bw)
    X = np.random.default_rng(1).standard_normal((2, T * Hs * Ws, d))
    ref = (X.reshape(2, T // bt, bt, Hs // bh, bh, Ws // bw, bw, d)
            .transpose(0, 1, 3, 5, 2, 4, 6, 7)
            .reshape(2, T * Hs * Ws, d))
    assert np.array_equal(O.reorder(X, g), ref)
    assert g.NB == (T // bt) * (Hs // bh) * (Ws // bw) and g.BS == 64


def test_workload_block_counts():
    # Block grids of the attention-layer shapes used for measurement.
    assert O.Geometry(16, 45, 80, 4, 5, 8).NB == 360
    assert O.Geometry(21, 30, 52, 3, 6, 8).NB == 245
    assert O.Geometry(21, 45, 80, 3, 5, 8).NB == 630
    _, nv = O.block_tables(O.Geometry(21, 30, 52, 3, 6, 8))
    assert sorted(set(nv.tolist())) == [72, 144]  # last block column holds 4 of 8 x
