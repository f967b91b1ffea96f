"""Pins for the oracle's inter-block estimator and Top-K / Top-P index search (§3.1, §3.3).

Brute force that does not sort (rank by counting, exact sums via math.fsum),
plus the selection invariants and a constructed case with a known answer.
"""
import math

import numpy as np
import pytest

from oracle import spade_oracle as O


def test_scores_match_explicit_loops():
    rng = np.random.default_rng(6)
    qbar, kbar = rng.standard_normal((2, 5, 7)), rng.standard_normal((2, 6, 7))
    s = O.block_scores(qbar, kbar, 0.25)
    for h in range(2):
        for i in range(5):
            for j in range(6):
                ref = math.fsum(qbar[h, i, c] * kbar[h, j, c] for c in range(7)) * 0.25
                assert abs(s[h, i, j] - ref) <= 1e-14 * max(1.0, abs(ref))


def _rank(s, j):
    """Position of block j in (score desc, index asc) order, by counting."""
    return sum(1 for l in range(len(s)) if s[l] > s[j] or (s[l] == s[j] and l < j))


def _rows(rng, n_rows, NB, ties=False):
    for _ in range(n_rows):
        s = rng.standard_normal(NB) * rng.uniform(0.1, 5)
        if ties:
            s = np.round(s, 0)  # many exact ties
        yield s


@pytest.mark.parametrize("ties", [False, True])
@pytest.mark.parametrize("NB", [1, 2, 8, 37])
def test_topk_matches_rank_counting(NB, ties):
    rng = np.random.default_rng(NB + 10 * ties)
    for s in _rows(rng, 20, NB, ties):
        for k in {1, 3, NB, NB + 5}:
            kept = O.select_row_topk(s, k)
            ref = sorted(j for j in range(NB) if _rank(s, j) < k)
            assert kept.tolist() == ref
            assert kept.size == min(k, NB)


@pytest.mark.parametrize("ties", [False, True])
@pytest.mark.parametrize("NB", [1, 2, 8, 37])
def test_topp_matches_bruteforce_prefix_mass(NB, ties):
    rng = np.random.default_rng(100 + NB + ties)
    for s in _rows(rng, 20, NB, ties):
        e = [math.exp(x - max(s)) for x in s]
        z = math.fsum(e)
        p = [x / z for x in e]
        ranked = sorted(range(NB), key=lambda j: _rank(s, j))
        for tau in (0.05, 0.5, 0.9, 0.999):
            masses = [math.fsum(p[j] for j in ranked[:m]) for m in range(1, NB + 1)]
            m_ref = next((m for m, v in enumerate(masses, 1) if v >= tau), NB)
            if any(abs(v - tau) < 1e-12 for v in masses):
                continue  # rounding-order band: not decidable against fsum
            kept = O.select_row_topp(s, tau)
            assert kept.tolist() == sorted(ranked[:m_ref])
            # invariants: mass reaches tau, and the prefix is the shortest one
            assert math.fsum(p[j] for j in kept) >= tau or kept.size == NB
            if kept.size > 1:
                assert masses[kept.size - 2] < tau


def test_topp_edge_values():
    s = np.array([0.3, 2.0, -1.0, 2.0, 0.0])
    assert O.select_row_topp(s, 1.0).tolist() == [0, 1, 2, 3, 4]  # tau = 1 keeps all
    assert O.select_row_topp(s, 1e-9).tolist() == [1]            # lowest index of the tied max
    flat = np.zeros(6)
    # equal scores: mass 1/6 each, ranked by index; 0.5 needs 3 blocks
    assert O.select_row_topp(flat, 0.5).tolist() == [0, 1, 2]
    assert O.select_row_topk(flat, 2).tolist() == [0, 1]


def test_orthogonal_block_means_select_the_diagonal():
    """kbar_j parallel to qbar_j and blocks mutually orthogonal -> top-1 is j = i."""
    rng = np.random.default_rng(7)
    NB, d = 6, 8
    basis = np.linalg.qr(rng.standard_normal((d, d)))[0][:NB]
    qbar = basis * rng.uniform(1, 2, (NB, 1))
    kbar = basis * rng.uniform(1, 2, (NB, 1))
    s = O.block_scores(qbar[None], kbar[None], 1 / math.sqrt(d))
    counts, idx = O.select(s, "topk", topk=1)
    assert counts.tolist() == [[1] * NB]
    assert idx[0, :, 0].tolist() == list(range(NB))
    assert (idx[0, :, 1:] == -1).all()


def test_select_layout_and_sparsity():
    rng = np.random.default_rng(8)
    s = rng.standard_normal((2, 3, 5, 5))
    counts, idx = O.select(s, "topp", tau=0.7)
    for c, row in zip(counts.ravel(), idx.reshape(-1, 5)):
        assert 1 <= c <= 5
        assert list(row[:c]) == sorted(row[:c]) and (row[c:] == -1).all()
    mask = O.block_mask(counts, idx)
    assert mask.sum() == counts.sum()
    assert math.isclose(O.block_sparsity(counts, 5), 1 - counts.sum() / (2 * 3 * 5 * 5))
