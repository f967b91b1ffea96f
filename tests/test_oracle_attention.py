"""Pins for the oracle's attention: Eq. (1) dense and Eq. (2) block-sparse (§2.2), whole path (§3.3)."""
import math

import numpy as np
import pytest
from scipy.special import logsumexp

from oracle import spade_oracle as O

GEOMS = [O.Geometry(4, 8, 8, 2, 4, 4), O.Geometry(5, 7, 9, 2, 3, 4)]


def _qkv(g, d=16, H=2, seed=0):
    rng = np.random.default_rng(seed)
    return [rng.standard_normal((1, H, g.N, d)) for _ in range(3)]


@pytest.mark.parametrize("g", GEOMS, ids=str)
@pytest.mark.parametrize("rule", [("topk", dict(topk=10 ** 6)), ("topp", dict(tau=1.0))])
def test_all_kept_equals_dense_attention(g, rule):
    """Keeping every block pair makes Eq. (2) equal Eq. (1)."""
    Q, K, V = _qkv(g)
    out = O.spade_attention(Q, K, V, g, rule[0], **rule[1])
    assert (out["counts"] == g.NB).all()
    ref = O.dense_attention(Q, K, V, 1 / math.sqrt(Q.shape[-1]))
    np.testing.assert_allclose(out["O"], ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("g", GEOMS, ids=str)
def test_diagonal_selection_equals_per_block_dense(g):
    Q, K, V = _qkv(g, seed=1)
    Qb, Kb, Vb = (O.reorder(a, g) for a in (Q, K, V))
    NB = g.NB
    counts = np.ones((1, 2, NB), np.int32)
    idx = np.full((1, 2, NB, NB), -1, np.int32)
    idx[..., 0] = np.arange(NB)
    Ob, _ = O.block_sparse_attention(Qb, Kb, Vb, counts, idx, g, 0.25)
    _, nv = O.block_tables(g)
    for i in range(NB):
        sl = slice(i * g.BS, i * g.BS + nv[i])
        ref = O.dense_attention(Qb[:, :, sl], Kb[:, :, sl], Vb[:, :, sl], 0.25)
        np.testing.assert_allclose(Ob[:, :, sl], ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("g", GEOMS, ids=str)
def test_matches_eq2_with_explicit_token_mask(g):
    """Eq. (2) in raster order with an explicit N x N additive mask M."""
    Q, K, V = _qkv(g, seed=2)
    out = O.spade_attention(Q, K, V, g, "topk", topk=3)
    scale = 1 / math.sqrt(Q.shape[-1])
    mask = O.block_mask(out["counts"], out["indices"])         # [1, H, NB, NB]
    pos = O.token_position(g)
    blk = pos // g.BS                                          # block of each raster token
    for h in range(2):
        M = np.where(mask[0, h][blk[:, None], blk[None, :]], 0.0, -np.inf)
        logits = Q[0, h] @ K[0, h].T * scale + M
        w = np.exp(logits - logits.max(1, keepdims=True))
        ref = (w / w.sum(1, keepdims=True)) @ V[0, h]
        np.testing.assert_allclose(out["O"][0, h], ref, rtol=0, atol=1e-12)
        # lse against scipy's logsumexp of the masked logits
        lse_raster = O.inverse_reorder(out["lse"][..., None], g)[0, h, :, 0]
        np.testing.assert_allclose(lse_raster, logsumexp(Q[0, h] @ K[0, h].T * scale + M, axis=1),
                                   rtol=0, atol=1e-12)


def test_softmax_weights_sum_to_one():
    """With V = 1 every output equals 1 (weights sum to one), whatever the mask."""
    g = GEOMS[1]
    Q, K, _ = _qkv(g, seed=3)
    out = O.spade_attention(Q, K, np.ones_like(Q), g, "topp", tau=0.6)
    np.testing.assert_allclose(out["O"], 1.0, rtol=0, atol=1e-12)


def test_padding_slots_of_output_are_zero_and_flops_count_valid_tokens():
    g = GEOMS[1]
    Q, K, V = _qkv(g, seed=4)
    out = O.spade_attention(Q, K, V, g, "topk", topk=2)
    slot_token, nv = O.block_tables(g)
    assert np.all(out["Ob"][..., slot_token < 0, :] == 0)
    ref = 0
    for h in range(2):
        for i in range(g.NB):
            for j in out["indices"][0, h, i, : out["counts"][0, h, i]]:
                ref += 4 * nv[i] * nv[j] * Q.shape[-1]
    assert O.kept_flops(out["counts"], out["indices"], g, Q.shape[-1]) == ref
