"""The oracle's pins must catch plausible mistakes.

Each case plants one mistake in the oracle (on the CPU, through monkeypatch)
and checks that at least one of the pin tests then fails.
"""
import math

import numpy as np
import pytest

from oracle import spade_oracle as O

from . import test_oracle_attention as TA
from . import test_oracle_geometry as TG
from . import test_oracle_selection as TS
from . import test_oracle_summaries as TM

G_RAGGED = O.Geometry(5, 7, 9, 2, 3, 4)


def _fails(fn, *args):
    try:
        fn(*args)
    except AssertionError:
        return True
    return False


def test_ties_broken_toward_higher_index_is_caught(monkeypatch):
    monkeypatch.setattr(O, "rank_order", lambda s: np.lexsort((-np.arange(s.shape[0]), -s)))
    assert _fails(TS.test_topk_matches_rank_counting, 8, True)


def test_mean_over_full_block_size_is_caught(monkeypatch):
    orig = O.block_tables

    def padded_counts(g):
        st, nv = orig(g)
        return st, np.full_like(nv, g.BS)
    monkeypatch.setattr(O, "block_tables", padded_counts)
    assert _fails(TM.test_means_match_direct_tile_slices, G_RAGGED)


def test_transposed_scores_are_caught(monkeypatch):
    monkeypatch.setattr(O, "block_scores",
                        lambda q, k, s: np.matmul(k, np.swapaxes(q, -1, -2)) * s)
    assert _fails(TS.test_scores_match_explicit_loops)


def test_missing_attention_scale_is_caught(monkeypatch):
    orig = O.block_sparse_attention
    monkeypatch.setattr(O, "block_sparse_attention",
                        lambda Qb, Kb, Vb, c, i, g, scale, rows=None: orig(Qb, Kb, Vb, c, i, g, 1.0, rows))
    assert _fails(TA.test_all_kept_equals_dense_attention, G_RAGGED, ("topk", dict(topk=10 ** 6)))


def test_topp_off_by_one_is_caught(monkeypatch):
    def keep_one_more(s, tau):
        NB = s.shape[0]
        if tau >= 1.0:
            return np.arange(NB)
        order = O.rank_order(s)
        cum = np.cumsum(O.row_softmax(s)[order])
        hit = np.nonzero(cum >= tau)[0]
        m = min(NB, int(hit[0]) + 2) if hit.size else NB
        return np.sort(order[:m])
    monkeypatch.setattr(O, "select_row_topp", keep_one_more)
    assert _fails(TS.test_topp_matches_bruteforce_prefix_mass, 8, False)


def test_slot_order_mistake_is_caught(monkeypatch):
    """Column-major slots inside a block (dx slowest) instead of raster."""
    def bad_tables(g):
        nT, nH, nW = g.grid
        st = np.full(g.NB * g.BS, -1, dtype=np.int64)
        nv = np.zeros(g.NB, dtype=np.int64)
        b = 0
        for tb in range(nT):
            for hb in range(nH):
                for wb in range(nW):
                    s = 0
                    for dx in range(g.bw):
                        for dy in range(g.bh):
                            for dt in range(g.bt):
                                t, y, x = tb * g.bt + dt, hb * g.bh + dy, wb * g.bw + dx
                                if t < g.T and y < g.Hs and x < g.Ws:
                                    st[b * g.BS + s] = (t * g.Hs + y) * g.Ws + x
                                    s += 1
                    nv[b] = s
                    b += 1
        return st, nv
    monkeypatch.setattr(O, "block_tables", bad_tables)
    assert _fails(TG.test_positions_match_independent_enumeration, G_RAGGED)


def test_sics_without_normalisation_is_caught(monkeypatch):
    monkeypatch.setattr(O, "_unit_rows", lambda Q: np.asarray(Q, dtype=np.float64))
    assert _fails(TM.test_sics_special_cases)


def test_softmax_without_max_shift_in_lse_is_caught(monkeypatch):
    orig = O.block_sparse_attention

    def lse_off(*a, **k):
        Ob, lse = orig(*a, **k)
        return Ob, lse + (lse != 0) * 0.5
    monkeypatch.setattr(O, "block_sparse_attention", lse_off)
    assert _fails(TA.test_matches_eq2_with_explicit_token_mask, G_RAGGED)


def test_last_maximum_wins_is_caught(monkeypatch):
    from . import test_oracle_sweep as TW

    def last_max(as_qk):
        per_head = np.asarray(as_qk).mean(axis=1)
        C = per_head.shape[0]
        choice = C - 1 - np.argmax(per_head[::-1], axis=0)
        return choice, per_head.max(axis=0)
    monkeypatch.setattr(O, "choose_schemes", last_max)
    assert _fails(TW.test_choice_table_by_hand)


def test_as_normalised_by_full_block_size_is_caught(monkeypatch):
    from . import test_oracle_sweep as TW

    def by_bs(sics, g):
        raw = sics.sum(axis=-1)
        return raw, raw / float(g.NB * g.BS ** 2)
    monkeypatch.setattr(O, "aggregation_score", by_bs)
    assert _fails(TW.test_ragged_tiles_score_one_too)


def test_group_output_in_wrong_heads_is_caught(monkeypatch):
    from . import test_oracle_sweep as TW
    orig = O.head_groups
    monkeypatch.setattr(O, "head_groups", lambda choice, C: [list(reversed(h)) for h in orig(choice, C)])
    orig_attn = O.spade_attention

    def shifted(Q, K, V, g, mode, **kw):
        r = orig_attn(Q, K, V, g, mode, **kw)
        r["O"] = np.roll(r["O"], 1, axis=1)
        return r
    monkeypatch.setattr(O, "spade_attention", shifted)
    assert _fails(TW.test_sweep_outputs_land_in_their_heads) or _fails(
        TW.test_sweep_keeping_every_block_is_dense_attention)
