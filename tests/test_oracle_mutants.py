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


# ---- full mask composition ----
from . import test_oracle_mask as TK  # noqa: E402


def test_dsa_taking_the_smaller_product_is_caught(monkeypatch):
    def dsa_min(qmax, qmin, kmax, kmin, scale):
        qt = (qmax + qmin) / 2.0
        out = np.empty(qt.shape[:-1] + (kmax.shape[-2],))
        for i in range(qt.shape[-2]):
            a = qt[..., i:i + 1, :]
            out[..., i, :] = np.minimum(a * kmax, a * kmin).sum(axis=-1)
        return out * scale
    monkeypatch.setattr(O, "dsa_scores", dsa_min)
    assert _fails(TK.test_dsa_bounds_every_key_and_is_reached_at_a_corner)


def test_dsa2_missing_a_corner_is_caught(monkeypatch):
    def three_corners(qmax, qmin, kmax, kmin, scale):
        out = np.empty(qmax.shape[:-1] + (kmax.shape[-2],))
        for i in range(qmax.shape[-2]):
            hi, lo = qmax[..., i:i + 1, :], qmin[..., i:i + 1, :]
            out[..., i, :] = np.stack([hi * kmax, hi * kmin, lo * kmax]).max(axis=0).sum(axis=-1)
        return out * scale
    monkeypatch.setattr(O, "dsa2_scores", three_corners)
    assert _fails(TK.test_dsa2_bounds_every_logit_of_the_pair)


def test_window_radius_off_by_one_is_caught(monkeypatch):
    def strict(g, w):
        if w is None or min(w) < 0:
            return np.zeros((g.NB, g.NB), dtype=bool)
        c = O.block_coords(g)
        return np.all(np.abs(c[:, None, :] - c[None, :, :]) < np.asarray(w) + 0, axis=-1)
    monkeypatch.setattr(O, "window_mask", strict)
    assert _fails(TK.test_window_row_counts_closed_form, (1, 1, 1))


def test_sink_counted_in_blocks_is_caught(monkeypatch):
    monkeypatch.setattr(O, "sink_blocks", lambda g, s: np.arange(g.NB) < s)
    assert _fails(TK.test_sink_blocks_by_token_count)


def test_intra_marking_the_most_coherent_is_caught(monkeypatch):
    orig = O.block_coherence
    monkeypatch.setattr(O, "block_coherence", lambda sics, g: -orig(sics, g))
    assert _fails(TK.test_intra_topk_table_by_hand)


def test_key_marks_broadcast_along_rows_is_caught(monkeypatch):
    orig = O.compose_mask
    monkeypatch.setattr(O, "compose_mask",
                        lambda inter, iq=None, ik=None, w=None, s=None:
                        orig(inter, iq, None, w, s) | (ik[..., :, None] if ik is not None else False))
    assert _fails(TK.test_composition_is_the_or_of_its_parts)


# ---- policy function ----
from . import test_oracle_policy as TP  # noqa: E402


def test_budgets_following_the_score_are_caught(monkeypatch):
    orig = O.policy_head_budgets
    monkeypatch.setattr(O, "policy_head_budgets",
                        lambda a, kd, NB: orig([1.0 / x for x in a], kd, NB))
    assert _fails(TP.test_budgets_fall_as_scores_rise_and_keep_the_total)


def test_warmup_rounded_down_is_caught(monkeypatch):
    def floor_warmup(step, n, task="t2v", turbo=False):
        if turbo:
            return step < 1
        return step < int(np.floor((0.30 if task == "t2v" else 0.25) * n))
    monkeypatch.setattr(O, "policy_dense", floor_warmup)
    assert _fails(TP.test_dense_warmup_steps, 50, "i2v", False, 12)


def test_tau_positively_correlated_with_the_score_is_caught(monkeypatch):
    orig = O.policy_head_tau

    def inverse(as_best, tau):  # spreads the dropped mass by 1 / AS instead of AS
        return orig([1.0 / a if a > 0 else 0.0 for a in as_best], tau)
    monkeypatch.setattr(O, "policy_head_tau", inverse)
    assert _fails(TP.test_head_tau_falls_as_scores_rise_and_keeps_the_mean)
