"""GPU parity of head grouping and the head-wise blocking choice against the fp64 oracle.

Covers the head-list form of spade_block_reorder (bit-exact gather into a
compact group tensor and scatter back into only the listed heads),
spade_aggregation_score and spade_choose_scheme (§3.2, Eq. (3)), and the
block-shape sweep end to end (choice, per-group selection, attention), small
and at the Hunyuan-Video attention-layer shape.
"""
import sys

import numpy as np
import pytest
import torch

from gen.workloads import SWEEP_CANDIDATES, workload
from oracle import spade_oracle as O
from paper_2608_03335_amd import spade as S
from paper_2608_03335_amd.pipeline import SweepPath

from . import _parity as P
from .test_oracle_sweep import _tile_constant_field

pytestmark = pytest.mark.gpu
DEV = "cuda"
# Aggregation scores are fp64 sums of fp64 SICS on both sides.
AS_REL = 1e-10
# Candidates whose scores for a head lie this close (relative) may swap.
CHOICE_REL = 1e-9


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _geom(cfg, H=None, shape=None):
    bt, bh, bw = shape or (cfg["bt"], cfg["bh"], cfg["bw"])
    return S.geom(cfg["B"], cfg["H"] if H is None else H, cfg["d"], cfg["T"], cfg["Hs"],
                  cfg["Ws"], bt, bh, bw)


@pytest.mark.parametrize("heads", [[3, 0, 4], [2], [4, 3, 2, 1, 0], []], ids=str)
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32], ids=["bf16", "fp32"])
def test_head_subset_reorder_bit_exact(heads, dtype):
    cfg = P.small_cfg(5, 7, 9, 2, 3, 4, d=64, H=5, B=2)
    _say("head subset reorder", heads, dtype)
    g, og = _geom(cfg), P.geometry(cfg)
    Q, _, _ = P.bf16_inputs(cfg)
    x = Q.to(dtype)
    iview = torch.int16 if dtype == torch.bfloat16 else torch.int32
    n = len(heads)
    xb = torch.full((cfg["B"], max(n, 1), g.NB * g.BS, cfg["d"]), float("nan"), dtype=dtype, device=DEV)
    S.spade_block_reorder(g, x, xb, heads=heads)
    fill = torch.randn(x.shape, device=DEV).to(dtype)
    y = fill.clone()
    S.spade_block_reorder(g, xb, y, inverse=True, heads=heads)
    torch.cuda.synchronize()
    if n:
        ref = O.reorder(x.view(iview).cpu().numpy()[:, heads], og)
        assert np.array_equal(xb.view(iview).cpu().numpy()[:, :n], ref)
    else:
        assert torch.isnan(xb.float()).all()      # nothing written
    others = [h for h in range(cfg["H"]) if h not in heads]
    assert torch.equal(y[:, heads].view(iview), x[:, heads].view(iview))
    assert torch.equal(y[:, others].view(iview), fill[:, others].view(iview))


@pytest.mark.parametrize("shape", [(2, 3, 4), (1, 8, 3), (5, 7, 7)], ids=str)
def test_aggregation_score(shape):
    cfg = P.small_cfg(5, 7, 9, *shape, d=128, H=3, B=2)
    _say("aggregation score", shape)
    g, og = _geom(cfg), P.geometry(cfg)
    Q, K, _ = P.bf16_inputs(cfg)
    Qb = torch.empty((2, 3, g.NB * g.BS, 128), dtype=torch.bfloat16, device=DEV)
    Kb = torch.empty_like(Qb)
    S.spade_block_reorder(g, Q, Qb)
    S.spade_block_reorder(g, K, Kb)
    f64 = dict(dtype=torch.float64, device=DEV)
    qbar, kbar = torch.empty((2, 3, g.NB, 128), **f64), torch.empty((2, 3, g.NB, 128), **f64)
    sq, sk = torch.empty((2, 3, g.NB), **f64), torch.empty((2, 3, g.NB), **f64)
    S.spade_summarize(g, Qb, Kb, qbar, kbar, sq, sk)
    aq, ak, aqk = (torch.empty((2, 3), **f64) for _ in range(3))
    S.spade_aggregation_score(g, sq, sk, aqk, aq, ak)
    torch.cuda.synchronize()
    _, ref_q = O.aggregation_score(O.block_sics(O.reorder(P.to_np64(Q), og), og), og)
    _, ref_k = O.aggregation_score(O.block_sics(O.reorder(P.to_np64(K), og), og), og)
    np.testing.assert_allclose(aq.cpu().numpy(), ref_q, rtol=AS_REL, atol=0)
    np.testing.assert_allclose(ak.cpu().numpy(), ref_k, rtol=AS_REL, atol=0)
    assert np.array_equal(aqk.cpu().numpy(), aq.cpu().numpy() + ak.cpu().numpy())


def test_choose_scheme_table_by_hand():
    as_qk = torch.tensor([
        [[1, 5, 0, -1], [1, 5, 0, -1]],
        [[2, 4, 0, -3], [4, 6, 0, -1]],
        [[2, 4, 1, -1], [2, 4, 0, -1]],
    ], dtype=torch.float64, device=DEV)
    choice = torch.full((4,), -7, dtype=torch.int32, device=DEV)
    best = torch.empty(4, dtype=torch.float64, device=DEV)
    S.spade_choose_scheme(as_qk, choice, best)
    torch.cuda.synchronize()
    assert choice.cpu().tolist() == [1, 0, 2, 0]
    assert best.cpu().tolist() == [3.0, 5.0, 0.5, -1.0]


@pytest.mark.parametrize("C,B,H", [(1, 1, 5), (5, 1, 37), (4, 3, 300)])
def test_choose_scheme_random(C, B, H):
    rng = np.random.default_rng(C * 1000 + H)
    table = rng.standard_normal((C, B, H))
    t = torch.from_numpy(table).to(DEV)
    choice = torch.empty(H, dtype=torch.int32, device=DEV)
    best = torch.empty(H, dtype=torch.float64, device=DEV)
    S.spade_choose_scheme(t, choice, best)
    torch.cuda.synchronize()
    ch, bst = O.choose_schemes(table)
    assert np.array_equal(choice.cpu().numpy(), ch)
    np.testing.assert_allclose(best.cpu().numpy(), bst, rtol=1e-14, atol=1e-15)


def _check_choice(as_gpu, as_ref, choice_gpu):
    """GPU AS table vs the oracle's; choice exact except near ties."""
    np.testing.assert_allclose(as_gpu, as_ref, rtol=AS_REL, atol=0)
    ch_ref, _ = O.choose_schemes(as_ref)
    per_head = as_ref.mean(axis=1)
    for h in np.flatnonzero(choice_gpu != ch_ref):
        a, b = per_head[choice_gpu[h], h], per_head[ch_ref[h], h]
        assert abs(a - b) <= CHOICE_REL * abs(b), f"head {h}: GPU chose {choice_gpu[h]}, oracle {ch_ref[h]}"
    return ch_ref


def _sweep_path(cfg, cands, sparsity, raster=False):
    return SweepPath(cfg["B"], cfg["H"], cfg["d"], cfg["T"], cfg["Hs"], cfg["Ws"], cands,
                     sparsity, device=DEV, raster=raster)


@pytest.mark.parametrize("d", [64, 128])
def test_sweep_tile_aligned_heads_end_to_end(d):
    """Heads whose Q/K are constant on one candidate's tiles choose that candidate;
    groups of 1-2 heads then run and land in their own output slots."""
    grid, cands, picks = (4, 8, 12), [(2, 4, 4), (4, 2, 6), (1, 8, 3)], (2, 0, 1, 0, 1)
    _say("sweep tile aligned", d)
    rng = np.random.default_rng(d)
    Qn = np.stack([_tile_constant_field(rng, grid, cands[c], d) for c in picks])[None]
    Kn = np.stack([_tile_constant_field(rng, grid, cands[c], d) for c in picks])[None]
    Qn, Kn = Qn * 0.5, Kn * 0.5
    Vn = rng.standard_normal(Qn.shape)
    Q, K, V = (torch.from_numpy(a).to(DEV).to(torch.bfloat16) for a in (Qn, Kn, Vn))
    cfg = dict(B=1, H=len(picks), d=d, T=grid[0], Hs=grid[1], Ws=grid[2])
    p = _sweep_path(cfg, cands, 0.5)
    p.run(Q, K, V)
    torch.cuda.synchronize()
    assert p.choice.cpu().tolist() == list(picks)
    ref = O.spade_sweep_attention(P.to_np64(Q), P.to_np64(K), P.to_np64(V), grid, cands, 0.5)
    assert ref["choice"].tolist() == list(picks)
    err = float(np.max(np.abs(P.to_np64(p.O) - ref["O"])))
    _say(f"  max-abs {err:.3e}")
    assert err <= P.ATTN_MAX_ABS


@pytest.mark.parametrize("sparsity", [0.7, 0.95])
def test_sweep_small_smooth_fields(sparsity):
    """Generator inputs on a ragged grid: choice, per-group selection and output."""
    grid, cands = (5, 8, 12), [(2, 4, 4), (4, 2, 6), (1, 8, 3), (5, 3, 5)]
    cfg = P.small_cfg(*grid, 2, 4, 4, d=128, H=6)
    cfg["aniso"] = [(2.5, 1, 1), (1, 2.5, 1), (1, 1, 2.5), (1, 1, 1), (2.5, 1, 1), (1, 1, 2.5)]
    _say("sweep smooth", sparsity)
    Q, K, V = P.bf16_inputs(cfg)
    p = _sweep_path(cfg, cands, sparsity)
    P.nan_fill(p.O)
    p.run(Q, K, V)
    torch.cuda.synchronize()
    q, k, v = (P.to_np64(x) for x in (Q, K, V))
    ref = O.spade_sweep_attention(q, k, v, grid, cands, sparsity)
    # the GPU's choice must be the oracle's, or one of a near-tie (checked here)
    _check_choice(p.as_qk.cpu().numpy(), ref["as_qk"], p.choice.cpu().numpy())
    # every group, under the GPU's own choice: selection against the oracle's, and the
    # attention against the oracle run on the GPU's lists, every element, every run
    ref_O = np.full(q.shape, np.nan)
    n_ex = 0
    for c, heads in p.work_list():
        g = O.Geometry(*grid, *cands[c])
        v_ = p.group_views(c, len(heads))
        qbar = O.block_means(O.reorder(q[:, heads], g), g)
        kbar = O.block_means(O.reorder(k[:, heads], g), g)
        s = O.block_scores(qbar, kbar, P.scale_of(128))
        c_o, i_o = O.select(s, "topk", topk=O.sweep_topk(sparsity, g.NB))
        cg, ig = v_["counts"].cpu().numpy(), v_["indices"].cpu().numpy()
        n_ex += P.compare_selection(s, c_o, i_o, cg, ig, "topk")
        ro, _ = P.oracle_attention_on_lists(q[:, heads], k[:, heads], v[:, heads], g, cg, ig,
                                            P.scale_of(128))
        ref_O[:, heads] = ro
    worst = P.finite_max_abs(P.to_np64(p.O), ref_O)
    _say(f"  groups {p.work_list()} exempt rows {n_ex} max-abs {worst:.3e}")
    assert worst <= P.ATTN_MAX_ABS


def test_sweep_full_hunyuan_shape():
    """Block-shape sweep at the Hunyuan-Video layer (24 heads, 57600 tokens, 4
    candidates, 85% sparsity), in the benchmark's launch configuration. Sampled
    heads: AS table, choice and per-group selection against the oracle; sampled
    query blocks of each group's attention; the scatter into the full output."""
    cfg = workload("hunyuan_sweep")
    sparsity, cands = 0.85, list(SWEEP_CANDIDATES)
    _say("sweep full hunyuan")
    Q, K, V = P.bf16_inputs(cfg)
    p = _sweep_path(cfg, cands, sparsity)
    P.nan_fill(p.O)
    p.run(Q, K, V)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(p.O).all()), "an output row was not written"
    heads = list(range(0, cfg["H"], 4))          # every 4th head: all four field types
    q, k = (P.to_np64(x[:, heads]) for x in (Q, K))
    grid = (cfg["T"], cfg["Hs"], cfg["Ws"])
    as_ref = np.stack([O.scheme_scores(q, k, O.Geometry(*grid, *c)) for c in cands])
    choice = p.choice.cpu().numpy()
    _check_choice(p.as_qk.cpu().numpy()[:, :, heads], as_ref, choice[heads])
    _say(f"  choice {choice.tolist()}")
    v = P.to_np64(V[:, heads])
    out = P.to_np64(p.O)
    worst = 0.0
    for c, grp in p.work_list():
        g = O.Geometry(*grid, *cands[c])
        vw = p.group_views(c, len(grp))
        sample = [j for j, h in enumerate(grp) if h in heads]
        if not sample:
            continue
        loc = [heads.index(grp[j]) for j in sample]
        qb, kb, vb = (O.reorder(a[:, loc], g) for a in (q, k, v))
        s = O.block_scores(O.block_means(qb, g), O.block_means(kb, g), P.scale_of(cfg["d"]))
        c_o, i_o = O.select(s, "topk", topk=O.sweep_topk(sparsity, g.NB))
        cg = vw["counts"].cpu().numpy()[:, sample]
        ig = vw["indices"].cpu().numpy()[:, sample]
        P.compare_selection(s, c_o, i_o, cg, ig, "topk")
        rows = P.sample_rows(1, len(sample), g.NB, 6, seed=c, must=[(0, 0, 0), (0, len(sample) - 1, g.NB - 1)])
        ref, _ = O.block_sparse_attention(qb, kb, vb, cg, ig, g, P.scale_of(cfg["d"]), rows=rows)
        got = P.to_np64(vw["O"][:, sample])
        _, nv = O.block_tables(g)
        pos = O.token_position(g)
        for (b, h, i) in rows:
            sl = slice(i * g.BS, i * g.BS + nv[i])
            worst = max(worst, P.finite_max_abs(got[b, h, sl], ref[b, h, sl]))
        # the group's blocked output went to its own heads of the raster output
        for j, jj in enumerate(sample):
            assert np.array_equal(out[:, grp[jj]], got[:, j][:, pos])
    _say(f"  attention max-abs over sampled query blocks: {worst:.3e}")
    assert worst <= P.ATTN_MAX_ABS


@pytest.mark.parametrize("case", ["small_d64", "small_d128_b2", "small_pair_b2", "hunyuan"])
def test_sweep_raster_multi_equals_grouped(case):
    """One multi-scheme raster call gives every head exactly the output of its
    group's blocked path (same rows, same arithmetic, same order)."""
    if case == "hunyuan":
        cfg, cands, sp = workload("hunyuan_sweep"), SWEEP_CANDIDATES, 0.85
    elif case == "small_pair_b2":
        # three 160-slot blockings (paired-wave kernel, different grids of blocks) beside a
        # 120-slot one, two batch elements (the per-batch head ranking)
        cfg = P.small_cfg(6, 15, 16, 1, 1, 1, d=64, H=4, B=2)
        cands, sp = [(2, 5, 16), (4, 5, 8), (5, 4, 8), (3, 5, 8)], 0.6
    elif case == "small_d64":
        cfg = P.small_cfg(6, 16, 20, 1, 1, 1, d=64, H=6)
        cands, sp = [(2, 4, 4), (3, 4, 5), (2, 8, 2), (1, 16, 4)], 0.6
    else:
        cfg = P.small_cfg(5, 11, 13, 1, 1, 1, d=128, H=5, B=2)
        cands, sp = [(2, 4, 4), (3, 4, 5), (5, 3, 3)], 0.7
    _say("raster multi sweep", case)
    Q, K, V = P.bf16_inputs(cfg)
    a = _sweep_path(cfg, cands, sp).run(Q, K, V)
    pb = _sweep_path(cfg, cands, sp, raster=True)
    b = pb.run(Q, K, V)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    if case == "small_pair_b2":  # some head ran on a 160-slot blocking
        assert any(int(c) < 3 for c in pb.choice.cpu())


# ---------------- one-pass candidate evaluation (spade_candidate_sics) ----------------
def _cand_sics(geoms, Q, K):
    sq = [torch.full((g.B, g.H, g.NB), float("nan"), dtype=torch.float64, device=DEV) for g in geoms]
    sk = [torch.full_like(t, float("nan")) for t in sq]
    S.spade_candidate_sics(geoms, Q, K, sq, sk)
    torch.cuda.synchronize()
    return sq, sk


@pytest.mark.parametrize("case", ["hunyuan_like_small", "ragged_d64_b2", "single", "mixed_ragged"])
def test_candidate_sics_matches_oracle_and_per_candidate_pass(case):
    """Every candidate's SICS from the one-pass call equals the oracle's closed form
    (rtol 1e-9) and the per-candidate pass of spade_block_summarize (rtol 1e-12);
    every output element is written (NaN-poisoned before)."""
    if case == "hunyuan_like_small":
        cfg, cands = P.small_cfg(16, 45, 24, 1, 1, 1, d=128, H=2), [(2, 8, 8), (4, 4, 8), (4, 5, 8), (8, 5, 4)]
    elif case == "ragged_d64_b2":
        cfg, cands = P.small_cfg(7, 13, 11, 1, 1, 1, d=64, H=3, B=2), [(2, 4, 4), (3, 4, 5), (2, 8, 2)]
    elif case == "single":
        cfg, cands = P.small_cfg(5, 9, 10, 1, 1, 1, d=128, H=2), [(2, 3, 4)]
    else:
        cfg, cands = P.small_cfg(6, 10, 15, 1, 1, 1, d=128, H=2), [(2, 3, 6), (4, 3, 3), (1, 6, 2)]
    _say("candidate sics", case)
    Q, K, _ = P.bf16_inputs(cfg)
    geoms = [_geom(cfg, shape=c) for c in cands]
    sq, sk = _cand_sics(geoms, Q, K)
    q, k = P.to_np64(Q), P.to_np64(K)
    for c, g in enumerate(geoms):
        og = O.Geometry(cfg["T"], cfg["Hs"], cfg["Ws"], *cands[c])
        for got, X in ((sq[c], q), (sk[c], k)):
            a = got.cpu().numpy()
            assert np.all(np.isfinite(a))
            np.testing.assert_allclose(a, O.block_sics(O.reorder(X, og), og), rtol=1e-9, atol=1e-9)
        pq = torch.empty_like(sq[c])
        pk = torch.empty_like(sk[c])
        S.spade_block_summarize(g, Q, K, sics_q=pq, sics_k=pk)
        torch.cuda.synchronize()
        np.testing.assert_allclose(sq[c].cpu().numpy(), pq.cpu().numpy(), rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(sk[c].cpu().numpy(), pk.cpu().numpy(), rtol=1e-12, atol=1e-12)
    again_q, again_k = _cand_sics(geoms, Q, K)
    for c in range(len(geoms)):  # fixed summation orders: bit for bit
        assert torch.equal(again_q[c], sq[c]) and torch.equal(again_k[c], sk[c])


def test_candidate_sics_full_hunyuan_sweep():
    """The sweep's four candidates at the Hunyuan-Video layer in one pass: against the
    per-candidate pass on every block of every head, the oracle on two heads, and the
    choice the sweep path makes with either evaluation."""
    cfg = workload("hunyuan_sweep")
    _say("candidate sics full hunyuan")
    Q, K, V = P.bf16_inputs(cfg)
    geoms = [_geom(cfg, shape=c) for c in SWEEP_CANDIDATES]
    sq, sk = _cand_sics(geoms, Q, K)
    for c, g in enumerate(geoms):
        pq, pk = torch.empty_like(sq[c]), torch.empty_like(sk[c])
        S.spade_block_summarize(g, Q, K, sics_q=pq, sics_k=pk)
        torch.cuda.synchronize()
        np.testing.assert_allclose(sq[c].cpu().numpy(), pq.cpu().numpy(), rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(sk[c].cpu().numpy(), pk.cpu().numpy(), rtol=1e-12, atol=1e-12)
        og = O.Geometry(cfg["T"], cfg["Hs"], cfg["Ws"], *SWEEP_CANDIDATES[c])
        for h in (0, cfg["H"] - 1):
            ref = O.block_sics(O.reorder(P.to_np64(Q[:, h:h + 1]), og), og)
            np.testing.assert_allclose(sq[c].cpu().numpy()[:, h:h + 1], ref, rtol=1e-9, atol=1e-9)
    one = SweepPath(cfg["B"], cfg["H"], cfg["d"], cfg["T"], cfg["Hs"], cfg["Ws"], SWEEP_CANDIDATES,
                    0.85, device=DEV)
    per = SweepPath(cfg["B"], cfg["H"], cfg["d"], cfg["T"], cfg["Hs"], cfg["Ws"], SWEEP_CANDIDATES,
                    0.85, device=DEV, one_pass=False)
    one.evaluate(Q, K)
    per.evaluate(Q, K)
    torch.cuda.synchronize()
    assert one.one_pass
    np.testing.assert_allclose(one.as_qk.cpu().numpy(), per.as_qk.cpu().numpy(), rtol=1e-12, atol=0)
    _check_choice(one.as_qk.cpu().numpy(), per.as_qk.cpu().numpy(), one.choice.cpu().numpy())


def test_candidate_sics_unsupported_falls_back():
    """Candidates whose common refinement exceeds the LDS are rejected with
    SPADE_ERR_UNSUPPORTED (nothing written); the sweep path then scores them one at a
    time and still matches the oracle's Aggregation Scores."""
    cfg = P.small_cfg(7, 11, 13, 1, 1, 1, d=128, H=2)
    cands = [(1, 1, 1), (7, 5, 7)]  # 7 x 5 x 7 cells of 1 KiB of fp64 sums per region
    _say("candidate sics fallback")
    Q, K, _ = P.bf16_inputs(cfg)
    geoms = [_geom(cfg, shape=c) for c in cands]
    sq = [torch.full((g.B, g.H, g.NB), -5.0, dtype=torch.float64, device=DEV) for g in geoms]
    sk = [torch.full_like(t, -5.0) for t in sq]
    with pytest.raises(S.SpadeError) as e:
        S.spade_candidate_sics(geoms, Q, K, sq, sk)
    assert e.value.status == S.SPADE_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert all(bool((t == -5.0).all()) for t in sq + sk)
    p = SweepPath(cfg["B"], cfg["H"], cfg["d"], cfg["T"], cfg["Hs"], cfg["Ws"], cands, 0.5, device=DEV)
    p.evaluate(Q, K)
    torch.cuda.synchronize()
    assert not p.one_pass
    q, k = P.to_np64(Q), P.to_np64(K)
    ref = np.stack([O.scheme_scores(q, k, O.Geometry(cfg["T"], cfg["Hs"], cfg["Ws"], *c)) for c in cands])
    np.testing.assert_allclose(p.as_qk.cpu().numpy(), ref, rtol=AS_REL, atol=0)
