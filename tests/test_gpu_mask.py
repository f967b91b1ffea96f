"""GPU parity of the full mask composition: spade_block_minmax and
spade_compose_select against the oracle (max/min Summarizer, DSA/DSA2
estimators, intra-block filter, local window, attention sink, per-head budgets).

Extremes are exact, so they are compared bit for bit. The composed lists are
checked in two parts: every block the oracle's intra/window/sink parts keep
must be kept, and outside those blocks the GPU's choice must be the oracle's
inter Top-K/Top-P selection, with the usual exemption for scores within 1e-6
relative of the row's cut. Intra thresholds are placed between the oracle's
coherence values, far from any of them, so the filter's decisions are exact.
"""
import sys

import numpy as np
import pytest
import torch

from oracle import spade_oracle as O
from paper_2608_03335_amd import spade as S
from paper_2608_03335_amd.pipeline import Scheme

from . import _parity as P
from .test_gpu_parity import _case, _geom, _path

pytestmark = pytest.mark.gpu
DEV = "cuda"
CASES = ["tiny", "ragged_d64", "ragged_d128", "bs144_tail", "w4_ragged", "one_block", "one_token"]


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _nan(shape, dtype=torch.float64):
    return torch.full(shape, float("nan"), dtype=dtype, device=DEV)


@pytest.mark.parametrize("name", CASES)
def test_minmax_exact_and_sics_equal_block_summarize(name):
    cfg = _case(name)
    _say("block_minmax", name)
    g, og = _geom(cfg), P.geometry(cfg)
    B, H, d = cfg["B"], cfg["H"], cfg["d"]
    Q, K, _ = P.bf16_inputs(cfg)
    ext = [_nan((B, H, g.NB, d)) for _ in range(4)]
    sq, sk, sq2, sk2 = (_nan((B, H, g.NB)) for _ in range(4))
    S.spade_block_minmax(g, Q, K, *ext, sq, sk)
    S.spade_block_summarize(g, Q, K, sics_q=sq2, sics_k=sk2)
    torch.cuda.synchronize()
    (qmax, qmin), (kmax, kmin) = (O.block_maxmin(O.reorder(P.to_np64(X), og), og) for X in (Q, K))
    for got, ref in zip(ext, (qmax, qmin, kmax, kmin)):
        assert np.array_equal(got.cpu().numpy(), ref)
    assert torch.equal(sq, sq2) and torch.equal(sk, sk2)


def test_minmax_head_list_matches_full_call():
    cfg = P.small_cfg(6, 11, 13, 3, 4, 5, d=128, H=3)
    _say("block_minmax head list")
    g = _geom(cfg)
    B, H, d = cfg["B"], 3, cfg["d"]
    Q, K, _ = P.bf16_inputs(cfg)
    full = [_nan((B, H, g.NB, d)) for _ in range(4)]
    S.spade_block_minmax(g, Q, K, *full)
    heads = (2, 0)
    part = [_nan((B, 2, g.NB, d)) for _ in range(4)]
    S.spade_block_minmax(g, Q, K, *part, heads=heads)
    torch.cuda.synchronize()
    for f, p in zip(full, part):
        assert torch.equal(p, f[:, list(heads)])


def _theta_between(c, q):
    """A threshold between two neighbouring coherence values near quantile q,
    at least 1e-9 away from every value."""
    v = np.unique(np.round(c.reshape(-1), 15))
    if v.size < 2:                      # one value (e.g. one-token blocks): mark nothing
        return float(0.5 * v[0])
    k = int(np.clip(np.floor(q * (v.size - 1)), 0, v.size - 2))
    gaps = np.diff(v)
    while gaps[k] < 1e-8 and k + 1 < gaps.size:
        k += 1
    theta = 0.5 * (v[k] + v[k + 1])
    assert np.min(np.abs(c - theta)) > 1e-9
    return float(theta)


def _schemes(cfg, Q, K):
    og = P.geometry(cfg)
    H, NB, Ws = cfg["H"], og.NB, cfg["Ws"]
    sq = O.block_sics(O.reorder(P.to_np64(Q), og), og)
    sk = O.block_sics(O.reorder(P.to_np64(K), og), og)
    coh = np.concatenate([O.block_coherence(sq, og).ravel(), O.block_coherence(sk, og).ravel()])
    theta = _theta_between(coh, 0.25)
    kin = max(1, NB // 4)
    return {
        "mean_plain": Scheme("mean", "topk", topk=3),
        "dsa_topk_intra_window_sink": Scheme("dsa", "topk", topk=2, intra="threshold",
                                             intra_theta=theta, window=(0, 1, 1), sink=Ws + 3),
        "dsa2_topp_intra_topk": Scheme("dsa2", "topp", tau=0.7, intra="topk", intra_topk=kin),
        "dsa_topk_per_head": Scheme("dsa", "topk", topk_per_head=tuple((3 * h) % NB + 1
                                                                      for h in range(H))),
        "mean_topp_per_head_window": Scheme("mean", "topp", tau_per_head=tuple(
            (1.0, 0.5, 0.3)[h % 3] for h in range(H)), window=(1, 0, 0)),
    }


def _oracle_spec(s: Scheme) -> O.MaskSpec:
    return O.MaskSpec(estimator=s.estimator, mode=s.mode, topk=s.topk, tau=s.tau,
                      topk_per_head=s.topk_per_head, tau_per_head=s.tau_per_head, intra=s.intra,
                      intra_theta=s.intra_theta, intra_topk=s.intra_topk,
                      window=s.window if min(s.window) >= 0 else None, sink=s.sink)


def _check_composed(cfg, scheme, ref, counts, indices):
    """Composed GPU lists against the oracle (see the module docstring)."""
    og = P.geometry(cfg)
    c_g, i_g = counts.cpu().numpy(), indices.cpu().numpy()
    NB = og.NB
    # the GPU lists: ascending, consistent with counts
    for idx in np.ndindex(*c_g.shape):
        row = i_g[idx][: c_g[idx]]
        assert np.all(np.diff(row) > 0) and (row.size == 0 or (row[0] >= 0 and row[-1] < NB))
    m_g = O.block_mask(c_g, np.where(i_g < 0, 0, i_g))
    win = O.window_mask(og, scheme.window) if min(scheme.window) >= 0 else None
    snk = O.sink_blocks(og, scheme.sink) if scheme.sink > 0 else None
    extra = O.compose_mask(np.zeros_like(m_g), ref["intra_q"], ref["intra_k"], win, snk)
    assert np.all(m_g[extra]), "a block the intra filter, window or sink keeps is missing"
    inter_o = O.block_mask(ref["inter_counts"], ref["inter_indices"])
    view = (m_g & ~extra) | (inter_o & extra)
    c_v, i_v = O.lists_from_mask(view)
    n_ex = 0
    for h in range(cfg["H"]):
        tau = scheme.tau_per_head[h] if scheme.tau_per_head is not None else scheme.tau
        sl = (slice(None), slice(h, h + 1))
        n_ex += P.compare_selection(ref["scores"][sl], ref["inter_counts"][sl],
                                    ref["inter_indices"][sl], c_v[sl], i_v[sl], scheme.mode, tau)
    return n_ex


@pytest.mark.parametrize("which", ["mean_plain", "dsa_topk_intra_window_sink", "dsa2_topp_intra_topk",
                                   "dsa_topk_per_head", "mean_topp_per_head_window"])
@pytest.mark.parametrize("name", CASES)
def test_compose_select_matches_oracle(name, which):
    cfg = _case(name)
    Q, K, V = P.bf16_inputs(cfg)
    scheme = _schemes(cfg, Q, K)[which]
    _say("compose_select", name, which)
    p = _path(cfg, virtual=True, scheme=scheme)
    scores = _nan((cfg["B"], cfg["H"], p.g.NB, p.g.NB))
    p.reorder_in(Q, K, V)
    S.spade_compose_select(p.g, p.spec, p.summ, p.counts, p.indices, scores)
    torch.cuda.synchronize()
    ref = O.composed_selection(P.to_np64(Q), P.to_np64(K), P.geometry(cfg), _oracle_spec(scheme),
                               P.scale_of(cfg["d"]))
    s_g = scores.cpu().numpy()
    tol = 1e-12 * max(1.0, float(np.max(np.abs(ref["scores"]))))
    assert np.max(np.abs(s_g - ref["scores"])) <= tol
    n_ex = _check_composed(cfg, scheme, ref, p.counts, p.indices)
    _say(f"  exempt rows {n_ex}")


@pytest.mark.parametrize("which", ["mean_plain", "dsa_topk_intra_window_sink", "dsa2_topp_intra_topk"])
@pytest.mark.parametrize("name", ["nb384", "many_blocks"])
def test_compose_select_wide_rows(name, which):
    """Rows of 257..512 and 513..1024 blocks (NB 384 and 1000): the selection kernel's
    wider register layouts, for every estimator, the intra filters and the window."""
    test_compose_select_matches_oracle(name, which)


@pytest.mark.parametrize("name", ["tiny", "ragged_d128", "w4_ragged"])
def test_compose_mean_plain_equals_estimate_select(name):
    cfg = _case(name)
    _say("compose == estimate_select", name)
    Q, K, V = P.bf16_inputs(cfg)
    for mode, topk, tau in (("topk", 3, 1.0), ("topp", 1, 0.8)):
        p = _path(cfg, virtual=True, scheme=Scheme("mean", mode, topk=topk, tau=tau))
        p.reorder_in(Q, K, V)
        p.select()
        c2, i2 = torch.full_like(p.counts, -7), torch.full_like(p.indices, -7)
        S.spade_estimate_select(p.g, p.qbar, p.kbar, p.mode, topk, tau, p.scale, c2, i2)
        torch.cuda.synchronize()
        assert torch.equal(p.counts, c2)
        for idx in np.ndindex(*c2.shape):
            n = int(c2[idx])
            assert torch.equal(p.indices[idx][:n], i2[idx][:n])


@pytest.mark.parametrize("name", ["tiny", "ragged_d64", "bs144_tail", "w4_ragged"])
def test_composed_path_matches_oracle(name):
    cfg = _case(name)
    Q, K, V = P.bf16_inputs(cfg)
    scheme = _schemes(cfg, Q, K)["dsa_topk_intra_window_sink"]
    _say("composed path", name)
    p = _path(cfg, virtual=True, scheme=scheme)
    P.nan_fill(p.O)
    out = p.run(Q, K, V)
    torch.cuda.synchronize()
    q, k, v = (P.to_np64(x) for x in (Q, K, V))
    og = P.geometry(cfg)
    ref = O.composed_selection(q, k, og, _oracle_spec(scheme), P.scale_of(cfg["d"]))
    n_ex = _check_composed(cfg, scheme, ref, p.counts, p.indices)
    # attention on the GPU's own lists, every element, every run
    ro, _ = P.oracle_attention_on_lists(q, k, v, og, p.counts.cpu().numpy(),
                                        p.indices.cpu().numpy(), P.scale_of(cfg["d"]))
    err = P.finite_max_abs(P.to_np64(out), ro)
    _say(f"  exempt rows {n_ex}, max-abs {err:.3e}")
    assert err <= P.ATTN_MAX_ABS


def test_compose_full_hunyuan_dsa():
    """The paper's experimental selection (DSA estimate, intra thresholding,
    inter Top-K) plus a spatial window, at the full Hunyuan-Video layer size."""
    from gen.workloads import workload
    cfg = workload("hunyuan")
    _say("compose full hunyuan dsa")
    Q, K, V = P.bf16_inputs(cfg)
    og = P.geometry(cfg)
    coh = np.concatenate([O.block_coherence(O.block_sics(O.reorder(P.to_np64(X), og), og), og).ravel()
                          for X in (Q, K)])
    theta = _theta_between(coh, 0.1)
    scheme = Scheme("dsa", "topk", topk=43, intra="threshold", intra_theta=theta, window=(0, 1, 1))
    p = _path(cfg, virtual=True, scheme=scheme)
    p.reorder_in(Q, K, V)
    p.select()
    torch.cuda.synchronize()
    ref = O.composed_selection(P.to_np64(Q), P.to_np64(K), og, _oracle_spec(scheme),
                               P.scale_of(cfg["d"]))
    n_ex = _check_composed(cfg, scheme, ref, p.counts, p.indices)
    kept = float(p.counts.sum()) / (cfg["H"] * og.NB * og.NB)
    _say(f"  exempt rows {n_ex}, kept fraction {kept:.3f}")
