"""GPU parity of the raster ("virtual blocking") attention call.

spade_sparse_attn_raster must equal spade_block_sparse_attn followed by the
inverse blocking, bit for bit (same rows, same arithmetic in the same order), on
the oracle's block lists; the whole virtual path must match the oracle.
"""
import sys

import numpy as np
import pytest
import torch

from oracle import spade_oracle as O
from paper_2608_03335_amd import spade as S

from . import _parity as P
from .test_gpu_parity import SMALL, _case, _geom, _oracle_selection, _path

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("name", SMALL)
def test_raster_equals_blocked_then_restore(name):
    cfg = dict(_case(name), B=2)
    _say("raster attention", name)
    g = _geom(cfg)
    Q, K, V = P.bf16_inputs(cfg)
    s, c, i = _oracle_selection(cfg, Q, K, cfg["mode"], cfg.get("topk"), cfg.get("tau"))
    counts = torch.from_numpy(c.astype(np.int32)).to(DEV)
    indices = torch.from_numpy(np.where(i < 0, 0, i).astype(np.int32)).to(DEV)
    p = _path(cfg, with_lse=True)
    p.reorder_in(Q, K, V)
    p.attend(counts, indices)
    p.restore()
    o = torch.full_like(Q, float("nan"))
    lse = torch.full((cfg["B"], cfg["H"], g.N), float("nan"), dtype=torch.float32, device=DEV)
    S.spade_sparse_attn_raster(g, Q, K, V, counts, indices, P.scale_of(cfg["d"]), o, lse,
                               workspace=p.ws)
    torch.cuda.synchronize()
    assert torch.equal(o.view(torch.int16), p.O.view(torch.int16))
    pos = torch.from_numpy(O.token_position(P.geometry(cfg))).to(DEV)
    assert torch.equal(lse, p.lse[:, :, pos])


@pytest.mark.parametrize("name", ["tiny", "ragged_d64", "bs144_tail", "one_block", "w4_ragged", "w6_ragged",
                                  "pp_bs129", "w3_ragged"])
def test_virtual_path_matches_oracle(name):
    """The whole virtual path: selection against the oracle's (cut exemptions
    allowed), and the attention output, NaN-poisoned before the call, against the
    oracle run on the GPU's own lists (every element, every run)."""
    cfg = _case(name)
    _say("virtual path", name)
    Q, K, V = P.bf16_inputs(cfg)
    p = _path(cfg, virtual=True, with_lse=True)
    P.nan_fill(p.O, p.lse)
    out = p.run(Q, K, V)
    torch.cuda.synchronize()
    og = P.geometry(cfg)
    q, k, v = (P.to_np64(x) for x in (Q, K, V))
    ref = O.spade_attention(q, k, v, og, cfg["mode"], topk=cfg.get("topk"), tau=cfg.get("tau"),
                            scale=P.scale_of(cfg["d"]))
    cg, ig = p.counts.cpu().numpy(), p.indices.cpu().numpy()
    n_ex = P.compare_selection(ref["scores"], ref["counts"], ref["indices"], cg, ig, cfg["mode"],
                               cfg.get("tau"))
    ro, rl = P.oracle_attention_on_lists(q, k, v, og, cg, ig, P.scale_of(cfg["d"]))
    err = P.finite_max_abs(P.to_np64(out), ro)
    assert P.finite_max_abs(p.lse.cpu().numpy(), rl) <= P.LSE_MAX_ABS
    _say(f"  exempt rows {n_ex}, max-abs {err:.3e}")
    assert err <= P.ATTN_MAX_ABS


def test_raster_full_hunyuan_equals_blocked():
    from gen.workloads import workload
    cfg = workload("hunyuan")
    _say("raster full hunyuan")
    Q, K, V = P.bf16_inputs(cfg)
    p = _path(cfg)
    p.run(Q, K, V)
    pv = _path(cfg, virtual=True)
    pv.run(Q, K, V)
    torch.cuda.synchronize()
    assert torch.equal(p.counts, pv.counts)
    assert torch.equal(p.O.view(torch.int16), pv.O.view(torch.int16))


@pytest.mark.parametrize("name,n_rows", [("wan13b", 16), ("hunyuan", 16), ("wan14b", 12)])
def test_full_shape_raster_path(name, n_rows):
    """The path bench.py times (raster form) at the full layer shapes, outputs
    NaN-poisoned before the call: every row's selection against the oracle; every
    output row finite; O and LSE of every query block of the head holding the
    heaviest row, and of sampled blocks (first and last included), recomputed by the
    oracle with the GPU's lists."""
    from gen.workloads import workload
    cfg = workload(name)
    _say("raster full shape", name)
    og = P.geometry(cfg)
    Q, K, V = P.bf16_inputs(cfg)
    p = _path(cfg, virtual=True, with_lse=True)
    P.nan_fill(p.O, p.lse)
    p.run(Q, K, V)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(p.O).all()), "an output row was not written"
    assert bool(torch.isfinite(p.lse).all()), "an LSE entry was not written"
    s, c, i = _oracle_selection(cfg, Q, K, cfg["mode"], cfg.get("topk"), cfg.get("tau"))
    cg, ig = p.counts.cpu().numpy(), p.indices.cpu().numpy()
    n_ex = P.compare_selection(s, c, i, cg, ig, cfg["mode"], cfg.get("tau"))
    _say(f"  selection rows exempt: {n_ex}")
    hb, hh = P.heaviest_head(cg)
    rows = P.sample_rows(cfg["B"], cfg["H"], og.NB, n_rows, seed=2,
                         must=[(0, 0, 0), (0, cfg["H"] - 1, og.NB - 1)])
    rows = sorted(set(rows) | {(hb, hh, r) for r in range(og.NB)})
    heads = sorted({h for _, h, _ in rows})
    sub = [(b, heads.index(h), i) for b, h, i in rows]
    q, k, v = (P.to_np64(x[:, heads]) for x in (Q, K, V))
    ro, rl = P.oracle_attention_on_lists(q, k, v, og, cg[:, heads], ig[:, heads],
                                         P.scale_of(cfg["d"]), rows=sub)
    worst = P.compare_rows_raster(P.to_np64(p.O[:, heads]), p.lse[:, heads].cpu().numpy(), ro, rl,
                                  og, sub)
    _say(f"  attention max-abs over {len(sub)} query blocks (head {hh} whole): {worst:.3e}")
    assert worst <= P.ATTN_MAX_ABS
