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


@pytest.mark.parametrize("name", ["tiny", "ragged_d64", "bs144_tail", "one_block", "w4_ragged", "w6_ragged"])
def test_virtual_path_matches_oracle(name):
    cfg = _case(name)
    _say("virtual path", name)
    Q, K, V = P.bf16_inputs(cfg)
    p = _path(cfg, virtual=True)
    out = p.run(Q, K, V)
    torch.cuda.synchronize()
    ref = O.spade_attention(P.to_np64(Q), P.to_np64(K), P.to_np64(V), P.geometry(cfg), cfg["mode"],
                            topk=cfg.get("topk"), tau=cfg.get("tau"), scale=P.scale_of(cfg["d"]))
    n_ex = P.compare_selection(ref["scores"], ref["counts"], ref["indices"], p.counts.cpu().numpy(),
                               p.indices.cpu().numpy(), cfg["mode"], cfg.get("tau"))
    if n_ex == 0:
        err = float(np.max(np.abs(P.to_np64(out) - ref["O"])))
        _say(f"  max-abs {err:.3e}")
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
    """The path bench.py times (raster form) at the full layer shapes: every row's
    selection against the oracle, and sampled query blocks (first and last included)
    recomputed by the oracle with the GPU's lists, O and LSE."""
    from gen.workloads import workload
    cfg = workload(name)
    _say("raster full shape", name)
    og = P.geometry(cfg)
    Q, K, V = P.bf16_inputs(cfg)
    p = _path(cfg, virtual=True, with_lse=True)
    p.run(Q, K, V)
    torch.cuda.synchronize()
    s, c, i = _oracle_selection(cfg, Q, K, cfg["mode"], cfg.get("topk"), cfg.get("tau"))
    n_ex = P.compare_selection(s, c, i, p.counts.cpu().numpy(), p.indices.cpu().numpy(),
                               cfg["mode"], cfg.get("tau"))
    _say(f"  selection rows exempt: {n_ex}")
    cg, ig = p.counts.cpu().numpy(), p.indices.cpu().numpy()
    rows = P.sample_rows(cfg["B"], cfg["H"], og.NB, n_rows, seed=2,
                         must=[(0, 0, 0), (0, cfg["H"] - 1, og.NB - 1)])
    heads = sorted({h for _, h, _ in rows})
    sub = [(b, heads.index(h), i) for b, h, i in rows]
    Qb, Kb, Vb = (O.reorder(P.to_np64(x[:, heads]), og) for x in (Q, K, V))
    ref, ref_lse = O.block_sparse_attention(Qb, Kb, Vb, cg[:, heads], ig[:, heads], og,
                                            P.scale_of(cfg["d"]), rows=sub)
    slot_token, nv = O.block_tables(og)
    got, got_lse = P.to_np64(p.O[:, heads]), p.lse[:, heads].cpu().numpy()
    worst = 0.0
    for (b, k, i) in sub:
        toks = slot_token[i * og.BS: i * og.BS + nv[i]]
        sl = slice(i * og.BS, i * og.BS + nv[i])
        worst = max(worst, float(np.max(np.abs(got[b, k, toks] - ref[b, k, sl]))))
        np.testing.assert_allclose(got_lse[b, k, toks], ref_lse[b, k, sl], atol=P.LSE_MAX_ABS, rtol=0)
    _say(f"  attention max-abs over {len(sub)} sampled query blocks: {worst:.3e}")
    assert worst <= P.ATTN_MAX_ABS
