"""The default path (summaries, selection, raster attention) and the allocation-free
attention call under HIP graph capture. The library allocates nothing and never
synchronises, so a captured call must replay exactly: every replay is compared with the
eager call, bit for bit, with its outputs poisoned, eager work and host synchronisations
between the replays. The first calls (which set each kernel's LDS limit and look up the
allocation-free call's scratch) run eagerly before the capture."""
import sys

import pytest
import torch

from paper_2608_03335_amd import spade as S
from paper_2608_03335_amd.pipeline import SpadePath

from . import _parity as P
from .test_gpu_parity import _case

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _live(counts, indices):
    """Indices with the entries past each row's count masked (they are not part of a list)."""
    NB = indices.shape[-1]
    live = torch.arange(NB, device=indices.device) < counts[..., None]
    return torch.where(live, indices, torch.full_like(indices, -1))


def _capture(fn):
    """fn captured in a graph after one warm-up call on a side stream."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        fn()
    torch.cuda.synchronize()
    return graph


@pytest.mark.parametrize("name", ["bs144_tail", "pp_ragged_d64", "w4_ragged", "many_blocks"])
def test_default_path_replays_exactly(name):
    cfg = _case(name)
    _say("graph capture, default path", name)
    Q, K, V = P.bf16_inputs(cfg, seed=11)
    p = SpadePath(cfg["B"], cfg["H"], cfg["d"], cfg["T"], cfg["Hs"], cfg["Ws"], cfg["bt"],
                  cfg["bh"], cfg["bw"], mode=cfg["mode"], topk=cfg.get("topk"),
                  tau=cfg.get("tau"), device=DEV, virtual=True, with_lse=True)
    p.run(Q, K, V)
    torch.cuda.synchronize()
    ref_o, ref_lse = p.O.clone(), p.lse.clone()
    ref_c, ref_i = p.counts.clone(), _live(p.counts, p.indices)
    graph = _capture(lambda: p.run(Q, K, V))
    for rep in range(3):
        P.nan_fill(p.O, p.lse)
        p.counts.fill_(-7)
        p.indices.fill_(-7)
        busy = (Q.float() * 2.0).sum()  # eager work between the replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.isfinite(busy)
        assert torch.equal(p.counts, ref_c), f"replay {rep}: counts"
        assert torch.equal(_live(p.counts, p.indices), ref_i), f"replay {rep}: indices"
        assert torch.equal(p.O.view(torch.int16), ref_o.view(torch.int16)), f"replay {rep}: O"
        assert torch.equal(p.lse, ref_lse), f"replay {rep}: lse"


@pytest.mark.parametrize("name", ["bs144_tail", "w4_ragged"])
def test_noalloc_attention_replays_exactly(name):
    cfg = dict(_case(name), B=2)
    _say("graph capture, allocation-free attention", name)
    g = S.geom(cfg["B"], cfg["H"], cfg["d"], cfg["T"], cfg["Hs"], cfg["Ws"], cfg["bt"], cfg["bh"],
               cfg["bw"])
    Q, K, V = P.bf16_inputs(cfg, seed=12)
    p = SpadePath(cfg["B"], cfg["H"], cfg["d"], cfg["T"], cfg["Hs"], cfg["Ws"], cfg["bt"],
                  cfg["bh"], cfg["bw"], mode=cfg["mode"], topk=cfg.get("topk"),
                  tau=cfg.get("tau"), device=DEV, virtual=True)
    p.reorder_in(Q, K, V)
    p.select()
    scale = P.scale_of(cfg["d"])
    o = torch.empty_like(Q)
    lse = torch.empty((cfg["B"], cfg["H"], g.N), dtype=torch.float32, device=DEV)
    S.spade_sparse_attn_raster_noalloc(g, Q, K, V, p.counts, p.indices, scale, o, lse)
    torch.cuda.synchronize()
    ref_o, ref_lse = o.clone(), lse.clone()
    graph = _capture(lambda: S.spade_sparse_attn_raster_noalloc(g, Q, K, V, p.counts, p.indices,
                                                                scale, o, lse))
    for rep in range(3):
        P.nan_fill(o, lse)
        # eager work between the replays: the regular call on the same lists
        o2 = torch.empty_like(Q)
        S.spade_sparse_attn_raster(g, Q, K, V, p.counts, p.indices, scale, o2, workspace=p.ws)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(o.view(torch.int16), ref_o.view(torch.int16)), f"replay {rep}: O"
        assert torch.equal(lse, ref_lse), f"replay {rep}: lse"
        assert torch.equal(o2.view(torch.int16), ref_o.view(torch.int16))
