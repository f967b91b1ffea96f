"""GPU parity of the fused blocking + Summarizer + SICS call (§3.3 optimisation (1)).

Its blocked copies must equal spade_block_reorder's bit for bit, and its
summaries must equal spade_summarize's bit for bit (the same fp64 reductions in
the same order), for every small geometry, with and without a head list and with
each output pair requested alone; and both must match the fp64 oracle.
"""
import sys

import numpy as np
import pytest
import torch

from oracle import spade_oracle as O
from paper_2608_03335_amd import spade as S

from . import _parity as P
from .test_gpu_parity import SMALL, _case, _geom

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _unfused(g, Q, K, heads, sics):
    """Reference on the GPU: head-list reorder, then spade_summarize."""
    n = Q.shape[1] if heads is None else len(heads)
    B, d = Q.shape[0], Q.shape[-1]
    gg = S.geom(B, n, d, g.T, g.Hs, g.Ws, g.bt, g.bh, g.bw)
    qb = torch.empty((B, n, g.NB * g.BS, d), dtype=torch.bfloat16, device=DEV)
    kb = torch.empty_like(qb)
    S.spade_block_reorder(g, Q, qb, heads=heads)
    S.spade_block_reorder(g, K, kb, heads=heads)
    f64 = dict(dtype=torch.float64, device=DEV)
    qbar, kbar = torch.empty((B, n, g.NB, d), **f64), torch.empty((B, n, g.NB, d), **f64)
    sq = torch.empty((B, n, g.NB), **f64) if sics else None
    sk = torch.empty((B, n, g.NB), **f64) if sics else None
    S.spade_summarize(gg, qb, kb, qbar, kbar, sq, sk)
    return qb, kb, qbar, kbar, sq, sk


@pytest.mark.parametrize("name", SMALL)
@pytest.mark.parametrize("heads", [None, "subset"])
def test_fused_equals_reorder_plus_summarize(name, heads):
    cfg = _case(name)
    cfg = dict(cfg, B=2)
    _say("fused", name, heads)
    g, og = _geom(cfg), P.geometry(cfg)
    Q, K, _ = P.bf16_inputs(cfg)
    hl = None if heads is None else list(reversed(range(cfg["H"])))[: max(1, cfg["H"] - 1)]
    n = cfg["H"] if hl is None else len(hl)
    B, d = cfg["B"], cfg["d"]
    ref = _unfused(g, Q, K, hl, sics=True)
    f64 = dict(dtype=torch.float64, device=DEV)
    qb = torch.full((B, n, g.NB * g.BS, d), float("nan"), dtype=torch.bfloat16, device=DEV)
    kb = torch.full_like(qb, float("nan"))
    qbar, kbar = torch.empty((B, n, g.NB, d), **f64), torch.empty((B, n, g.NB, d), **f64)
    sq, sk = torch.empty((B, n, g.NB), **f64), torch.empty((B, n, g.NB), **f64)
    S.spade_block_summarize(g, Q, K, qb, kb, qbar, kbar, sq, sk, heads=hl)
    # summaries only (no blocked writes), and SICS only
    qbar2, kbar2 = torch.empty_like(qbar), torch.empty_like(kbar)
    S.spade_block_summarize(g, Q, K, qbar=qbar2, kbar=kbar2, heads=hl)
    sq3, sk3 = torch.empty_like(sq), torch.empty_like(sk)
    S.spade_block_summarize(g, Q, K, sics_q=sq3, sics_k=sk3, heads=hl)
    torch.cuda.synchronize()
    for a, b in ((qb, ref[0]), (kb, ref[1])):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    for a, b in ((qbar, ref[2]), (kbar, ref[3]), (qbar2, ref[2]), (kbar2, ref[3]),
                 (sq, ref[4]), (sk, ref[5]), (sq3, ref[4]), (sk3, ref[5])):
        assert torch.equal(a, b)
    # and the oracle
    sel = list(range(cfg["H"])) if hl is None else hl
    for X, xbar, sics in ((Q, qbar, sq), (K, kbar, sk)):
        Xb = O.reorder(P.to_np64(X)[:, sel], og)
        r = O.block_means(Xb, og)
        assert np.max(np.abs(xbar.cpu().numpy() - r)) <= 1e-12 * (1 + np.max(np.abs(r)))
        np.testing.assert_allclose(sics.cpu().numpy(), O.block_sics(Xb, og), rtol=1e-9, atol=1e-9)
