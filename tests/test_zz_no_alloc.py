"""The allocation-free raster attention entry point, through the C ABI.

spade_sparse_attn_raster_noalloc keeps its schedule scratch in the library's own
per-GPU array instead of a caller workspace; its outputs must equal
spade_sparse_attn_raster's bit for bit. Two calls in a row on the shared array, the
second on a smaller problem, then the first problem again (the array keeps the
last call's contents, which must not matter)."""
import sys

import numpy as np
import pytest
import torch

from paper_2608_03335_amd import spade as S

from . import _parity as P

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _case(T, Hs, Ws, bt, bh, bw, d, H, B, seed):
    cfg = P.small_cfg(T, Hs, Ws, bt, bh, bw, d=d, H=H, B=B)
    g = S.geom(B, H, d, T, Hs, Ws, bt, bh, bw)
    Q, K, V = P.bf16_inputs(cfg, seed=seed)
    rng = np.random.default_rng(seed)
    NB = g.NB
    counts = rng.integers(1, NB + 1, size=(B, H, NB)).astype(np.int32)
    idx = np.zeros((B, H, NB, NB), np.int32)
    for r in np.ndindex(B, H, NB):
        idx[r][: counts[r]] = np.sort(rng.choice(NB, counts[r], replace=False))
    return g, Q, K, V, torch.from_numpy(counts).to(DEV), torch.from_numpy(idx).to(DEV)


def _both(g, Q, K, V, c, i):
    scale = P.scale_of(g.d)
    o_ref = torch.full_like(Q, float("nan"))
    l_ref = torch.full((g.B, g.H, g.N), float("nan"), dtype=torch.float32, device=DEV)
    ws = torch.empty(max(S.spade_attn_workspace_bytes(g), 1), dtype=torch.uint8, device=DEV)
    S.spade_sparse_attn_raster(g, Q, K, V, c, i, scale, o_ref, l_ref, workspace=ws)
    o = torch.full_like(Q, float("nan"))
    lse = torch.full_like(l_ref, float("nan"))
    S.spade_sparse_attn_raster_noalloc(g, Q, K, V, c, i, scale, o, lse)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(o).all()) and bool(torch.isfinite(lse).all())
    assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16))
    assert torch.equal(lse, l_ref)
    return o


def test_noalloc_equals_workspace_call_twice_then_smaller():
    # first: 160-slot blocks (paired kernel), 3 heads x 2 batch elements, ragged grid
    big = _case(7, 11, 19, 4, 5, 8, 128, 3, 2, seed=11)
    # second, smaller: 120-slot blocks (single-member kernel), 2 heads, d = 64
    small = _case(5, 9, 13, 3, 5, 8, 64, 2, 1, seed=12)
    _say("noalloc: big")
    first = _both(*big)
    _say("noalloc: smaller")
    _both(*small)
    _say("noalloc: big again")
    again = _both(*big)
    assert torch.equal(first.view(torch.int16), again.view(torch.int16))


def test_noalloc_host_errors_match():
    g = S.geom(1, 2, 96, 4, 8, 8, 2, 4, 4)  # d = 96: unsupported on both entry points
    t = torch.zeros(2 * 256 * 96, dtype=torch.bfloat16, device=DEV)
    c = torch.zeros(2 * 8, dtype=torch.int32, device=DEV)
    i = torch.zeros(2 * 8 * 8, dtype=torch.int32, device=DEV)
    for fn, extra in ((S.spade_sparse_attn_raster_noalloc, {}),
                      (S.spade_sparse_attn_raster, {"workspace": c})):
        with pytest.raises(S.SpadeError) as e:
            fn(g, t, t, t, c, i, 0.1, t, **extra)
        assert e.value.status == S.SPADE_ERR_UNSUPPORTED
    g2 = S.geom(1, 2, 128, 4, 8, 8, 2, 4, 4)
    t2 = torch.zeros(2 * 256 * 128, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(S.SpadeError) as e:  # a bad scale is rejected before any launch
        S.spade_sparse_attn_raster_noalloc(g2, t2, t2, t2, c, i, -1.0, t2)
    assert e.value.status == S.SPADE_ERR_INVALID_ARG
