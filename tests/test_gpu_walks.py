"""Kept-walk lengths of the 5-tile attention kernels, element-wise against the oracle.

Blocks of 160 slots at d = 128 run the software-pipelined kernel: one barrier per
window of four chunks, chunk c in ring slot c mod 9, the fifth row tile split over
four waves by chunk index mod 4 and merged by log-sum-exp. Every residue of the walk
length modulo 4 and 9, and walks shorter than one window, must give Eq. (2) on the
given lists. The grid is ragged on every axis, so some query blocks hold fewer than
129 real rows (the fifth tile, or more, has no rows) and some key blocks fill only
one or two chunks.
"""
import numpy as np
import pytest
import torch

from oracle import spade_oracle as O
from paper_2608_03335_amd import spade as S

from . import _parity as P

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _lists(NB, H, seed):
    """Row i of head h keeps (i + 5 h) mod 14 random blocks, ascending; one row of head 0
    keeps every block and one keeps none."""
    rng = np.random.default_rng(seed)
    counts = np.zeros((1, H, NB), np.int32)
    idx = np.zeros((1, H, NB, NB), np.int32)
    for h in range(H):
        for i in range(NB):
            k = (i + 5 * h) % 14
            counts[0, h, i] = k
            idx[0, h, i, :k] = np.sort(rng.choice(NB, k, replace=False))
    counts[0, 0, 1] = NB
    idx[0, 0, 1] = np.arange(NB)
    counts[0, 0, 2] = 0
    return counts, idx


@pytest.mark.parametrize("raster", [True, False], ids=["raster", "blocked"])
def test_five_tile_walk_lengths(raster):
    # blocks 4 x 5 x 8 (160 slots) over a 9 x 13 x 25 grid: extents (4, 4, 1) x (5, 5, 3)
    # x (8, 8, 8, 1), so real rows per query block range from 3 to 160
    cfg = P.small_cfg(9, 13, 25, 4, 5, 8, d=128, H=3, B=1)
    og = P.geometry(cfg)
    g = S.geom(cfg["B"], cfg["H"], cfg["d"], cfg["T"], cfg["Hs"], cfg["Ws"], cfg["bt"],
               cfg["bh"], cfg["bw"])
    NB, BS = g.NB, g.BS
    assert BS == 160 and NB == 36
    Q, K, V = P.bf16_inputs(cfg, seed=11)
    counts, idx = _lists(NB, cfg["H"], seed=11)
    c = torch.from_numpy(counts).to(DEV)
    i = torch.from_numpy(idx).to(DEV)
    scale = P.scale_of(cfg["d"])
    ws = torch.empty(max(S.spade_attn_workspace_bytes(g), 1), dtype=torch.uint8, device=DEV)
    lse = torch.full((1, cfg["H"], g.N if raster else NB * BS), float("nan"),
                     dtype=torch.float32, device=DEV)
    if raster:
        o = torch.full_like(Q, float("nan"))
        S.spade_sparse_attn_raster(g, Q, K, V, c, i, scale, o, lse, workspace=ws)
    else:
        blk = [torch.empty((1, cfg["H"], NB * BS, cfg["d"]), dtype=torch.bfloat16, device=DEV)
               for _ in range(3)]
        for x, xb in zip((Q, K, V), blk):
            S.spade_block_reorder(g, x, xb)
        ob = torch.full_like(blk[0], float("nan"))
        S.spade_block_sparse_attn(g, *blk, c, i, scale, ob, lse, workspace=ws)
        o = torch.full_like(Q, float("nan"))
        S.spade_block_reorder(g, ob, o, inverse=True)
    torch.cuda.synchronize()
    got = P.to_np64(o)
    got_lse = lse.cpu().numpy().astype(np.float64)
    if not raster:
        got_lse = got_lse[:, :, O.token_position(og)]
    empty = [(0, h, r) for h in range(cfg["H"]) for r in range(NB) if counts[0, h, r] == 0]
    rows = [(0, h, r) for h in range(cfg["H"]) for r in range(NB) if counts[0, h, r] > 0]
    ref_o, ref_l = P.oracle_attention_on_lists(P.to_np64(Q), P.to_np64(K), P.to_np64(V), og,
                                               counts, idx, scale, rows=rows)
    for (b, h, r) in empty:
        toks = P.row_tokens(og, r)
        assert np.all(got[b, h, toks] == 0) and np.all(np.isneginf(got_lse[b, h, toks]))
    worst = P.compare_rows_raster(got, got_lse, ref_o, ref_l, og, rows)
    print(f"max-abs {worst:.3e} over {len(rows)} query blocks", flush=True)
    assert worst <= P.ATTN_MAX_ABS
