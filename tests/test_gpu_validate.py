"""Device check of block lists (spade_validate_lists) and the binding's debug mode.

The lists are the block mask in the row-wise form the attention walks (§3.3
optimisation (3)): per query block, its kept key blocks in ascending order. Well-formed
lists must pass; planted faults (a count outside [0, NB], an index outside [0, NB), an
order that does not strictly ascend) must be reported with the lowest failing row and
the union of the failure bits. Entries past a row's count are not part of the list."""
import sys

import numpy as np
import pytest
import torch

from paper_2608_03335_amd import spade as S

from . import _parity as P

pytestmark = pytest.mark.gpu
DEV = "cuda"
CLEAN = [0, 2**31 - 1, 0, 0]


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _lists(g, seed):
    rng = np.random.default_rng(seed)
    NB = g.NB
    counts = rng.integers(0, NB + 1, size=(g.B, g.H, NB)).astype(np.int32)
    idx = rng.integers(-7, 3 * NB, size=(g.B, g.H, NB, NB)).astype(np.int32)  # junk past counts
    for r in np.ndindex(g.B, g.H, NB):
        idx[r][: counts[r]] = np.sort(rng.choice(NB, counts[r], replace=False))
    return counts, idx


def _report(g, counts, idx):
    rep = torch.full((4,), -99, dtype=torch.int32, device=DEV)
    c = torch.from_numpy(np.ascontiguousarray(counts)).to(DEV)
    i = torch.from_numpy(np.ascontiguousarray(idx)).to(DEV)
    S.spade_validate_lists(g, c, i, rep)
    torch.cuda.synchronize()
    return rep.cpu().tolist()


SHAPES = [  # (B, H, T, Hs, Ws, bt, bh, bw): NB 2, 27, 100 (ragged grids)
    (1, 1, 2, 4, 4, 2, 4, 2),
    (2, 3, 5, 9, 10, 2, 4, 4),
    (1, 2, 10, 10, 10, 1, 1, 10),
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_well_formed_lists_pass(shape):
    B, H, T, Hs, Ws, bt, bh, bw = shape
    g = S.geom(B, H, 64, T, Hs, Ws, bt, bh, bw)
    _say(f"validate well-formed lists {shape} NB={g.NB}")
    counts, idx = _lists(g, seed=1)
    assert _report(g, counts, idx) == CLEAN


def test_planted_faults_are_reported():
    g = S.geom(2, 3, 64, 5, 9, 10, 2, 4, 4)
    NB = g.NB
    _say(f"validate planted faults NB={NB}")
    counts, idx = _lists(g, seed=2)
    flat_c = counts.reshape(-1)
    flat_i = idx.reshape(-1, NB)
    rows = {}
    # count above NB, count below 0
    flat_c[40] = NB + 1
    rows[40] = S.SPADE_LIST_BAD_COUNT
    flat_c[7] = -1
    rows[7] = S.SPADE_LIST_BAD_COUNT
    # an index outside [0, NB) inside the list
    flat_c[101] = 5
    flat_i[101, :5] = [0, 3, NB, NB + 1, NB + 2]
    rows[101] = S.SPADE_LIST_BAD_INDEX
    flat_c[55] = 3
    flat_i[55, :3] = [-1, 2, 4]
    rows[55] = S.SPADE_LIST_BAD_INDEX
    # descending pair, and a repeated block (not strictly ascending)
    flat_c[130] = 4
    flat_i[130, :4] = [1, 5, 4, 9]
    rows[130] = S.SPADE_LIST_NOT_ASCENDING
    flat_c[131] = 2
    flat_i[131, :2] = [6, 6]
    rows[131] = S.SPADE_LIST_NOT_ASCENDING
    rep = _report(g, counts, idx)
    assert rep == [len(rows), min(rows), S.SPADE_LIST_BAD_COUNT | S.SPADE_LIST_BAD_INDEX
                   | S.SPADE_LIST_NOT_ASCENDING, 0]
    # each fault alone: the row and its bit
    for r, bit in rows.items():
        c1, i1 = _lists(g, seed=2)
        c1.reshape(-1)[r] = flat_c[r]
        i1.reshape(-1, NB)[r] = flat_i[r]
        assert _report(g, c1, i1) == [1, r, bit, 0], r


def test_fault_past_the_first_wave_width():
    g = S.geom(1, 1, 64, 10, 10, 10, 1, 1, 10)  # NB = 100
    NB = g.NB
    _say(f"validate a late fault NB={NB}")
    counts = np.full((1, 1, NB), NB, np.int32)
    idx = np.broadcast_to(np.arange(NB, dtype=np.int32), (1, 1, NB, NB)).copy()
    assert _report(g, counts, idx) == CLEAN
    idx[0, 0, 17, 90] = idx[0, 0, 17, 89]  # entry 90: lane 26 of the second pass over the row
    idx[0, 0, 42, 99] = NB
    assert _report(g, counts, idx) == [2, 17, S.SPADE_LIST_NOT_ASCENDING | S.SPADE_LIST_BAD_INDEX,
                                       0]


def test_empty_problem_clears_the_report():
    g = S.geom(0, 3, 64, 5, 9, 10, 2, 4, 4)
    rep = torch.full((4,), -99, dtype=torch.int32, device=DEV)
    S.spade_validate_lists(g, None, None, rep)
    torch.cuda.synchronize()
    assert rep.cpu().tolist() == CLEAN


def test_debug_mode_raises_on_malformed_lists(monkeypatch):
    T, Hs, Ws, bt, bh, bw = 5, 9, 10, 2, 4, 4
    cfg = P.small_cfg(T, Hs, Ws, bt, bh, bw, d=64, H=2, B=1)
    g = S.geom(1, 2, 64, T, Hs, Ws, bt, bh, bw)
    _say(f"validate debug mode NB={g.NB}")
    Q, K, V = P.bf16_inputs(cfg, seed=3)
    counts, idx = _lists(g, seed=3)
    c = torch.from_numpy(counts).to(DEV)
    i = torch.from_numpy(idx).to(DEV)
    scale = P.scale_of(g.d)
    ws = torch.empty(max(S.spade_attn_workspace_bytes(g), 1), dtype=torch.uint8, device=DEV)
    o0 = torch.empty_like(Q)
    S.spade_sparse_attn_raster(g, Q, K, V, c, i, scale, o0, workspace=ws)
    monkeypatch.setenv("SPADE_DEBUG_VALIDATE", "1")
    o1 = torch.empty_like(Q)
    S.spade_sparse_attn_raster(g, Q, K, V, c, i, scale, o1, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(o0, o1)  # the check changes nothing on good lists
    bad = c.clone()
    bad[0, 1, 3] = g.NB + 2
    with pytest.raises(S.SpadeError, match="1 rows fail, the first is row 30"):
        S.spade_sparse_attn_raster(g, Q, K, V, bad, i, scale, o1, workspace=ws)
    with pytest.raises(S.SpadeError, match="malformed block lists"):
        S.spade_sparse_attn_raster_noalloc(g, Q, K, V, bad, i, scale, o1)
