"""Host-side checks of the figures bench.py reports (CPU; no GPU call).

- Kept FLOPs, the numerator of the roofline's `achieved` figure: the two matmuls of
  Eq. (2) cost 4·d FLOP per kept (query token, key token) pair. bench.py sums
  4·d·n_i·n_j over the kept block pairs; here the same total comes from counting token
  pairs under the token-level mask that the block lists induce, with each token's
  block taken from the oracle's slot tables (ragged edge blocks, two batch elements,
  list entries past each row's count left as garbage).
- Real tokens per block, the weights of that sum, against the oracle's block tables.
- A request for more than one GPU ends with status 2 and a message.
"""
import os
import subprocess
import sys
from types import SimpleNamespace

import numpy as np
import pytest
import torch

import bench
import oracle.spade_oracle as O
from paper_2608_03335_amd.pipeline import block_valid_counts

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

GEOMS = [
    (5, 11, 20, 2, 4, 9),   # ragged in every dimension
    (4, 8, 8, 2, 4, 4),     # no ragged block
    (3, 7, 13, 3, 7, 13),   # one block holding the whole grid
    (1, 1, 1, 1, 1, 1),     # one token
]


def _geom(T, Hs, Ws, bt, bh, bw):
    return (O.Geometry(T, Hs, Ws, bt, bh, bw),
            SimpleNamespace(T=T, Hs=Hs, Ws=Ws, bt=bt, bh=bh, bw=bw))


def _random_lists(rng, B, H, NB):
    """Ascending kept lists of random length; entries past the count are garbage."""
    counts = rng.integers(0, NB + 1, size=(B, H, NB))
    counts[0, 0, 0] = NB  # one full row
    counts[-1, -1, -1] = 0  # one empty row
    indices = rng.integers(-5, NB + 5, size=(B, H, NB, NB))
    for idx in np.ndindex(B, H, NB):
        c = counts[idx]
        indices[idx][:c] = np.sort(rng.choice(NB, size=c, replace=False))
    return counts, indices


@pytest.mark.parametrize("shape", GEOMS)
def test_block_token_counts_match_the_oracle_tables(shape):
    og, hg = _geom(*shape)
    _, n_valid = O.block_tables(og)
    np.testing.assert_array_equal(block_valid_counts(hg), n_valid)


@pytest.mark.parametrize("shape", GEOMS)
@pytest.mark.parametrize("d", [64, 128])
def test_kept_flops_count_token_pairs(shape, d):
    og, hg = _geom(*shape)
    rng = np.random.default_rng(sum(shape) * 7 + d)
    B, H, NB = 2, 3, og.NB
    counts, indices = _random_lists(rng, B, H, NB)

    # token -> block from the oracle's slot table, then the token-level mask
    slot_token, _ = O.block_tables(og)
    blk = np.empty(og.N, dtype=np.int64)
    live = slot_token >= 0
    blk[slot_token[live]] = np.nonzero(live)[0] // og.BS
    pairs = 0
    for b in range(B):
        for h in range(H):
            bm = O.block_mask(counts[b, h][None], indices[b, h][None])[0]  # [NB, NB]
            pairs += int(bm[blk[:, None], blk[None, :]].sum())
    expected = 4.0 * d * pairs

    nvalid = torch.from_numpy(block_valid_counts(hg))
    got = bench.kept_flops_lists(torch.from_numpy(counts.astype(np.int32)),
                                 torch.from_numpy(indices.astype(np.int32)), nvalid, d)
    assert got == expected


def test_dense_mask_flops_are_the_dense_attention_count():
    og, hg = _geom(5, 11, 20, 2, 4, 9)
    NB, d = og.NB, 128
    counts = np.full((1, 1, NB), NB, dtype=np.int32)
    indices = np.broadcast_to(np.arange(NB, dtype=np.int32), (1, 1, NB, NB)).copy()
    nvalid = torch.from_numpy(block_valid_counts(hg))
    got = bench.kept_flops_lists(torch.from_numpy(counts), torch.from_numpy(indices), nvalid, d)
    assert got == 4.0 * d * og.N * og.N  # Eq. (1): QK^T and PV over every token pair


def test_several_gpus_are_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       cwd=ROOT, capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


@pytest.mark.parametrize("bt,bh,bw,d,nb,kernel", [
    (4, 5, 8, 128, 360, "attn_sw_kernel"),     # Hunyuan's blocks: the software-pipelined kernel
    (3, 6, 8, 128, 245, "attn_sw_kernel"),     # 144 slots, five tiles
    (4, 5, 8, 128, 3824, "attn_sw_kernel"),    # the longest kept list its 9-chunk ring leaves room for
    (4, 5, 8, 128, 3825, "attn_pp_kernel"),    # one more: the paired kernel's 8-chunk ring
    (4, 5, 8, 64, 360, "attn_pp_kernel"),      # d = 64: the paired kernel
    (4, 5, 8, 128, 7928, "attn_pp_kernel"),
    (4, 5, 8, 128, 7929, "attn_kernel"),       # past the paired kernel's list space
    (3, 5, 8, 128, 630, "attn_kernel"),        # 120 slots (four tiles)
])
def test_kernel_label_follows_the_dispatch(bt, bh, bw, d, nb, kernel):
    """The bench names the kernel the library launches: the LDS budgets of the 5-tile
    kernels (ring + slot table + per-slot key counts + kept list <= 160 KB)."""
    g = SimpleNamespace(bt=bt, bh=bh, bw=bw, d=d, NB=nb)
    assert bench.attn_kernel_label(g).split()[1] == kernel
