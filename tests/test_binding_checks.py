"""The binding's tensor checks: every pointer it hands to the C ABI comes from a
contiguous GPU tensor of the declared element type and at least the size the
geometry implies. The checks run before any library call, so they are exercised
here on CPU tensors (the device check comes last)."""
import pytest
import torch

from paper_2608_03335_amd import spade as S

G = S.spade_geom(1, 2, 128, 4, 8, 8, 2, 4, 4)   # B H d T Hs Ws bt bh bw: N 256, NB 8, BS 32
N, NB, BS = 256, 8, 32


def _raster(dtype=torch.bfloat16, n=None):
    return torch.zeros(n if n is not None else 2 * N * 128, dtype=dtype)


def _raises(match, fn, *a, **kw):
    with pytest.raises(S.SpadeError, match=match) as e:
        fn(*a, **kw)
    assert e.value.status == S.SPADE_ERR_INVALID_ARG


def test_reorder_rejects_other_element_types():
    for dt in (torch.float16, torch.float64, torch.int32):
        _raises("bfloat16 or float32", S.spade_block_reorder, G, _raster(dt), _raster(dt))


def test_reorder_checks_both_sides_against_the_geometry():
    blocked = 2 * NB * BS * 128
    _raises("x holds", S.spade_block_reorder, G, _raster(n=2 * N * 128 - 1), _raster(n=blocked))
    _raises("y holds", S.spade_block_reorder, G, _raster(), _raster(n=blocked - 1))
    _raises("y must be torch.bfloat16", S.spade_block_reorder, G, _raster(),
            _raster(torch.float32, blocked))
    # a head list shrinks the blocked side to its heads
    _raises("GPU tensor", S.spade_block_reorder, G, _raster(), _raster(n=NB * BS * 128),
            heads=[1])


def test_attention_checks_every_tensor():
    q = _raster()
    counts = torch.zeros(2 * NB, dtype=torch.int32)
    idx = torch.zeros(2 * NB * NB, dtype=torch.int32)
    o = _raster()
    call = S.spade_sparse_attn_raster
    _raises("q must be torch.bfloat16", call, G, q.float(), q, q, counts, idx, 0.1, o)
    _raises("counts must be torch.int32", call, G, q, q, q, counts.long(), idx, 0.1, o)
    _raises("indices holds", call, G, q, q, q, counts, idx[:-1], 0.1, o)
    _raises("o must be contiguous", call, G, q, q, q, counts, idx, 0.1,
            o.view(2, -1).t())
    _raises("lse holds", call, G, q, q, q, counts, idx, 0.1, o,
            lse=torch.zeros(2 * N - 1, dtype=torch.float32))
    _raises("GPU tensor", call, G, q, q, q, counts, idx, 0.1, o)
    blocked = torch.zeros(2 * NB * BS * 128, dtype=torch.bfloat16)
    _raises("lse must be torch.float32", S.spade_block_sparse_attn, G, blocked, blocked, blocked,
            counts, idx, 0.1, blocked, lse=torch.zeros(2 * NB * BS, dtype=torch.float64))


def test_selection_and_summary_checks():
    summ = torch.zeros(2 * NB * 128, dtype=torch.float64)
    counts = torch.zeros(2 * NB, dtype=torch.int32)
    idx = torch.zeros(2 * NB * NB, dtype=torch.int32)
    _raises("qbar must be torch.float64", S.spade_estimate_select, G, summ.float(), summ,
            S.SPADE_TOPK, 2, 1.0, 0.1, counts, idx)
    _raises("scores holds", S.spade_estimate_select, G, summ, summ, S.SPADE_TOPK, 2, 1.0, 0.1,
            counts, idx, scores=torch.zeros(5, dtype=torch.float64))
    _raises("sics_q holds", S.spade_block_summarize, G, _raster(), _raster(),
            sics_q=torch.zeros(2 * NB - 1, dtype=torch.float64),
            sics_k=torch.zeros(2 * NB, dtype=torch.float64))
    _raises("qmax must be torch.float64", S.spade_block_minmax, G, _raster(), _raster(),
            summ.float(), summ, summ, summ)
    _raises("qbar must be torch.float64", S.summaries, qbar=summ.float())
    _raises("topk_per_head must be torch.int32", S.mask_spec,
            topk_per_head=torch.zeros(2, dtype=torch.int64))
    _raises("k_out holds", S.spade_policy_budgets, torch.zeros(4, dtype=torch.float64), 8, NB,
            torch.zeros(3, dtype=torch.int32))


def test_multi_checks_head_lists():
    q = _raster()
    good = (0, torch.zeros(NB, dtype=torch.int32), torch.zeros(NB * NB, dtype=torch.int32), 0, 0)
    short = (0, torch.zeros(NB, dtype=torch.int32), torch.zeros(NB * NB - 1, dtype=torch.int32),
             0, 0)
    wide = (0, torch.zeros(NB, dtype=torch.int64), torch.zeros(NB * NB, dtype=torch.int32), 0, 0)
    call = S.spade_sparse_attn_raster_multi
    _raises(r"heads\[1\] indices", call, [G], [good, short], q, q, q, 0.1, q)
    _raises(r"heads\[0\] counts", call, [G], [wide, good], q, q, q, 0.1, q)


def test_multi_checks_table_length_and_batch_spans():
    q = _raster()
    good = (0, torch.zeros(NB, dtype=torch.int32), torch.zeros(NB * NB, dtype=torch.int32), 0, 0)
    call = S.spade_sparse_attn_raster_multi
    # one entry per head of geometry 0, no fewer and no more
    _raises("heads has 1 entries", call, [G], [good], q, q, q, 0.1, q)
    _raises("heads has 3 entries", call, [G], [good] * 3, q, q, q, 0.1, q)
    # B = 2: batch 1's lists start a stride after batch 0's and must lie in the storage
    G2 = S.spade_geom(2, 2, 128, 4, 8, 8, 2, 4, 4)
    q2 = _raster(n=2 * 2 * N * 128)
    cstore = torch.zeros(2 * NB, dtype=torch.int32)
    istore = torch.zeros(2 * NB * NB, dtype=torch.int32)
    ok = (0, cstore[:NB], istore[:NB * NB], NB, NB * NB)
    far_c = (0, cstore[:NB], istore[:NB * NB], NB + 1, NB * NB)
    far_i = (0, cstore[:NB], istore[:NB * NB], NB, NB * NB + 1)
    late = (0, cstore[NB:], istore[NB * NB:], NB, NB * NB)  # batch 0 at the storage's end
    _raises(r"heads\[0\] counts: the batch strides", call, [G2], [far_c, ok], q2, q2, q2, 0.1, q2)
    _raises(r"heads\[1\] indices: the batch strides", call, [G2], [ok, far_i], q2, q2, q2, 0.1, q2)
    _raises(r"heads\[0\] counts: the batch strides", call, [G2], [late, ok], q2, q2, q2, 0.1, q2)
    # a valid table passes every check up to the device one
    _raises("GPU tensor", call, [G2], [ok, ok], q2, q2, q2, 0.1, q2)
