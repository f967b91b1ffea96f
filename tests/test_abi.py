"""The C-ABI library loads, exports every declared symbol, and rejects bad arguments on the host.

No compute call is made here: every call below fails validation before any HIP
launch, so these run without a GPU.
"""
import ctypes
import os
import re

import pytest

from paper_2608_03335_amd import spade as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "spade.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(spade_[a-z_]+)\s*\(", text)))


def test_header_declares_the_path_calls():
    names = _declared()
    for n in ("spade_block_reorder", "spade_summarize", "spade_estimate_select",
              "spade_block_sparse_attn", "spade_aggregation_score", "spade_choose_scheme",
              "spade_block_summarize"):
        assert n in names


def test_library_exports_every_declared_symbol():
    L = S.lib()
    for name in _declared():
        assert hasattr(L, name), name
    assert set(_declared()) == set(S.EXPORTED)


def _g(**kw):
    base = dict(B=1, H=2, d=128, T=4, Hs=8, Ws=8, bt=2, bh=4, bw=4)
    base.update(kw)
    return S.spade_geom(*[base[k] for k in ("B", "H", "d", "T", "Hs", "Ws", "bt", "bh", "bw")])


NULL = None
FAKE = ctypes.c_void_p(0x1000)      # aligned, never dereferenced (validation fails first)
MISALIGNED = ctypes.c_void_p(0x1008)


def _status(fn, *args):
    st = fn(*args)
    msg = S.lib().spade_last_error().decode()
    return st, msg


def test_status_strings():
    L = S.lib()
    assert L.spade_status_string(0) == b"SPADE_OK"
    assert L.spade_status_string(3) == b"SPADE_ERR_WORKSPACE"
    assert L.spade_status_string(99) == b"SPADE_ERR_UNKNOWN"


@pytest.mark.parametrize("kw,expect", [
    (dict(d=96), S.SPADE_ERR_UNSUPPORTED),
    (dict(bt=0), S.SPADE_ERR_INVALID_ARG),
    (dict(B=-1), S.SPADE_ERR_INVALID_ARG),
    (dict(bt=8, bh=8, bw=8), S.SPADE_ERR_UNSUPPORTED),   # BS = 512 > 256
])
def test_geometry_validation(kw, expect):
    L = S.lib()
    g = _g(**kw)
    st, msg = _status(L.spade_block_reorder, ctypes.byref(g), FAKE, FAKE, 0, 0, None, 0, None)
    assert st == expect and msg


def test_reorder_argument_errors():
    L = S.lib()
    g = _g()
    assert L.spade_block_reorder(None, FAKE, FAKE, 0, 0, None, 0, None) == S.SPADE_ERR_INVALID_ARG
    assert L.spade_block_reorder(ctypes.byref(g), NULL, FAKE, 0, 0, None, 0, None) == S.SPADE_ERR_INVALID_ARG
    assert L.spade_block_reorder(ctypes.byref(g), FAKE, FAKE, 0, 0, None, 0, None) == S.SPADE_ERR_INVALID_ARG  # alias
    assert L.spade_block_reorder(ctypes.byref(g), FAKE, MISALIGNED, 0, 0, None, 0, None) == S.SPADE_ERR_INVALID_ARG
    assert L.spade_block_reorder(ctypes.byref(g), FAKE, ctypes.c_void_p(0x2000), 7, 0, None, 0, None) == S.SPADE_ERR_INVALID_ARG
    assert L.spade_block_reorder(ctypes.byref(g), FAKE, ctypes.c_void_p(0x2000), 0, 2, None, 0, None) == S.SPADE_ERR_INVALID_ARG


def _heads(*hs):
    return (ctypes.c_int32 * max(len(hs), 1))(*hs)


@pytest.mark.parametrize("heads,n,expect", [
    (None, 1, S.SPADE_ERR_INVALID_ARG),            # null list needs n_heads == 0
    ((0, 2), 2, S.SPADE_ERR_INVALID_ARG),           # head 2 outside [0, H=2)
    ((1, -1), 2, S.SPADE_ERR_INVALID_ARG),          # negative head
    ((1, 1), 2, S.SPADE_ERR_INVALID_ARG),           # duplicate
    ((0,), -1, S.SPADE_ERR_INVALID_ARG),            # negative count
    (tuple(range(65)), 65, S.SPADE_ERR_INVALID_ARG),  # more than 64 heads
    ((1,), 0, S.SPADE_OK),                          # empty list: nothing to move
])
def test_reorder_head_list_errors(heads, n, expect):
    L = S.lib()
    g = _g(H=2) if n != 65 else _g(H=100)
    arr = None if heads is None else _heads(*heads)
    for inverse in (0, 1):
        st = L.spade_block_reorder(ctypes.byref(g), FAKE, ctypes.c_void_p(0x2000), 0, inverse,
                                   arr, n, None)
        assert st == expect, (heads, n, inverse)


def test_block_summarize_errors():
    L = S.lib()
    g = _g()
    B2 = ctypes.c_void_p(0x2000)
    call = lambda *a: L.spade_block_summarize(ctypes.byref(g), *a)
    # pairs must come together; something must be requested
    assert call(FAKE, B2, FAKE, NULL, NULL, NULL, NULL, NULL, None, 0, None) == S.SPADE_ERR_INVALID_ARG
    assert call(FAKE, B2, NULL, NULL, FAKE, NULL, NULL, NULL, None, 0, None) == S.SPADE_ERR_INVALID_ARG
    assert call(FAKE, B2, NULL, NULL, NULL, NULL, FAKE, NULL, None, 0, None) == S.SPADE_ERR_INVALID_ARG
    assert call(FAKE, B2, NULL, NULL, NULL, NULL, NULL, NULL, None, 0, None) == S.SPADE_ERR_INVALID_ARG
    # null or misaligned inputs, aliasing outputs
    assert call(NULL, B2, NULL, NULL, FAKE, FAKE, NULL, NULL, None, 0, None) == S.SPADE_ERR_INVALID_ARG
    assert call(FAKE, MISALIGNED, NULL, NULL, FAKE, FAKE, NULL, NULL, None, 0, None) == S.SPADE_ERR_INVALID_ARG
    assert call(FAKE, B2, FAKE, ctypes.c_void_p(0x3000), NULL, NULL, NULL, NULL, None, 0, None) == S.SPADE_ERR_INVALID_ARG
    # head list checks as for the reorder
    assert call(FAKE, B2, NULL, NULL, FAKE, FAKE, NULL, NULL, _heads(0, 2), 2, None) == S.SPADE_ERR_INVALID_ARG
    assert call(FAKE, B2, NULL, NULL, FAKE, FAKE, NULL, NULL, None, 1, None) == S.SPADE_ERR_INVALID_ARG
    assert L.spade_block_summarize(ctypes.byref(_g(d=96)), FAKE, B2, NULL, NULL, FAKE, FAKE, NULL,
                                   NULL, None, 0, None) == S.SPADE_ERR_UNSUPPORTED


def test_aggregation_and_choice_errors():
    L = S.lib()
    g = _g()
    assert L.spade_aggregation_score(ctypes.byref(g), FAKE, NULL, NULL, NULL, FAKE, None) == S.SPADE_ERR_INVALID_ARG
    assert L.spade_aggregation_score(ctypes.byref(g), FAKE, FAKE, FAKE, FAKE, NULL, None) == S.SPADE_ERR_INVALID_ARG
    assert L.spade_aggregation_score(ctypes.byref(_g(d=96)), FAKE, FAKE, NULL, NULL, FAKE, None) == S.SPADE_ERR_UNSUPPORTED
    assert L.spade_choose_scheme(FAKE, 0, 1, 2, FAKE, NULL, None) == S.SPADE_ERR_INVALID_ARG
    assert L.spade_choose_scheme(FAKE, 1025, 1, 2, FAKE, NULL, None) == S.SPADE_ERR_INVALID_ARG
    assert L.spade_choose_scheme(FAKE, 2, -1, 2, FAKE, NULL, None) == S.SPADE_ERR_INVALID_ARG
    assert L.spade_choose_scheme(NULL, 2, 1, 2, FAKE, NULL, None) == S.SPADE_ERR_INVALID_ARG
    assert L.spade_choose_scheme(FAKE, 2, 1, 2, NULL, NULL, None) == S.SPADE_ERR_INVALID_ARG
    assert L.spade_choose_scheme(NULL, 2, 0, 2, NULL, NULL, None) == S.SPADE_OK
    assert L.spade_choose_scheme(NULL, 2, 1, 0, NULL, NULL, None) == S.SPADE_OK


def test_empty_problem_is_a_no_op():
    L = S.lib()
    for kw in (dict(B=0), dict(H=0), dict(T=0)):
        g = _g(**kw)
        assert L.spade_block_reorder(ctypes.byref(g), NULL, NULL, 0, 0, None, 0, None) == S.SPADE_OK
        assert L.spade_summarize(ctypes.byref(g), NULL, NULL, NULL, NULL, NULL, NULL, None) == S.SPADE_OK
        assert L.spade_aggregation_score(ctypes.byref(g), NULL, NULL, NULL, NULL, NULL, None) == S.SPADE_OK
        assert L.spade_block_summarize(ctypes.byref(g), NULL, NULL, NULL, NULL, FAKE, FAKE, NULL, NULL,
                                       None, 0, None) == S.SPADE_OK
        assert L.spade_estimate_select(ctypes.byref(g), NULL, NULL, 0, 1, 0.0, 1.0, NULL, NULL, NULL, None) == S.SPADE_OK
        assert L.spade_attn_workspace_bytes(ctypes.byref(g)) == 0
        assert L.spade_block_sparse_attn(ctypes.byref(g), NULL, NULL, NULL, NULL, NULL, 1.0,
                                         NULL, NULL, NULL, 0, None) == S.SPADE_OK


def test_summarize_errors():
    L = S.lib()
    g = _g()
    assert L.spade_summarize(ctypes.byref(g), FAKE, NULL, FAKE, FAKE, NULL, NULL, None) == S.SPADE_ERR_INVALID_ARG
    assert L.spade_summarize(ctypes.byref(g), FAKE, FAKE, FAKE, FAKE, FAKE, NULL, None) == S.SPADE_ERR_INVALID_ARG


@pytest.mark.parametrize("mode,topk,tau,scale,expect", [
    (2, 1, 0.5, 1.0, S.SPADE_ERR_INVALID_ARG),
    (S.SPADE_TOPK, 0, 0.5, 1.0, S.SPADE_ERR_INVALID_ARG),
    (S.SPADE_TOPP, 1, 0.0, 1.0, S.SPADE_ERR_INVALID_ARG),
    (S.SPADE_TOPP, 1, 1.5, 1.0, S.SPADE_ERR_INVALID_ARG),
    (S.SPADE_TOPP, 1, float("nan"), 1.0, S.SPADE_ERR_INVALID_ARG),
    (S.SPADE_TOPK, 1, 0.5, 0.0, S.SPADE_ERR_INVALID_ARG),
    (S.SPADE_TOPK, 1, 0.5, float("inf"), S.SPADE_ERR_INVALID_ARG),
])
def test_select_parameter_errors(mode, topk, tau, scale, expect):
    L = S.lib()
    g = _g()
    st = L.spade_estimate_select(ctypes.byref(g), FAKE, FAKE, mode, topk, tau, scale, FAKE, FAKE, NULL, None)
    assert st == expect


def test_select_block_count_limit():
    L = S.lib()
    g = _g(T=64, Hs=64, Ws=64, bt=2, bh=2, bw=2)  # NB = 32768 > 1024
    st = L.spade_estimate_select(ctypes.byref(g), FAKE, FAKE, 0, 1, 0.5, 1.0, FAKE, FAKE, NULL, None)
    assert st == S.SPADE_ERR_UNSUPPORTED


def test_attention_block_count_limit():
    L = S.lib()
    g = _g(T=64, Hs=64, Ws=64, bt=1, bh=2, bw=2)  # NB = 65536 > 16384
    st = L.spade_block_sparse_attn(ctypes.byref(g), FAKE, FAKE, FAKE, FAKE, FAKE, 0.125, FAKE,
                                   NULL, FAKE, 0, None)
    assert st == S.SPADE_ERR_UNSUPPORTED


def test_attention_workspace_and_pointer_errors():
    L = S.lib()
    g = _g()
    need = L.spade_attn_workspace_bytes(ctypes.byref(g))
    st = L.spade_block_sparse_attn(ctypes.byref(g), FAKE, FAKE, NULL, FAKE, FAKE, 0.125, FAKE,
                                   NULL, FAKE, need, None)
    assert st == S.SPADE_ERR_INVALID_ARG
    if need > 0:
        st = L.spade_block_sparse_attn(ctypes.byref(g), FAKE, FAKE, FAKE, FAKE, FAKE, 0.125, FAKE,
                                       NULL, FAKE, need - 1, None)
        assert st == S.SPADE_ERR_WORKSPACE
    st = L.spade_block_sparse_attn(ctypes.byref(g), FAKE, FAKE, FAKE, FAKE, FAKE, -1.0, FAKE,
                                   NULL, FAKE, need, None)
    assert st == S.SPADE_ERR_INVALID_ARG
    # the ranked work order: 16 bytes per (batch, head) pair (keys, order, and the
    # first items a multi-scheme launch keeps)
    assert need == g.B * g.H * 16
    st = L.spade_block_sparse_attn(ctypes.byref(g), FAKE, FAKE, FAKE, FAKE, FAKE, 0.125, FAKE,
                                   NULL, NULL, need, None)
    assert st == S.SPADE_ERR_WORKSPACE
    st = L.spade_block_sparse_attn(ctypes.byref(g), FAKE, FAKE, FAKE, FAKE, FAKE, 0.125, FAKE,
                                   NULL, MISALIGNED, need, None)
    assert st == S.SPADE_ERR_WORKSPACE


def test_python_binding_raises_with_message():
    g = _g(d=96)
    with pytest.raises(S.SpadeError, match="head dim"):
        S._check(S.lib().spade_block_reorder(ctypes.byref(g), FAKE, FAKE, 0, 0, None, 0, None))


def _summ(**kw):
    f = dict(qbar=0x1000, kbar=0x1000, qmax=0x1000, qmin=0x1000, kmax=0x1000, kmin=0x1000,
             sics_q=0x1000, sics_k=0x1000)
    f.update(kw)
    return S.spade_summaries(*[f[k] for k in ("qbar", "kbar", "qmax", "qmin", "kmax", "kmin",
                                              "sics_q", "sics_k")])


def _spec(**kw):
    f = dict(estimator=S.SPADE_EST_DSA, mode=S.SPADE_TOPK, topk=4, tau=0.9, scale=0.1)
    f.update(kw)
    return S.mask_spec(**f)


@pytest.mark.parametrize("spec,summ,expect", [
    (dict(estimator=3), {}, S.SPADE_ERR_INVALID_ARG),
    (dict(mode=2), {}, S.SPADE_ERR_INVALID_ARG),
    (dict(topk=0), {}, S.SPADE_ERR_INVALID_ARG),
    (dict(mode=S.SPADE_TOPP, tau=0.0), {}, S.SPADE_ERR_INVALID_ARG),
    (dict(mode=S.SPADE_TOPP, tau=1.5), {}, S.SPADE_ERR_INVALID_ARG),
    (dict(scale=0.0), {}, S.SPADE_ERR_INVALID_ARG),
    (dict(intra=3), {}, S.SPADE_ERR_INVALID_ARG),
    (dict(intra=S.SPADE_INTRA_TOPK, intra_topk=-1), {}, S.SPADE_ERR_INVALID_ARG),
    (dict(intra=S.SPADE_INTRA_THRESHOLD, intra_theta=float("nan")), {}, S.SPADE_ERR_INVALID_ARG),
    (dict(sink_tokens=-1), {}, S.SPADE_ERR_INVALID_ARG),
    (dict(), dict(kmin=None), S.SPADE_ERR_INVALID_ARG),            # DSA needs max and min
    (dict(estimator=S.SPADE_EST_MEAN), dict(qbar=None), S.SPADE_ERR_INVALID_ARG),
    (dict(intra=S.SPADE_INTRA_THRESHOLD, intra_theta=0.5), dict(sics_k=None),
     S.SPADE_ERR_INVALID_ARG),
    (dict(), dict(qmax=0x1008), S.SPADE_ERR_INVALID_ARG),          # misaligned summary
])
def test_compose_select_errors(spec, summ, expect):
    L = S.lib()
    g = _g()
    st = L.spade_compose_select(ctypes.byref(g), ctypes.byref(_spec(**spec)), ctypes.byref(_summ(**summ)),
                                FAKE, FAKE, NULL, None)
    assert st == expect, S.lib().spade_last_error().decode()


def test_compose_select_null_structs_and_limits():
    L = S.lib()
    g = _g()
    assert L.spade_compose_select(ctypes.byref(g), None, ctypes.byref(_summ()), FAKE, FAKE, NULL,
                                  None) == S.SPADE_ERR_INVALID_ARG
    assert L.spade_compose_select(ctypes.byref(g), ctypes.byref(_spec()), None, FAKE, FAKE, NULL,
                                  None) == S.SPADE_ERR_INVALID_ARG
    assert L.spade_compose_select(ctypes.byref(g), ctypes.byref(_spec()), ctypes.byref(_summ()),
                                  NULL, FAKE, NULL, None) == S.SPADE_ERR_INVALID_ARG
    big = _g(T=64, Hs=64, Ws=64, bt=2, bh=2, bw=4)               # NB = 32*32*16 > 1024
    assert L.spade_compose_select(ctypes.byref(big), ctypes.byref(_spec()), ctypes.byref(_summ()),
                                  FAKE, FAKE, NULL, None) == S.SPADE_ERR_UNSUPPORTED
    empty = _g(B=0)
    assert L.spade_compose_select(ctypes.byref(empty), ctypes.byref(_spec()), ctypes.byref(_summ()),
                                  NULL, NULL, NULL, None) == S.SPADE_OK


def test_block_minmax_errors():
    L = S.lib()
    g = _g()
    args = [FAKE] * 6
    assert L.spade_block_minmax(ctypes.byref(g), *args[:5], NULL, NULL, NULL, None, 0,
                                None) == S.SPADE_ERR_INVALID_ARG     # kmin missing
    assert L.spade_block_minmax(ctypes.byref(g), *args, FAKE, NULL, None, 0,
                                None) == S.SPADE_ERR_INVALID_ARG     # one SICS output only
    assert L.spade_block_minmax(ctypes.byref(g), MISALIGNED, *args[1:], NULL, NULL, None, 0,
                                None) == S.SPADE_ERR_INVALID_ARG
    bad = _heads(0, 0)
    assert L.spade_block_minmax(ctypes.byref(g), *args, NULL, NULL, bad, 2,
                                None) == S.SPADE_ERR_INVALID_ARG     # duplicate head
    assert L.spade_block_minmax(ctypes.byref(_g(H=0)), NULL, NULL, NULL, NULL, NULL, NULL, NULL,
                                NULL, None, 0, None) == S.SPADE_OK


def test_policy_budgets_errors():
    L = S.lib()
    ok = L.spade_policy_budgets
    assert ok(FAKE, -1, None, 0, 4, 10, FAKE, None) == S.SPADE_ERR_INVALID_ARG      # negative H
    assert ok(FAKE, 4, None, 0, 0, 10, FAKE, None) == S.SPADE_ERR_INVALID_ARG       # k_dyn < 1
    assert ok(FAKE, 4, None, 0, 4, 0, FAKE, None) == S.SPADE_ERR_INVALID_ARG        # NB < 1
    assert ok(NULL, 4, None, 0, 4, 10, FAKE, None) == S.SPADE_ERR_INVALID_ARG       # null input
    assert ok(FAKE, 4, _heads(0, 4), 2, 4, 10, FAKE, None) == S.SPADE_ERR_INVALID_ARG  # head 4 >= H
    assert ok(FAKE, 4, _heads(1, 1), 2, 4, 10, FAKE, None) == S.SPADE_ERR_INVALID_ARG  # duplicate
    assert ok(NULL, 0, None, 0, 4, 10, NULL, None) == S.SPADE_OK                     # H = 0: no-op


def test_candidate_sics_errors():
    L = S.lib()
    fn = L.spade_candidate_sics
    P2 = (ctypes.c_void_p * 2)(0x1000, 0x1000)
    g1, g2 = _g(), _g(bt=1, bh=8, bw=2)
    two = (S.spade_geom * 2)(g1, g2)
    assert fn(two, 0, FAKE, FAKE, P2, P2, None) == S.SPADE_ERR_INVALID_ARG      # no geometry
    assert fn(two, 9, FAKE, FAKE, P2, P2, None) == S.SPADE_ERR_INVALID_ARG      # above 8
    other = (S.spade_geom * 2)(g1, _g(T=5, bt=1, bh=8, bw=2))
    assert fn(other, 2, FAKE, FAKE, P2, P2, None) == S.SPADE_ERR_INVALID_ARG    # grids differ
    assert fn(two, 2, NULL, FAKE, P2, P2, None) == S.SPADE_ERR_INVALID_ARG      # null q
    assert fn(two, 2, MISALIGNED, FAKE, P2, P2, None) == S.SPADE_ERR_INVALID_ARG
    P0 = (ctypes.c_void_p * 2)(0x1000, 0)
    assert fn(two, 2, FAKE, FAKE, P0, P2, None) == S.SPADE_ERR_INVALID_ARG      # null sics_q[1]
    # pairwise coprime extents: the common region is cut into too many cells
    big = _g(T=64, Hs=64, Ws=64)
    coprime = (S.spade_geom * 4)(*[S.spade_geom(1, 2, 128, 64, 64, 64, e, 1, 1) for e in (7, 11, 13, 17)])
    st, msg = _status(fn, coprime, 4, FAKE, FAKE, (ctypes.c_void_p * 4)(*[0x1000] * 4),
                      (ctypes.c_void_p * 4)(*[0x1000] * 4), None)
    assert st == S.SPADE_ERR_UNSUPPORTED and "cells" in msg, msg
    del big
    empty = (S.spade_geom * 1)(_g(B=0))
    assert fn(empty, 1, NULL, NULL, NULL, NULL, None) == S.SPADE_OK              # empty: no-op


def test_policy_tau_errors():
    ok = S.lib().spade_policy_tau
    assert ok(FAKE, -1, None, 0, 0.9, FAKE, None) == S.SPADE_ERR_INVALID_ARG        # negative H
    assert ok(FAKE, 4, None, 0, 0.0, FAKE, None) == S.SPADE_ERR_INVALID_ARG         # tau = 0
    assert ok(FAKE, 4, None, 0, 1.5, FAKE, None) == S.SPADE_ERR_INVALID_ARG         # tau > 1
    assert ok(FAKE, 4, None, 0, float("nan"), FAKE, None) == S.SPADE_ERR_INVALID_ARG
    assert ok(FAKE, 4, None, 0, 0.9, NULL, None) == S.SPADE_ERR_INVALID_ARG         # null output
    assert ok(FAKE, 4, _heads(0, 4), 2, 0.9, FAKE, None) == S.SPADE_ERR_INVALID_ARG  # head 4 >= H
    assert ok(NULL, 0, None, 0, 0.9, NULL, None) == S.SPADE_OK                      # H = 0: no-op


def test_multi_scheme_attention_errors():
    L = S.lib()
    g1, g2 = _g(), _g(bt=1, bh=8, bw=2)
    geoms = (S.spade_geom * 2)(g1, g2)
    heads = (S.spade_head_lists * 2)(S.spade_head_lists(0, 0x1000, 0x1000, 0, 0),
                                     S.spade_head_lists(1, 0x1000, 0x1000, 0, 0))
    call = lambda gs, n, hs, scale=0.1: L.spade_sparse_attn_raster_multi(  # noqa: E731
        gs, n, hs, FAKE, FAKE, FAKE, scale, FAKE, NULL, NULL, 0, None)
    assert call(geoms, 0, heads) == S.SPADE_ERR_INVALID_ARG                  # no geometry
    assert call(geoms, 9, heads) == S.SPADE_ERR_INVALID_ARG                  # more than 8
    assert call(geoms, 2, heads, scale=0.0) == S.SPADE_ERR_INVALID_ARG
    other = (S.spade_geom * 2)(g1, _g(T=6))                                  # different grid
    assert call(other, 2, heads) == S.SPADE_ERR_INVALID_ARG
    bad = (S.spade_head_lists * 2)(S.spade_head_lists(0, 0x1000, 0x1000, 0, 0),
                                   S.spade_head_lists(2, 0x1000, 0x1000, 0, 0))
    assert call(geoms, 2, bad) == S.SPADE_ERR_INVALID_ARG                    # scheme 2 of 2
    nul = (S.spade_head_lists * 2)(S.spade_head_lists(0, 0x1000, 0x1000, 0, 0),
                                   S.spade_head_lists(1, 0, 0x1000, 0, 0))
    assert call(geoms, 2, nul) == S.SPADE_ERR_INVALID_ARG                    # null counts
    assert call(geoms, 2, None) == S.SPADE_ERR_INVALID_ARG
    many = (S.spade_geom * 1)(_g(H=65))
    assert call(many, 1, heads) == S.SPADE_ERR_UNSUPPORTED                   # H > 64
    empty = (S.spade_geom * 1)(_g(B=0))
    assert call(empty, 1, None) == S.SPADE_OK
    # the workspace of the per-launch head ranking
    need = L.spade_attn_workspace_bytes(ctypes.byref(g1))
    assert need == g1.B * g1.H * 16
    ws_call = lambda ws, n: L.spade_sparse_attn_raster_multi(  # noqa: E731
        geoms, 2, heads, FAKE, FAKE, FAKE, 0.1, FAKE, NULL, ws, n, None)
    assert ws_call(NULL, need) == S.SPADE_ERR_WORKSPACE
    assert ws_call(FAKE, need - 1) == S.SPADE_ERR_WORKSPACE
    assert ws_call(MISALIGNED, need) == S.SPADE_ERR_WORKSPACE


def test_validate_lists_errors():
    fn = S.lib().spade_validate_lists
    g = _g()
    assert fn(ctypes.byref(g), FAKE, FAKE, NULL, None) == S.SPADE_ERR_INVALID_ARG   # null report
    assert fn(ctypes.byref(g), NULL, FAKE, FAKE, None) == S.SPADE_ERR_INVALID_ARG   # null counts
    assert fn(ctypes.byref(g), FAKE, NULL, FAKE, None) == S.SPADE_ERR_INVALID_ARG   # null indices
    assert fn(ctypes.byref(_g(d=96)), FAKE, FAKE, FAKE, None) == S.SPADE_ERR_UNSUPPORTED
    assert fn(ctypes.byref(_g(bt=0)), FAKE, FAKE, FAKE, None) == S.SPADE_ERR_INVALID_ARG
    # one-token blocks, d = 64: 65535 * 33792 rows > 2^31 - 1, tensors still within limits
    big = _g(B=1, H=65535, d=64, T=32, Hs=32, Ws=33, bt=1, bh=1, bw=1)
    st, msg = _status(fn, ctypes.byref(big), FAKE, FAKE, FAKE, None)
    assert st == S.SPADE_ERR_UNSUPPORTED and "rows" in msg
