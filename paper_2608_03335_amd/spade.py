"""Thin ctypes binding of libspade.so: same names as the C ABI, argument marshalling only.

Tensors are torch tensors used as device buffers; every step of the path runs in
the library's HIP kernels. Each function raises SpadeError when the library
returns a non-OK status. Calls are asynchronous on the given HIP stream
(default: torch's current stream).
"""
from __future__ import annotations

import ctypes
import os

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libspade.so")

SPADE_OK, SPADE_ERR_INVALID_ARG, SPADE_ERR_UNSUPPORTED, SPADE_ERR_WORKSPACE, SPADE_ERR_HIP = range(5)
SPADE_BF16, SPADE_FP32 = 0, 1
SPADE_TOPK, SPADE_TOPP = 0, 1
SPADE_EST_MEAN, SPADE_EST_DSA, SPADE_EST_DSA2 = 0, 1, 2
SPADE_INTRA_NONE, SPADE_INTRA_THRESHOLD, SPADE_INTRA_TOPK = 0, 1, 2

EXPORTED = ("spade_block_reorder", "spade_summarize", "spade_block_summarize",
            "spade_aggregation_score",
            "spade_choose_scheme", "spade_estimate_select", "spade_block_minmax",
            "spade_compose_select", "spade_policy_budgets", "spade_attn_workspace_bytes",
            "spade_block_sparse_attn", "spade_sparse_attn_raster",
            "spade_sparse_attn_raster_multi", "spade_status_string",
            "spade_last_error")
MAX_HEAD_LIST = 64


class SpadeError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{message} (status {status})")
        self.status = status


class spade_geom(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("B", "H", "d", "T", "Hs", "Ws", "bt", "bh", "bw")]

    @property
    def BS(self) -> int:
        return self.bt * self.bh * self.bw

    @property
    def NB(self) -> int:
        return (-(-self.T // self.bt)) * (-(-self.Hs // self.bh)) * (-(-self.Ws // self.bw))

    @property
    def N(self) -> int:
        return self.T * self.Hs * self.Ws


def geom(B, H, d, T, Hs, Ws, bt, bh, bw) -> spade_geom:
    return spade_geom(B, H, d, T, Hs, Ws, bt, bh, bw)


class spade_head_lists(ctypes.Structure):
    _fields_ = [("scheme", ctypes.c_int32), ("counts", ctypes.c_void_p),
                ("indices", ctypes.c_void_p), ("counts_bstride", ctypes.c_int64),
                ("indices_bstride", ctypes.c_int64)]


class spade_summaries(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("qbar", "kbar", "qmax", "qmin", "kmax", "kmin",
                                               "sics_q", "sics_k")]


class spade_mask_spec(ctypes.Structure):
    _fields_ = [("estimator", ctypes.c_int32), ("mode", ctypes.c_int32), ("topk", ctypes.c_int32),
                ("tau", ctypes.c_double), ("scale", ctypes.c_double),
                ("topk_per_head", ctypes.c_void_p), ("tau_per_head", ctypes.c_void_p),
                ("intra", ctypes.c_int32), ("intra_topk", ctypes.c_int32),
                ("intra_theta", ctypes.c_double), ("window", ctypes.c_int32 * 3),
                ("sink_tokens", ctypes.c_int64)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libspade.so; raise if it has not been built (no fallback exists)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with "
                               "`python -m paper_2608_03335_amd.build_lib`")
        L = ctypes.CDLL(_LIB_PATH)
        vp, i32, f64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_double, ctypes.c_size_t
        G = ctypes.POINTER(spade_geom)
        sig = {
            "spade_block_reorder": (i32, [G, vp, vp, i32, i32, ctypes.POINTER(i32), i32, vp]),
            "spade_summarize": (i32, [G, vp, vp, vp, vp, vp, vp, vp]),
            "spade_block_summarize": (i32, [G, vp, vp, vp, vp, vp, vp, vp, vp,
                                            ctypes.POINTER(i32), i32, vp]),
            "spade_aggregation_score": (i32, [G, vp, vp, vp, vp, vp, vp]),
            "spade_choose_scheme": (i32, [vp, i32, i32, i32, vp, vp, vp]),
            "spade_estimate_select": (i32, [G, vp, vp, i32, i32, f64, f64, vp, vp, vp, vp]),
            "spade_block_minmax": (i32, [G, vp, vp, vp, vp, vp, vp, vp, vp,
                                         ctypes.POINTER(i32), i32, vp]),
            "spade_compose_select": (i32, [G, ctypes.POINTER(spade_mask_spec),
                                           ctypes.POINTER(spade_summaries), vp, vp, vp, vp]),
            "spade_policy_budgets": (i32, [vp, i32, ctypes.POINTER(i32), i32, i32, i32, vp, vp]),
            "spade_attn_workspace_bytes": (sz, [G]),
            "spade_block_sparse_attn": (i32, [G, vp, vp, vp, vp, vp, f64, vp, vp, vp, sz, vp]),
            "spade_sparse_attn_raster": (i32, [G, vp, vp, vp, vp, vp, f64, vp, vp, vp, sz, vp]),
            "spade_sparse_attn_raster_multi": (i32, [G, i32, ctypes.POINTER(spade_head_lists), vp,
                                                     vp, vp, f64, vp, vp, vp, sz, vp]),
            "spade_status_string": (ctypes.c_char_p, [i32]),
            "spade_last_error": (ctypes.c_char_p, []),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype, fn.argtypes = res, args
        _lib = L
    return _lib


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _s(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _check(status: int):
    if status != SPADE_OK:
        L = lib()
        raise SpadeError(status, f"{L.spade_status_string(status).decode()}: "
                                 f"{L.spade_last_error().decode()}")


def _head_list(heads):
    if heads is None:
        return None, 0
    hs = [int(h) for h in heads]
    return (ctypes.c_int32 * max(len(hs), 1))(*hs), len(hs)


def spade_block_reorder(g: spade_geom, x, y, inverse: bool = False, heads=None, stream=None):
    """heads: None (all heads) or a sequence of head indices (the group's heads)."""
    dtype = SPADE_BF16 if x.dtype == torch.bfloat16 else SPADE_FP32
    arr, n = _head_list(heads)
    _check(lib().spade_block_reorder(ctypes.byref(g), _p(x), _p(y), dtype, int(inverse), arr, n,
                                     _s(stream)))


def spade_summarize(g: spade_geom, qb, kb, qbar, kbar, sics_q=None, sics_k=None, stream=None):
    _check(lib().spade_summarize(ctypes.byref(g), _p(qb), _p(kb), _p(qbar), _p(kbar),
                                 _p(sics_q), _p(sics_k), _s(stream)))


def spade_block_summarize(g: spade_geom, q, k, qb=None, kb=None, qbar=None, kbar=None,
                          sics_q=None, sics_k=None, heads=None, stream=None):
    arr, n = _head_list(heads)
    _check(lib().spade_block_summarize(ctypes.byref(g), _p(q), _p(k), _p(qb), _p(kb), _p(qbar),
                                       _p(kbar), _p(sics_q), _p(sics_k), arr, n, _s(stream)))


def spade_aggregation_score(g: spade_geom, sics_q, sics_k, as_qk, as_q=None, as_k=None,
                            stream=None):
    _check(lib().spade_aggregation_score(ctypes.byref(g), _p(sics_q), _p(sics_k), _p(as_q),
                                         _p(as_k), _p(as_qk), _s(stream)))


def spade_choose_scheme(as_qk, choice, best=None, stream=None):
    """as_qk: fp64 [C, B, H] device tensor; choice: int32 [H]; best: fp64 [H] or None."""
    C, B, H = as_qk.shape
    _check(lib().spade_choose_scheme(_p(as_qk), int(C), int(B), int(H), _p(choice), _p(best),
                                     _s(stream)))


def spade_estimate_select(g: spade_geom, qbar, kbar, mode: int, topk: int, tau: float,
                          scale: float, counts, indices, scores=None, stream=None):
    _check(lib().spade_estimate_select(ctypes.byref(g), _p(qbar), _p(kbar), int(mode), int(topk),
                                       float(tau), float(scale), _p(counts), _p(indices),
                                       _p(scores), _s(stream)))


def spade_block_minmax(g: spade_geom, q, k, qmax, qmin, kmax, kmin, sics_q=None, sics_k=None,
                       heads=None, stream=None):
    arr, n = _head_list(heads)
    _check(lib().spade_block_minmax(ctypes.byref(g), _p(q), _p(k), _p(qmax), _p(qmin), _p(kmax),
                                    _p(kmin), _p(sics_q), _p(sics_k), arr, n, _s(stream)))


def mask_spec(estimator=SPADE_EST_MEAN, mode=SPADE_TOPK, topk=0, tau=1.0, scale=1.0,
              topk_per_head=None, tau_per_head=None, intra=SPADE_INTRA_NONE, intra_topk=0,
              intra_theta=0.0, window=(-1, -1, -1), sink_tokens=0) -> spade_mask_spec:
    """topk_per_head / tau_per_head: None or device tensors (int32 / fp64, [H]); the
    caller keeps them alive until the call has run on its stream."""
    return spade_mask_spec(int(estimator), int(mode), int(topk), float(tau), float(scale),
                           None if topk_per_head is None else topk_per_head.data_ptr(),
                           None if tau_per_head is None else tau_per_head.data_ptr(),
                           int(intra), int(intra_topk), float(intra_theta),
                           (ctypes.c_int32 * 3)(*[int(w) for w in window]), int(sink_tokens))


def summaries(qbar=None, kbar=None, qmax=None, qmin=None, kmax=None, kmin=None, sics_q=None,
              sics_k=None) -> spade_summaries:
    ptr = lambda t: None if t is None else t.data_ptr()  # noqa: E731
    return spade_summaries(ptr(qbar), ptr(kbar), ptr(qmax), ptr(qmin), ptr(kmax), ptr(kmin),
                           ptr(sics_q), ptr(sics_k))


def spade_compose_select(g: spade_geom, spec: spade_mask_spec, summ: spade_summaries, counts,
                         indices, scores=None, stream=None):
    _check(lib().spade_compose_select(ctypes.byref(g), ctypes.byref(spec), ctypes.byref(summ),
                                      _p(counts), _p(indices), _p(scores), _s(stream)))


def spade_sparse_attn_raster_multi(geoms, heads, q, k, v, scale: float, o, lse=None,
                                   workspace=None, stream=None):
    """geoms: sequence of spade_geom; heads: per head (scheme, counts, indices,
    counts_bstride, indices_bstride) with counts/indices device tensors (views at
    batch 0 of the head)."""
    ga = (spade_geom * len(geoms))(*geoms)
    ha = (spade_head_lists * max(len(heads), 1))(
        *[spade_head_lists(int(c), cn.data_ptr(), ix.data_ptr(), int(cs), int(xs))
          for c, cn, ix, cs, xs in heads])
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().spade_sparse_attn_raster_multi(ga, len(geoms), ha, _p(q), _p(k), _p(v),
                                                float(scale), _p(o), _p(lse), _p(workspace),
                                                nbytes, _s(stream)))


def spade_policy_budgets(as_best, k_dyn: int, NB: int, k_out, heads=None, stream=None):
    """as_best: fp64 [H] device tensor; k_out: int32 [len(heads) or H] device tensor."""
    arr, n = _head_list(heads)
    _check(lib().spade_policy_budgets(_p(as_best), int(as_best.numel()), arr, n, int(k_dyn),
                                      int(NB), _p(k_out), _s(stream)))


def spade_attn_workspace_bytes(g: spade_geom) -> int:
    return int(lib().spade_attn_workspace_bytes(ctypes.byref(g)))


def spade_block_sparse_attn(g: spade_geom, qb, kb, vb, counts, indices, scale: float, ob,
                            lse=None, workspace=None, stream=None):
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().spade_block_sparse_attn(ctypes.byref(g), _p(qb), _p(kb), _p(vb), _p(counts),
                                         _p(indices), float(scale), _p(ob), _p(lse),
                                         _p(workspace), nbytes, _s(stream)))


def spade_sparse_attn_raster(g: spade_geom, q, k, v, counts, indices, scale: float, o, lse=None,
                             workspace=None, stream=None):
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().spade_sparse_attn_raster(ctypes.byref(g), _p(q), _p(k), _p(v), _p(counts),
                                          _p(indices), float(scale), _p(o), _p(lse),
                                          _p(workspace), nbytes, _s(stream)))
