"""Thin ctypes binding of libspade.so: same names as the C ABI, argument marshalling only.

Tensors are torch tensors used as device buffers; every step of the path runs in
the library's HIP kernels. Each function raises SpadeError when the library
returns a non-OK status. Calls are asynchronous on the given HIP stream
(default: torch's current stream).

The C ABI sees plain pointers and cannot tell a host buffer, a strided view, the
wrong element type or a short buffer from a good one, so the binding checks each
tensor before passing its pointer: on the GPU, contiguous, of the element type
the header declares and at least as large as the geometry implies (raising
SpadeError with SPADE_ERR_INVALID_ARG otherwise).
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
SPADE_TASK_T2V, SPADE_TASK_I2V = 0, 1
SPADE_LIST_BAD_COUNT, SPADE_LIST_BAD_INDEX, SPADE_LIST_NOT_ASCENDING = 1, 2, 4

EXPORTED = ("spade_block_reorder", "spade_summarize", "spade_block_summarize",
            "spade_candidate_sics", "spade_aggregation_score",
            "spade_choose_scheme", "spade_estimate_select", "spade_block_minmax",
            "spade_compose_select", "spade_policy_budgets", "spade_policy_tau",
            "spade_policy_dense", "spade_policy_split", "spade_attn_workspace_bytes",
            "spade_block_sparse_attn", "spade_sparse_attn_raster",
            "spade_sparse_attn_raster_multi", "spade_sparse_attn_raster_noalloc",
            "spade_validate_lists", "spade_status_string",
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
            "spade_candidate_sics": (i32, [G, i32, vp, vp, ctypes.POINTER(vp), ctypes.POINTER(vp),
                                           vp]),
            "spade_choose_scheme": (i32, [vp, i32, i32, i32, vp, vp, vp]),
            "spade_estimate_select": (i32, [G, vp, vp, i32, i32, f64, f64, vp, vp, vp, vp]),
            "spade_block_minmax": (i32, [G, vp, vp, vp, vp, vp, vp, vp, vp,
                                         ctypes.POINTER(i32), i32, vp]),
            "spade_compose_select": (i32, [G, ctypes.POINTER(spade_mask_spec),
                                           ctypes.POINTER(spade_summaries), vp, vp, vp, vp]),
            "spade_policy_budgets": (i32, [vp, i32, ctypes.POINTER(i32), i32, i32, i32, vp, vp]),
            "spade_policy_tau": (i32, [vp, i32, ctypes.POINTER(i32), i32, f64, vp, vp]),
            "spade_policy_dense": (i32, [i32, i32, i32, i32, ctypes.POINTER(i32)]),
            "spade_policy_split": (i32, [i32, i32, ctypes.POINTER(i32), ctypes.POINTER(i32),
                                         ctypes.POINTER(i32)]),
            "spade_attn_workspace_bytes": (sz, [G]),
            "spade_block_sparse_attn": (i32, [G, vp, vp, vp, vp, vp, f64, vp, vp, vp, sz, vp]),
            "spade_sparse_attn_raster": (i32, [G, vp, vp, vp, vp, vp, f64, vp, vp, vp, sz, vp]),
            "spade_sparse_attn_raster_noalloc": (i32, [G, vp, vp, vp, vp, vp, f64, vp, vp, vp]),
            "spade_sparse_attn_raster_multi": (i32, [G, i32, ctypes.POINTER(spade_head_lists), vp,
                                                     vp, vp, f64, vp, vp, vp, sz, vp]),
            "spade_validate_lists": (i32, [G, vp, vp, vp, vp]),
            "spade_status_string": (ctypes.c_char_p, [i32]),
            "spade_last_error": (ctypes.c_char_p, []),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype, fn.argtypes = res, args
        _lib = L
    return _lib


BF16, F32, F64, I32 = torch.bfloat16, torch.float32, torch.float64, torch.int32


class _Args:
    """Checked device pointers of one call's tensors. Element type, layout and size
    are checked as each tensor is added (None passes as NULL; dtype None: any;
    numel None: unchecked), the device of all of them just before the call, so an
    argument mistake is reported before a placement one."""

    def __init__(self):
        self.host = None

    def __call__(self, t, dtype, numel, name):
        if t is None:
            return None
        if not isinstance(t, torch.Tensor):
            raise SpadeError(SPADE_ERR_INVALID_ARG, f"{name} must be a torch tensor")
        if dtype is not None and t.dtype != dtype:
            raise SpadeError(SPADE_ERR_INVALID_ARG, f"{name} must be {dtype} (got {t.dtype})")
        if not t.is_contiguous():
            raise SpadeError(SPADE_ERR_INVALID_ARG, f"{name} must be contiguous")
        if numel is not None and t.numel() < numel:
            raise SpadeError(SPADE_ERR_INVALID_ARG,
                             f"{name} holds {t.numel()} elements, {numel} needed")
        if not t.is_cuda and self.host is None:
            self.host = name
        return ctypes.c_void_p(t.data_ptr())

    def ready(self):
        if self.host is not None:
            raise SpadeError(SPADE_ERR_INVALID_ARG, f"{self.host} must be a GPU tensor")

    def run(self, fn, *args):
        """Calls fn once every tensor has passed; the stream (the last argument, as
        given by the caller) is resolved only then."""
        self.ready()
        return fn(*args[:-1], _s(args[-1]))


class _Dims:
    """Element counts of the tensors of one geometry (n: heads of the call), or
    None everywhere when the geometry is invalid (the library then rejects it)."""

    def __init__(self, g: spade_geom, n=None):
        ok = min(g.bt, g.bh, g.bw) >= 1 and min(g.B, g.H, g.T, g.Hs, g.Ws) >= 0
        nb = ((-(-g.T // g.bt)) * (-(-g.Hs // g.bh)) * (-(-g.Ws // g.bw))) if ok else 0
        bh = g.B * (g.H if n is None else n)
        full = g.B * g.H
        N = g.T * g.Hs * g.Ws
        BS = g.bt * g.bh * g.bw
        v = (lambda x: x if ok else None)  # noqa: E731
        self.raster = v(full * N * g.d)          # raster [B,H,N,d]
        self.raster_rows = v(full * N)           # raster [B,H,N]
        self.blocked = v(bh * nb * BS * g.d)     # blocked [B,n,NB*BS,d]
        self.blocked_rows = v(bh * nb * BS)      # blocked [B,n,NB*BS]
        self.summ = v(bh * nb * g.d)             # [B,n,NB,d]
        self.per_block = v(bh * nb)              # [B,n,NB]
        self.pairs = v(bh * nb * nb)             # [B,n,NB,NB]
        self.per_head = v(bh)                    # [B,n]
        self.NB = nb


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
    if not isinstance(x, torch.Tensor) or x.dtype not in (BF16, F32):
        raise SpadeError(SPADE_ERR_INVALID_ARG, "x must be a bfloat16 or float32 tensor")
    a = _Args()
    arr, n = _head_list(heads)
    D = _Dims(g, n if heads is not None else None)
    src, dst = (D.blocked, D.raster) if inverse else (D.raster, D.blocked)
    dtype = SPADE_BF16 if x.dtype == BF16 else SPADE_FP32
    _check(a.run(lib().spade_block_reorder, ctypes.byref(g), a(x, x.dtype, src, "x"),
                 a(y, x.dtype, dst, "y"), dtype, int(inverse), arr, n, stream))


def spade_summarize(g: spade_geom, qb, kb, qbar, kbar, sics_q=None, sics_k=None, stream=None):
    a = _Args()
    D = _Dims(g)
    _check(a.run(lib().spade_summarize, ctypes.byref(g), a(qb, BF16, D.blocked, "qb"),
                 a(kb, BF16, D.blocked, "kb"), a(qbar, F64, D.summ, "qbar"),
                 a(kbar, F64, D.summ, "kbar"), a(sics_q, F64, D.per_block, "sics_q"),
                 a(sics_k, F64, D.per_block, "sics_k"), stream))


def spade_block_summarize(g: spade_geom, q, k, qb=None, kb=None, qbar=None, kbar=None,
                          sics_q=None, sics_k=None, heads=None, stream=None):
    a = _Args()
    arr, n = _head_list(heads)
    D = _Dims(g, n if heads is not None else None)
    _check(a.run(lib().spade_block_summarize, ctypes.byref(g), a(q, BF16, D.raster, "q"),
                 a(k, BF16, D.raster, "k"), a(qb, BF16, D.blocked, "qb"),
                 a(kb, BF16, D.blocked, "kb"), a(qbar, F64, D.summ, "qbar"),
                 a(kbar, F64, D.summ, "kbar"), a(sics_q, F64, D.per_block, "sics_q"),
                 a(sics_k, F64, D.per_block, "sics_k"), arr, n, stream))


def spade_candidate_sics(geoms, q, k, sics_q, sics_k, stream=None):
    """geoms: sequence of spade_geom; sics_q / sics_k: per candidate a fp64 [B,H,NB_c]
    device tensor. Raises SpadeError(SPADE_ERR_UNSUPPORTED) when the candidates'
    common refinement does not fit (score them one at a time then)."""
    a = _Args()
    if len(sics_q) != len(geoms) or len(sics_k) != len(geoms):
        raise SpadeError(SPADE_ERR_INVALID_ARG, "one sics_q and one sics_k tensor per geometry")
    ga = (spade_geom * max(len(geoms), 1))(*geoms)
    D = _Dims(geoms[0]) if len(geoms) else None
    pq = (ctypes.c_void_p * max(len(geoms), 1))(
        *[_value(a(t, F64, _Dims(g).per_block, f"sics_q[{c}]")) for c, (g, t) in
          enumerate(zip(geoms, sics_q))])
    pk = (ctypes.c_void_p * max(len(geoms), 1))(
        *[_value(a(t, F64, _Dims(g).per_block, f"sics_k[{c}]")) for c, (g, t) in
          enumerate(zip(geoms, sics_k))])
    _check(a.run(lib().spade_candidate_sics, ga, len(geoms),
                 a(q, BF16, D.raster if D else None, "q"), a(k, BF16, D.raster if D else None, "k"),
                 pq, pk, stream))


def spade_aggregation_score(g: spade_geom, sics_q, sics_k, as_qk, as_q=None, as_k=None,
                            stream=None):
    a = _Args()
    D = _Dims(g)
    _check(a.run(lib().spade_aggregation_score, ctypes.byref(g),
                 a(sics_q, F64, D.per_block, "sics_q"), a(sics_k, F64, D.per_block, "sics_k"),
                 a(as_q, F64, D.per_head, "as_q"), a(as_k, F64, D.per_head, "as_k"),
                 a(as_qk, F64, D.per_head, "as_qk"), stream))


def spade_choose_scheme(as_qk, choice, best=None, stream=None):
    """as_qk: fp64 [C, B, H] device tensor; choice: int32 [H]; best: fp64 [H] or None."""
    a = _Args()
    C, B, H = as_qk.shape
    _check(a.run(lib().spade_choose_scheme, a(as_qk, F64, None, "as_qk"), int(C), int(B), int(H),
                 a(choice, I32, H, "choice"), a(best, F64, H, "best"), stream))


def spade_estimate_select(g: spade_geom, qbar, kbar, mode: int, topk: int, tau: float,
                          scale: float, counts, indices, scores=None, stream=None):
    a = _Args()
    D = _Dims(g)
    _check(a.run(lib().spade_estimate_select, ctypes.byref(g), a(qbar, F64, D.summ, "qbar"),
                 a(kbar, F64, D.summ, "kbar"), int(mode), int(topk), float(tau), float(scale),
                 a(counts, I32, D.per_block, "counts"), a(indices, I32, D.pairs, "indices"),
                 a(scores, F64, D.pairs, "scores"), stream))


def spade_block_minmax(g: spade_geom, q, k, qmax, qmin, kmax, kmin, sics_q=None, sics_k=None,
                       heads=None, stream=None):
    a = _Args()
    arr, n = _head_list(heads)
    D = _Dims(g, n if heads is not None else None)
    _check(a.run(lib().spade_block_minmax, ctypes.byref(g), a(q, BF16, D.raster, "q"),
                 a(k, BF16, D.raster, "k"), a(qmax, F64, D.summ, "qmax"),
                 a(qmin, F64, D.summ, "qmin"), a(kmax, F64, D.summ, "kmax"),
                 a(kmin, F64, D.summ, "kmin"), a(sics_q, F64, D.per_block, "sics_q"),
                 a(sics_k, F64, D.per_block, "sics_k"), arr, n, stream))


def _value(p):
    return None if p is None else p.value


def mask_spec(estimator=SPADE_EST_MEAN, mode=SPADE_TOPK, topk=0, tau=1.0, scale=1.0,
              topk_per_head=None, tau_per_head=None, intra=SPADE_INTRA_NONE, intra_topk=0,
              intra_theta=0.0, window=(-1, -1, -1), sink_tokens=0) -> spade_mask_spec:
    """topk_per_head / tau_per_head: None or device tensors (int32 / fp64, [H]); the
    caller keeps them alive until the call has run on its stream."""
    a = _Args()
    tk = a(topk_per_head, I32, None, "topk_per_head")
    tu = a(tau_per_head, F64, None, "tau_per_head")
    a.ready()
    return spade_mask_spec(int(estimator), int(mode), int(topk), float(tau), float(scale),
                           _value(tk), _value(tu), int(intra), int(intra_topk),
                           float(intra_theta), (ctypes.c_int32 * 3)(*[int(w) for w in window]),
                           int(sink_tokens))


def summaries(qbar=None, kbar=None, qmax=None, qmin=None, kmax=None, kmin=None, sics_q=None,
              sics_k=None) -> spade_summaries:
    """Device fp64 summary tensors of one selection call (None: not given)."""
    a = _Args()
    ptrs = [_value(a(t, F64, None, name)) for t, name in (
        (qbar, "qbar"), (kbar, "kbar"), (qmax, "qmax"), (qmin, "qmin"), (kmax, "kmax"),
        (kmin, "kmin"), (sics_q, "sics_q"), (sics_k, "sics_k"))]
    a.ready()
    return spade_summaries(*ptrs)


def spade_compose_select(g: spade_geom, spec: spade_mask_spec, summ: spade_summaries, counts,
                         indices, scores=None, stream=None):
    a = _Args()
    D = _Dims(g)
    _check(a.run(lib().spade_compose_select, ctypes.byref(g), ctypes.byref(spec),
                 ctypes.byref(summ), a(counts, I32, D.per_block, "counts"),
                 a(indices, I32, D.pairs, "indices"), a(scores, F64, D.pairs, "scores"),
                 stream))


def _storage_span(t, elems: int, name: str):
    """The view t must have `elems` elements of its storage from its first element on."""
    if not isinstance(t, torch.Tensor):
        return
    avail = t.untyped_storage().nbytes() // t.element_size() - t.storage_offset()
    if elems > avail:
        raise SpadeError(SPADE_ERR_INVALID_ARG,
                         f"{name}: the batch strides reach {elems} elements, storage holds {avail}")


def spade_sparse_attn_raster_multi(geoms, heads, q, k, v, scale: float, o, lse=None,
                                   workspace=None, stream=None):
    """geoms: sequence of spade_geom; heads: per head (scheme, counts, indices,
    counts_bstride, indices_bstride) with counts/indices device tensors (views at
    batch 0 of the head, at least NB and NB*NB elements of its blocking)."""
    a = _Args()
    ga = (spade_geom * len(geoms))(*geoms)
    heads = list(heads)
    # the library reads one entry per head of geometry 0: a short table would make it
    # read past the array (and hand garbage list pointers to the kernel)
    if len(geoms) and len(heads) != geoms[0].H:
        raise SpadeError(SPADE_ERR_INVALID_ARG,
                         f"heads has {len(heads)} entries, geometry 0 has H={geoms[0].H}")
    B = geoms[0].B if len(geoms) else 0
    rows = []
    for h, (c, cn, ix, cs, xs) in enumerate(heads):
        nb = _Dims(geoms[int(c)]).NB if 0 <= int(c) < len(geoms) else None
        pc = a(cn, I32, nb, f"heads[{h}] counts")
        pi = a(ix, I32, None if nb is None else nb * nb, f"heads[{h}] indices")
        if nb is not None and B > 1:
            # batch element b's lists start cs (xs) elements after batch 0's: the whole
            # span must lie inside the tensor's storage
            _storage_span(cn, (B - 1) * int(cs) + nb, f"heads[{h}] counts")
            _storage_span(ix, (B - 1) * int(xs) + nb * nb, f"heads[{h}] indices")
        rows.append(spade_head_lists(int(c), _value(pc), _value(pi), int(cs), int(xs)))
    ha = (spade_head_lists * max(len(rows), 1))(*rows)
    D = _Dims(geoms[0]) if len(geoms) else None
    n_rast = D.raster if D else None
    n_rows = D.raster_rows if D else None
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(a.run(lib().spade_sparse_attn_raster_multi, ga, len(geoms), ha,
                 a(q, BF16, n_rast, "q"), a(k, BF16, n_rast, "k"), a(v, BF16, n_rast, "v"),
                 float(scale), a(o, BF16, n_rast, "o"), a(lse, F32, n_rows, "lse"),
                 a(workspace, None, None, "workspace"), nbytes, stream))


def spade_policy_budgets(as_best, k_dyn: int, NB: int, k_out, heads=None, stream=None):
    """as_best: fp64 [H] device tensor; k_out: int32 [len(heads) or H] device tensor."""
    a = _Args()
    arr, n = _head_list(heads)
    H = int(as_best.numel())
    _check(a.run(lib().spade_policy_budgets, a(as_best, F64, None, "as_best"), H, arr, n,
                 int(k_dyn), int(NB), a(k_out, I32, n if heads is not None else H, "k_out"),
                 stream))


def spade_policy_tau(as_best, tau: float, tau_out, heads=None, stream=None):
    """as_best: fp64 [H] device tensor; tau_out: fp64 [len(heads) or H] device tensor."""
    a = _Args()
    arr, n = _head_list(heads)
    H = int(as_best.numel())
    _check(a.run(lib().spade_policy_tau, a(as_best, F64, None, "as_best"), H, arr, n, float(tau),
                 a(tau_out, F64, n if heads is not None else H, "tau_out"), stream))


def spade_policy_dense(step: int, n_steps: int, task: int = SPADE_TASK_T2V,
                       turbo: bool = False) -> bool:
    """Host call: does denoising step `step` of n_steps run full attention?"""
    out = ctypes.c_int32(0)
    _check(lib().spade_policy_dense(int(step), int(n_steps), int(task), int(bool(turbo)),
                                    ctypes.byref(out)))
    return bool(out.value)


def spade_policy_split(k_total: int, func: int):
    """Host call: (window radii or None, window blocks, dynamic k) for k_total blocks."""
    w = (ctypes.c_int32 * 3)()
    wb, kd = ctypes.c_int32(0), ctypes.c_int32(0)
    _check(lib().spade_policy_split(int(k_total), int(func), w, ctypes.byref(wb),
                                    ctypes.byref(kd)))
    radii = tuple(int(x) for x in w)
    return (None if radii[0] < 0 else radii), int(wb.value), int(kd.value)


def spade_attn_workspace_bytes(g: spade_geom) -> int:
    return int(lib().spade_attn_workspace_bytes(ctypes.byref(g)))


def spade_validate_lists(g: spade_geom, counts, indices, report, stream=None):
    """report: int32 [4] device tensor: failing rows, lowest failing row, OR of the
    SPADE_LIST_* bits, 0 (see spade.h)."""
    a = _Args()
    D = _Dims(g)
    _check(a.run(lib().spade_validate_lists, ctypes.byref(g),
                 a(counts, I32, D.per_block, "counts"), a(indices, I32, D.pairs, "indices"),
                 a(report, I32, 4, "report"), stream))


def _debug_validate(g: spade_geom, counts, indices, stream):
    """With SPADE_DEBUG_VALIDATE=1 in the environment, the single-geometry attention
    calls first check their lists on the device and raise SpadeError on a malformed
    row (this waits for the stream)."""
    if os.environ.get("SPADE_DEBUG_VALIDATE", "0") != "1":
        return
    dev = counts.device if isinstance(counts, torch.Tensor) else None
    report = torch.empty(4, dtype=I32, device=dev)
    spade_validate_lists(g, counts, indices, report, stream)
    if stream is None or hasattr(stream, "synchronize"):
        (stream or torch.cuda.current_stream(dev)).synchronize()
    else:
        torch.cuda.synchronize(dev)
    bad, first, bits, _ = (int(x) for x in report.cpu())
    if bad:
        raise SpadeError(SPADE_ERR_INVALID_ARG,
                         f"malformed block lists: {bad} rows fail, the first is row {first}, "
                         f"failure bits {bits:#x}")


def spade_block_sparse_attn(g: spade_geom, qb, kb, vb, counts, indices, scale: float, ob,
                            lse=None, workspace=None, stream=None):
    _debug_validate(g, counts, indices, stream)
    a = _Args()
    D = _Dims(g)
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(a.run(lib().spade_block_sparse_attn, ctypes.byref(g), a(qb, BF16, D.blocked, "qb"),
                 a(kb, BF16, D.blocked, "kb"), a(vb, BF16, D.blocked, "vb"),
                 a(counts, I32, D.per_block, "counts"), a(indices, I32, D.pairs, "indices"),
                 float(scale), a(ob, BF16, D.blocked, "ob"), a(lse, F32, D.blocked_rows, "lse"),
                 a(workspace, None, None, "workspace"), nbytes, stream))


def spade_sparse_attn_raster(g: spade_geom, q, k, v, counts, indices, scale: float, o, lse=None,
                             workspace=None, stream=None):
    _debug_validate(g, counts, indices, stream)
    a = _Args()
    D = _Dims(g)
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(a.run(lib().spade_sparse_attn_raster, ctypes.byref(g), a(q, BF16, D.raster, "q"),
                 a(k, BF16, D.raster, "k"), a(v, BF16, D.raster, "v"),
                 a(counts, I32, D.per_block, "counts"), a(indices, I32, D.pairs, "indices"),
                 float(scale), a(o, BF16, D.raster, "o"), a(lse, F32, D.raster_rows, "lse"),
                 a(workspace, None, None, "workspace"), nbytes, stream))


def spade_sparse_attn_raster_noalloc(g: spade_geom, q, k, v, counts, indices, scale: float, o,
                                     lse=None, stream=None):
    """spade_sparse_attn_raster with the library's own per-GPU scratch (no workspace)."""
    _debug_validate(g, counts, indices, stream)
    a = _Args()
    D = _Dims(g)
    _check(a.run(lib().spade_sparse_attn_raster_noalloc, ctypes.byref(g),
                 a(q, BF16, D.raster, "q"), a(k, BF16, D.raster, "k"), a(v, BF16, D.raster, "v"),
                 a(counts, I32, D.per_block, "counts"), a(indices, I32, D.pairs, "indices"),
                 float(scale), a(o, BF16, D.raster, "o"), a(lse, F32, D.raster_rows, "lse"),
                 stream))
