"""Buffers + the C-ABI calls of one sparse attention pass (paper §3.3 order).

blocking (Q, K, V) -> summaries -> estimate + select -> block-sparse attention
-> restore layout. By default the blocking of Q and K and their summaries are
one fused call (spade_block_summarize, §3.3 optimisation (1)); `fused=False`
issues spade_block_reorder x3 + spade_summarize instead. With `virtual=True`
nothing is copied into the blocked layout: the summaries are read straight from
the raster Q, K and the attention gathers its rows from, and writes O back to,
the raster tensors (spade_sparse_attn_raster). A `Scheme` selects the full mask
composition instead of the plain Top-K/Top-P rule (spade_block_minmax for the
DSA estimators' summaries, spade_compose_select). All buffers are allocated once
here (torch, device memory); `run` only issues the library calls on one stream,
with no host sync.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np
import torch

from . import spade as S


@dataclass
class Scheme:
    """One head-wise sparsity scheme (§3.1): estimator expression, inter-block
    Top-K/Top-P value (optionally per head), intra-block filter, local-window
    radii in blocks and attention-sink length in tokens."""
    estimator: str = "mean"          # "mean" | "dsa" | "dsa2"
    mode: str = "topk"               # "topk" | "topp"
    topk: int = 1
    tau: float = 1.0
    topk_per_head: tuple | None = None
    tau_per_head: tuple | None = None
    intra: str | None = None         # None | "threshold" | "topk"
    intra_theta: float = 0.0
    intra_topk: int = 0
    window: tuple = (-1, -1, -1)
    sink: int = 0

    @property
    def extremes(self) -> bool:
        return self.estimator != "mean"


def _device_array(x, dtype, dev):
    """None, a device tensor (used as is) or a sequence (copied to the device)."""
    if x is None or isinstance(x, torch.Tensor):
        return x
    return torch.tensor(x, dtype=dtype, device=dev)


_EST = {"mean": S.SPADE_EST_MEAN, "dsa": S.SPADE_EST_DSA, "dsa2": S.SPADE_EST_DSA2}
_INTRA = {None: S.SPADE_INTRA_NONE, "threshold": S.SPADE_INTRA_THRESHOLD, "topk": S.SPADE_INTRA_TOPK}


def block_valid_counts(g) -> np.ndarray:
    """Real tokens per block (T-major block order): product of the clipped extents."""
    def extents(n, b):
        nb = -(-n // b)
        return np.minimum(b, n - b * np.arange(nb))
    et, eh, ew = extents(g.T, g.bt), extents(g.Hs, g.bh), extents(g.Ws, g.bw)
    return (et[:, None, None] * eh[None, :, None] * ew[None, None, :]).reshape(-1).astype(np.int64)


class SpadePath:
    def __init__(self, B, H, d, T, Hs, Ws, bt, bh, bw, *, mode="topp", topk=None, tau=None,
                 scale=None, device="cuda", with_sics=False, with_lse=False, fused=True,
                 virtual=False, scheme: Scheme | None = None):
        self.g = S.geom(B, H, d, T, Hs, Ws, bt, bh, bw)
        self.scheme = scheme
        if scheme is not None:
            mode, topk, tau = scheme.mode, scheme.topk, scheme.tau
            with_sics = with_sics or scheme.intra is not None
        self.virtual = bool(virtual)
        self.fused = bool(fused) or self.virtual
        self._qkv = None
        self.mode = S.SPADE_TOPP if mode == "topp" else S.SPADE_TOPK
        self.topk = int(topk or 0)
        self.tau = float(tau if tau is not None else 1.0)
        self.scale = float(scale if scale is not None else 1.0 / math.sqrt(d))
        g, dev = self.g, device
        NB, BS = g.NB, g.BS
        bf = torch.bfloat16
        blocked = (0,) if self.virtual else (B, H, NB * BS, d)
        self.Qb = torch.empty(blocked, dtype=bf, device=dev)
        self.Kb = torch.empty_like(self.Qb)
        self.Vb = torch.empty_like(self.Qb)
        self.Ob = torch.empty_like(self.Qb)
        self.O = torch.empty((B, H, g.N, d), dtype=bf, device=dev)
        self.qbar = torch.empty((B, H, NB, d), dtype=torch.float64, device=dev)
        self.kbar = torch.empty_like(self.qbar)
        self.sics_q = torch.empty((B, H, NB), dtype=torch.float64, device=dev) if with_sics else None
        self.sics_k = torch.empty_like(self.sics_q) if with_sics else None
        self.ext = None  # (qmax, qmin, kmax, kmin) for the DSA estimators
        self.spec = None
        if scheme is not None:
            if scheme.extremes:
                self.ext = tuple(torch.empty((B, H, NB, d), dtype=torch.float64, device=dev)
                                 for _ in range(4))
            self._topk_h = _device_array(scheme.topk_per_head, torch.int32, dev)
            self._tau_h = _device_array(scheme.tau_per_head, torch.float64, dev)
            self.spec = S.mask_spec(_EST[scheme.estimator], self.mode, self.topk, self.tau,
                                    self.scale, self._topk_h, self._tau_h, _INTRA[scheme.intra],
                                    scheme.intra_topk, scheme.intra_theta, scheme.window,
                                    scheme.sink)
            self.summ = S.summaries(self.qbar, self.kbar, *(self.ext or (None,) * 4),
                                    self.sics_q, self.sics_k)
        self.counts = torch.empty((B, H, NB), dtype=torch.int32, device=dev)
        self.indices = torch.empty((B, H, NB, NB), dtype=torch.int32, device=dev)
        lse_rows = g.N if self.virtual else NB * BS
        self.lse = torch.empty((B, H, lse_rows), dtype=torch.float32, device=dev) if with_lse else None
        nws = S.spade_attn_workspace_bytes(g)
        self.ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)

    # individual stages, so they can be timed separately
    def reorder_in(self, Q, K, V, stream=None):
        """Blocking of Q, K, V; in fused mode also the summaries of Q and K; in
        virtual mode only the summaries (the raster tensors are kept for attend)."""
        if self.ext is not None:  # DSA estimators: extremes (+ SICS) from the raster tensors
            S.spade_block_minmax(self.g, Q, K, *self.ext, self.sics_q, self.sics_k, stream=stream)
            if self.virtual:
                self._qkv = (Q, K, V)
                return
            for x, y in ((Q, self.Qb), (K, self.Kb), (V, self.Vb)):
                S.spade_block_reorder(self.g, x, y, inverse=False, stream=stream)
            return
        if self.virtual:
            S.spade_block_summarize(self.g, Q, K, qbar=self.qbar, kbar=self.kbar,
                                    sics_q=self.sics_q, sics_k=self.sics_k, stream=stream)
            self._qkv = (Q, K, V)
            return
        if self.fused:
            S.spade_block_summarize(self.g, Q, K, self.Qb, self.Kb, self.qbar, self.kbar,
                                    self.sics_q, self.sics_k, stream=stream)
            S.spade_block_reorder(self.g, V, self.Vb, inverse=False, stream=stream)
            return
        for x, y in ((Q, self.Qb), (K, self.Kb), (V, self.Vb)):
            S.spade_block_reorder(self.g, x, y, inverse=False, stream=stream)

    def summarize(self, stream=None):
        """Summaries of the blocked Q, K (already produced by reorder_in in fused mode)."""
        if self.fused or self.ext is not None:
            return
        S.spade_summarize(self.g, self.Qb, self.Kb, self.qbar, self.kbar, self.sics_q,
                          self.sics_k, stream=stream)

    def select(self, stream=None):
        if self.spec is not None:
            S.spade_compose_select(self.g, self.spec, self.summ, self.counts, self.indices,
                                   stream=stream)
            return
        S.spade_estimate_select(self.g, self.qbar, self.kbar, self.mode, self.topk, self.tau,
                                self.scale, self.counts, self.indices, stream=stream)

    def attend(self, counts=None, indices=None, stream=None):
        if self.virtual:
            Q, K, V = self._qkv
            S.spade_sparse_attn_raster(self.g, Q, K, V,
                                       self.counts if counts is None else counts,
                                       self.indices if indices is None else indices,
                                       self.scale, self.O, self.lse, self.ws, stream=stream)
            return
        S.spade_block_sparse_attn(self.g, self.Qb, self.Kb, self.Vb,
                                  self.counts if counts is None else counts,
                                  self.indices if indices is None else indices,
                                  self.scale, self.Ob, self.lse, self.ws, stream=stream)

    def restore(self, stream=None):
        if self.virtual:  # the attention already wrote O in raster order
            return
        S.spade_block_reorder(self.g, self.Ob, self.O, inverse=True, stream=stream)

    def run(self, Q, K, V, stream=None):
        self.reorder_in(Q, K, V, stream)
        self.summarize(stream)
        self.select(stream)
        self.attend(stream=stream)
        self.restore(stream)
        return self.O


def _chunks(heads, n):
    return [heads[i:i + n] for i in range(0, len(heads), n)]


class SweepPath:
    """Head-wise blocking choice over candidate schemes, then one path per head group.

    Evaluation (§3.2): for every candidate, SICS of Q and K straight from the
    raster tensors (fused call, nothing written in blocked layout), the
    normalised Aggregation Score, then the per-head argmax on the device. The
    choice is read back to the host (the one sync) to form the head groups; each
    group then runs the fused blocking + summaries of Q, K with its head list
    (§3.3 (1), (2)), the blocking of V, Top-K selection with
    k = max(1, round((1 - s) NB)), block-sparse attention and the inverse
    blocking into the full output. With `raster=True` (at most 64 heads) the
    groups compute only their summaries and block lists, and one multi-scheme
    call (spade_sparse_attn_raster_multi) attends every head from the raster
    tensors under its own blocking and writes O in raster order.
    """

    def __init__(self, B, H, d, T, Hs, Ws, candidates, sparsity, *, scale=None, device="cuda",
                 policy=None, raster=False, tau=None, one_pass=True):
        self.B, self.H, self.d = B, H, d
        self.raster = bool(raster)
        if self.raster and H > S.MAX_HEAD_LIST:
            raise ValueError(f"raster sweep supports at most {S.MAX_HEAD_LIST} heads")
        self.policy = policy  # None: uniform k per group; else the policy function's budgets
        # row rule of the groups: Top-K with k = max(1, round((1 - s) NB)) (tau None), or
        # Top-P with mass tau (the policy then spreads the mass over the heads, and the
        # Top-K budget only sizes its static window)
        self.tau = None if tau is None else float(tau)
        # candidate evaluation in one pass over Q and K (spade_candidate_sics)
        self.one_pass = bool(one_pass)
        self.shapes = [tuple(c) for c in candidates]
        self.sparsity = float(sparsity)
        self.scale = float(scale if scale is not None else 1.0 / math.sqrt(d))
        self.geoms = [S.geom(B, H, d, T, Hs, Ws, *c) for c in self.shapes]
        bf, f64, dev = torch.bfloat16, torch.float64, device
        self.topk = [max(1, int(math.floor((1.0 - self.sparsity) * g.NB + 0.5))) for g in self.geoms]
        # evaluation buffers, one set per candidate (all heads): SICS only
        self.ev = [dict(sics_q=torch.empty((B, H, g.NB), dtype=f64, device=dev),
                        sics_k=torch.empty((B, H, g.NB), dtype=f64, device=dev))
                   for g in self.geoms]
        C = len(self.geoms)
        self.as_qk = torch.empty((C, B, H), dtype=f64, device=dev)
        self.choice = torch.empty(H, dtype=torch.int32, device=dev)
        self.best = torch.empty(H, dtype=f64, device=dev)
        # group buffers: flat storage for up to min(H, 64) heads per candidate,
        # viewed as a contiguous [B, n, ...] tensor for a group of n heads
        cap = min(H, S.MAX_HEAD_LIST)
        self.gb = []
        for g in self.geoms:
            rows = 0 if self.raster else g.NB * g.BS  # the raster sweep blocks nothing
            self.gb.append(dict(
                Q=torch.empty(B * cap * rows * d, dtype=bf, device=dev),
                K=torch.empty(B * cap * rows * d, dtype=bf, device=dev),
                V=torch.empty(B * cap * rows * d, dtype=bf, device=dev),
                O=torch.empty(B * cap * rows * d, dtype=bf, device=dev),
                qbar=torch.empty(B * cap * g.NB * d, dtype=f64, device=dev),
                kbar=torch.empty(B * cap * g.NB * d, dtype=f64, device=dev),
                counts=torch.empty(B * cap * g.NB, dtype=torch.int32, device=dev),
                indices=torch.empty(B * cap * g.NB * g.NB, dtype=torch.int32, device=dev),
                k_heads=torch.empty(cap, dtype=torch.int32, device=dev),
                tau_heads=torch.empty(cap, dtype=f64, device=dev)))
        self.ws = torch.empty(max(max(S.spade_attn_workspace_bytes(g) for g in self.geoms), 1),
                              dtype=torch.uint8, device=dev)
        self.O = torch.empty((B, H, T * Hs * Ws, d), dtype=bf, device=dev)

    def evaluate(self, Q, K, stream=None):
        """SICS of every candidate (one pass over Q and K when the candidates' common
        refinement fits, else one pass per candidate), the Aggregation Scores, and the
        per-head choice."""
        if self.one_pass:
            try:
                S.spade_candidate_sics(self.geoms, Q, K, [e["sics_q"] for e in self.ev],
                                       [e["sics_k"] for e in self.ev], stream=stream)
            except S.SpadeError as err:
                if err.status != S.SPADE_ERR_UNSUPPORTED:
                    raise
                self.one_pass = False
        if not self.one_pass:
            for g, e in zip(self.geoms, self.ev):
                S.spade_block_summarize(g, Q, K, sics_q=e["sics_q"], sics_k=e["sics_k"],
                                        stream=stream)
        for c, (g, e) in enumerate(zip(self.geoms, self.ev)):
            S.spade_aggregation_score(g, e["sics_q"], e["sics_k"], self.as_qk[c], stream=stream)
        S.spade_choose_scheme(self.as_qk, self.choice, self.best, stream=stream)

    def groups(self, stream=None):
        """Host copy of the choice (waits for `stream`) -> ascending head list per candidate."""
        if stream is not None:
            stream.synchronize()
        ch = self.choice.cpu().tolist()
        return [[h for h in range(self.H) if ch[h] == c] for c in range(len(self.geoms))]

    def group_views(self, c, n):
        g = self.geoms[c]
        gg = S.geom(self.B, n, self.d, g.T, g.Hs, g.Ws, g.bt, g.bh, g.bw)
        b, rows, NB = self.gb[c], g.NB * g.BS, g.NB
        v = dict(g=gg)
        for k in ("Q", "K", "V", "O"):  # blocked group tensors (none in raster mode)
            v[k] = None if self.raster else b[k][: self.B * n * rows * self.d].view(
                self.B, n, rows, self.d)
        for k in ("qbar", "kbar"):
            v[k] = b[k][: self.B * n * NB * self.d].view(self.B, n, NB, self.d)
        v["counts"] = b["counts"][: self.B * n * NB].view(self.B, n, NB)
        v["indices"] = b["indices"][: self.B * n * NB * NB].view(self.B, n, NB, NB)
        return v

    # group stages, separately callable so they can be timed
    def group_select(self, c, heads, Q, K, V, stream=None):
        g, v = self.geoms[c], self.group_views(c, len(heads))
        if self.raster:
            S.spade_block_summarize(g, Q, K, qbar=v["qbar"], kbar=v["kbar"], heads=heads,
                                    stream=stream)
        else:
            S.spade_block_summarize(g, Q, K, v["Q"], v["K"], v["qbar"], v["kbar"], heads=heads,
                                    stream=stream)
            S.spade_block_reorder(g, V, v["V"], heads=heads, stream=stream)
        if self.policy is None:
            mode = S.SPADE_TOPK if self.tau is None else S.SPADE_TOPP
            S.spade_estimate_select(v["g"], v["qbar"], v["kbar"], mode, self.topk[c],
                                    1.0 if self.tau is None else self.tau, self.scale,
                                    v["counts"], v["indices"], stream=stream)
            return v
        if self.tau is None:
            # the policy function: static window + per-head k from the Selected AS (§3.1)
            kh = self.gb[c]["k_heads"][: len(heads)]
            sc = self.policy.scheme(self.topk[c], g.NB, self.best, kh, heads=heads, stream=stream)
            spec = S.mask_spec(S.SPADE_EST_MEAN, S.SPADE_TOPK, sc.topk, 1.0, self.scale, kh, None,
                               S.SPADE_INTRA_NONE, 0, 0.0, sc.window, 0)
        else:
            # Top-P: the same window, and per-head mass from the Selected AS
            th = self.gb[c]["tau_heads"][: len(heads)]
            sc = self.policy.scheme_topp(self.tau, self.topk[c], self.best, th, heads=heads,
                                         stream=stream)
            spec = S.mask_spec(S.SPADE_EST_MEAN, S.SPADE_TOPP, 1, self.tau, self.scale, None, th,
                               S.SPADE_INTRA_NONE, 0, 0.0, sc.window, 0)
        v["scheme"] = sc
        S.spade_compose_select(v["g"], spec, S.summaries(v["qbar"], v["kbar"]), v["counts"],
                               v["indices"], stream=stream)
        return v

    def group_attend(self, c, v, stream=None):
        S.spade_block_sparse_attn(v["g"], v["Q"], v["K"], v["V"], v["counts"], v["indices"],
                                  self.scale, v["O"], None, self.ws, stream=stream)

    def group_restore(self, c, heads, v, stream=None):
        S.spade_block_reorder(self.geoms[c], v["O"], self.O, inverse=True, heads=heads,
                              stream=stream)

    def attend_all(self, selected, Q, K, V, stream=None):
        """Raster mode: one multi-scheme call over every head; `selected` holds the
        (candidate, heads, views) of each group."""
        table = [None] * self.H
        for c, heads, v in selected:
            NB, n = self.geoms[c].NB, len(heads)
            for k, h in enumerate(heads):
                table[h] = (c, v["counts"][0, k], v["indices"][0, k], n * NB, n * NB * NB)
        S.spade_sparse_attn_raster_multi(self.geoms, table, Q, K, V, self.scale, self.O,
                                         workspace=self.ws, stream=stream)

    def work_list(self, stream=None):
        """[(candidate, heads)] with every group split into chunks of <= 64 heads."""
        return [(c, hs) for c, grp in enumerate(self.groups(stream))
                for hs in _chunks(grp, S.MAX_HEAD_LIST)]

    def run(self, Q, K, V, stream=None):
        self.evaluate(Q, K, stream)
        if self.raster:
            selected = [(c, heads, self.group_select(c, heads, Q, K, V, stream))
                        for c, heads in self.work_list(stream)]
            self.attend_all(selected, Q, K, V, stream)
            return self.O
        for c, heads in self.work_list(stream):
            v = self.group_select(c, heads, Q, K, V, stream)
            self.group_attend(c, v, stream)
            self.group_restore(c, heads, v, stream)
        return self.O
