"""Buffers + the five C-ABI calls of one sparse attention pass (paper §3.3 order).

blocking (Q, K, V) -> summaries -> estimate + select -> block-sparse attention
-> restore layout. All buffers are allocated once here (torch, device memory);
`run` only issues the library calls on one stream, with no host sync.
"""
from __future__ import annotations

import math

import numpy as np
import torch

from . import spade as S


def block_valid_counts(g) -> np.ndarray:
    """Real tokens per block (T-major block order): product of the clipped extents."""
    def extents(n, b):
        nb = -(-n // b)
        return np.minimum(b, n - b * np.arange(nb))
    et, eh, ew = extents(g.T, g.bt), extents(g.Hs, g.bh), extents(g.Ws, g.bw)
    return (et[:, None, None] * eh[None, :, None] * ew[None, None, :]).reshape(-1).astype(np.int64)


class SpadePath:
    def __init__(self, B, H, d, T, Hs, Ws, bt, bh, bw, *, mode="topp", topk=None, tau=None,
                 scale=None, device="cuda", with_sics=False, with_lse=False):
        self.g = S.geom(B, H, d, T, Hs, Ws, bt, bh, bw)
        self.mode = S.SPADE_TOPP if mode == "topp" else S.SPADE_TOPK
        self.topk = int(topk or 0)
        self.tau = float(tau if tau is not None else 1.0)
        self.scale = float(scale if scale is not None else 1.0 / math.sqrt(d))
        g, dev = self.g, device
        NB, BS = g.NB, g.BS
        bf = torch.bfloat16
        self.Qb = torch.empty((B, H, NB * BS, d), dtype=bf, device=dev)
        self.Kb = torch.empty_like(self.Qb)
        self.Vb = torch.empty_like(self.Qb)
        self.Ob = torch.empty_like(self.Qb)
        self.O = torch.empty((B, H, g.N, d), dtype=bf, device=dev)
        self.qbar = torch.empty((B, H, NB, d), dtype=torch.float64, device=dev)
        self.kbar = torch.empty_like(self.qbar)
        self.sics_q = torch.empty((B, H, NB), dtype=torch.float64, device=dev) if with_sics else None
        self.sics_k = torch.empty_like(self.sics_q) if with_sics else None
        self.counts = torch.empty((B, H, NB), dtype=torch.int32, device=dev)
        self.indices = torch.empty((B, H, NB, NB), dtype=torch.int32, device=dev)
        self.lse = torch.empty((B, H, NB * BS), dtype=torch.float32, device=dev) if with_lse else None
        nws = S.spade_attn_workspace_bytes(g)
        self.ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)

    # individual stages, so they can be timed separately
    def reorder_in(self, Q, K, V, stream=None):
        for x, y in ((Q, self.Qb), (K, self.Kb), (V, self.Vb)):
            S.spade_block_reorder(self.g, x, y, inverse=False, stream=stream)

    def summarize(self, stream=None):
        S.spade_summarize(self.g, self.Qb, self.Kb, self.qbar, self.kbar, self.sics_q,
                          self.sics_k, stream=stream)

    def select(self, stream=None):
        S.spade_estimate_select(self.g, self.qbar, self.kbar, self.mode, self.topk, self.tau,
                                self.scale, self.counts, self.indices, stream=stream)

    def attend(self, counts=None, indices=None, stream=None):
        S.spade_block_sparse_attn(self.g, self.Qb, self.Kb, self.Vb,
                                  self.counts if counts is None else counts,
                                  self.indices if indices is None else indices,
                                  self.scale, self.Ob, self.lse, self.ws, stream=stream)

    def restore(self, stream=None):
        S.spade_block_reorder(self.g, self.Ob, self.O, inverse=True, stream=stream)

    def run(self, Q, K, V, stream=None):
        self.reorder_in(Q, K, V, stream)
        self.summarize(stream)
        self.select(stream)
        self.attend(stream=stream)
        self.restore(stream)
        return self.O
