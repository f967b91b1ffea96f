"""Helpers shared by the GPU parity tests: inputs, oracle conversions, comparators."""
from __future__ import annotations

import math

import numpy as np
import torch

from gen.workloads import make_inputs, workload
from oracle import spade_oracle as O

# Attention parity bar: bf16 inputs, fp32 accumulation, bf16 output.
ATTN_MAX_ABS = 2e-2
# Log-sum-exp: the kernel's softmax denominator sums the bf16-rounded weights that
# also feed the P*V product (relative error <= 2^-9 each, same sign at worst), so
# |lse - lse_exact| <= log(1 + 2^-9) plus fp32 rounding of the sum; 4e-3 covers it.
LSE_MAX_ABS = 4e-3
# Selection: memberships may differ only for blocks whose score lies within this
# relative distance of the row's cut (or, for Top-P, where the prefix mass at the
# boundary lies within it of tau).
SELECT_REL = 1e-6


def to_np64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def geometry(cfg) -> O.Geometry:
    return O.Geometry(cfg["T"], cfg["Hs"], cfg["Ws"], cfg["bt"], cfg["bh"], cfg["bw"])


def bf16_inputs(cfg, seed=0, device="cuda"):
    """Seeded Q, K, V rounded to bf16 on `device`."""
    Q, K, V = make_inputs(cfg, seed=seed, device=device)
    return tuple(x.to(torch.bfloat16) for x in (Q, K, V))


def small_cfg(T, Hs, Ws, bt, bh, bw, d=128, H=2, B=1, gain=2.5, freq=0.05, **kw):
    """A workload dict for an arbitrary small grid (same generator recipe)."""
    cfg = dict(B=B, H=H, d=d, T=T, Hs=Hs, Ws=Ws, bt=bt, bh=bh, bw=bw, N=T * Hs * Ws,
               mode="topp", topk=None, tau=0.9, aniso=(1.0, 1.0, 1.0),
               head_gains=[gain] * H, head_freqs=[freq * (1 + 0.5 * h) for h in range(H)])
    cfg.update(kw)
    return cfg


def compare_selection(scores, c_o, i_o, c_g, i_g, mode, tau=None, rel=SELECT_REL):
    """Row-by-row comparison of kept sets. Returns (n_exempt_rows, worst_message).

    Raises AssertionError on a difference that no exemption covers. scores are the
    oracle's fp64 [.., NB, NB]; counts/indices as the library lays them out.
    """
    lead = c_o.shape
    n_exempt = 0
    for idx in np.ndindex(*lead):
        ko = i_o[idx][: c_o[idx]]
        kg = i_g[idx][: c_g[idx]]
        assert np.all(np.diff(kg) > 0), f"row {idx}: GPU indices not strictly ascending"
        if c_o[idx] == c_g[idx] and np.array_equal(ko, kg):
            continue
        s = scores[idx]
        order = O.rank_order(s)
        m_o = int(c_o[idx])
        cut = s[order[m_o - 1]]
        diff = np.setxor1d(ko, kg)
        if np.all(np.abs(s[diff] - cut) <= rel * abs(cut)):
            n_exempt += 1
            continue
        if mode == "topp":
            m_g = int(c_g[idx])
            same_prefix = np.array_equal(np.sort(order[:m_g]), kg)
            cum = np.cumsum(O.row_softmax(s)[order])
            lo, hi = min(m_o, m_g), max(m_o, m_g)
            # prefix masses that decided the boundary between the two counts
            near = all(abs(cum[m - 1] - tau) <= rel for m in range(max(lo, 1), hi + 1))
            if same_prefix and near:
                n_exempt += 1
                continue
        raise AssertionError(f"row {idx}: oracle kept {ko.tolist()} GPU kept {kg.tolist()}")
    return n_exempt


def sample_rows(B, H, NB, n, seed=0, must=()):
    rng = np.random.default_rng(seed)
    rows = {tuple(r) for r in must}
    while len(rows) < min(n, B * H * NB):
        rows.add((int(rng.integers(B)), int(rng.integers(H)), int(rng.integers(NB))))
    return sorted(rows)


def scale_of(d):
    return 1.0 / math.sqrt(d)


def nan_fill(*tensors):
    """Poison output buffers before a call: a row the kernel skips stays NaN."""
    for t in tensors:
        if t is not None and t.is_floating_point():
            t.fill_(float("nan"))


def finite_max_abs(got, ref) -> float:
    """max |got - ref| over every element, failing on any non-finite GPU value
    (Python's max() would silently drop a NaN)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    bad = ~np.isfinite(got)
    assert not bad.any(), f"{int(bad.sum())} non-finite GPU values (first at {np.argwhere(bad)[0].tolist()})"
    return float(np.max(np.abs(got - ref))) if got.size else 0.0


def oracle_attention_on_lists(q, k, v, og, counts, indices, scale, rows=None):
    """Eq. (2) by the oracle with the given block lists (normally the GPU's own),
    on fp64 raster q, k, v [B, H, N, d]. Returns (O, lse) in raster order
    [B, H, N, d] / [B, H, N]; with `rows` only those query blocks are computed."""
    Qb, Kb, Vb = (O.reorder(x, og) for x in (q, k, v))
    ob, lb = O.block_sparse_attention(Qb, Kb, Vb, counts, indices, og, scale, rows=rows)
    pos = O.token_position(og)
    return ob[:, :, pos], lb[:, :, pos]


def row_tokens(og, i) -> np.ndarray:
    """Raster tokens of query block i's real slots."""
    slot_token, nv = O.block_tables(og)
    return slot_token[i * og.BS: i * og.BS + nv[i]]


def compare_rows_raster(got_o, got_lse, ref_o, ref_lse, og, rows):
    """Element-wise attention check of the listed query blocks (b, h, i) on raster
    outputs; returns the worst max-abs. Every compared value must be finite."""
    worst = 0.0
    for (b, h, i) in rows:
        toks = row_tokens(og, i)
        worst = max(worst, finite_max_abs(got_o[b, h, toks], ref_o[b, h, toks]))
        if got_lse is not None:
            d = finite_max_abs(got_lse[b, h, toks], ref_lse[b, h, toks])
            assert d <= LSE_MAX_ABS, f"lse of row {(b, h, i)} off by {d:.3e}"
    return worst


def heaviest_head(counts) -> tuple:
    """(b, h) of the pair holding the row with the most kept blocks (ties: first)."""
    c = np.asarray(counts)
    b, h, _ = np.unravel_index(int(np.argmax(c)), c.shape)
    return int(b), int(h)
