"""Plain fp64 CPU oracle of SPADE's block-sparse attention hot path.

TEST INFRASTRUCTURE ONLY. This module is the slow, obviously-correct reference
that the GPU path is checked against. Only the test suite, the smoke check and
the benchmark's CPU-baseline leg may import it; the library never does, and it
shares no code with the GPU kernels.

Paper: "SPADE: An Input-Adaptive Sparse Attention Engine for Fast Video
Diffusion Models Inference" (arXiv 2608.03335). What the path computes, in the
paper's order (§3.3, Head-wise Sparse Attention):

  1. blocking: rearrange tokens into 3D blocks of a blocking scheme
     (§3.1, Fig. 3: t x h x w tiles, order T, H, W);
  2. Summarizer: one vector per Q/K block, here the mean (MEAN-SPADE, §3.1);
  3. inter-block Estimator: block-pair importance from the summaries' dot
     products (§3.3);
  4. Top-K / Top-P filtering of each query block's row (§3.1 utility
     parameters, §3.3);
  5. block-sparse attention, Eq. (2): softmax(QK^T/sqrt(d) + M) V with M = 0
     on kept block pairs and -inf elsewhere;
  6. restore the original token layout (§3.3).
Plus the intra-block aggregation measure SICS, Eq. (4) and Eq. (5) / Alg. 1
(§3.2), and the Aggregation Score, Eq. (3).

Readings where the paper is silent (each is a stated choice):
  * tokens are flattened T-major, n = (t*Hs + y)*Ws + x;
  * blocks are numbered T-major over the ceil-sized block grid; inside a block
    the valid tokens come first, in raster order of (dt, dy, dx); the remaining
    slots up to BS are zero padding;
  * block means average valid tokens only; padded keys never receive weight;
  * the estimator score is <qbar_i, kbar_j> / sqrt(d);
  * rows are ranked by (score descending, block index ascending);
  * Top-P keeps the shortest prefix of that ranking whose softmax mass over the
    row's block scores reaches tau (at least one block); tau >= 1 keeps all;
  * kept indices are reported in ascending block order;
  * a candidate blocking is scored by AS(Q) + AS(K), each normalised by
    sum_b n_b^2 so that block sizes and padding compare; a head's score is its
    batch mean; the first candidate with the highest score wins;
  * the block-shape sweep keeps k = max(1, round((1 - s) NB)) blocks per row
    for a target block sparsity s.
Readings of the full mask composition (§3.1 vDiT-SSR, §3.3; the figure that
defines the DSA estimators is not part of the text, so those two are readings
that no printed value pins — "parity unpinned" with respect to the paper; the
tests pin them to the bounds they are built to be):
  * max/min Summarizer: elementwise max and min over each block's real tokens;
  * DSA estimate: with q~ = (q_max + q_min) / 2, scale * sum_c max(q~_c k_max_c,
    q~_c k_min_c), the largest <q~, k> over the box spanned by block j's keys;
  * DSA2 estimate: scale * sum_c of the largest of the four products of
    {q_max_c, q_min_c} and {k_max_c, k_min_c}: the largest <q, k> over both
    blocks' boxes, so it bounds every logit of the block pair from above;
  * intra-block filter (the intra-top value): a block's coherence is
    SICS / n_b^2 (the mean pairwise cosine similarity, self pairs included);
    the filter marks incoherent blocks, whose summary is least trustworthy:
    coherence < theta (threshold mode) or the k least coherent blocks of the
    head (Top-K mode, ties to the lower index). A marked Q block keeps its whole
    row and a marked K block its whole column (intra scores broadcast and
    OR-combined with the inter selection);
  * local window (w_t, w_h, w_w) in block units: key block j is kept for query
    block i when their block-grid coordinates differ by at most w on each axis;
    a negative radius disables the window;
  * attention sink of s tokens: every query block keeps the key blocks holding
    any of the first s raster tokens;
  * the mask is the OR of the inter Top-K/Top-P selection (computed on the inter
    scores alone) and the parts above; per-head k or tau values (the policy's
    head-wise budgets) replace the scalar ones.
Readings of the policy function (§3.1 policy function; §4 configurations and the
policy study), which the paper describes by its effect only:
  * warm-up: the first ceil(0.30 n) denoising steps (text-to-video) or
    ceil(0.25 n) (image-to-video) of n use full attention; Turbo only step 0;
  * budget split: of k_total blocks per row, a static share (1/31 for Func 0,
    whose dynamic:static budget is 30:1; 0.2 for Func 1, ~80% dynamic) goes to
    the largest window of a fixed ladder of radii that fits in it; the dynamic
    Top-K keeps the rest, k_dyn = k_total - window size;
  * AS-guided budgets: head h gets k_h = clamp(floor(H k_dyn w_h / W + 1/2), 1, NB)
    with w_h = 1 / AS_h (budget negatively correlated with the Selected
    Aggregation Score; w_h = 0 when AS_h <= 0) and W the sum of the w_h in head
    order (W = 0: every head gets clamp(k_dyn, 1, NB));
  * for Top-P schemes the budget is the mass: head h keeps tau_h = 1 - e_h with
    the dropped mass e_h = H (1 - tau) AS_h / S proportional to its score (S the
    sum of the positive scores in head order; AS_h <= 0 drops nothing; S = 0:
    tau for every head), so the mean dropped mass stays 1 - tau.

Every array here is float64 (inputs are upcast first). Shapes: Q, K, V are
[B, H, N, d]; blocked tensors are [B, H, NB*BS, d].
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


# --------------------------------------------------------------------------
# Geometry (§3.1 blocking scheme, Fig. 3; §2.1 flattening of the latent grid)
# --------------------------------------------------------------------------
@dataclass(frozen=True)
class Geometry:
    T: int
    Hs: int
    Ws: int
    bt: int
    bh: int
    bw: int

    @property
    def N(self) -> int:
        return self.T * self.Hs * self.Ws

    @property
    def BS(self) -> int:
        return self.bt * self.bh * self.bw

    @property
    def grid(self):
        return (-(-self.T // self.bt), -(-self.Hs // self.bh), -(-self.Ws // self.bw))

    @property
    def NB(self) -> int:
        nT, nH, nW = self.grid
        return nT * nH * nW


def block_tables(g: Geometry):
    """Enumerate every block and its valid tokens.

    Returns (slot_token, n_valid):
      slot_token[p] for p in [0, NB*BS): the raster token index stored at padded
        position p, or -1 for a padding slot;
      n_valid[b]: number of real tokens in block b.
    Blocks are visited in T-major order of the block grid; within a block the
    tokens are visited in raster order of (dt, dy, dx) and placed in consecutive
    slots, so real tokens come first.
    """
    nT, nH, nW = g.grid
    BS = g.BS
    slot_token = np.full(g.NB * BS, -1, dtype=np.int64)
    n_valid = np.zeros(g.NB, dtype=np.int64)
    b = 0
    for tb in range(nT):
        for hb in range(nH):
            for wb in range(nW):
                s = 0
                for dt in range(g.bt):
                    for dy in range(g.bh):
                        for dx in range(g.bw):
                            t, y, x = tb * g.bt + dt, hb * g.bh + dy, wb * g.bw + dx
                            if t < g.T and y < g.Hs and x < g.Ws:
                                slot_token[b * BS + s] = (t * g.Hs + y) * g.Ws + x
                                s += 1
                n_valid[b] = s
                b += 1
    return slot_token, n_valid


def token_position(g: Geometry) -> np.ndarray:
    """pos[n] = padded position of raster token n (inverse of slot_token)."""
    slot_token, _ = block_tables(g)
    pos = np.empty(g.N, dtype=np.int64)
    valid = slot_token >= 0
    pos[slot_token[valid]] = np.nonzero(valid)[0]
    return pos


# --------------------------------------------------------------------------
# Blocking (layout transform) and its inverse (§3.3: Q, K, V enter the
# blocked layout before attention, and the output returns to raster order)
# --------------------------------------------------------------------------
def reorder(X: np.ndarray, g: Geometry) -> np.ndarray:
    """Raster [.., N, d] -> blocked [.., NB*BS, d]; padding slots are zero."""
    slot_token, _ = block_tables(g)
    out = np.zeros(X.shape[:-2] + (g.NB * g.BS, X.shape[-1]), dtype=X.dtype)
    valid = slot_token >= 0
    out[..., valid, :] = X[..., slot_token[valid], :]
    return out


def inverse_reorder(Xb: np.ndarray, g: Geometry) -> np.ndarray:
    """Blocked [.., NB*BS, d] -> raster [.., N, d] (padding slots dropped)."""
    return Xb[..., token_position(g), :]


# --------------------------------------------------------------------------
# Summarizer: mean over each block's valid tokens (§3.1, MEAN-SPADE)
# --------------------------------------------------------------------------
def block_means(Xb: np.ndarray, g: Geometry) -> np.ndarray:
    """[B, H, NB*BS, d] -> [B, H, NB, d], mean over valid slots only."""
    _, n_valid = block_tables(g)
    Xb = np.asarray(Xb, dtype=np.float64)
    out = np.empty(Xb.shape[:-2] + (g.NB, Xb.shape[-1]), dtype=np.float64)
    for b in range(g.NB):
        rows = Xb[..., b * g.BS: b * g.BS + n_valid[b], :]
        out[..., b, :] = rows.sum(axis=-2) / n_valid[b]
    return out


# --------------------------------------------------------------------------
# SICS (§3.2): sum of all pairwise cosine similarities inside one block.
# Three forms that must agree: Eq. (4) directly; Eq. (5)'s split into the n
# self-pairs plus twice the sum over ordered pairs a < b; and the squared norm
# of the sum of unit vectors, which Eq. (5)'s expansion equals term by term.
# --------------------------------------------------------------------------
def _unit_rows(Q: np.ndarray) -> np.ndarray:
    Q = np.asarray(Q, dtype=np.float64)
    nrm = np.sqrt((Q * Q).sum(axis=-1, keepdims=True))
    safe = np.where(nrm > 0, nrm, 1.0)
    return np.where(nrm > 0, Q / safe, 0.0)  # a zero vector contributes nothing


def sics_pairwise(Q: np.ndarray) -> float:
    """Eq. (4): sum_a sum_b q_a.q_b / (|q_a| |q_b|) for one block [n, d]."""
    U = _unit_rows(Q)
    n = U.shape[0]
    total = 0.0
    for a in range(n):
        for b in range(n):
            total += float(U[a] @ U[b])
    return total


def sics_prefix(Q: np.ndarray) -> float:
    """Eq. (5) split: n + 2 * sum_{a<b} <q^_a, q^_b>, the pair sum taken as each
    unit row dotted with the exclusive prefix sum of the rows before it.

    A zero row has no unit vector: it adds neither a pair term nor a self term.
    """
    U = _unit_rows(Q)
    before = np.cumsum(U, axis=0) - U          # sum of the unit rows preceding each row
    pairs = float(np.einsum("jd,jd->", before, U))
    selfs = int(np.count_nonzero(np.any(U != 0, axis=1)))
    return selfs + 2.0 * pairs


def sics_closed(Q: np.ndarray) -> float:
    """|| sum_k q_k/|q_k| ||^2, the O(n d) form of Eq. (4)."""
    s = _unit_rows(Q).sum(axis=0)
    return float(s @ s)


def block_sics(Xb: np.ndarray, g: Geometry, form: str = "closed") -> np.ndarray:
    """[B, H, NB*BS, d] -> [B, H, NB] SICS of each block's valid rows."""
    fn = {"closed": sics_closed, "prefix": sics_prefix, "pairwise": sics_pairwise}[form]
    _, n_valid = block_tables(g)
    lead = Xb.shape[:-2]
    out = np.empty(lead + (g.NB,), dtype=np.float64)
    for idx in np.ndindex(*lead):
        for b in range(g.NB):
            out[idx + (b,)] = fn(Xb[idx + (slice(b * g.BS, b * g.BS + n_valid[b]),)])
    return out


def aggregation_score(sics: np.ndarray, g: Geometry):
    """Eq. (3): AS = sum over blocks of SICS (last axis), raw and normalised.

    The normalised form divides by sum_b n_b^2 (the value when every block's
    vectors are parallel) so that candidates with different block sizes or
    padding are comparable; for equal, unpadded blocks it is a constant factor
    and leaves the per-head argmax of Eq. (3) unchanged.
    """
    _, n_valid = block_tables(g)
    raw = sics.sum(axis=-1)
    return raw, raw / float((n_valid.astype(np.float64) ** 2).sum())


def scheme_scores(Q, K, g: Geometry) -> np.ndarray:
    """Per-(batch, head) score of one candidate blocking: AS_norm(Q) + AS_norm(K).

    §3.2 builds the candidates' scores from Q and K blocked under each scheme;
    Eq. (3) defines AS for Q as the sum of block SICS, and K is treated alike.
    """
    Q, K = np.asarray(Q, np.float64), np.asarray(K, np.float64)
    _, as_q = aggregation_score(block_sics(reorder(Q, g), g), g)
    _, as_k = aggregation_score(block_sics(reorder(K, g), g), g)
    return as_q + as_k


def choose_schemes(as_qk: np.ndarray):
    """Selected Blocking Scheme per head (§3.2): highest AS wins.

    as_qk: [C, B, H] candidate scores. A head's score for candidate c is its mean
    over the batch, so one scheme serves the head in every batch element; ties go
    to the lower candidate index. Returns (choice [H] int, best [H]).
    """
    per_head = np.asarray(as_qk, np.float64).mean(axis=1)        # [C, H]
    choice = np.zeros(per_head.shape[1], dtype=np.int64)
    best = per_head[0].copy()
    for c in range(1, per_head.shape[0]):                        # first maximum wins
        better = per_head[c] > best
        choice[better], best[better] = c, per_head[c][better]
    return choice, best


def head_groups(choice: np.ndarray, C: int):
    """Head grouping (§3.3 (2)): ascending head list per candidate (may be empty)."""
    return [[int(h) for h in np.flatnonzero(np.asarray(choice) == c)] for c in range(C)]


def sweep_topk(sparsity: float, NB: int) -> int:
    """Blocks kept per query row for a target block sparsity s: max(1, round((1-s) NB))."""
    return max(1, int(np.floor((1.0 - sparsity) * NB + 0.5)))


def spade_sweep_attention(Q, K, V, grid, block_shapes, sparsity: float, scale=None):
    """Head-wise blocking choice among candidates, then each head group's path.

    For every candidate (bt, bh, bw): blocking of Q and K, SICS, normalised AS
    (Eq. (3)); each head takes its best candidate (§3.2); heads sharing a scheme
    form a group (§3.3 (2)) that runs blocking -> means -> scores -> Top-K with
    k = sweep_topk(sparsity, NB) -> Eq. (2) -> restore, into the full output.
    grid = (T, Hs, Ws). Returns dict(O, choice, best, as_qk, groups, per-group
    counts/indices).
    """
    Q, K, V = (np.asarray(a, dtype=np.float64) for a in (Q, K, V))
    d = Q.shape[-1]
    scale = 1.0 / np.sqrt(d) if scale is None else scale
    geoms = [Geometry(*grid, *bs) for bs in block_shapes]
    as_qk = np.stack([scheme_scores(Q, K, g) for g in geoms])     # [C, B, H]
    choice, best = choose_schemes(as_qk)
    groups = head_groups(choice, len(geoms))
    O = np.zeros_like(Q)
    per_group = []
    for c, heads in enumerate(groups):
        if not heads:
            per_group.append(None)
            continue
        g = geoms[c]
        r = spade_attention(Q[:, heads], K[:, heads], V[:, heads], g, "topk",
                            topk=sweep_topk(sparsity, g.NB), scale=scale)
        O[:, heads] = r["O"]
        per_group.append(dict(heads=heads, counts=r["counts"], indices=r["indices"],
                              topk=sweep_topk(sparsity, g.NB)))
    return dict(O=O, choice=choice, best=best, as_qk=as_qk, groups=groups, per_group=per_group)


# --------------------------------------------------------------------------
# Inter-block estimator (§3.3): importance of block pair (i, j) from summaries
# --------------------------------------------------------------------------
def block_scores(qbar: np.ndarray, kbar: np.ndarray, scale: float) -> np.ndarray:
    """[.., NB, d] x [.., NB, d] -> [.., NB, NB]: <qbar_i, kbar_j> * scale."""
    return np.matmul(qbar, np.swapaxes(kbar, -1, -2)) * scale


# --------------------------------------------------------------------------
# Top-K / Top-P index search (§3.1 utility parameters; §3.3 filtering)
# --------------------------------------------------------------------------
def rank_order(s: np.ndarray) -> np.ndarray:
    """Block indices of one row ordered by (score descending, index ascending)."""
    j = np.arange(s.shape[0])
    return np.lexsort((j, -s))


def row_softmax(s: np.ndarray) -> np.ndarray:
    e = np.exp(s - s.max())
    return e / e.sum()


def select_row_topk(s: np.ndarray, k: int) -> np.ndarray:
    """Ascending indices of the min(k, NB) highest-ranked blocks."""
    return np.sort(rank_order(s)[: min(k, s.shape[0])])


def select_row_topp(s: np.ndarray, tau: float) -> np.ndarray:
    """Ascending indices of the shortest ranked prefix whose mass reaches tau.

    The mass of block j is its softmax weight over the row's scores; the prefix
    mass is accumulated left to right in rank order. At least one block is
    kept. With tau >= 1 every block is kept (exact softmax weights are all
    positive, so no proper prefix reaches 1). If rounding keeps the running sum
    below tau to the end, every block is kept.
    """
    NB = s.shape[0]
    if tau >= 1.0:
        return np.arange(NB)
    order = rank_order(s)
    cum = np.cumsum(row_softmax(s)[order])  # sequential, left to right
    hit = np.nonzero(cum >= tau)[0]
    m = int(hit[0]) + 1 if hit.size else NB
    return np.sort(order[:m])


def select(scores: np.ndarray, mode: str, topk: int | None = None, tau: float | None = None):
    """Apply the row rule to every (b, h, i) row of [B, H, NB, NB] scores.

    Returns counts [B, H, NB] int32 and indices [B, H, NB, NB] int32 whose
    first counts[..] entries are the kept blocks, ascending; the rest are -1.
    """
    lead = scores.shape[:-1]
    NB = scores.shape[-1]
    counts = np.zeros(lead, dtype=np.int32)
    indices = np.full(lead + (NB,), -1, dtype=np.int32)
    for idx in np.ndindex(*lead):
        row = scores[idx]
        kept = select_row_topk(row, topk) if mode == "topk" else select_row_topp(row, tau)
        counts[idx] = kept.size
        indices[idx + (slice(0, kept.size),)] = kept
    return counts, indices


def block_mask(counts: np.ndarray, indices: np.ndarray) -> np.ndarray:
    """Binary [.., NB, NB] mask from counts + index lists."""
    NB = indices.shape[-1]
    mask = np.zeros(indices.shape[:-1] + (NB,), dtype=bool)
    for idx in np.ndindex(*counts.shape):
        mask[idx + (indices[idx][: counts[idx]],)] = True
    return mask


# --------------------------------------------------------------------------
# Attention: Eq. (1) dense and Eq. (2) block-sparse
# --------------------------------------------------------------------------
def dense_attention(Q, K, V, scale: float):
    """Eq. (1) on [.., N, d]: softmax(Q K^T * scale) V, max-subtracted, fp64."""
    Q, K, V = (np.asarray(a, dtype=np.float64) for a in (Q, K, V))
    logits = np.matmul(Q, np.swapaxes(K, -1, -2)) * scale
    logits -= logits.max(axis=-1, keepdims=True)
    w = np.exp(logits)
    w /= w.sum(axis=-1, keepdims=True)
    return np.matmul(w, V)


def block_sparse_attention(Qb, Kb, Vb, counts, indices, g: Geometry, scale: float,
                           rows=None):
    """Eq. (2) on blocked tensors, one query block at a time.

    For query block i of head (b, h), the keys are the valid slots of the kept
    blocks S_i (ascending). Returns (Ob, lse): Ob [B, H, NB*BS, d] with padding
    query slots left at 0, lse [B, H, NB*BS] (natural log of the softmax
    denominator, including the max), 0 at padding slots.

    rows: optional iterable of (b, h, i) to compute only those query blocks
    (the others stay 0); used for sampled checks at full size.
    """
    _, n_valid = block_tables(g)
    BS = g.BS
    B, H = Qb.shape[:2]
    d = Qb.shape[-1]
    Ob = np.zeros((B, H, g.NB * BS, d), dtype=np.float64)
    lse = np.zeros((B, H, g.NB * BS), dtype=np.float64)
    todo = rows if rows is not None else np.ndindex(B, H, g.NB)
    for (b, h, i) in todo:
        kept = indices[b, h, i, : counts[b, h, i]]
        q = np.asarray(Qb[b, h, i * BS: i * BS + n_valid[i]], dtype=np.float64)
        ks = np.concatenate([np.asarray(Kb[b, h, j * BS: j * BS + n_valid[j]], dtype=np.float64)
                             for j in kept])
        vs = np.concatenate([np.asarray(Vb[b, h, j * BS: j * BS + n_valid[j]], dtype=np.float64)
                             for j in kept])
        logits = (q @ ks.T) * scale
        mx = logits.max(axis=1, keepdims=True)
        w = np.exp(logits - mx)
        z = w.sum(axis=1, keepdims=True)
        Ob[b, h, i * BS: i * BS + n_valid[i]] = (w @ vs) / z
        lse[b, h, i * BS: i * BS + n_valid[i]] = (mx + np.log(z))[:, 0]
    return Ob, lse


# --------------------------------------------------------------------------
# Max/min Summarizer and the DSA / DSA2 inter-estimators (§3.1 Summarizer and
# Estimator Expressions; DSA-SPADE is the variant the experiments run, §4)
# --------------------------------------------------------------------------
def block_maxmin(Xb: np.ndarray, g: Geometry):
    """[B, H, NB*BS, d] -> (max, min), each [B, H, NB, d], over valid slots only."""
    _, n_valid = block_tables(g)
    Xb = np.asarray(Xb, dtype=np.float64)
    shape = Xb.shape[:-2] + (g.NB, Xb.shape[-1])
    mx, mn = np.empty(shape), np.empty(shape)
    for b in range(g.NB):
        rows = Xb[..., b * g.BS: b * g.BS + n_valid[b], :]
        mx[..., b, :] = rows.max(axis=-2)
        mn[..., b, :] = rows.min(axis=-2)
    return mx, mn


def dsa_scores(qmax, qmin, kmax, kmin, scale: float) -> np.ndarray:
    """DSA estimate [.., NB, NB]: per channel the larger of q~*k_max and q~*k_min,
    summed over channels, with q~ the midpoint of the query block's range."""
    qt = (qmax + qmin) / 2.0
    out = np.empty(qt.shape[:-1] + (kmax.shape[-2],))
    for i in range(qt.shape[-2]):
        a = qt[..., i:i + 1, :]
        out[..., i, :] = np.maximum(a * kmax, a * kmin).sum(axis=-1)
    return out * scale


def dsa2_scores(qmax, qmin, kmax, kmin, scale: float) -> np.ndarray:
    """DSA2 estimate [.., NB, NB]: per channel the largest product of a query
    extreme and a key extreme, summed over channels."""
    out = np.empty(qmax.shape[:-1] + (kmax.shape[-2],))
    for i in range(qmax.shape[-2]):
        hi, lo = qmax[..., i:i + 1, :], qmin[..., i:i + 1, :]
        corners = np.stack([hi * kmax, hi * kmin, lo * kmax, lo * kmin])
        out[..., i, :] = corners.max(axis=0).sum(axis=-1)
    return out * scale


# --------------------------------------------------------------------------
# Intra-block filter, local window, attention sink and their composition with
# the inter selection (§3.1 sparsity-ratio scheme and utility parameters; §3.3:
# intra scores broadcast and OR-combined with the inter scores, the result
# united with the local-window and attention-sink masks)
# --------------------------------------------------------------------------
def block_coherence(sics: np.ndarray, g: Geometry) -> np.ndarray:
    """SICS / n_b^2 per block: 1 when every vector of the block is parallel."""
    _, n_valid = block_tables(g)
    return np.asarray(sics, dtype=np.float64) / (n_valid.astype(np.float64) ** 2)


def intra_marks(sics: np.ndarray, g: Geometry, mode: str, theta=None, k=None) -> np.ndarray:
    """Boolean [.., NB]: the blocks the intra-block filter marks (incoherent ones)."""
    c = block_coherence(sics, g)
    if mode == "threshold":
        return c < theta
    assert mode == "topk"
    marks = np.zeros(c.shape, dtype=bool)
    j = np.arange(c.shape[-1])
    for idx in np.ndindex(*c.shape[:-1]):
        order = np.lexsort((j, c[idx]))          # coherence ascending, index ascending
        marks[idx + (order[: min(k, c.shape[-1])],)] = True
    return marks


def block_coords(g: Geometry) -> np.ndarray:
    """[NB, 3] block-grid coordinates (tb, hb, wb) of every block, T-major order."""
    nT, nH, nW = g.grid
    return np.array([(tb, hb, wb) for tb in range(nT) for hb in range(nH) for wb in range(nW)],
                    dtype=np.int64)


def window_mask(g: Geometry, w) -> np.ndarray:
    """[NB, NB]: key block j within the (w_t, w_h, w_w) block window of query block i."""
    if w is None or min(w) < 0:
        return np.zeros((g.NB, g.NB), dtype=bool)
    c = block_coords(g)
    diff = np.abs(c[:, None, :] - c[None, :, :])
    return np.all(diff <= np.asarray(w, dtype=np.int64), axis=-1)


def sink_blocks(g: Geometry, s: int) -> np.ndarray:
    """[NB]: blocks holding at least one of the first s raster tokens."""
    slot_token, n_valid = block_tables(g)
    marks = np.zeros(g.NB, dtype=bool)
    for b in range(g.NB):
        toks = slot_token[b * g.BS: b * g.BS + n_valid[b]]
        marks[b] = bool(np.any(toks < s))
    return marks


@dataclass(frozen=True)
class MaskSpec:
    """What one selection call composes (§3.1 sparsity-ratio scheme)."""
    estimator: str = "mean"            # "mean" | "dsa" | "dsa2"
    mode: str = "topk"                 # inter rule: "topk" | "topp"
    topk: int | None = None
    tau: float | None = None
    topk_per_head: tuple | None = None  # [H] budgets replacing topk
    tau_per_head: tuple | None = None   # [H] budgets replacing tau
    intra: str | None = None           # None | "threshold" | "topk"
    intra_theta: float | None = None
    intra_topk: int | None = None
    window: tuple | None = None        # (w_t, w_h, w_w) block radii
    sink: int = 0                      # attention-sink length in tokens


def select_per_head(scores: np.ndarray, spec: MaskSpec):
    """The inter rule on [B, H, NB, NB] scores, with per-head k or tau if given."""
    H = scores.shape[1]
    counts = np.zeros(scores.shape[:-1], dtype=np.int32)
    indices = np.full(scores.shape, -1, dtype=np.int32)
    for h in range(H):
        k = spec.topk_per_head[h] if spec.topk_per_head is not None else spec.topk
        t = spec.tau_per_head[h] if spec.tau_per_head is not None else spec.tau
        c, ix = select(scores[:, h:h + 1], spec.mode, topk=k, tau=t)
        counts[:, h:h + 1], indices[:, h:h + 1] = c, ix
    return counts, indices


def compose_mask(inter: np.ndarray, intra_q=None, intra_k=None, window=None, sink=None):
    """[B, H, NB, NB] OR of the inter mask, the broadcast intra marks (rows for
    Q, columns for K), the window [NB, NB] and the sink columns [NB]."""
    m = inter.copy()
    if intra_q is not None:
        m |= intra_q[..., :, None]
    if intra_k is not None:
        m |= intra_k[..., None, :]
    if window is not None:
        m |= window
    if sink is not None:
        m |= sink
    return m


def lists_from_mask(mask: np.ndarray):
    """counts [.., NB] and ascending index lists [.., NB, NB] (-1 padded) of a mask."""
    NB = mask.shape[-1]
    counts = mask.sum(axis=-1).astype(np.int32)
    indices = np.full(mask.shape, -1, dtype=np.int32)
    for idx in np.ndindex(*mask.shape[:-1]):
        kept = np.nonzero(mask[idx])[0]
        indices[idx + (slice(0, kept.size),)] = kept
    assert indices.shape[-1] == NB
    return counts, indices


def composed_selection(Q, K, g: Geometry, spec: MaskSpec, scale=None) -> dict:
    """Blocking -> Summarizer -> estimator -> inter rule -> intra filter, window
    and sink -> OR -> block lists (§3.3 order)."""
    Q, K = (np.asarray(a, dtype=np.float64) for a in (Q, K))
    scale = 1.0 / np.sqrt(Q.shape[-1]) if scale is None else scale
    Qb, Kb = reorder(Q, g), reorder(K, g)
    out = {}
    if spec.estimator == "mean":
        qbar, kbar = block_means(Qb, g), block_means(Kb, g)
        s = block_scores(qbar, kbar, scale)
        out.update(qbar=qbar, kbar=kbar)
    else:
        (qmax, qmin), (kmax, kmin) = block_maxmin(Qb, g), block_maxmin(Kb, g)
        est = dsa_scores if spec.estimator == "dsa" else dsa2_scores
        s = est(qmax, qmin, kmax, kmin, scale)
        out.update(qmax=qmax, qmin=qmin, kmax=kmax, kmin=kmin)
    ci, ii = select_per_head(s, spec)
    inter = block_mask(ci, ii)
    iq = ik = None
    if spec.intra is not None:
        sq, sk = block_sics(Qb, g), block_sics(Kb, g)
        iq = intra_marks(sq, g, spec.intra, spec.intra_theta, spec.intra_topk)
        ik = intra_marks(sk, g, spec.intra, spec.intra_theta, spec.intra_topk)
        out.update(sics_q=sq, sics_k=sk)
    win = window_mask(g, spec.window) if spec.window is not None else None
    snk = sink_blocks(g, spec.sink) if spec.sink > 0 else None
    mask = compose_mask(inter, iq, ik, win, snk)
    counts, indices = lists_from_mask(mask)
    out.update(scores=s, inter_counts=ci, inter_indices=ii, intra_q=iq, intra_k=ik,
               mask=mask, counts=counts, indices=indices, Qb=Qb, Kb=Kb)
    return out


def spade_attention_composed(Q, K, V, g: Geometry, spec: MaskSpec, scale=None) -> dict:
    """The whole path with the composed mask: selection, Eq. (2), restore."""
    V = np.asarray(V, dtype=np.float64)
    scale = 1.0 / np.sqrt(V.shape[-1]) if scale is None else scale
    r = composed_selection(Q, K, g, spec, scale)
    Ob, lse = block_sparse_attention(r["Qb"], r["Kb"], reorder(V, g), r["counts"],
                                     r["indices"], g, scale)
    r.update(O=inverse_reorder(Ob, g), Ob=Ob, lse=lse)
    return r


# --------------------------------------------------------------------------
# Policy function (§3.1: head-wise sparsity-ratio schemes from the inference
# state and the Selected Aggregation Score; §4: Func 0 / Func 1 budgets, dense
# warm-up steps, Turbo)
# --------------------------------------------------------------------------
WINDOW_LADDER = ((0, 0, 0), (0, 0, 1), (0, 1, 1), (1, 1, 1), (1, 1, 2), (1, 2, 2), (2, 2, 2))
STATIC_SHARE = {0: 1.0 / 31.0, 1: 0.2}


def policy_dense(step: int, n_steps: int, task: str = "t2v", turbo: bool = False) -> bool:
    """Whether denoising step `step` (0-based) of n_steps runs full attention."""
    if turbo:
        return step < 1
    frac = 0.30 if task == "t2v" else 0.25
    return step < int(np.ceil(frac * n_steps - 1e-9))


def window_size(w) -> int:
    return (2 * w[0] + 1) * (2 * w[1] + 1) * (2 * w[2] + 1)


def policy_split(k_total: int, func: int):
    """(window radii or None, window size, k_dyn) for a per-row budget of k_total."""
    k_static = int(np.floor(k_total * STATIC_SHARE[func] + 0.5))
    fits = [w for w in WINDOW_LADDER if window_size(w) <= k_static]
    if not fits:
        return None, 0, k_total
    w = fits[-1]
    return w, window_size(w), k_total - window_size(w)


def policy_head_budgets(as_best, k_dyn: int, NB: int) -> np.ndarray:
    """Per-head dynamic k, negatively correlated with the Selected AS (see header)."""
    as_best = [float(a) for a in as_best]
    H = len(as_best)
    w = [1.0 / a if a > 0.0 else 0.0 for a in as_best]   # no score: no extra budget
    W = 0.0
    for x in w:                      # head order, one addition at a time
        W += x
    if not W > 0.0:                  # no head has a score: the flat budget
        return np.full(H, min(max(k_dyn, 1), NB), dtype=np.int32)
    total = float(H) * float(k_dyn)
    return np.array([min(max(int(np.floor(total * x / W + 0.5)), 1), NB) for x in w],
                    dtype=np.int32)


def policy_head_tau(as_best, tau: float) -> np.ndarray:
    """Per-head Top-P mass for a Top-P scheme, negatively correlated with the
    Selected AS (reading): the dropped mass 1 - tau is spread over the heads in
    proportion to their score, e_h = (H (1 - tau)) * AS_h / S with S the sum of the
    positive scores in head order, and tau_h = 1 - e_h. The mean dropped mass stays
    1 - tau; a head with AS <= 0 drops nothing (tau_h = 1); S = 0 gives every head
    tau. tau_h may fall to or below 0, which keeps only the top block."""
    a = [max(float(x), 0.0) for x in as_best]
    H = len(a)
    S = 0.0
    for x in a:                      # head order, one addition at a time
        S += x
    if not S > 0.0:
        return np.full(H, float(tau))
    total = float(H) * (1.0 - float(tau))
    return np.array([1.0 - total * x / S for x in a], dtype=np.float64)


# --------------------------------------------------------------------------
# Whole path and work counters
# --------------------------------------------------------------------------
def spade_attention(Q, K, V, g: Geometry, mode: str, topk=None, tau=None, scale=None):
    """blocking -> means -> scores -> selection -> Eq. (2) -> restore layout."""
    Q, K, V = (np.asarray(a, dtype=np.float64) for a in (Q, K, V))
    d = Q.shape[-1]
    scale = 1.0 / np.sqrt(d) if scale is None else scale
    Qb, Kb, Vb = reorder(Q, g), reorder(K, g), reorder(V, g)
    qbar, kbar = block_means(Qb, g), block_means(Kb, g)
    s = block_scores(qbar, kbar, scale)
    counts, indices = select(s, mode, topk=topk, tau=tau)
    Ob, lse = block_sparse_attention(Qb, Kb, Vb, counts, indices, g, scale)
    return dict(O=inverse_reorder(Ob, g), Ob=Ob, lse=lse, qbar=qbar, kbar=kbar,
                scores=s, counts=counts, indices=indices)


def kept_flops(counts, indices, g: Geometry, d: int) -> float:
    """Matmul FLOPs of the kept work: sum over kept (i, j) of 4 * n_i * n_j * d."""
    _, n_valid = block_tables(g)
    total = 0
    for idx in np.ndindex(*counts.shape):
        i = idx[-1]
        kept = indices[idx][: counts[idx]]
        total += 4 * int(n_valid[i]) * int(n_valid[kept].sum()) * d
    return float(total)


def block_sparsity(counts, NB: int) -> float:
    return 1.0 - float(np.asarray(counts, dtype=np.float64).sum()) / (counts.size * NB)
