"""Workload definitions: attention-layer shapes of the video DiTs the paper runs.

Each entry gives the grid (T, Hs, Ws), heads H, head dim d, the 3D block
(bt, bh, bw), the selection rule, and the generator constants (gain and
per-head bandwidth) chosen so that the selection lands near the sparsity the
paper reports (about 85% block sparsity for Hunyuan-Video at 720p, Table 2).
The generator constants are input recipe, not method parameters.
"""
from __future__ import annotations

import numpy as np


def _logspace_heads(H: int, f_lo: float, f_hi: float):
    return list(np.geomspace(f_lo, f_hi, H)) if H > 1 else [f_lo]


WORKLOADS = {
    # Small case the oracle finishes instantly: 2 heads, 8 blocks of 32 tokens.
    "tiny": dict(B=1, H=2, d=64, T=4, Hs=8, Ws=8, bt=2, bh=4, bw=4,
                 mode="topk", topk=3, tau=None, gain=1.0, freqs=[0.08, 0.15],
                 aniso=(1.0, 1.0, 1.0), in_dtype="fp32"),
    # Wan 2.1 1.3B, 480p, 81 frames: 21 latent frames of 30 x 52 tokens.
    "wan13b": dict(B=1, H=12, d=128, T=21, Hs=30, Ws=52, bt=3, bh=6, bw=8,
                   mode="topp", topk=None, tau=0.9, gain=2.6, freqs=None,
                   f_lo=0.030, f_hi=0.030, aniso=(1.0, 1.0, 1.0), in_dtype="bf16"),
    # Hunyuan-Video, 720p, 61 frames: 16 latent frames of 45 x 80 tokens.
    "hunyuan": dict(B=1, H=24, d=128, T=16, Hs=45, Ws=80, bt=4, bh=5, bw=8,
                    mode="topp", topk=None, tau=0.9, gain=None, g_lo=2.15, g_hi=3.3,
                    freqs=None, f_cycle=(0.015, 0.03, 0.06), aniso=(1.0, 1.0, 1.0),
                    in_dtype="bf16"),
    # Wan 2.1 14B, 720p, 81 frames: 21 latent frames of 45 x 80 tokens; half the
    # heads local (narrow field), half near-global (wide field).
    "wan14b": dict(B=1, H=40, d=128, T=21, Hs=45, Ws=80, bt=3, bh=5, bw=8,
                   mode="topp", topk=None, tau=0.9, gain=None, freqs=None,
                   split_heads=dict(local=(2.9, 0.03), wide=(2.5, 0.08)),
                   aniso=(1.0, 1.0, 1.0), in_dtype="bf16"),
    # Hunyuan-Video shape for the block-shape sweep: heads cycle through fields
    # that vary fastest along t, y, x or evenly, so different candidates win.
    "hunyuan_sweep": dict(B=1, H=24, d=128, T=16, Hs=45, Ws=80, bt=4, bh=5, bw=8,
                          mode="topk", topk=None, tau=None, gain=None, g_lo=2.15, g_hi=3.3,
                          freqs=None, f_cycle=(0.015, 0.03, 0.06),
                          aniso_cycle=((2.5, 1.0, 1.0), (1.0, 2.5, 1.0), (1.0, 1.0, 2.5),
                                       (1.0, 1.0, 1.0)),
                          in_dtype="bf16"),
}

# The experiments' selection (DSA estimate, intra-block thresholding, inter Top-K)
# plus a static spatial window, with budgets of roughly 80% dynamic and 20%
# static blocks at about 85% block sparsity: k dynamic blocks per row and a
# (0, 1, 1) window of up to 9 blocks. The coherence bound sits near the 1st
# percentile of this generator's block coherence for the layer (seed 0), so the
# filter marks about 1% of the blocks (mostly in the wide-field heads).
DSA_SCHEMES = {
    "hunyuan": dict(topk=43, window=(0, 1, 1), intra_theta=0.41),
    "wan13b": dict(topk=27, window=(0, 1, 1), intra_theta=0.62),
    "wan14b": dict(topk=76, window=(0, 1, 1), intra_theta=0.27),
}

# Blocking-scheme candidates of the block-shape sweep (two of 128 tokens, two
# of 160) and its target block sparsities.
SWEEP_CANDIDATES = ((2, 8, 8), (4, 4, 8), (4, 5, 8), (8, 5, 4))
SWEEP_SPARSITIES = (0.70, 0.85, 0.95)


def _split(cfg: dict, k: int):
    H = cfg["H"]
    half = H // 2
    sp = cfg["split_heads"]
    return [sp["local"][k]] * half + [sp["wide"][k]] * (H - half)


def head_gains(cfg: dict):
    H = cfg["H"]
    if cfg.get("split_heads"):
        return _split(cfg, 0)
    if cfg.get("gain") is not None:
        return [float(cfg["gain"])] * H
    return _logspace_heads(H, cfg["g_lo"], cfg["g_hi"])


def head_freqs(cfg: dict):
    H = cfg["H"]
    if cfg.get("freqs") is not None:
        return list(cfg["freqs"])
    if cfg.get("f_cycle") is not None:
        cyc = cfg["f_cycle"]
        return [cyc[h % len(cyc)] for h in range(H)]
    if cfg.get("split_heads"):
        return _split(cfg, 1)
    return _logspace_heads(H, cfg["f_lo"], cfg["f_hi"])


def workload(name: str, **overrides) -> dict:
    cfg = dict(WORKLOADS[name])
    cfg.update(overrides)
    cfg["name"] = name
    cfg["N"] = cfg["T"] * cfg["Hs"] * cfg["Ws"]
    cfg["head_freqs"] = head_freqs(cfg)
    cfg["head_gains"] = head_gains(cfg)
    if cfg.get("aniso_cycle") is not None:
        cyc = cfg["aniso_cycle"]
        cfg["aniso"] = [tuple(cyc[h % len(cyc)]) for h in range(cfg["H"])]
    return cfg


def make_inputs(cfg: dict, *, seed: int = 0, device="cpu"):
    """fp32 Q, K, V for a workload (callers round to bf16 themselves)."""
    from .synth import smooth_field_qkv
    return smooth_field_qkv(cfg["B"], cfg["H"], cfg["T"], cfg["Hs"], cfg["Ws"], cfg["d"],
                            seed=seed, gain_qk=cfg["head_gains"], freqs=cfg["head_freqs"],
                            aniso=cfg["aniso"], device=device)
