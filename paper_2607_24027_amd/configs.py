"""Workload shapes for the routed-attention hot path.

Each workload mirrors a transformer attention shape from the paper's evaluation
(Section 4, "Models" and "Implementation Details"): a video DiT at 480p and 720p,
an image DiT with appended text tokens, and a small fp32 case for exhaustive
checks.  Inputs are synthetic (see ``synth.py``); the routing cutoff ``beta`` for
each workload is calibrated offline on the CPU reference and stored in
``betas.json`` next to this file.
"""
from __future__ import annotations

import json
import os
from dataclasses import dataclass, field
from typing import Optional, Tuple


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    d: int
    dtype: str                      # "bf16" or "f32"
    grid: Tuple[int, ...]           # token grid, raster order (T,H,W) or (H,W)
    block_q: int
    block_k: int
    target_kept: float              # target fraction of routable blocks kept
    seed: int
    length_scale: Tuple[float, float] = (2.0, 8.0)
    text_tokens: int = 0            # appended N(0,1) tokens, always kept exactly

    @property
    def N(self) -> int:
        n = 1
        for g in self.grid:
            n *= g
        return n + self.text_tokens

    @property
    def NQ(self) -> int:
        return -(-self.N // self.block_q)

    @property
    def NK(self) -> int:
        return -(-self.N // self.block_k)

    @property
    def dense_flop(self) -> float:
        """4*B*H*N^2*d: the dense-equivalent work of one forward (QK^T and PV)."""
        return 4.0 * self.B * self.H * self.N * self.N * self.d


TINY = Workload("tiny", B=1, H=2, d=64, dtype="f32", grid=(4, 16, 32),
                block_q=64, block_k=64, target_kept=0.30, seed=0)
VIDEO_480P = Workload("video480p", B=1, H=12, d=128, dtype="bf16", grid=(21, 30, 52),
                      block_q=128, block_k=64, target_kept=0.25, seed=1)
VIDEO_720P = Workload("video720p", B=1, H=40, d=128, dtype="bf16", grid=(21, 45, 80),
                      block_q=128, block_k=64, target_kept=0.20, seed=2)
IMAGE_2K = Workload("image", B=2, H=24, d=128, dtype="bf16", grid=(128, 128),
                    block_q=64, block_k=64, target_kept=0.35, seed=3,
                    length_scale=(4.0, 16.0), text_tokens=512)

WORKLOADS = {w.name: w for w in (TINY, VIDEO_480P, VIDEO_720P, IMAGE_2K)}

# Kept-fraction sweep at the 720p shape (1.0 means beta = -inf, i.e. dense routing).
SWEEP_KEPT = (1.0, 0.50, 0.25, 0.10, 0.05)

_BETA_FILE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "betas.json")


def load_betas() -> dict:
    """Calibrated cutoffs: {"<workload>@<kept>": beta}.  Missing file -> {}."""
    try:
        with open(_BETA_FILE) as f:
            return json.load(f)
    except FileNotFoundError:
        return {}


def beta_for(workload: Workload, kept: Optional[float] = None, threshold_mode: str = "exact") -> float:
    """Calibrated cutoff for a kept fraction, for the exact or the diagonal threshold estimator."""
    kept = workload.target_kept if kept is None else kept
    if kept >= 1.0:
        return float("-inf")
    key = f"{workload.name}@{kept:.2f}" + ("" if threshold_mode == "exact" else f"/{threshold_mode}")
    betas = load_betas()
    if key not in betas:
        raise KeyError(f"no calibrated beta for {key}; run oracle/calibrate_beta.py")
    return float(betas[key])
