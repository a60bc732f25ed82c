"""Seeded synthetic Q/K/V with the structure of video/image DiT attention inputs.

This module holds no attention arithmetic: it only draws the inputs that both the
GPU path and the CPU reference consume.

Recipe (one independent stream per (batch, head), from
``numpy.random.SeedSequence(seed).spawn(B*H)`` with PCG64):

* tokens lie on a raster-ordered grid, index ``n = (t*Hg + h)*Wg + w`` (video) or
  ``n = h*Wg + w`` (image); text tokens, if any, are appended at the tail;
* a length scale ``l ~ U[lo, hi]`` grid cells per head;
* M = 8 random Fourier features of the grid position: frequencies
  ``omega_m ~ N(0, l^-2 I)``, phases ``phi_m ~ U[0, 2pi)``,
  ``f_m(p) = sqrt(2/M) sin(omega_m . p + phi_m)``;
* one projection ``P ~ N(0,1)^{M x d}`` shared by Q and K, so that smooth-field
  structure shows up in the block-pooled logits (the attention locality that the
  paper's routing exploits);
* ``Q = F P + 0.5 eps_Q``, ``K = F P + 0.5 eps_K``, ``V ~ N(0,1)``;
* text tokens: Q, K, V ~ N(0,1).

Values are drawn in float32 and rounded once to the workload dtype (bf16 by
round-to-nearest-even, or kept as f32).
"""
from __future__ import annotations

import os
from concurrent.futures import ProcessPoolExecutor
from typing import Optional, Sequence, Tuple

import numpy as np

N_FEATURES = 8
NOISE = 0.5


def _grid_positions(grid: Sequence[int]) -> np.ndarray:
    axes = [np.arange(g, dtype=np.float64) for g in grid]
    mesh = np.meshgrid(*axes, indexing="ij")
    return np.stack([m.reshape(-1) for m in mesh], axis=1)  # [prod(grid), ndim]


def _head_qkv(args) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    seed_seq, grid, text_tokens, d, lo, hi = args
    rng = np.random.Generator(np.random.PCG64(seed_seq))
    pos = _grid_positions(grid)
    n_img = pos.shape[0]
    n = n_img + text_tokens
    ell = rng.uniform(lo, hi)
    omega = rng.standard_normal((N_FEATURES, pos.shape[1])) / ell
    phase = rng.uniform(0.0, 2.0 * np.pi, size=N_FEATURES)
    proj = rng.standard_normal((N_FEATURES, d))
    feats = np.sqrt(2.0 / N_FEATURES) * np.sin(pos @ omega.T + phase)
    field = (feats @ proj).astype(np.float32)
    q = np.empty((n, d), np.float32)
    k = np.empty((n, d), np.float32)
    q[:n_img] = field + NOISE * rng.standard_normal((n_img, d), dtype=np.float32)
    k[:n_img] = field + NOISE * rng.standard_normal((n_img, d), dtype=np.float32)
    v = rng.standard_normal((n, d), dtype=np.float32)
    if text_tokens:
        q[n_img:] = rng.standard_normal((text_tokens, d), dtype=np.float32)
        k[n_img:] = rng.standard_normal((text_tokens, d), dtype=np.float32)
    return q, k, v


def make_qkv(workload, heads: Optional[Sequence[Tuple[int, int]]] = None,
             workers: int = 0):
    """Return (q, k, v) as CPU torch tensors of shape [B, H, N, d] in the
    workload dtype (torch.bfloat16 or torch.float32).

    ``heads``: optional list of (b, h) to fill; other heads are left zero (used
    by tests that only need a few heads of a large shape).
    ``workers``: >1 generates heads in a process pool.
    """
    import torch

    w = workload
    tdtype = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    children = np.random.SeedSequence(w.seed).spawn(w.B * w.H)
    want = [(b, h) for b in range(w.B) for h in range(w.H)] if heads is None else list(heads)
    out = [torch.zeros((w.B, w.H, w.N, w.d), dtype=tdtype) for _ in range(3)]
    jobs = [(children[b * w.H + h], w.grid, w.text_tokens, w.d, *w.length_scale) for b, h in want]
    if workers and workers > 1 and len(jobs) > 1:
        with ProcessPoolExecutor(max_workers=min(workers, len(jobs))) as ex:
            results = list(ex.map(_head_qkv, jobs))
    else:
        results = [_head_qkv(j) for j in jobs]
    for (b, h), arrs in zip(want, results):
        for t, a in zip(out, arrs):
            t[b, h] = torch.from_numpy(a).to(tdtype)
    return tuple(out)


def default_workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(n, 16))
