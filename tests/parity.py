"""Helpers shared by the GPU parity tests: tolerances, metrics and small
synthetic workloads."""
from __future__ import annotations

import math

import numpy as np

from paper_2607_24027_amd.configs import Workload

# Output tolerances against the fp64 oracle.
BF16_MAX_ABS, BF16_MEAN_REL = 2e-2, 2e-3
F32_MAX_ABS, F32_MEAN_REL = 1e-4, 1e-5


def to_np(t) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def errors(gpu: np.ndarray, ref: np.ndarray):
    ok = ~np.isnan(ref)
    diff = np.abs(gpu[ok] - ref[ok])
    return float(diff.max()), float(diff.sum() / max(np.abs(ref[ok]).sum(), 1e-300))


def assert_output_close(gpu: np.ndarray, ref: np.ndarray, dtype: str, what: str = ""):
    max_abs, mean_rel = errors(gpu, ref)
    if dtype == "bf16":
        tol = (BF16_MAX_ABS, BF16_MEAN_REL)
    else:
        tol = (F32_MAX_ABS, F32_MEAN_REL)
    assert max_abs <= tol[0] and mean_rel <= tol[1], \
        f"{what}: max-abs {max_abs:.3e} (tol {tol[0]:.0e}), mean-rel {mean_rel:.3e} (tol {tol[1]:.0e})"
    return max_abs, mean_rel


def assert_mask_matches(gpu_mask: np.ndarray, ora_mask: np.ndarray, s_hat: np.ndarray, tau: np.ndarray,
                        band: float = 1e-3):
    """Bit-exact outside |s_hat - tau| < band; returns the number of in-band flips."""
    diff = gpu_mask != ora_mask
    near = np.abs(s_hat - tau[..., None]) < band
    outside = diff & ~near
    assert not outside.any(), f"{int(outside.sum())} mask flips outside the {band} band"
    return int((diff & near).sum())


def small_workload(name, grid, d, bq, dtype="bf16", text_tokens=0, H=2, B=1, seed=11):
    return Workload(name, B=B, H=H, d=d, dtype=dtype, grid=grid, block_q=bq, block_k=64,
                    target_kept=0.3, seed=seed, text_tokens=text_tokens)


def finite_beta(beta):
    return not math.isinf(beta)
