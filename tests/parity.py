"""Helpers shared by the GPU parity tests: tolerances, metrics and small
synthetic workloads."""
from __future__ import annotations

import math
import os
from concurrent.futures import ProcessPoolExecutor

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


# --------------------------------------------------------------------------- whole heads, in parallel
# The oracle evaluates a head query block by query block.  Its exponentials and key gathers
# run on one core, so whole heads of the large workloads are evaluated as (head, block range)
# jobs in a process pool, one BLAS thread per worker.  The arrays reach the workers through
# fork (copy-on-write), not through pickling.
_JOB_DATA = {}


def _limit_blas_threads():
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)
    except Exception:  # pragma: no cover - threadpoolctl is optional
        pass


def _oracle_job(job):
    from oracle import sol_attn_oracle as ora
    h, lo, hi = job
    d = _JOB_DATA
    mask = None if d["mask"] is None else d["mask"][h][None, None]
    res = ora.forward(d["q"][h][None, None], d["k"][h][None, None], d["v"][h][None, None], d["block_q"],
                      d["block_k"], d["beta"], d["mode"], keep_tail_tokens=d["keep"],
                      query_blocks=list(range(lo, hi)), mask=mask)
    r0, r1 = lo * d["block_q"], min(hi * d["block_q"], d["q"].shape[1])
    return h, r0, r1, res["out"][0, 0, r0:r1]


def pool_workers() -> int:
    """Worker processes for oracle jobs: the CPU share of one GPU (at most 12), at least 1."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(n, 12))


def oracle_whole_heads(q, k, v, block_q, block_k, beta, mode, mask=None, keep_tail_tokens=0, workers=None):
    """Oracle outputs of every row of the given heads.

    q, k, v: [H', N, d] float arrays (the heads to evaluate, input values as given to the GPU);
    mask: [H', NQ, NKr] selection to use instead of routing, or None.  Returns [H', N, d] float64.
    """
    workers = workers or pool_workers()
    hn, n, _ = q.shape
    nq = -(-n // block_q)
    per = max(1, -(-nq * hn // workers))              # one job per worker (each pools its head)
    jobs = [(h, lo, min(lo + per, nq)) for h in range(hn) for lo in range(0, nq, per)]
    _JOB_DATA.update(q=q, k=k, v=v, mask=mask, block_q=block_q, block_k=block_k, beta=beta, mode=mode,
                     keep=keep_tail_tokens)
    out = np.full(q.shape, np.nan)
    try:
        if workers > 1:
            with ProcessPoolExecutor(max_workers=workers, initializer=_limit_blas_threads) as ex:
                results = list(ex.map(_oracle_job, jobs))
        else:
            results = [_oracle_job(j) for j in jobs]
    finally:
        _JOB_DATA.clear()
    for h, r0, r1, rows in results:
        out[h, r0:r1] = rows
    return out
