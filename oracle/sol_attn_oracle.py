"""Plain fp64 CPU oracle for the Sol-Attn forward pass.

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call this module.  It imports
nothing from the GPU library and the GPU library imports nothing from it.

Everything is computed in float64 from the (bf16 or f32) input values, in the
order the paper states the method, with numpy matmuls as the only library steps.

Notation (Section 2 "Preliminaries", Section 3 "Methodology"):
    Q_i, K_j, V_j    query block i / key-value block j (rows of the sequence)
    Qbar_i, Kbar_j   token means of a block                      (Eq. block_proxy)
    s_hat_ij         block proxy score Qbar_i . Kbar_j            (Eq. block_proxy)
    mu_i, sigma_i    mean / std of the proxy row s_hat_i          (Eq. threshold_routing)
    tau_i            mu_i + beta * sigma_i                        (Eq. threshold_routing)
    S_i, U_i         selected / unselected key blocks of row i
    D_i, N_i         combined softmax denominator / numerator     (Eqs. solattn_denominator,
                                                                   solattn_numerator)

Readings of the paper used here (each is listed with its reason in the design
notes of the repository):
  * the softmax scale 1/sqrt(d), which the paper omits from Eq. dense_attn, is
    applied to the exact logits and to the proxies alike;
  * proxy statistics use the population normaliser 1/N (Appendix, threshold
    variance derivation) over the routable key blocks only;
  * selection is strict: s_hat_ij > tau_i; beta = -inf keeps every routable block
    and beta = +inf keeps none (the +-inf cases never evaluate inf * sigma);
  * a ragged last block is averaged over its valid tokens and its multiplicity in
    Eq. solattn_denominator is its valid-token count n_j instead of the block size B;
  * V_hat_j in Eq. solattn_numerator is the sum of V over the block's valid tokens;
  * ``keep_tail_tokens`` trailing tokens (text tokens of an MMDiT; Appendix,
    "Generation Configurations") form forced key blocks that are always computed
    exactly and take no part in routing statistics;
  * a row with no term at all (only possible without the correction) outputs 0.
"""
from __future__ import annotations

import math
from concurrent.futures import ProcessPoolExecutor
from typing import Optional, Sequence

import numpy as np

MODES = ("dense", "sparse", "sparse_no_correction")
THRESHOLD_MODES = ("exact", "diagonal")
BAND = 1e-3


# ---------------------------------------------------------------------------
# Pooling and routing (Section 3.1, Eqs. block_proxy and threshold_routing)
# ---------------------------------------------------------------------------

def block_counts(n_tokens: int, block: int) -> np.ndarray:
    """Valid-token count of every block of ``block`` consecutive tokens."""
    nb = -(-n_tokens // block)
    counts = np.full(nb, block, dtype=np.int64)
    counts[-1] = n_tokens - (nb - 1) * block
    return counts


def pool_means(x: np.ndarray, block: int):
    """Token means of consecutive blocks (Eq. block_proxy: Mean along tokens).

    x: [..., N, d].  Returns (means [..., NB, d] float64, counts [NB]).
    """
    x = np.asarray(x, dtype=np.float64)
    n = x.shape[-2]
    counts = block_counts(n, block)
    means = np.empty(x.shape[:-2] + (len(counts), x.shape[-1]), dtype=np.float64)
    for j, c in enumerate(counts):
        means[..., j, :] = x[..., j * block: j * block + c, :].mean(axis=-2)
    return means, counts


def proxy_scores(qbar: np.ndarray, kbar: np.ndarray, scale: float) -> np.ndarray:
    """s_hat_ij = scale * Qbar_i . Kbar_j (Eq. block_proxy)."""
    return scale * (qbar @ np.swapaxes(kbar, -1, -2))


def row_stats(s_hat: np.ndarray):
    """Mean and population standard deviation of each proxy row, straight from
    their definitions (Eq. threshold_routing; Appendix variance derivation)."""
    mu = s_hat.mean(axis=-1)
    sigma = np.sqrt(((s_hat - mu[..., None]) ** 2).mean(axis=-1))
    return mu, sigma


def row_stats_from_moments(qbar: np.ndarray, kbar: np.ndarray, scale: float):
    """The same statistics from the first and second pooled-key moments
    (Eq. threshold_stats_exact), without forming the proxy row."""
    nk = kbar.shape[-2]
    mean_k = kbar.mean(axis=-2)                                   # [..., d]
    second = np.swapaxes(kbar, -1, -2) @ kbar / nk                # [..., d, d]
    mu = scale * np.einsum("...id,...d->...i", qbar, mean_k)
    quad = np.einsum("...id,...de,...ie->...i", qbar, second, qbar)
    var = scale * scale * quad - mu * mu
    return mu, np.sqrt(np.maximum(var, 0.0))


def diagonal_sigma(qbar: np.ndarray, kbar: np.ndarray, scale: float):
    """Diagonal-covariance estimate of sigma_i (Appendix, Eq. appendix_diagonal_threshold):
    v_K = mean_j(Kbar_j * Kbar_j) - mu_K * mu_K over the pooled keys given (the routable
    ones), sigma_i^2 = scale^2 * (Qbar_i * Qbar_i) . v_K."""
    mean_k = kbar.mean(axis=-2)
    v_k = (kbar * kbar).mean(axis=-2) - mean_k * mean_k
    var = scale * scale * ((qbar * qbar) @ v_k[..., None])[..., 0]
    return np.sqrt(np.maximum(var, 0.0))


def thresholds(mu: np.ndarray, sigma: np.ndarray, beta: float) -> np.ndarray:
    """tau_i = mu_i + beta * sigma_i (Eq. threshold_routing), with beta = -inf
    meaning keep all and beta = +inf meaning keep none."""
    if beta == -math.inf:
        return np.full_like(mu, -np.inf)
    if beta == math.inf:
        return np.full_like(mu, np.inf)
    return mu + beta * sigma


def route(s_hat: np.ndarray, tau: np.ndarray) -> np.ndarray:
    """S_i = {j : s_hat_ij > tau_i} (Eq. threshold_routing)."""
    return s_hat > tau[..., None]


def route_topk(s_hat: np.ndarray, k: int) -> np.ndarray:
    """Top-k routing, the fixed-budget baseline of Section 2: the k largest proxies of
    each row (ties go to the lower key-block index)."""
    order = np.argsort(-s_hat, axis=-1, kind="stable")
    mask = np.zeros(s_hat.shape, dtype=bool)
    np.put_along_axis(mask, order[..., :min(k, s_hat.shape[-1])], True, axis=-1)
    return mask


def route_topp(s_hat: np.ndarray, p: float) -> np.ndarray:
    """Top-p routing, the cumulative-mass baseline of Section 2: over the block softmax
    p_hat_i = Softmax(s_hat_i) (Eq. block_proxy), the shortest prefix of blocks in
    decreasing proxy order (ties to the lower index) whose mass reaches p; a block is kept
    when the mass of the blocks before it is below p."""
    order = np.argsort(-s_hat, axis=-1, kind="stable")
    srt = np.take_along_axis(s_hat, order, axis=-1)
    w = np.exp(srt - srt[..., :1])
    mass = w / w.sum(axis=-1, keepdims=True)
    before = np.cumsum(mass, axis=-1) - mass
    keep_sorted = before < p
    mask = np.zeros(s_hat.shape, dtype=bool)
    np.put_along_axis(mask, order, keep_sorted, axis=-1)
    return mask


# ---------------------------------------------------------------------------
# Combined softmax terms (Section 3.2, Eqs. solattn_denominator / numerator)
# ---------------------------------------------------------------------------

def exact_terms(q_rows, keys, values, scale, shift):
    """Exact-branch contributions of a set of keys to each row:
    D = sum_u exp(scale q.k_u - shift),  N = sum_u exp(scale q.k_u - shift) v_u."""
    w = np.exp(scale * (q_rows @ keys.T) - shift[:, None])
    return w.sum(axis=1), w @ values


def approx_terms(q_rows, kbar_blocks, vhat_blocks, counts, scale, shift):
    """Zeroth-order contributions of unselected blocks (Eq. zeroth_order_expansion
    kept to its first term): D = sum_j n_j exp(scale q.Kbar_j - shift),
    N = sum_j exp(scale q.Kbar_j - shift) Vhat_j with Vhat_j the block's value sum."""
    w = np.exp(scale * (q_rows @ kbar_blocks.T) - shift[:, None])
    return w @ counts.astype(np.float64), w @ vhat_blocks


def _forward_head(args):
    (qh, kh, vh, block_q, block_k, beta, mode, n_forced, qblocks, mask_h, threshold_mode) = args
    qh = np.asarray(qh, dtype=np.float64)
    kh = np.asarray(kh, dtype=np.float64)
    vh = np.asarray(vh, dtype=np.float64)
    n, d = qh.shape
    scale = 1.0 / math.sqrt(d)
    qbar, _ = pool_means(qh, block_q)
    kbar, kcounts = pool_means(kh, block_k)
    nk = len(kcounts)
    nkr = nk - n_forced
    vhat = np.stack([vh[j * block_k: j * block_k + c].sum(axis=0) for j, c in enumerate(kcounts)])

    s_hat = proxy_scores(qbar, kbar[:nkr], scale)
    mu, sigma = row_stats(s_hat)
    if threshold_mode == "diagonal":
        sigma = diagonal_sigma(qbar, kbar[:nkr], scale)
    tau = thresholds(mu, sigma, beta)
    sel = route(s_hat, tau) if mask_h is None else np.asarray(mask_h, dtype=bool)
    band = int(np.count_nonzero(np.abs(s_hat - tau[:, None]) < BAND))

    out = np.full((n, d), np.nan)
    forced = list(range(nkr, nk))
    for i in qblocks:
        r0, r1 = i * block_q, min((i + 1) * block_q, n)
        q_rows = qh[r0:r1]
        if mode == "dense":
            exact_blocks, approx_blocks = list(range(nk)), []
        else:
            exact_blocks = [j for j in range(nkr) if sel[i, j]] + forced
            approx_blocks = [j for j in range(nkr) if not sel[i, j]] if mode == "sparse" else []
        key_idx = np.concatenate([np.arange(j * block_k, j * block_k + kcounts[j]) for j in exact_blocks]) \
            if exact_blocks else np.zeros(0, dtype=np.int64)
        ab = np.asarray(approx_blocks, dtype=np.int64)
        # Row shift for overflow safety: the largest exponent of any term.
        cand = []
        if key_idx.size:
            cand.append((scale * (q_rows @ kh[key_idx].T)).max(axis=1))
        if ab.size:
            cand.append((scale * (q_rows @ kbar[ab].T) + np.log(kcounts[ab])).max(axis=1))
        if not cand:
            out[r0:r1] = 0.0
            continue
        shift = np.max(np.stack(cand), axis=0)
        den = np.zeros(r1 - r0)
        num = np.zeros((r1 - r0, d))
        if key_idx.size:
            dd, nn = exact_terms(q_rows, kh[key_idx], vh[key_idx], scale, shift)
            den += dd
            num += nn
        if ab.size:
            dd, nn = approx_terms(q_rows, kbar[ab], vhat[ab], kcounts[ab], scale, shift)
            den += dd
            num += nn
        out[r0:r1] = num / den[:, None]
    return out, sel, s_hat, tau, mu, sigma, band


def forward(q, k, v, block_q: int, block_k: int, beta: float, mode: str,
            keep_tail_tokens: int = 0, query_blocks: Optional[Sequence[int]] = None,
            mask: Optional[np.ndarray] = None, heads: Optional[Sequence] = None,
            workers: int = 0, threshold_mode: str = "exact") -> dict:
    """Sol-Attn forward pass for q, k, v of shape [B, H, N, d].

    mode: "dense" (Eq. dense_attn), "sparse" (exact selected blocks plus the
    zeroth-order correction for unselected ones, Eqs. solattn_denominator and
    solattn_numerator) or "sparse_no_correction" (Eq. block_sparse_attn with the
    routed block mask).
    query_blocks: optional subset of query blocks to evaluate (other rows NaN).
    mask: optional [B, H, NQ, NK_routable] selection to use instead of routing.
    heads: optional list of (b, h) to evaluate (other heads NaN / empty).
    threshold_mode: "exact" (sigma_i from the full proxy row, equal to Eq.
    threshold_stats_exact) or "diagonal" (Appendix, Eq. appendix_diagonal_threshold).

    Returns a dict with out [B,H,N,d] float64, mask [B,H,NQ,NKr] bool, s_hat, tau,
    mu, sigma, frac [B,H] (kept fraction of routable pairs; 1.0 for dense) and
    band [B,H] (pairs with |s_hat - tau| < 1e-3).
    """
    if mode not in MODES:
        raise ValueError(f"mode must be one of {MODES}")
    if threshold_mode not in THRESHOLD_MODES:
        raise ValueError(f"threshold_mode must be one of {THRESHOLD_MODES}")
    q = np.asarray(q)
    k = np.asarray(k)
    v = np.asarray(v)
    B, H, n, d = q.shape
    if keep_tail_tokens % block_k:
        raise ValueError("keep_tail_tokens must be a multiple of block_k")
    n_forced = keep_tail_tokens // block_k
    nq = -(-n // block_q)
    nk = -(-n // block_k)
    nkr = nk - n_forced
    qblocks = list(range(nq)) if query_blocks is None else list(query_blocks)
    head_list = [(b, h) for b in range(B) for h in range(H)] if heads is None else list(heads)

    jobs = [(q[b, h], k[b, h], v[b, h], block_q, block_k, beta, mode, n_forced, qblocks,
             None if mask is None else mask[b, h], threshold_mode) for b, h in head_list]
    if workers and workers > 1 and len(jobs) > 1:
        with ProcessPoolExecutor(max_workers=min(workers, len(jobs))) as ex:
            results = list(ex.map(_forward_head, jobs))
    else:
        results = [_forward_head(j) for j in jobs]

    res = {
        "out": np.full((B, H, n, d), np.nan),
        "mask": np.zeros((B, H, nq, nkr), dtype=bool),
        "s_hat": np.full((B, H, nq, nkr), np.nan),
        "tau": np.full((B, H, nq), np.nan),
        "mu": np.full((B, H, nq), np.nan),
        "sigma": np.full((B, H, nq), np.nan),
        "frac": np.full((B, H), np.nan),
        "band": np.zeros((B, H), dtype=np.int64),
    }
    for (b, h), (out, sel, s_hat, tau, mu, sigma, band) in zip(head_list, results):
        res["out"][b, h] = out
        res["mask"][b, h] = sel
        res["s_hat"][b, h] = s_hat
        res["tau"][b, h] = tau
        res["mu"][b, h] = mu
        res["sigma"][b, h] = sigma
        res["frac"][b, h] = 1.0 if mode == "dense" else sel.mean()
        res["band"][b, h] = band
    return res


def routing(q, k, block_q: int, block_k: int, beta: float, keep_tail_tokens: int = 0,
            threshold_mode: str = "exact") -> dict:
    """Routing only (pool -> proxies -> row statistics -> thresholds -> mask) for
    all heads; cheap enough for the full 720p map."""
    q = np.asarray(q)
    k = np.asarray(k)
    d = q.shape[-1]
    scale = 1.0 / math.sqrt(d)
    n_forced = keep_tail_tokens // block_k
    qbar, _ = pool_means(q, block_q)
    kbar, _ = pool_means(k, block_k)
    nkr = kbar.shape[-2] - n_forced
    s_hat = proxy_scores(qbar, kbar[..., :nkr, :], scale)
    mu, sigma = row_stats(s_hat)
    if threshold_mode == "diagonal":
        sigma = diagonal_sigma(qbar, kbar[..., :nkr, :], scale)
    tau = thresholds(mu, sigma, beta)
    sel = route(s_hat, tau)
    band = np.count_nonzero(np.abs(s_hat - tau[..., None]) < BAND, axis=(-1, -2))
    return {"mask": sel, "s_hat": s_hat, "tau": tau, "mu": mu, "sigma": sigma,
            "frac": sel.mean(axis=(-1, -2)), "band": band, "qbar": qbar, "kbar": kbar}


def frac_selected(mask: np.ndarray) -> np.ndarray:
    """Per-(b,h) fraction of routable (query block, key block) pairs selected."""
    return mask.mean(axis=(-1, -2))
