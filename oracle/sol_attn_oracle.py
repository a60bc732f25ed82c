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
  * a row with no term at all (only possible without the correction) outputs 0;
  * causal masks (an extension the Appendix names as future work: row-dependent masks
    need centring and multiplicity over valid keys).  With granule G, key s is visible
    to query t iff s < min((t // G + 1) G, N): G = 1 is token-causal attention, G = a
    frame's token count is frame-causal attention.  Key blocks visible to every row of
    a query block are its routable blocks: mu_i and sigma_i are taken over them only and
    their multiplicity is their full valid-token count.  Key blocks visible to some rows
    only are computed exactly under the token mask, like forced blocks; blocks visible
    to none are skipped.
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


# ---------------------------------------------------------------------------
# Causal masks (extension: the Appendix's row-dependent masks)
# ---------------------------------------------------------------------------

def causal_limits(n_tokens: int, granule: int) -> np.ndarray:
    """lim[t] = min((t // G + 1) * G, N): query t sees exactly the keys s < lim[t]."""
    t = np.arange(n_tokens, dtype=np.int64)
    return np.minimum((t // granule + 1) * granule, n_tokens)


def causal_block_ranges(n_tokens: int, block_q: int, block_k: int, granule: int):
    """Per query block i, (r_i, e_i): key blocks [0, r_i) are visible to every row of
    the block (its routable blocks), [r_i, e_i) to some rows only, [e_i, NK) to none.
    Visibility is a prefix of the keys and lim[t] grows with t, so the first row of a
    block fixes r_i and its last row fixes e_i."""
    lim = causal_limits(n_tokens, granule)
    kcounts = block_counts(n_tokens, block_k)
    kend = np.arange(len(kcounts)) * block_k + kcounts          # exclusive end of each key block
    kstart = np.arange(len(kcounts)) * block_k
    nq = -(-n_tokens // block_q)
    r = np.empty(nq, dtype=np.int64)
    e = np.empty(nq, dtype=np.int64)
    for i in range(nq):
        lo = lim[i * block_q]
        hi = lim[min((i + 1) * block_q, n_tokens) - 1]
        r[i] = int(np.count_nonzero(kend <= lo))
        e[i] = int(np.count_nonzero(kstart < hi))
    return r, e


def causal_row_stats(s_hat: np.ndarray, r: np.ndarray):
    """mu_i and sigma_i over the routable prefix j < r_i of each proxy row (population
    normaliser 1/r_i, as for the full row); NaN where r_i = 0."""
    valid = np.arange(s_hat.shape[-1])[None, :] < r[:, None]
    cnt = np.where(r > 0, r, 1).astype(np.float64)
    mu = np.where(valid, s_hat, 0.0).sum(axis=-1) / cnt
    var = np.where(valid, (s_hat - mu[..., None]) ** 2, 0.0).sum(axis=-1) / cnt
    mu = np.where(r > 0, mu, np.nan)
    return mu, np.where(r > 0, np.sqrt(var), np.nan)


def causal_route(s_hat: np.ndarray, tau: np.ndarray, r: np.ndarray) -> np.ndarray:
    """S_i = {j < r_i : s_hat_ij > tau_i}."""
    valid = np.arange(s_hat.shape[-1])[None, :] < r[:, None]
    with np.errstate(invalid="ignore"):
        return valid & (s_hat > tau[..., None])


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

def exact_logits(q_rows, keys, scale, visible=None):
    """Exact logits scale * q.k_u of each row against a set of keys, -inf where the row does not
    see the key (``visible`` [rows, keys], causal masks)."""
    lg = scale * (q_rows @ keys.T)
    if visible is not None:
        lg = np.where(visible, lg, -np.inf)
    return lg


def exact_terms(q_rows, keys, values, scale, shift, visible=None, logits=None):
    """Exact-branch contributions of a set of keys to each row:
    D = sum_u exp(scale q.k_u - shift),  N = sum_u exp(scale q.k_u - shift) v_u,
    the sums running over the keys a row sees (``visible`` [rows, keys], causal masks).
    ``logits``: the same rows' exact_logits(q_rows, keys, scale, visible), if already formed."""
    if logits is None:
        logits = exact_logits(q_rows, keys, scale, visible)
    w = np.exp(logits - shift[:, None])
    if visible is not None:
        w = np.where(visible, w, 0.0)
    return w.sum(axis=1), w @ values


def approx_terms(q_rows, kbar_blocks, vhat_blocks, counts, scale, shift):
    """Zeroth-order contributions of unselected blocks (Eq. zeroth_order_expansion
    kept to its first term): D = sum_j n_j exp(scale q.Kbar_j - shift),
    N = sum_j exp(scale q.Kbar_j - shift) Vhat_j with Vhat_j the block's value sum."""
    w = np.exp(scale * (q_rows @ kbar_blocks.T) - shift[:, None])
    return w @ counts.astype(np.float64), w @ vhat_blocks


def _forward_head(args):
    (qh, kh, vh, block_q, block_k, beta, mode, n_forced, qblocks, mask_h, threshold_mode, granule) = args
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
    if granule:
        lim = causal_limits(n, granule)
        r_blk, e_blk = causal_block_ranges(n, block_q, block_k, granule)
        mu, sigma = causal_row_stats(s_hat, r_blk)
    else:
        r_blk = np.full(len(qbar), nkr, dtype=np.int64)
        e_blk = np.full(len(qbar), nk, dtype=np.int64)
        mu, sigma = row_stats(s_hat)
        if threshold_mode == "diagonal":
            sigma = diagonal_sigma(qbar, kbar[:nkr], scale)
    tau = thresholds(mu, sigma, beta)
    if mask_h is not None:
        sel = np.asarray(mask_h, dtype=bool)
    else:
        sel = causal_route(s_hat, tau, r_blk) if granule else route(s_hat, tau)
    routable = np.arange(nkr)[None, :] < r_blk[:, None]
    with np.errstate(invalid="ignore"):
        band = int(np.count_nonzero(routable & (np.abs(s_hat - tau[:, None]) < BAND)))

    out = np.full((n, d), np.nan)
    for i in qblocks:
        r0, r1 = i * block_q, min((i + 1) * block_q, n)
        q_rows = qh[r0:r1]
        ri, ei = int(r_blk[i]), int(e_blk[i])
        forced = list(range(ri, ei)) if granule else list(range(nkr, nk))
        if mode == "dense":
            exact_blocks, approx_blocks = list(range(ei)), []
        else:
            exact_blocks = [j for j in range(ri) if sel[i, j]] + forced
            approx_blocks = [j for j in range(ri) if not sel[i, j]] if mode == "sparse" else []
        key_idx = np.concatenate([np.arange(j * block_k, j * block_k + kcounts[j]) for j in exact_blocks]) \
            if exact_blocks else np.zeros(0, dtype=np.int64)
        visible = key_idx[None, :] < lim[r0:r1, None] if granule else None
        ab = np.asarray(approx_blocks, dtype=np.int64)
        # Row shift for overflow safety: the largest exponent of any term.
        cand = []
        lg = None
        if key_idx.size:
            lg = exact_logits(q_rows, kh[key_idx], scale, visible)
            cand.append(lg.max(axis=1))
        if ab.size:
            cand.append((scale * (q_rows @ kbar[ab].T) + np.log(kcounts[ab])).max(axis=1))
        if not cand:
            out[r0:r1] = 0.0
            continue
        shift = np.max(np.stack(cand), axis=0)
        empty = ~np.isfinite(shift)        # causal rows with no visible term (no correction)
        shift = np.where(empty, 0.0, shift)
        den = np.zeros(r1 - r0)
        num = np.zeros((r1 - r0, d))
        if key_idx.size:
            dd, nn = exact_terms(q_rows, None, vh[key_idx], scale, shift, visible, logits=lg)
            den += dd
            num += nn
        if ab.size:
            dd, nn = approx_terms(q_rows, kbar[ab], vhat[ab], kcounts[ab], scale, shift)
            den += dd
            num += nn
        with np.errstate(invalid="ignore", divide="ignore"):
            out[r0:r1] = np.where(den[:, None] > 0, num / np.where(den > 0, den, 1.0)[:, None], 0.0)
    return out, sel, s_hat, tau, mu, sigma, band, int(r_blk.sum())


def forward(q, k, v, block_q: int, block_k: int, beta: float, mode: str,
            keep_tail_tokens: int = 0, query_blocks: Optional[Sequence[int]] = None,
            mask: Optional[np.ndarray] = None, heads: Optional[Sequence] = None,
            workers: int = 0, threshold_mode: str = "exact", causal_granule: int = 0) -> dict:
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
    causal_granule: 0 for bidirectional attention, G >= 1 for the causal mask
    s < min((t // G + 1) G, N) (statistics over each query block's routable prefix).

    Returns a dict with out [B,H,N,d] float64, mask [B,H,NQ,NKr] bool, s_hat, tau,
    mu, sigma, frac [B,H] (kept fraction of routable pairs; 1.0 for dense) and
    band [B,H] (routable pairs with |s_hat - tau| < 1e-3).
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
    if causal_granule < 0:
        raise ValueError("causal_granule must be >= 0")
    if causal_granule and (keep_tail_tokens or threshold_mode != "exact"):
        raise ValueError("causal masks take no forced tail and the exact threshold estimator only")
    n_forced = keep_tail_tokens // block_k
    nq = -(-n // block_q)
    nk = -(-n // block_k)
    nkr = nk - n_forced
    qblocks = list(range(nq)) if query_blocks is None else list(query_blocks)
    head_list = [(b, h) for b in range(B) for h in range(H)] if heads is None else list(heads)

    jobs = [(q[b, h], k[b, h], v[b, h], block_q, block_k, beta, mode, n_forced, qblocks,
             None if mask is None else mask[b, h], threshold_mode, causal_granule) for b, h in head_list]
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
    for (b, h), (out, sel, s_hat, tau, mu, sigma, band, n_routable) in zip(head_list, results):
        res["out"][b, h] = out
        res["mask"][b, h] = sel
        res["s_hat"][b, h] = s_hat
        res["tau"][b, h] = tau
        res["mu"][b, h] = mu
        res["sigma"][b, h] = sigma
        res["frac"][b, h] = 1.0 if mode == "dense" else sel.sum() / max(n_routable, 1)
        res["band"][b, h] = band
    return res


def routing(q, k, block_q: int, block_k: int, beta: float, keep_tail_tokens: int = 0,
            threshold_mode: str = "exact", causal_granule: int = 0) -> dict:
    """Routing only (pool -> proxies -> row statistics -> thresholds -> mask) for
    all heads; cheap enough for the full 720p map.  With causal_granule > 0 the
    statistics and the mask cover each query block's routable prefix only."""
    q = np.asarray(q)
    k = np.asarray(k)
    d = q.shape[-1]
    scale = 1.0 / math.sqrt(d)
    n_forced = keep_tail_tokens // block_k
    qbar, _ = pool_means(q, block_q)
    kbar, _ = pool_means(k, block_k)
    nkr = kbar.shape[-2] - n_forced
    s_hat = proxy_scores(qbar, kbar[..., :nkr, :], scale)
    if causal_granule:
        if keep_tail_tokens or threshold_mode != "exact":
            raise ValueError("causal masks take no forced tail and the exact threshold estimator only")
        r_blk, _ = causal_block_ranges(q.shape[-2], block_q, block_k, causal_granule)
        mu, sigma = causal_row_stats(s_hat.reshape(-1, nkr), np.tile(r_blk, s_hat.size // (len(r_blk) * nkr)))
        mu, sigma = mu.reshape(s_hat.shape[:-1]), sigma.reshape(s_hat.shape[:-1])
        tau = thresholds(mu, sigma, beta)
        routable = np.arange(nkr)[None, :] < r_blk[:, None]
        with np.errstate(invalid="ignore"):
            sel = routable & (s_hat > tau[..., None])
        n_routable = float(r_blk.sum())
    else:
        mu, sigma = row_stats(s_hat)
        if threshold_mode == "diagonal":
            sigma = diagonal_sigma(qbar, kbar[..., :nkr, :], scale)
        tau = thresholds(mu, sigma, beta)
        sel = route(s_hat, tau)
        routable = np.ones(s_hat.shape[-2:], dtype=bool)
        n_routable = float(routable.size)
    with np.errstate(invalid="ignore"):
        band = np.count_nonzero(routable & (np.abs(s_hat - tau[..., None]) < BAND), axis=(-1, -2))
    return {"mask": sel, "s_hat": s_hat, "tau": tau, "mu": mu, "sigma": sigma,
            "frac": sel.sum(axis=(-1, -2)) / n_routable, "band": band, "qbar": qbar, "kbar": kbar,
            "routable": routable}

