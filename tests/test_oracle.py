"""Pins for the fp64 CPU oracle: checks against facts the paper and the
mathematics fix, independent of the oracle's own formulas."""
import json
import math
import os
from statistics import NormalDist

import numpy as np
import pytest
import torch
from hypothesis import given, settings
from hypothesis import strategies as st

from oracle import sol_attn_oracle as ora

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rand_qkv(rng, B=1, H=2, N=200, d=16, qscale=1.0):
    q = rng.standard_normal((B, H, N, d)) * qscale
    k = rng.standard_normal((B, H, N, d))
    v = rng.standard_normal((B, H, N, d))
    return q, k, v


def smooth_qkv(rng, B=1, H=2, N=256, d=16):
    """Block-correlated inputs so that routing is far from uniform."""
    t = np.arange(N)[:, None] / 24.0
    f = rng.standard_normal((4, d))
    base = np.sin(t * np.array([1.0, 0.6, 0.3, 0.15]) + rng.uniform(0, 6, 4)) @ f
    q = base + 0.5 * rng.standard_normal((B, H, N, d))
    k = base + 0.5 * rng.standard_normal((B, H, N, d))
    v = rng.standard_normal((B, H, N, d))
    return q, k, v


# --------------------------------------------------------------------------- pooling

def test_pool_means_closed_form_ramp():
    # x[n] = n in every feature: the mean of tokens [a, b) is (a + b - 1) / 2,
    # including the ragged last block of 5 tokens (Eq. block_proxy, valid tokens only).
    n, blk = 69, 16
    x = np.repeat(np.arange(n, dtype=np.float64)[:, None], 3, axis=1)
    means, counts = ora.pool_means(x, blk)
    assert counts.tolist() == [16, 16, 16, 16, 5]
    for j, c in enumerate(counts):
        a = j * blk
        assert np.all(means[j] == (a + a + c - 1) / 2.0)


# --------------------------------------------------------------------------- dense path

@pytest.mark.parametrize("bq,bk,n", [(64, 64, 200), (32, 16, 131), (128, 64, 256)])
def test_dense_matches_library_sdpa(bq, bk, n):
    rng = np.random.default_rng(1)
    q, k, v = rand_qkv(rng, N=n)
    res = ora.forward(q, k, v, bq, bk, 0.5, "dense")
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v)).numpy()
    assert np.max(np.abs(res["out"] - ref)) < 1e-12


def test_beta_minus_inf_reproduces_dense_exactly():
    rng = np.random.default_rng(2)
    q, k, v = smooth_qkv(rng, N=200)
    dense = ora.forward(q, k, v, 64, 32, 0.0, "dense")["out"]
    for mode in ("sparse", "sparse_no_correction"):
        res = ora.forward(q, k, v, 64, 32, -math.inf, mode)
        assert res["mask"].all()
        assert np.array_equal(res["out"], dense)
        assert np.all(res["frac"] == 1.0)


# --------------------------------------------------------------------------- routing

def test_proxy_equals_true_logit_for_blockwise_constant_inputs():
    rng = np.random.default_rng(3)
    n, d, bq, bk = 96, 8, 32, 16
    qb = rng.standard_normal((n // bq, d))
    kb = rng.standard_normal((n // bk, d))
    q = np.repeat(qb, bq, axis=0)
    k = np.repeat(kb, bk, axis=0)
    scale = 1 / math.sqrt(d)
    qbar, _ = ora.pool_means(q, bq)
    kbar, _ = ora.pool_means(k, bk)
    s_hat = ora.proxy_scores(qbar, kbar, scale)
    true = scale * q @ k.T
    for i in range(n // bq):
        for j in range(n // bk):
            blk = true[i * bq:(i + 1) * bq, j * bk:(j + 1) * bk]
            assert np.max(np.abs(blk - s_hat[i, j])) < 1e-12


def test_moment_form_matches_direct_row_statistics():
    # Eq. threshold_stats_exact (moments of the pooled keys) against the row
    # statistics of the materialised proxy row.
    rng = np.random.default_rng(4)
    qbar = rng.standard_normal((2, 3, 40, 32)) + 0.3
    kbar = rng.standard_normal((2, 3, 300, 32)) * 0.7 + 1.1
    scale = 1 / math.sqrt(32)
    mu_d, sd_d = ora.row_stats(ora.proxy_scores(qbar, kbar, scale))
    mu_m, sd_m = ora.row_stats_from_moments(qbar, kbar, scale)
    assert np.max(np.abs(mu_m - mu_d) / np.abs(mu_d).max()) < 1e-10
    assert np.max(np.abs(sd_m - sd_d) / sd_d) < 1e-9


def test_chunked_thresholding_recovers_full_row_set():
    # Streaming the pooled keys in chunks of C and thresholding each chunk gives
    # the same set as thresholding the whole row (Section 3.2, chunk-wise
    # on-the-fly thresholding); C changes nothing.
    rng = np.random.default_rng(5)
    q, k, _ = smooth_qkv(rng, N=512)
    r = ora.routing(q, k, 32, 16, 0.4)
    scale = 1 / math.sqrt(q.shape[-1])
    nk = r["kbar"].shape[-2]
    for c in (1, 7, 64, nk):
        sel = np.zeros_like(r["mask"])
        for t0 in range(0, nk, c):
            chunk = ora.proxy_scores(r["qbar"], r["kbar"][..., t0:t0 + c, :], scale)
            sel[..., t0:t0 + c] = chunk > r["tau"][..., None]
        assert np.array_equal(sel, r["mask"])


def test_topk_and_topp_brute_force():
    # The routing baselines written out by hand on tiny rows: top-k keeps the k largest
    # (ties to the lower index); top-p keeps blocks while the softmax mass before them
    # (in decreasing order) is below p.
    rows = np.array([[0.5, 2.0, -1.0, 2.0, 0.3],
                     [1.0, 1.0, 1.0, 1.0, 1.0],
                     [3.0, 0.0, 0.0, -2.0, 1.0]])
    assert ora.route_topk(rows, 2).tolist() == [[False, True, False, True, False],
                                                  [True, True, False, False, False],
                                                  [True, False, False, False, True]]
    for p in (0.05, 0.3, 0.5, 0.9, 0.999, 1.0):
        got = ora.route_topp(rows, p)
        for r, row in enumerate(rows):
            order = sorted(range(len(row)), key=lambda j: (-row[j], j))
            z = sum(math.exp(x) for x in row)
            acc, want = 0.0, [False] * len(row)
            for j in order:
                if acc < p:
                    want[j] = True
                acc += math.exp(row[j]) / z
            assert got[r].tolist() == want, (p, r)


def hadamard(n):
    h = np.array([[1.0]])
    while h.shape[0] < n:
        h = np.block([[h, h], [h, -h]])
    return h


def test_diagonal_threshold_equals_exact_for_uncorrelated_pooled_keys():
    # Appendix, Eq. appendix_diagonal_threshold keeps only the diagonal of the
    # pooled-key covariance.  Block keys built from the columns of a Hadamard
    # matrix (orthogonal, zero-mean except the constant first column) have an
    # exactly diagonal covariance, so the diagonal estimate must equal the exact
    # standard deviation of the materialised proxy row.
    rng = np.random.default_rng(40)
    d, bk, bq = 16, 4, 8
    colscale = rng.uniform(0.5, 2.0, d)
    kbar = hadamard(d) * colscale                       # 16 blocks x 16 dims
    k = np.repeat(kbar, bk, axis=0)[None, None]         # block-constant keys
    q = rng.standard_normal((1, 1, 6 * bq, d))
    ex = ora.routing(q, k, bq, bk, 0.7)
    dg = ora.routing(q, k, bq, bk, 0.7, threshold_mode="diagonal")
    assert np.max(np.abs(dg["sigma"] - ex["sigma"])) < 1e-12
    assert np.array_equal(dg["mask"], ex["mask"])


def test_diagonal_threshold_brute_force():
    # sigma_i^2 = s^2 * sum_d Qbar_id^2 * (1/N) sum_j (Kbar_jd - mean_d)^2, written
    # out with plain loops on a tiny case.
    rng = np.random.default_rng(41)
    d, bk, bq, n = 6, 4, 5, 37
    q = rng.standard_normal((1, 1, n, d))
    k = rng.standard_normal((1, 1, n, d)) + rng.standard_normal(d)
    r = ora.routing(q, k, bq, bk, 0.3, threshold_mode="diagonal")
    qh, kh = q[0, 0], k[0, 0]
    kb = [[sum(kh[t, c] for t in range(j, min(j + bk, n))) / (min(j + bk, n) - j) for c in range(d)]
          for j in range(0, n, bk)]
    nk = len(kb)
    mean = [sum(kb[j][c] for j in range(nk)) / nk for c in range(d)]
    var = [sum((kb[j][c] - mean[c]) ** 2 for j in range(nk)) / nk for c in range(d)]
    s = 1 / math.sqrt(d)
    for i, i0 in enumerate(range(0, n, bq)):
        rows = range(i0, min(i0 + bq, n))
        qb = [sum(qh[t, c] for t in rows) / len(rows) for c in range(d)]
        sig = math.sqrt(s * s * sum(qb[c] ** 2 * var[c] for c in range(d)))
        assert abs(r["sigma"][0, 0, i] - sig) < 1e-12
        mu = s * sum(qb[c] * mean[c] for c in range(d))
        assert abs(r["tau"][0, 0, i] - (mu + 0.3 * sig)) < 1e-12


def test_diagonal_threshold_differs_for_correlated_keys():
    # With two perfectly correlated key dimensions the off-diagonal covariance is
    # large, and dropping it must change sigma (the flag is not a no-op).
    rng = np.random.default_rng(42)
    d, bk = 8, 4
    base = rng.standard_normal((64, 1))
    kbar = np.concatenate([base, base, 0.1 * rng.standard_normal((64, d - 2))], axis=1)
    k = np.repeat(kbar, bk, axis=0)[None, None]
    q = np.ones((1, 1, 16, d))
    ex = ora.routing(q, k, 8, bk, 0.5)
    dg = ora.routing(q, k, 8, bk, 0.5, threshold_mode="diagonal")
    assert np.min(np.abs(dg["sigma"] - ex["sigma"]) / ex["sigma"]) > 0.2


@pytest.mark.parametrize("beta", [0.0, 0.5, 1.0, 1.5])
def test_kept_density_follows_gaussian_tail(beta):
    # Keys constant within each block with iid N(0, I) block values make every
    # proxy row exactly Gaussian, so the kept fraction is 1 - Phi(beta)
    # (Section 3.1, rho_G(beta) = 1 - Phi(beta)).
    rng = np.random.default_rng(6)
    d, bk, nk, bq, nq = 16, 4, 4096, 8, 8
    k = np.repeat(rng.standard_normal((nk, d)), bk, axis=0)[None, None]
    q = rng.standard_normal((1, 1, bq * nq, d))
    r = ora.routing(q, k, bq, bk, beta)
    expected = 1.0 - NormalDist().cdf(beta)
    assert abs(float(r["frac"][0, 0]) - expected) < 0.015


def test_zero_spread_selects_nothing_for_finite_beta():
    rng = np.random.default_rng(7)
    d = 8
    k = np.tile(rng.standard_normal((1, d)), (128, 1))[None, None]
    q = rng.standard_normal((1, 1, 128, d))
    for beta in (-2.0, 0.0, 1.0):
        r = ora.routing(q, k, 32, 16, beta)
        assert np.all(r["sigma"] < 1e-12)
        assert not r["mask"].any()
    assert ora.routing(q, k, 32, 16, -math.inf)["mask"].all()
    assert not ora.routing(q, k, 32, 16, math.inf)["mask"].any()


# --------------------------------------------------------------------------- closed forms

def _brute_force_rows(q, k, v, scale, key_mask=None):
    """Softmax attention by explicit loops (one row at a time)."""
    n, d = q.shape
    out = np.zeros((n, d))
    for r in range(n):
        logits = [scale * sum(q[r, c] * k[u, c] for c in range(d)) for u in range(k.shape[0])]
        keep = [u for u in range(k.shape[0]) if key_mask is None or key_mask[u]]
        if not keep:
            continue
        m = max(logits[u] for u in keep)
        w = {u: math.exp(logits[u] - m) for u in keep}
        z = sum(w.values())
        for c in range(d):
            out[r, c] = sum(w[u] * v[u, c] for u in keep) / z
    return out


@pytest.mark.parametrize("beta", [-0.3, 0.4, 1.2, math.inf])
def test_sparse_equals_dense_over_block_mean_keys(beta):
    # Closed form of the zeroth-order correction: for query block i, the sparse
    # output is exact softmax attention in which every key of an unselected block
    # j is replaced by Kbar_j (values unchanged), because
    # sum_u exp(q.Kbar_j) v_u = exp(q.Kbar_j) Vhat_j  (Eqs. solattn_denominator,
    # solattn_numerator).  The no-correction output is Eq. block_sparse_attn.
    rng = np.random.default_rng(8)
    n, d, bq, bk = 88, 6, 32, 16          # ragged query (24) and key (8) tails
    q, k, v = smooth_qkv(rng, B=1, H=1, N=n, d=d)
    scale = 1 / math.sqrt(d)
    sp = ora.forward(q, k, v, bq, bk, beta, "sparse")
    nc = ora.forward(q, k, v, bq, bk, beta, "sparse_no_correction")
    mask = sp["mask"][0, 0]
    assert np.array_equal(mask, nc["mask"][0, 0])
    kh, vh, qh = k[0, 0], v[0, 0], q[0, 0]
    for i in range(mask.shape[0]):
        rows = slice(i * bq, min((i + 1) * bq, n))
        kmod = kh.copy()
        keymask = np.zeros(n, dtype=bool)
        for j in range(mask.shape[1]):
            ks = slice(j * bk, min((j + 1) * bk, n))
            if mask[i, j]:
                keymask[ks] = True
            else:
                kmod[ks] = kh[ks].mean(axis=0)
        want_sp = _brute_force_rows(qh[rows], kmod, vh, scale)
        want_nc = _brute_force_rows(qh[rows], kh, vh, scale, keymask)
        assert np.max(np.abs(sp["out"][0, 0, rows] - want_sp)) < 1e-12
        assert np.max(np.abs(nc["out"][0, 0, rows] - want_nc)) < 1e-12


@settings(max_examples=40, deadline=None, derandomize=True)
@given(n=st.integers(1, 60), bq=st.sampled_from([4, 8, 16, 32]), bk=st.sampled_from([4, 8, 16]),
       d=st.integers(1, 4), forced=st.integers(0, 2), seed=st.integers(0, 10**6),
       beta=st.one_of(st.floats(-2.0, 2.0), st.just(math.inf), st.just(-math.inf)))
def test_closed_form_over_random_shapes(n, bq, bk, d, forced, seed, beta):
    # The closed form of both sparse modes (see test_sparse_equals_dense_over_block_mean_keys)
    # over random lengths, block sizes and forced tails: forced key blocks are always exact,
    # an unselected routable block enters the corrected output through its mean key with
    # its values unchanged, and the uncorrected output sees the kept keys only (a row with
    # none is zero).
    nk = -(-n // bk)
    keep = forced * bk
    if keep >= n or nk - forced < 1 or keep % bk or (n - keep) <= 0:
        keep = 0
    rng = np.random.default_rng(seed)
    q, k, v = smooth_qkv(rng, B=1, H=1, N=n, d=d)
    scale = 1 / math.sqrt(d)
    sp = ora.forward(q, k, v, bq, bk, beta, "sparse", keep_tail_tokens=keep)
    nc = ora.forward(q, k, v, bq, bk, beta, "sparse_no_correction", keep_tail_tokens=keep)
    mask = sp["mask"][0, 0]
    nkr = mask.shape[1]
    assert nkr == nk - keep // bk
    kh, vh, qh = k[0, 0], v[0, 0], q[0, 0]
    for i in range(mask.shape[0]):
        rows = slice(i * bq, min((i + 1) * bq, n))
        kmod = kh.copy()
        keymask = np.zeros(n, dtype=bool)
        keymask[nkr * bk:] = True                    # forced tail
        for j in range(nkr):
            ks = slice(j * bk, min((j + 1) * bk, n))
            if mask[i, j]:
                keymask[ks] = True
            else:
                kmod[ks] = kh[ks].mean(axis=0)
        want_sp = _brute_force_rows(qh[rows], kmod, vh, scale)
        want_nc = _brute_force_rows(qh[rows], kh, vh, scale, keymask)
        assert np.max(np.abs(sp["out"][0, 0, rows] - want_sp)) < 1e-11
        assert np.max(np.abs(nc["out"][0, 0, rows] - want_nc)) < 1e-11


def test_correction_is_exact_for_blockwise_constant_keys():
    # delta_u = 0 inside every key block makes the zeroth-order term exact
    # (Appendix, approximation error), so sparse == dense for every beta, while
    # dropping blocks (no correction) changes the output.
    rng = np.random.default_rng(9)
    n, d, bq, bk = 192, 16, 64, 32
    kb = rng.standard_normal((1, 2, n // bk, d))
    k = np.repeat(kb, bk, axis=2)
    q = rng.standard_normal((1, 2, n, d)) + np.repeat(kb, bk, axis=2)
    v = rng.standard_normal((1, 2, n, d))
    dense = ora.forward(q, k, v, bq, bk, 0.0, "dense")["out"]
    for beta in (-1.0, 0.0, 0.7, 2.0, math.inf):
        sp = ora.forward(q, k, v, bq, bk, beta, "sparse")
        assert np.max(np.abs(sp["out"] - dense)) < 1e-12
    nc = ora.forward(q, k, v, bq, bk, 0.7, "sparse_no_correction")
    assert not nc["mask"].all()
    assert np.max(np.abs(nc["out"] - dense)) > 1e-3


@pytest.mark.parametrize("mode", ora.MODES)
def test_weights_sum_to_one(mode):
    # V == 1 gives O == 1: the exact and approximate weights share one
    # normaliser (Eqs. solattn_denominator, solattn_numerator); without the
    # correction a row with no selected block is 0.
    rng = np.random.default_rng(10)
    q, k, _ = smooth_qkv(rng, N=160)
    v = np.ones_like(q)
    res = ora.forward(q, k, v, 32, 16, 1.0, mode)
    if mode == "sparse_no_correction":
        for b, h in np.ndindex(res["mask"].shape[:2]):
            for i in range(res["mask"].shape[2]):
                rows = res["out"][b, h, i * 32:(i + 1) * 32]
                want = 1.0 if res["mask"][b, h, i].any() else 0.0
                assert np.max(np.abs(rows - want)) < 1e-13
    else:
        assert np.max(np.abs(res["out"] - 1.0)) < 1e-13


def test_error_bound_of_zeroth_order_term():
    # Appendix, Eq. appendix_approximation_error: with a = q.Kbar, delta_u =
    # q.(k_u - Kbar) and eta = max|delta_u|,
    #   0 <= D - D~ <= 1/2 exp(a + eta) sum delta_u^2,
    #   ||N - N~|| <= exp(a + eta) sum |delta_u| ||v_u||.
    rng = np.random.default_rng(11)
    d, blk, scale = 16, 64, 1 / math.sqrt(16)
    for trial in range(20):
        spread = [0.02, 0.1, 0.5][trial % 3]
        q_rows = rng.standard_normal((8, d))
        kc = rng.standard_normal(d)
        keys = kc + spread * rng.standard_normal((blk, d))
        vals = rng.standard_normal((blk, d))
        shift = np.zeros(8)
        D, N = ora.exact_terms(q_rows, keys, vals, scale, shift)
        kbar = keys.mean(axis=0, keepdims=True)
        Dt, Nt = ora.approx_terms(q_rows, kbar, vals.sum(axis=0, keepdims=True),
                                  np.array([blk]), scale, shift)
        a = scale * q_rows @ kbar[0]
        delta = scale * q_rows @ (keys - kbar).T
        eta = np.abs(delta).max(axis=1)
        bound_d = 0.5 * np.exp(a + eta) * (delta ** 2).sum(axis=1)
        bound_n = np.exp(a + eta) * (np.abs(delta) @ np.linalg.norm(vals, axis=1))
        gap = D - Dt
        assert np.all(gap >= -1e-12 * D)
        assert np.all(gap <= bound_d * (1 + 1e-9) + 1e-300)
        assert np.all(np.linalg.norm(N - Nt, axis=1) <= bound_n * (1 + 1e-9))


# --------------------------------------------------------------------------- invariances

def test_key_shift_invariance():
    # Adding one vector to every key shifts each proxy row and each logit row by
    # a per-row constant: the mask and all outputs are unchanged.
    rng = np.random.default_rng(12)
    q, k, v = smooth_qkv(rng, N=200)
    c = rng.standard_normal(q.shape[-1])
    for mode in ora.MODES:
        a = ora.forward(q, k, v, 64, 32, 0.3, mode)
        b = ora.forward(q, k + c, v, 64, 32, 0.3, mode)
        assert np.array_equal(a["mask"], b["mask"])
        assert np.max(np.abs(a["out"] - b["out"])) < 1e-10


def test_query_scale_keeps_mask():
    rng = np.random.default_rng(13)
    q, k, _ = smooth_qkv(rng, N=256)
    a = ora.routing(q, k, 32, 16, 0.6)
    b = ora.routing(q * 3.7, k, 32, 16, 0.6)
    assert np.array_equal(a["mask"], b["mask"])


def test_key_block_permutation_invariance():
    rng = np.random.default_rng(14)
    n, bk = 256, 32
    q, k, v = smooth_qkv(rng, N=n)
    perm = rng.permutation(n // bk)
    idx = np.concatenate([np.arange(p * bk, (p + 1) * bk) for p in perm])
    for mode in ora.MODES:
        a = ora.forward(q, k, v, 64, bk, 0.2, mode)
        b = ora.forward(q, k[..., idx, :], v[..., idx, :], 64, bk, 0.2, mode)
        assert np.array_equal(a["mask"][..., perm], b["mask"])
        assert np.max(np.abs(a["out"] - b["out"])) < 1e-12


# --------------------------------------------------------------------------- forced tail blocks

def test_forced_tail_blocks_exact_and_excluded_from_statistics():
    rng = np.random.default_rng(15)
    n_img, n_txt, d, bq, bk = 192, 64, 8, 64, 32
    q, k, v = smooth_qkv(rng, B=1, H=1, N=n_img + n_txt, d=d)
    res = ora.forward(q, k, v, bq, bk, 0.8, "sparse_no_correction", keep_tail_tokens=n_txt)
    # statistics and mask over the routable blocks only
    r = ora.routing(q[..., :n_img, :], k[..., :n_img, :], bq, bk, 0.8)
    qbar, _ = ora.pool_means(q, bq)
    kbar, _ = ora.pool_means(k[..., :n_img, :], bk)
    s_hat = ora.proxy_scores(qbar, kbar, 1 / math.sqrt(d))
    mu, sd = ora.row_stats(s_hat)
    assert res["mask"].shape[-1] == n_img // bk
    assert np.array_equal(res["mask"], s_hat > (mu + 0.8 * sd)[..., None])
    assert r["mask"].shape[-1] == res["mask"].shape[-1]
    # text keys always exact: compare with brute force over selected + text keys
    scale = 1 / math.sqrt(d)
    for i in range(res["mask"].shape[2]):
        rows = slice(i * bq, min((i + 1) * bq, n_img + n_txt))
        keymask = np.zeros(n_img + n_txt, dtype=bool)
        keymask[n_img:] = True
        for j in np.nonzero(res["mask"][0, 0, i])[0]:
            keymask[j * bk:(j + 1) * bk] = True
        want = _brute_force_rows(q[0, 0, rows], k[0, 0], v[0, 0], scale, keymask)
        assert np.max(np.abs(res["out"][0, 0, rows] - want)) < 1e-12


# --------------------------------------------------------------------------- worked example

def test_hand_example():
    g = json.load(open(os.path.join(GOLDEN, "hand_example.json")))
    e = math.e
    q = np.array(g["q"])[None, None, :, None]
    v = np.array(g["v"])[None, None, :, None]

    c1 = g["case_equal_blocks"]
    k = np.array(c1["k"])[None, None, :, None]
    sp = ora.forward(q, k, v, 4, 2, c1["beta"], "sparse")
    assert np.allclose(sp["s_hat"][0, 0, 0], c1["s_hat"], atol=1e-15)
    assert abs(sp["mu"][0, 0, 0] - c1["mu"]) < 1e-15 and sp["sigma"][0, 0, 0] < 1e-15
    assert sp["mask"][0, 0, 0].tolist() == c1["mask"]
    assert np.allclose(sp["out"], c1["sparse_value"], atol=1e-14)
    dense = (1 + 2 * e**2 + 3 * e + 4 * e) / (1 + e**2 + 2 * e)
    assert np.allclose(ora.forward(q, k, v, 4, 2, 0.0, "dense")["out"], dense, atol=1e-14)
    nc = ora.forward(q, k, v, 4, 2, c1["beta"], "sparse_no_correction")
    assert np.all(nc["out"] == c1["no_correction_value"])

    c2 = g["case_one_selected"]
    k = np.array(c2["k"])[None, None, :, None]
    sp = ora.forward(q, k, v, 4, 2, c2["beta"], "sparse")
    assert np.allclose(sp["s_hat"][0, 0, 0], c2["s_hat"], atol=1e-15)
    assert abs(sp["mu"][0, 0, 0] - c2["mu"]) < 1e-15 and abs(sp["sigma"][0, 0, 0] - c2["sigma"]) < 1e-15
    assert sp["mask"][0, 0, 0].tolist() == c2["mask"]
    assert np.allclose(sp["out"], (1 + 2 * e**2 + 7) / (1 + e**2 + 2), atol=1e-14)
    nc = ora.forward(q, k, v, 4, 2, c2["beta"], "sparse_no_correction")
    assert np.allclose(nc["out"], (1 + 2 * e**2) / (1 + e**2), atol=1e-14)
    dn = ora.forward(q, k, v, 4, 2, c2["beta"], "dense")
    assert np.allclose(dn["out"], (1 + 2 * e**2 + 3 / e + 4 * e) / (1 + e**2 + 1 / e + e), atol=1e-14)


# --------------------------------------------------------------------------- causal masks

def causal_sdpa(q, k, v, granule):
    n = q.shape[-2]
    t = np.arange(n)
    allowed = t[None, :] < np.minimum((t[:, None] // granule + 1) * granule, n)
    return torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v),
        attn_mask=torch.from_numpy(allowed)).numpy()


@pytest.mark.parametrize("bq,bk,n,g", [(32, 16, 131, 1), (64, 64, 200, 1), (32, 16, 150, 40), (64, 16, 97, 13)])
def test_causal_dense_and_full_selection_match_library_sdpa(bq, bk, n, g):
    # Dense mode and beta = -inf (every routable block exact, partial blocks under the token
    # mask) must both equal masked softmax attention from the library.
    rng = np.random.default_rng(30)
    q, k, v = rand_qkv(rng, N=n)
    ref = causal_sdpa(q, k, v, g)
    for mode, beta in (("dense", 0.3), ("sparse", -math.inf), ("sparse_no_correction", -math.inf)):
        res = ora.forward(q, k, v, bq, bk, beta, mode, causal_granule=g)
        assert np.max(np.abs(res["out"] - ref)) < 1e-12, mode


def test_causal_block_ranges_brute_force():
    # Classify every (query block, key block) pair by checking every (query, key) token
    # pair: routable = seen by all rows, partial = seen by some rows.
    for n, bq, bk, g in ((37, 8, 4, 1), (37, 8, 4, 3), (50, 16, 8, 20), (64, 16, 16, 16), (29, 8, 4, 100)):
        r, e = ora.causal_block_ranges(n, bq, bk, g)
        nq, nk = -(-n // bq), -(-n // bk)
        for i in range(nq):
            rows = range(i * bq, min((i + 1) * bq, n))
            full, some = [], []
            for j in range(nk):
                keys = range(j * bk, min((j + 1) * bk, n))
                seen = [(s // g) <= (t // g) for t in rows for s in keys]
                full.append(all(seen))
                some.append(any(seen))
            assert full == [j < r[i] for j in range(nk)], (n, bq, bk, g, i)
            assert some == [j < e[i] for j in range(nk)], (n, bq, bk, g, i)


def _brute_causal(q, k, v, bq, bk, g, beta, mode):
    """Pure-Python loops for one head: visibility from (s // g) <= (t // g), block
    means, proxies, mean/std over the key blocks every row of the query block sees,
    strict selection, then per-row exact terms over the visible keys of selected and
    partially visible blocks plus n_j exp(q.Kbar_j) terms for unselected routable blocks."""
    n, d = len(q), len(q[0])
    sc = 1.0 / math.sqrt(d)
    nq, nk = -(-n // bq), -(-n // bk)

    def mean_rows(x, a, b):
        return [sum(x[t][c] for t in range(a, b)) / (b - a) for c in range(d)]

    def dot(a, b):
        return sum(x * y for x, y in zip(a, b))

    def vis(t, s):
        return (s // g) <= (t // g)

    kb = [(j * bk, min((j + 1) * bk, n)) for j in range(nk)]
    kbar = [mean_rows(k, a, b) for a, b in kb]
    out = [[0.0] * d for _ in range(n)]
    mask = [[False] * nk for _ in range(nq)]
    for i in range(nq):
        r0, r1 = i * bq, min((i + 1) * bq, n)
        qbar = mean_rows(q, r0, r1)
        full = [all(vis(t, s) for t in range(r0, r1) for s in range(a, b)) for a, b in kb]
        some = [any(vis(t, s) for t in range(r0, r1) for s in range(a, b)) for a, b in kb]
        routable = [j for j in range(nk) if full[j]]
        if routable:
            sh = {j: sc * dot(qbar, kbar[j]) for j in routable}
            mu = sum(sh.values()) / len(sh)
            sig = math.sqrt(sum((x - mu) ** 2 for x in sh.values()) / len(sh))
            tau = -math.inf if beta == -math.inf else (math.inf if beta == math.inf else mu + beta * sig)
            for j in routable:
                mask[i][j] = sh[j] > tau
        for t in range(r0, r1):
            terms = []   # (log weight, value vector)
            for j in range(nk):
                a, b = kb[j]
                exact = some[j] and (mode == "dense" or not full[j] or mask[i][j])
                if exact:
                    for s in range(a, b):
                        if vis(t, s):
                            terms.append((sc * dot(q[t], k[s]), v[s]))
                elif full[j] and mode == "sparse":
                    vsum = [sum(v[s][c] for s in range(a, b)) for c in range(d)]
                    terms.append((sc * dot(q[t], kbar[j]) + math.log(b - a), [x / (b - a) for x in vsum]))
            if terms:
                m = max(lw for lw, _ in terms)
                den = sum(math.exp(lw - m) for lw, _ in terms)
                out[t] = [sum(math.exp(lw - m) * vec[c] for lw, vec in terms) / den for c in range(d)]
    return np.array(out), np.array(mask)


@pytest.mark.parametrize("g", [1, 3, 12])
@pytest.mark.parametrize("mode", ["sparse", "sparse_no_correction", "dense"])
def test_causal_forward_brute_force(g, mode):
    rng = np.random.default_rng(31)
    n, d, bq, bk = 37, 4, 8, 4
    q, k, v = smooth_qkv(rng, B=1, H=1, N=n, d=d)
    for beta in (0.0, 0.7):
        res = ora.forward(q, k, v, bq, bk, beta, mode, causal_granule=g)
        out, mask = _brute_causal(q[0, 0].tolist(), k[0, 0].tolist(), v[0, 0].tolist(), bq, bk, g, beta, mode)
        assert np.max(np.abs(res["out"][0, 0] - out)) < 1e-12
        if mode != "dense":
            assert (res["mask"][0, 0] == mask).all()


def test_causal_granule_covering_the_sequence_is_bidirectional():
    rng = np.random.default_rng(32)
    q, k, v = smooth_qkv(rng, N=150)
    for mode in ("sparse", "sparse_no_correction"):
        a = ora.forward(q, k, v, 32, 16, 0.4, mode)
        b = ora.forward(q, k, v, 32, 16, 0.4, mode, causal_granule=150)
        assert (a["mask"] == b["mask"]).all()
        assert np.max(np.abs(a["out"] - b["out"])) < 1e-13


@pytest.mark.parametrize("g", [1, 24])
def test_causal_outputs_ignore_future_keys(g):
    # Rows of a query block must not depend on keys or values it cannot see: neither
    # through the exact terms, nor through the routing statistics (centring over the
    # visible blocks only), nor through the correction.  The future keys are pushed
    # along the mean query so that their proxies, and any statistic that includes them,
    # move far.
    rng = np.random.default_rng(33)
    n, bq, bk = 256, 32, 8
    q, k, v = smooth_qkv(rng, N=n)
    cut = 160
    k2, v2 = k.copy(), v.copy()
    qdir = q.mean(axis=-2, keepdims=True)
    k2[..., cut:, :] += 4.0 * qdir + rng.standard_normal(k2[..., cut:, :].shape)
    v2[..., cut:, :] = rng.standard_normal(v2[..., cut:, :].shape)
    lim = ora.causal_limits(n, g)
    keep = [i for i in range(-(-n // bq)) if lim[min((i + 1) * bq, n) - 1] <= cut]
    assert len(keep) >= 4
    for mode in ("sparse", "sparse_no_correction"):
        a = ora.forward(q, k, v, bq, bk, 0.5, mode, causal_granule=g)
        b = ora.forward(q, k2, v2, bq, bk, 0.5, mode, causal_granule=g)
        rows = np.concatenate([np.arange(i * bq, min((i + 1) * bq, n)) for i in keep])
        assert (a["mask"][:, :, keep] == b["mask"][:, :, keep]).all()
        assert np.max(np.abs(a["out"][:, :, rows] - b["out"][:, :, rows])) < 1e-13


def test_causal_weights_sum_to_one():
    rng = np.random.default_rng(34)
    q, k, _ = smooth_qkv(rng, N=130)
    v = np.ones_like(q)
    for g in (1, 20):
        for mode in ("sparse", "dense"):
            res = ora.forward(q, k, v, 32, 16, 0.8, mode, causal_granule=g)
            assert np.max(np.abs(res["out"] - 1.0)) < 1e-12


def test_causal_routing_matches_forward():
    rng = np.random.default_rng(35)
    q, k, v = smooth_qkv(rng, N=200)
    r = ora.routing(q, k, 32, 16, 0.6, causal_granule=5)
    f = ora.forward(q, k, v, 32, 16, 0.6, "sparse", causal_granule=5)
    assert (r["mask"] == f["mask"]).all()
    assert np.allclose(r["tau"], f["tau"], equal_nan=True)
    assert np.allclose(r["frac"], f["frac"])


# --------------------------------------------------------------------------- planted mistakes

def test_pins_catch_a_dropped_multiplicity(monkeypatch):
    # A plausible slip (multiplicity 1 instead of n_j in Eq. solattn_denominator)
    # must break the normalisation pin.
    rng = np.random.default_rng(16)
    q, k, _ = smooth_qkv(rng, N=128)
    v = np.ones_like(q)
    orig = ora.approx_terms

    def wrong(q_rows, kbar_blocks, vhat_blocks, counts, scale, shift):
        return orig(q_rows, kbar_blocks, vhat_blocks, np.ones_like(counts), scale, shift)

    monkeypatch.setattr(ora, "approx_terms", wrong)
    res = ora.forward(q, k, v, 32, 16, 0.5, "sparse")
    assert np.max(np.abs(res["out"] - 1.0)) > 1e-2


def test_pins_catch_an_uncentred_diagonal_estimate(monkeypatch):
    # A plausible slip in Eq. appendix_diagonal_threshold (forgetting to subtract
    # mu_K * mu_K) must break the uncorrelated-keys pin: the constant Hadamard
    # column then contributes.
    def wrong(qbar, kbar, scale):
        v_k = (kbar * kbar).mean(axis=-2)
        return np.sqrt(scale * scale * ((qbar * qbar) @ v_k[..., None])[..., 0])

    monkeypatch.setattr(ora, "diagonal_sigma", wrong)
    with pytest.raises(AssertionError):
        test_diagonal_threshold_equals_exact_for_uncorrelated_pooled_keys()


def test_pins_catch_a_flipped_threshold_sign():
    rng = np.random.default_rng(17)
    d, bk, nk = 16, 4, 2048
    k = np.repeat(rng.standard_normal((nk, d)), bk, axis=0)[None, None]
    q = rng.standard_normal((1, 1, 64, d))
    r = ora.routing(q, k, 8, bk, 1.0)
    wrong = r["s_hat"] > (r["mu"] - 1.0 * r["sigma"])[..., None]
    expected = 1.0 - NormalDist().cdf(1.0)
    assert abs(float(r["frac"][0, 0]) - expected) < 0.015
    assert abs(float(wrong.mean()) - expected) > 0.5


def test_pins_catch_causal_statistics_over_the_whole_row(monkeypatch):
    # A plausible slip (centring the proxies over every key block instead of the
    # visible ones) must break the future-keys pin.
    monkeypatch.setattr(ora, "causal_row_stats", lambda s_hat, r: ora.row_stats(s_hat))
    with pytest.raises(AssertionError):
        test_causal_outputs_ignore_future_keys(1)
