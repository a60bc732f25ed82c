"""GPU parity: the HIP path (through the C ABI) against the fp64 CPU oracle.

Small shapes are compared element by element over every output; the full
workload shapes (in the launch configuration the benchmark times) are compared on
the complete selection mask and on sampled query blocks of sampled heads.
"""
import math

import numpy as np
import pytest
import torch

from oracle import sol_attn_oracle as ora
from paper_2607_24027_amd import binding as sb
from paper_2607_24027_amd import configs, synth
from tests.parity import (assert_mask_matches, assert_output_close, oracle_whole_heads, small_workload, to_np)

pytestmark = pytest.mark.gpu

INF = math.inf


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    sb.lib()  # fail loudly if the library is missing
    return torch.device("cuda:0")


SMALL = {
    # name: (grid, d, block_q, dtype, text tokens)
    "bf16_d128_q128": ((5, 10, 100), 128, 128, "bf16", 0),     # N=5000: NQ=40 (tail 8), NK=79 (tail 8), 2 chunks
    "bf16_d64_q64_text": ((4, 20, 64), 64, 64, "bf16", 512),   # N=5632: 8 forced text blocks
    "bf16_d128_q64_text": ((60, 70), 128, 64, "bf16", 576),    # 2D grid, N=4776: ragged text tail
    "f32_d64_q64": ((4, 16, 32), 64, 64, "f32", 0),            # the tiny workload shape
    "f32_d128_q128": ((3, 10, 41), 128, 128, "f32", 0),        # N=1230, ragged
}
_cache = {}


def small_inputs(name):
    if name not in _cache:
        grid, d, bq, dtype, text = SMALL[name]
        w = small_workload(name, grid, d, bq, dtype=dtype, text_tokens=text)
        _cache[name] = (w, synth.make_qkv(w))
    return _cache[name]


def run_gpu(dev, w, q, k, v, beta, mode, want_mask=True, threshold_mode="exact", outputs_defined=True):
    qd, kd, vd = (t.to(dev) for t in (q, k, v))
    nkr = w.NK - w.text_tokens // 64
    mw = sb.mask_words(nkr)
    mask = torch.zeros((w.B, w.H, w.NQ, mw), dtype=torch.int32, device=dev) if want_mask else None
    counts = torch.full((w.B, w.H), -1, dtype=torch.int32, device=dev)
    # NaN-filled output: every row must be written by whichever workgroup claimed its query block
    # (the kernels hand out query blocks through work queues, in a data-dependent order)
    out = torch.full_like(qd, math.nan)
    sb.forward(qd, kd, vd, w.block_q, 64, beta, mode, keep_tail_tokens=w.text_tokens, out=out,
               counts=counts, mask_out=mask, threshold_mode=threshold_mode)
    torch.cuda.synchronize()
    if outputs_defined:
        assert bool(torch.isfinite(out).all()), f"{w.name}/{mode}: rows left unwritten"
    gmask = None
    if want_mask and mode != "dense":
        gmask = sb.unpack_mask(mask.cpu().numpy().view(np.uint32), nkr)
    return out, gmask, counts.cpu().numpy().view(np.uint32)


@pytest.mark.parametrize("name", list(SMALL))
@pytest.mark.parametrize("mode,beta", [("dense", 0.0), ("sparse", 0.8), ("sparse", -INF), ("sparse", INF),
                                       ("sparse_no_correction", 0.8), ("sparse_no_correction", -INF),
                                       ("sparse_no_correction", INF), ("sparse", 0.0)])
def test_forward_parity_small(dev, name, mode, beta):
    w, (q, k, v) = small_inputs(name)
    print(f"[parity] {name} mode={mode} beta={beta}", flush=True)
    out, gmask, counts = run_gpu(dev, w, q, k, v, beta, mode)
    qn, kn, vn = to_np(q), to_np(k), to_np(v)
    ref = ora.forward(qn, kn, vn, w.block_q, 64, beta, mode, keep_tail_tokens=w.text_tokens)
    if mode != "dense":
        flips = assert_mask_matches(gmask, ref["mask"], ref["s_hat"], ref["tau"])
        if flips:
            ref = ora.forward(qn, kn, vn, w.block_q, 64, beta, mode, keep_tail_tokens=w.text_tokens, mask=gmask)
        assert np.array_equal(counts, gmask.sum(axis=(2, 3)))
    else:
        nkr = w.NK - w.text_tokens // 64
        assert np.all(counts == w.NQ * nkr)
    assert_output_close(to_np(out), ref["out"], w.dtype, f"{name}/{mode}/{beta}")


@pytest.mark.parametrize("name", ["bf16_d128_q128", "f32_d64_q64", "bf16_d64_q64_text"])
def test_pool_blocks_parity(dev, name):
    w, (q, k, v) = small_inputs(name)
    qbar, kbar, vbar = sb.pool_blocks(q.to(dev), k.to(dev), v.to(dev), w.block_q, 64)
    torch.cuda.synchronize()
    for got, x, blk in ((qbar, q, w.block_q), (kbar, k, 64), (vbar, v, 64)):
        want, _ = ora.pool_means(to_np(x), blk)
        np.testing.assert_allclose(to_np(got), want, rtol=1e-5, atol=2e-6)


def test_pool_blocks_long_blocks(dev):
    # The pooling entry point takes any block size; blocks longer than 128 rows take the
    # row-by-row tail path.
    w, (q, k, v) = small_inputs("bf16_d128_q128")
    for blk in (200, 1000):
        qbar, _, _ = sb.pool_blocks(q.to(dev), k.to(dev), v.to(dev), blk, 64)
        torch.cuda.synchronize()
        want, _ = ora.pool_means(to_np(q), blk)
        np.testing.assert_allclose(to_np(qbar), want, rtol=1e-5, atol=2e-6)


EDGE = {
    # name: (grid, d, block_q, dtype, text tokens, B, H)
    "n1": ((1, 1), 128, 128, "bf16", 0, 1, 1),            # one token: one query and one key block
    "n63": ((7, 9), 64, 64, "bf16", 0, 1, 2),             # one ragged block of each kind
    "n65": ((5, 13), 128, 128, "bf16", 0, 2, 3),          # B=2, H=3; a 1-token last key block
    "one_routable": ((1, 64), 128, 64, "bf16", 64, 1, 2), # N=128 with 64 text tokens: one routable block
    "f32_n100": ((10, 10), 64, 128, "f32", 0, 2, 1),      # f32 path, ragged, B=2
    "split_tail13": ((5, 41), 128, 64, "bf16", 0, 1, 2),  # d=128, 64-row blocks: last key block 13 keys,
                                                          # its second 32-key half empty
    "split_tail32": ((4, 40), 128, 64, "bf16", 0, 2, 1),  # last key block exactly one 32-key half
}


@pytest.mark.parametrize("name", list(EDGE))
@pytest.mark.parametrize("mode,beta", [("dense", 0.0), ("sparse", 0.5), ("sparse", -INF),
                                       ("sparse_no_correction", 0.5), ("sparse_no_correction", -0.3)])
def test_forward_parity_edge_shapes(dev, name, mode, beta):
    grid, d, bq, dtype, text, B, H = EDGE[name]
    w = small_workload(name, grid, d, bq, dtype=dtype, text_tokens=text, H=H, B=B, seed=23)
    q, k, v = synth.make_qkv(w)
    print(f"[parity] edge {name} N={w.N} mode={mode} beta={beta}", flush=True)
    out, gmask, counts = run_gpu(dev, w, q, k, v, beta, mode)
    qn, kn, vn = to_np(q), to_np(k), to_np(v)
    ref = ora.forward(qn, kn, vn, w.block_q, 64, beta, mode, keep_tail_tokens=w.text_tokens)
    if mode != "dense":
        flips = assert_mask_matches(gmask, ref["mask"], ref["s_hat"], ref["tau"])
        if flips:
            ref = ora.forward(qn, kn, vn, w.block_q, 64, beta, mode, keep_tail_tokens=w.text_tokens, mask=gmask)
        assert np.array_equal(counts, gmask.sum(axis=(2, 3)))
    assert_output_close(to_np(out), ref["out"], w.dtype, f"edge {name}/{mode}/{beta}")


def random_case(seed):
    """A seeded random forward configuration: shape, block sizes, dtype, text tail, cutoff, mode."""
    rng = np.random.default_rng(1000 + seed)
    d = int(rng.choice([64, 128]))
    bq = int(rng.choice([64, 128]))
    dtype = "f32" if rng.random() < 0.2 else "bf16"
    n_img = int(rng.integers(1, 6000))
    shape = int(rng.integers(1, 4))                       # 1D, 2D or 3D token grid
    if shape == 1:
        grid = (n_img,)
    elif shape == 2:
        a = int(rng.integers(1, 80))
        grid = (a, max(1, n_img // a))
    else:
        a, b = int(rng.integers(1, 12)), int(rng.integers(1, 30))
        grid = (a, b, max(1, n_img // (a * b)))
    text = 64 * int(rng.integers(1, 9)) if (dtype == "bf16" and rng.random() < 0.3) else 0
    B, H = int(rng.integers(1, 3)), int(rng.integers(1, 4))
    r = rng.random()
    beta = -INF if r < 0.1 else (INF if r < 0.2 else float(np.round(rng.uniform(-1.0, 2.0), 3)))
    mode = str(rng.choice(["dense", "sparse", "sparse_no_correction"]))
    return grid, d, bq, dtype, text, B, H, beta, mode


@pytest.mark.parametrize("seed", range(24))
def test_forward_parity_random_shapes(dev, seed):
    # Seeded random configurations (any token count, ragged tails, 1D/2D/3D grids, text tails,
    # both dtypes and block heights, cutoffs from -inf to +inf), element by element.
    grid, d, bq, dtype, text, B, H, beta, mode = random_case(seed)
    w = small_workload(f"rand{seed}", grid, d, bq, dtype=dtype, text_tokens=text, H=H, B=B, seed=50 + seed)
    print(f"[parity] random {seed}: grid={grid} N={w.N} d={d} bq={bq} {dtype} text={text} B={B} H={H} "
          f"beta={beta} {mode}", flush=True)
    q, k, v = synth.make_qkv(w)
    out, gmask, counts = run_gpu(dev, w, q, k, v, beta, mode)
    qn, kn, vn = to_np(q), to_np(k), to_np(v)
    ref = ora.forward(qn, kn, vn, w.block_q, 64, beta, mode, keep_tail_tokens=w.text_tokens)
    if mode != "dense":
        flips = assert_mask_matches(gmask, ref["mask"], ref["s_hat"], ref["tau"])
        if flips:
            ref = ora.forward(qn, kn, vn, w.block_q, 64, beta, mode, keep_tail_tokens=w.text_tokens, mask=gmask)
        assert np.array_equal(counts, gmask.sum(axis=(2, 3)))
    assert_output_close(to_np(out), ref["out"], w.dtype, f"random {seed}")


@pytest.mark.parametrize("nq", [4096, 4100])
def test_query_block_order_limits(dev, nq):
    # The sparse kernels take the query blocks of each head in an order computed on the GPU
    # for up to 4096 blocks per head (every rank-sort slot of a thread in use at 4096) and in
    # the identity order above that.  d = 64, block_q = 64: N = 64 * nq tokens, one head;
    # complete mask, sampled query blocks, every output row written.
    w = small_workload(f"order{nq}", (nq, 64), 64, 64, H=1)
    q, k, v = synth.make_qkv(w)
    print(f"[parity] query-block order limit NQ={nq} N={w.N}", flush=True)
    r = ora.routing(to_np(q), to_np(k), w.block_q, 64, 0.8)
    for mode in ("sparse", "sparse_no_correction"):
        out, gmask, counts = run_gpu(dev, w, q, k, v, 0.8, mode)
        assert_mask_matches(gmask, r["mask"], r["s_hat"], r["tau"])
        assert np.array_equal(counts, gmask.sum(axis=(2, 3)))
        qblocks = [0, 1, nq // 3, nq // 2, nq - 1]
        ref = ora.forward(to_np(q), to_np(k), to_np(v), w.block_q, 64, 0.8, mode, query_blocks=qblocks, mask=gmask)
        rows = np.concatenate([np.arange(i * w.block_q, min((i + 1) * w.block_q, w.N)) for i in qblocks])
        got = out.float().cpu().numpy().astype(np.float64)
        assert_output_close(got[:, :, rows], ref["out"][:, :, rows], w.dtype, f"order{nq}/{mode}")


@pytest.mark.parametrize("name", ["bf16_d128_q128", "f32_d64_q64"])
@pytest.mark.parametrize("beta", [0.8, -0.5, -INF, INF])
def test_thresholds_parity(dev, name, beta):
    w, (q, k, v) = small_inputs(name)
    qbar, kbar, _ = sb.pool_blocks(q.to(dev), k.to(dev), v.to(dev), w.block_q, 64)
    tau, mu, sigma = sb.thresholds(qbar, kbar, beta)
    torch.cuda.synchronize()
    scale = 1 / math.sqrt(w.d)
    s_hat = ora.proxy_scores(to_np(qbar), to_np(kbar), scale)
    mu_r, sd_r = ora.row_stats(s_hat)
    np.testing.assert_allclose(to_np(mu), mu_r, atol=1e-5, rtol=1e-5)
    np.testing.assert_allclose(to_np(sigma), sd_r, atol=1e-5, rtol=1e-5)
    tau_r = ora.thresholds(mu_r, sd_r, beta)
    if math.isinf(beta):
        assert np.array_equal(to_np(tau), tau_r)
    else:
        np.testing.assert_allclose(to_np(tau), tau_r, atol=1e-5, rtol=1e-5)


@pytest.mark.parametrize("name", ["bf16_d128_q128", "f32_d64_q64", "bf16_d64_q64_text", "bf16_d128_q64_text"])
@pytest.mark.parametrize("mode", ["sparse", "sparse_no_correction"])
def test_forward_parity_diagonal_threshold(dev, name, mode):
    # Appendix, Eq. appendix_diagonal_threshold selected through SOL_THRESHOLD_DIAGONAL.
    w, (q, k, v) = small_inputs(name)
    beta = 0.8
    print(f"[parity] {name} mode={mode} diagonal thresholds", flush=True)
    out, gmask, counts = run_gpu(dev, w, q, k, v, beta, mode, threshold_mode="diagonal")
    qn, kn, vn = to_np(q), to_np(k), to_np(v)
    ref = ora.forward(qn, kn, vn, w.block_q, 64, beta, mode, keep_tail_tokens=w.text_tokens,
                      threshold_mode="diagonal")
    flips = assert_mask_matches(gmask, ref["mask"], ref["s_hat"], ref["tau"])
    if flips:
        ref = ora.forward(qn, kn, vn, w.block_q, 64, beta, mode, keep_tail_tokens=w.text_tokens, mask=gmask)
    assert np.array_equal(counts, gmask.sum(axis=(2, 3)))
    assert_output_close(to_np(out), ref["out"], w.dtype, f"{name}/{mode}/diagonal")


@pytest.mark.parametrize("name", ["bf16_d128_q128", "f32_d64_q64"])
@pytest.mark.parametrize("beta", [0.8, -INF])
def test_thresholds_parity_diagonal(dev, name, beta):
    w, (q, k, v) = small_inputs(name)
    qbar, kbar, _ = sb.pool_blocks(q.to(dev), k.to(dev), v.to(dev), w.block_q, 64)
    tau, mu, sigma = sb.thresholds(qbar, kbar, beta, threshold_mode="diagonal")
    torch.cuda.synchronize()
    scale = 1 / math.sqrt(w.d)
    qb, kb = to_np(qbar), to_np(kbar)
    mu_r, _ = ora.row_stats(ora.proxy_scores(qb, kb, scale))
    sd_r = ora.diagonal_sigma(qb, kb, scale)
    np.testing.assert_allclose(to_np(mu), mu_r, atol=1e-5, rtol=1e-5)
    np.testing.assert_allclose(to_np(sigma), sd_r, atol=1e-5, rtol=1e-5)
    tau_r = ora.thresholds(mu_r, sd_r, beta)
    if math.isinf(beta):
        assert np.array_equal(to_np(tau), tau_r)
    else:
        np.testing.assert_allclose(to_np(tau), tau_r, atol=1e-5, rtol=1e-5)


@pytest.mark.parametrize("name", ["bf16_d128_q128", "bf16_d128_q64_text", "bf16_d64_q64_text"])
def test_beta_minus_inf_is_bitwise_dense(dev, name):
    # every routable block selected: the exact tiles are all key blocks in increasing order, as in
    # dense mode, so the two outputs agree bit for bit (any query-block height and key split)
    w, (q, k, v) = small_inputs(name)
    dense, _, _ = run_gpu(dev, w, q, k, v, 0.0, "dense", want_mask=False)
    for mode in ("sparse", "sparse_no_correction"):
        out, gmask, counts = run_gpu(dev, w, q, k, v, -INF, mode)
        assert gmask.all()
        assert torch.equal(out, dense)


@pytest.mark.parametrize("name", ["bf16_d128_q128", "bf16_d64_q64_text"])
@pytest.mark.parametrize("qf,kf,modes", [(2e-5, 5e4, ("sparse_no_correction",)),
                                         (1.0, 1e-6, ("sparse", "sparse_no_correction"))],
                         ids=["large_keys", "subnormal_keys"])
def test_routing_outside_the_f16_normal_range(dev, name, qf, kf, modes):
    # Routing takes f32 proxies from the f32 pooled means, while the pre-pass also writes f16
    # copies of the pooled keys (read by the correction tiles only).  Inputs at both ends of the
    # f16 range must leave the selection and the no-correction outputs unaffected:
    # * keys x5e4, queries x2e-5: the logits keep their scale, most pooled-key rows have a
    #   component past the f16 range (65504) and the pooled queries are f16 subnormals (the range
    #   contract on k applies to SOL_SPARSE only, so only the no-correction mode runs);
    # * keys x1e-6: the pooled keys are f16 subnormals, and the proxies scale by 1e-6.
    # The mask must match the oracle's routing, with the band scaled as the proxies are, and the
    # outputs the oracle's.
    w, (q, k, v) = small_inputs(name)
    q = (q.float() * qf).to(q.dtype)
    k = (k.float() * kf).to(k.dtype)
    kbar = np.abs(ora.pool_means(to_np(k), 64)[0])
    if kf > 1:
        assert (kbar > 65504).any(axis=-1).mean() > 0.3
    else:
        assert np.median(kbar) < 2.0 ** -14   # below the smallest normal f16
    qn, kn, vn = to_np(q), to_np(k), to_np(v)
    for mode in modes:
        for beta in (0.8, -0.3):
            print(f"[parity] {name} q x{qf} k x{kf} {mode} beta={beta}", flush=True)
            out, gmask, counts = run_gpu(dev, w, q, k, v, beta, mode)
            ref = ora.forward(qn, kn, vn, w.block_q, 64, beta, mode, keep_tail_tokens=w.text_tokens)
            flips = assert_mask_matches(gmask, ref["mask"], ref["s_hat"], ref["tau"], band=1e-3 * qf * kf)
            if flips:
                ref = ora.forward(qn, kn, vn, w.block_q, 64, beta, mode, keep_tail_tokens=w.text_tokens,
                                  mask=gmask)
            assert np.array_equal(counts, gmask.sum(axis=(2, 3)))
            assert_output_close(to_np(out), ref["out"], w.dtype, f"{name}/q x{qf} k x{kf}/{mode}/{beta}")
    if kf > 1:
        # SOL_SPARSE with pooled keys past the f16 range is outside its contract: the correction
        # tiles' f16 pooled keys overflow, so its outputs are not defined.  What stays defined is
        # what the f32 routing produces: the mask and the counts.
        out, gmask, counts = run_gpu(dev, w, q, k, v, 0.8, "sparse", outputs_defined=False)
        ref = ora.routing(qn, kn, w.block_q, 64, 0.8, keep_tail_tokens=w.text_tokens)
        assert_mask_matches(gmask, ref["mask"], ref["s_hat"], ref["tau"], band=1e-3 * qf * kf)
        assert np.array_equal(counts, gmask.sum(axis=(2, 3)))


def test_no_correction_with_nothing_selected_is_zero(dev):
    w, (q, k, v) = small_inputs("bf16_d128_q128")
    out, gmask, counts = run_gpu(dev, w, q, k, v, INF, "sparse_no_correction")
    assert not gmask.any() and not counts.any()
    assert torch.count_nonzero(out) == 0


def test_short_form_and_stats(dev):
    w, (q, k, v) = small_inputs("bf16_d128_q128")
    qd, kd, vd = (t.to(dev) for t in (q, k, v))
    ref, gmask, counts = run_gpu(dev, w, q, k, v, 0.8, "sparse")
    out = torch.empty_like(qd)
    sb.forward_short(qd, kd, vd, out, w.block_q, 64, 0.8, "sparse")
    frac = sb.stats(w.B, w.H)
    assert torch.equal(out, ref)
    nkr = w.NK
    np.testing.assert_allclose(frac, (gmask.sum(axis=(2, 3)) / (w.NQ * nkr)).ravel(), rtol=1e-6)


def test_stats_per_counts_buffer(dev):
    # Two forwards in flight on two streams, each with its own counts buffer: sol_attn_stats
    # returns each one's own per-head fractions (with the shape of the forward that wrote it),
    # and refuses counts = NULL when the thread's last forward used caller-owned counts.
    wa, (qa, ka, va) = small_inputs("bf16_d128_q128")
    wb, (qb, kb, vb) = small_inputs("bf16_d64_q64_text")
    ra, ma, _ = run_gpu(dev, wa, qa, ka, va, 0.8, "sparse")
    rb, mb, _ = run_gpu(dev, wb, qb, kb, vb, 0.3, "sparse_no_correction")
    want_a = (ma.sum(axis=(2, 3)) / (wa.NQ * wa.NK)).ravel()
    want_b = (mb.sum(axis=(2, 3)) / (wb.NQ * (wb.NK - wb.text_tokens // 64))).ravel()
    ca = torch.zeros((wa.B, wa.H), dtype=torch.int32, device=dev)
    cb = torch.zeros((wb.B, wb.H), dtype=torch.int32, device=dev)
    dev_in = [tuple(t.to(dev) for t in x) for x in ((qa, ka, va), (qb, kb, vb))]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]   # default priority
    ws = [torch.empty(sb.workspace_bytes(w.B, w.H, w.N, w.d, w.block_q, 64, m, sb.SOL_BF16, w.text_tokens),
                      dtype=torch.uint8, device=dev) for w, m in ((wa, "sparse"), (wb, "sparse_no_correction"))]
    torch.cuda.synchronize()
    with torch.cuda.stream(streams[0]):
        sb.forward(*dev_in[0], wa.block_q, 64, 0.8, "sparse", counts=ca, workspace=ws[0])
    with torch.cuda.stream(streams[1]):
        sb.forward(*dev_in[1], wb.block_q, 64, 0.3, "sparse_no_correction", keep_tail_tokens=wb.text_tokens,
                   counts=cb, workspace=ws[1])
    np.testing.assert_allclose(sb.stats(wb.B, wb.H, counts=cb), want_b, rtol=1e-6)
    np.testing.assert_allclose(sb.stats(wa.B, wa.H, counts=ca), want_a, rtol=1e-6)
    with pytest.raises(sb.SolAttnError) as ei:   # the last forward on this thread wrote caller counts
        sb.stats(wb.B, wb.H)
    assert ei.value.code == sb.SOL_ERR_NO_DATA
    import ctypes
    arr = (ctypes.c_float * 2)()   # B/H other than those of the forward that wrote ca (1, 2)
    assert sb.lib().sol_attn_stats(ctypes.cast(arr, ctypes.c_void_p), 2, 1, ca.data_ptr()) == sb.SOL_ERR_NO_DATA
    torch.cuda.synchronize()


def test_caller_workspace(dev):
    w, (q, k, v) = small_inputs("bf16_d64_q64_text")
    qd, kd, vd = (t.to(dev) for t in (q, k, v))
    ref = sb.forward(qd, kd, vd, w.block_q, 64, 0.8, "sparse", keep_tail_tokens=w.text_tokens)
    nbytes = sb.workspace_bytes(w.B, w.H, w.N, w.d, w.block_q, 64, "sparse", sb.SOL_BF16, w.text_tokens)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    out = sb.forward(qd, kd, vd, w.block_q, 64, 0.8, "sparse", keep_tail_tokens=w.text_tokens, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(out, ref)
    with pytest.raises(sb.SolAttnError) as ei:
        sb.forward(qd, kd, vd, w.block_q, 64, 0.8, "sparse", keep_tail_tokens=w.text_tokens, workspace=ws[: nbytes // 2])
    assert ei.value.code == sb.SOL_ERR_WORKSPACE


@pytest.mark.parametrize("name", ["bf16_d128_q128", "bf16_d128_q64_text"])
def test_deterministic(dev, name):
    w, (q, k, v) = small_inputs(name)
    a, _, _ = run_gpu(dev, w, q, k, v, 0.8, "sparse")
    b, _, _ = run_gpu(dev, w, q, k, v, 0.8, "sparse")
    assert torch.equal(a, b)


# --------------------------------------------------------------------------- many heads, every row
# 96 queue positions per XCD: a third of the query blocks start their exact tiles at a nonzero
# phase, the persistent workgroups run more than one block each and may take blocks from other
# XCDs' queues; every output row is compared with the oracle.
_many = {}


def many_heads_inputs():
    if not _many:
        w = small_workload("many_heads", (16, 128), 128, 128, H=24, B=2, seed=31)
        _many["w"] = w
        _many["qkv"] = synth.make_qkv(w)
    return _many["w"], _many["qkv"]


@pytest.mark.parametrize("mode,beta", [("sparse", 0.5), ("sparse_no_correction", 0.8), ("dense", 0.0)])
def test_forward_parity_many_heads(dev, mode, beta):
    w, (q, k, v) = many_heads_inputs()
    print(f"[parity] many heads B={w.B} H={w.H} N={w.N} mode={mode} beta={beta}", flush=True)
    out, gmask, counts = run_gpu(dev, w, q, k, v, beta, mode)
    qn, kn, vn = to_np(q), to_np(k), to_np(v)
    ref = ora.forward(qn, kn, vn, w.block_q, 64, beta, mode)
    if mode != "dense":
        flips = assert_mask_matches(gmask, ref["mask"], ref["s_hat"], ref["tau"])
        if flips:
            ref = ora.forward(qn, kn, vn, w.block_q, 64, beta, mode, mask=gmask)
        assert np.array_equal(counts, gmask.sum(axis=(2, 3)))
    assert_output_close(to_np(out), ref["out"], w.dtype, f"many_heads/{mode}/{beta}")


def test_many_heads_beta_minus_inf_is_bitwise_dense(dev):
    w, (q, k, v) = many_heads_inputs()
    dense, _, _ = run_gpu(dev, w, q, k, v, 0.0, "dense", want_mask=False)
    out, gmask, _ = run_gpu(dev, w, q, k, v, -INF, "sparse")
    assert gmask.all()
    assert torch.equal(out, dense)


def test_concurrent_streams_own_workspaces(dev):
    # Two forwards in flight at once on two streams, each with its own workspace (which holds the
    # pre-pass results and the work-queue counters) and counts: both match the sequential results
    # bit for bit.
    w, (q, k, v) = many_heads_inputs()
    qd, kd, vd = (t.to(dev) for t in (q, k, v))
    ref_s = sb.forward(qd, kd, vd, w.block_q, 64, 0.5, "sparse")
    ref_d = sb.forward(qd, kd, vd, w.block_q, 64, 0.0, "dense")
    ws = [torch.empty(sb.workspace_bytes(w.B, w.H, w.N, w.d, w.block_q, 64, m, sb.SOL_BF16, 0), dtype=torch.uint8,
                      device=dev) for m in ("sparse", "dense")]
    counts = [torch.zeros((w.B, w.H), dtype=torch.int32, device=dev) for _ in range(2)]
    outs = [torch.full_like(qd, math.nan) for _ in range(2)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]   # default priority
    torch.cuda.synchronize()
    for _ in range(3):
        with torch.cuda.stream(streams[0]):
            sb.forward(qd, kd, vd, w.block_q, 64, 0.5, "sparse", out=outs[0], workspace=ws[0], counts=counts[0])
        with torch.cuda.stream(streams[1]):
            sb.forward(qd, kd, vd, w.block_q, 64, 0.0, "dense", out=outs[1], workspace=ws[1], counts=counts[1])
    torch.cuda.synchronize()
    assert torch.equal(outs[0], ref_s)
    assert torch.equal(outs[1], ref_d)


# --------------------------------------------------------------------------- full workload shapes

@pytest.fixture(scope="module", params=["video480p", "image", "video720p"])
def full(request, dev):
    w = configs.WORKLOADS[request.param]
    print(f"[parity] generating {w.name}", flush=True)
    q, k, v = synth.make_qkv(w, workers=synth.default_workers())
    beta = configs.beta_for(w)
    print(f"[parity] oracle routing {w.name}", flush=True)
    r = ora.routing(q.float().numpy(), k.float().numpy(), w.block_q, 64, beta, keep_tail_tokens=w.text_tokens)
    yield w, (q, k, v), beta, r
    del q, k, v, r


@pytest.mark.parametrize("mode", ["sparse", "sparse_no_correction", "dense"])
def test_full_size_sampled(dev, full, mode):
    w, (q, k, v), beta, r = full
    print(f"[parity] full {w.name} mode={mode}", flush=True)
    out, gmask, counts = run_gpu(dev, w, q, k, v, beta, mode)
    heads = [(0, 0), (w.B - 1, w.H - 1)]
    # 480p and image: every query block of both heads; 720p (whose whole heads are compared at
    # every cutoff of the kept-fraction sweep): first, second, middle and ragged last block
    qblocks = sorted({0, 1, w.NQ // 2, w.NQ - 1}) if w.name == "video720p" else list(range(w.NQ))
    mask_for_oracle = None
    if mode != "dense":
        flips = assert_mask_matches(gmask, r["mask"], r["s_hat"], r["tau"])
        print(f"[parity] {w.name}: {flips} in-band mask flips of {gmask.size}", flush=True)
        assert np.array_equal(counts, gmask.sum(axis=(2, 3)))
        mask_for_oracle = gmask
    hb, hh = [b for b, _ in heads], [h for _, h in heads]
    qs, ks, vs = (x[hb, hh].float().numpy() for x in (q, k, v))
    sub_mask = None if mask_for_oracle is None else mask_for_oracle[hb, hh]
    got = out[hb, hh].float().cpu().numpy().astype(np.float64)[None]
    rows = np.concatenate([np.arange(i * w.block_q, min((i + 1) * w.block_q, w.N)) for i in qblocks])
    if len(qblocks) == w.NQ:   # whole heads: (head, block range) jobs in a process pool
        ref_out = oracle_whole_heads(qs, ks, vs, w.block_q, 64, beta, mode, mask=sub_mask,
                                     keep_tail_tokens=w.text_tokens)[None]
    else:
        ref_out = ora.forward(qs[None], ks[None], vs[None], w.block_q, 64, beta, mode, keep_tail_tokens=w.text_tokens,
                              query_blocks=qblocks, mask=None if sub_mask is None else sub_mask[None])["out"]
    ref = {"out": ref_out}
    max_abs, mean_rel = assert_output_close(got[:, :, rows], ref["out"][:, :, rows], w.dtype, f"{w.name}/{mode}")
    print(f"[parity] {w.name} {mode}: {len(qblocks)} query blocks of heads {heads}, max-abs {max_abs:.3e}, "
          f"mean-rel {mean_rel:.3e}", flush=True)


def test_full_size_diagonal_threshold_mask(dev, full):
    # The diagonal estimator at its own calibrated cutoff (same target density): GPU mask
    # against the oracle's diagonal routing on every pair (bit-exact outside the 1e-3
    # band), and its agreement with the exact estimator's mask.
    w, (q, k, v), _, r = full
    beta = configs.beta_for(w, threshold_mode="diagonal")
    _, gmask, counts = run_gpu(dev, w, q, k, v, beta, "sparse_no_correction", threshold_mode="diagonal")
    rd = ora.routing(q.float().numpy(), k.float().numpy(), w.block_q, 64, beta, keep_tail_tokens=w.text_tokens,
                     threshold_mode="diagonal")
    flips = assert_mask_matches(gmask, rd["mask"], rd["s_hat"], rd["tau"])
    agree = float((rd["mask"] == r["mask"]).mean())
    print(f"[parity] {w.name} diagonal thresholds: kept {float(rd['mask'].mean()):.4f} (exact "
          f"{float(r['mask'].mean()):.4f}), mask agreement with exact {agree:.4f}, {flips} in-band flips",
          flush=True)
    assert np.array_equal(counts, gmask.sum(axis=(2, 3)))


# --------------------------------------------------------------------------- routing baselines

def check_baseline_masks(gmask, ref_mask, s_hat, rule):
    """GPU top-k / top-p mask against the oracle's on the same proxies: differences only at
    near-ties of the cut (proxies within 1e-3 of the smallest kept one)."""
    diff = gmask != ref_mask
    if rule == "topk":
        assert np.array_equal(gmask.sum(-1), ref_mask.sum(-1))
    else:
        assert np.all(np.abs(gmask.sum(-1).astype(np.int64) - ref_mask.sum(-1)) <= 2)
    cut = np.where(ref_mask, s_hat, np.inf).min(axis=-1, keepdims=True)
    near = np.abs(s_hat - cut) < 1e-3
    assert not (diff & ~near).any(), f"{int((diff & ~near).sum())} baseline mask differences away from the cut"
    return int(diff.sum())


@pytest.mark.parametrize("name", ["bf16_d128_q128", "f32_d64_q64", "bf16_d64_q64_text"])
@pytest.mark.parametrize("rule,param", [("topk", 1), ("topk", 7), ("topk", 25), ("topp", 0.05), ("topp", 0.5),
                                        ("topp", 0.95), ("topp", 1.0)])
def test_route_materialized_small(dev, name, rule, param):
    w, (q, k, v) = small_inputs(name)
    nkr = w.NK - w.text_tokens // 64
    if rule == "topk" and param > nkr:
        pytest.skip("k larger than the routable blocks")
    qbar, kbar, _ = sb.pool_blocks(q.to(dev), k.to(dev), v.to(dev), w.block_q, 64)
    prox, mask = sb.route_materialized(qbar, kbar, rule, param, nk_routable=nkr)
    torch.cuda.synchronize()
    s_hat = ora.proxy_scores(to_np(qbar), to_np(kbar)[:, :, :nkr], 1 / math.sqrt(w.d))
    np.testing.assert_allclose(to_np(prox), s_hat, atol=1e-5, rtol=1e-5)
    gmask = sb.unpack_mask(mask.cpu().numpy().view(np.uint32), nkr)
    ref = ora.route_topk(s_hat, param) if rule == "topk" else ora.route_topp(s_hat, param)
    check_baseline_masks(gmask, ref, s_hat, rule)


def test_route_materialized_full_720p(dev):
    w = configs.WORKLOADS["video720p"]
    q, k, v = synth.make_qkv(w, heads=[(0, 0), (0, 1)], workers=synth.default_workers())
    q, k, v = q[:, :2].contiguous(), k[:, :2].contiguous(), v[:, :2].contiguous()
    qbar, kbar, _ = sb.pool_blocks(q.to(dev), k.to(dev), v.to(dev), w.block_q, 64)
    s_hat = ora.proxy_scores(to_np(qbar), to_np(kbar), 1 / math.sqrt(w.d))
    for rule, param in (("topk", 177), ("topp", 0.32)):
        _, mask = sb.route_materialized(qbar, kbar, rule, param)
        torch.cuda.synchronize()
        gmask = sb.unpack_mask(mask.cpu().numpy().view(np.uint32), w.NK)
        ref = ora.route_topk(s_hat, param) if rule == "topk" else ora.route_topp(s_hat, param)
        n = check_baseline_masks(gmask, ref, s_hat, rule)
        print(f"[parity] 720p {rule}({param}): {n} near-cut differences, kept {gmask.mean():.4f}", flush=True)
