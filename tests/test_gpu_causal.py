"""GPU parity of routed attention under causal masks (sol_attn_forward_causal) against the
fp64 oracle: masks bit-exact outside the 1e-3 band of the threshold, outputs within the
bf16 / f32 tolerances, counts and stats over each query block's routable blocks."""
import math

import numpy as np
import pytest
import torch

from oracle import sol_attn_oracle as ora
from paper_2607_24027_amd import binding as sb
from paper_2607_24027_amd import configs, synth
from tests.parity import assert_mask_matches, assert_output_close, small_workload, to_np

pytestmark = pytest.mark.gpu

INF = math.inf


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    sb.lib()  # fail loudly if the library is missing
    return torch.device("cuda:0")


CASES = {
    # name: (grid, d, block_q, dtype, causal granule)
    "bf16_d128_q128_token": ((5, 10, 100), 128, 128, "bf16", 1),        # N=5000, ragged blocks
    "bf16_d128_q128_frame": ((5, 10, 100), 128, 128, "bf16", 1000),     # one frame = 1000 tokens
    "bf16_d128_q128_whole": ((5, 10, 100), 128, 128, "bf16", 5000),     # G = N: bidirectional
    "bf16_d64_q64_g7": ((4, 20, 70), 64, 64, "bf16", 7),                # N=5600, granule off the blocks
    "bf16_d128_q64_row": ((60, 70), 128, 64, "bf16", 70),               # 2D grid, one image row per step
    "f32_d64_q64_token": ((4, 16, 32), 64, 64, "f32", 1),
    "f32_d128_q128_g41": ((3, 10, 41), 128, 128, "f32", 41),            # N=1230
}
_cache = {}


def inputs(name):
    if name not in _cache:
        grid, d, bq, dtype, g = CASES[name]
        w = small_workload(name, grid, d, bq, dtype=dtype, seed=29)
        _cache[name] = (w, g, synth.make_qkv(w))
    return _cache[name]


def routable_pairs(w, g):
    r, _ = ora.causal_block_ranges(w.N, w.block_q, 64, g)
    return int(r.sum())


_last_counts = {}   # device counts of the last run_causal call, for sol_attn_stats


def run_causal(dev, w, g, q, k, v, beta, mode):
    qd, kd, vd = (t.to(dev) for t in (q, k, v))
    mask = torch.zeros((w.B, w.H, w.NQ, sb.mask_words(w.NK)), dtype=torch.int32, device=dev)
    counts = torch.full((w.B, w.H), -1, dtype=torch.int32, device=dev)
    out = sb.forward(qd, kd, vd, w.block_q, 64, beta, mode, counts=counts, mask_out=mask, causal_granule=g)
    torch.cuda.synchronize()
    _last_counts["t"] = counts
    gmask = sb.unpack_mask(mask.cpu().numpy().view(np.uint32), w.NK) if mode != "dense" else None
    return out, gmask, counts.cpu().numpy().view(np.uint32)


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("mode,beta", [("dense", 0.0), ("sparse", 0.8), ("sparse", -INF), ("sparse", INF),
                                       ("sparse_no_correction", 0.8), ("sparse_no_correction", -INF),
                                       ("sparse", 0.0)])
def test_causal_parity_small(dev, name, mode, beta):
    w, g, (q, k, v) = inputs(name)
    print(f"[causal] {name} G={g} mode={mode} beta={beta}", flush=True)
    out, gmask, counts = run_causal(dev, w, g, q, k, v, beta, mode)
    qn, kn, vn = to_np(q), to_np(k), to_np(v)
    ref = ora.forward(qn, kn, vn, w.block_q, 64, beta, mode, causal_granule=g)
    if mode != "dense":
        flips = assert_mask_matches(gmask, ref["mask"], ref["s_hat"], ref["tau"])
        if flips:
            ref = ora.forward(qn, kn, vn, w.block_q, 64, beta, mode, causal_granule=g, mask=gmask)
        assert np.array_equal(counts, gmask.sum(axis=(2, 3)))
        frac = np.array(sb.stats(w.B, w.H, counts=_last_counts["t"])).reshape(w.B, w.H)
        np.testing.assert_allclose(frac, gmask.sum(axis=(2, 3)) / routable_pairs(w, g), rtol=1e-6)
    else:
        assert np.all(counts == routable_pairs(w, g))
    assert_output_close(to_np(out), ref["out"], w.dtype, f"causal {name}/{mode}/{beta}")


def random_causal_case(seed):
    """A seeded random causal configuration: token grid, block sizes, dtype, granule, cutoff, mode."""
    rng = np.random.default_rng(2000 + seed)
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
    n = int(np.prod(grid))
    r = rng.random()
    g = 1 if r < 0.3 else (n if r < 0.4 else int(rng.integers(1, n + 1)))   # token, bidirectional, any
    B, H = int(rng.integers(1, 3)), int(rng.integers(1, 4))
    r = rng.random()
    beta = -INF if r < 0.1 else (INF if r < 0.2 else float(np.round(rng.uniform(-1.0, 2.0), 3)))
    mode = str(rng.choice(["dense", "sparse", "sparse_no_correction"]))
    return grid, d, bq, dtype, g, B, H, beta, mode


@pytest.mark.parametrize("seed", range(24))
def test_causal_parity_random_shapes(dev, seed):
    # Seeded random causal configurations (any token count, ragged tails, 1D/2D/3D grids, granules
    # from one token to the whole sequence, both dtypes and block heights, cutoffs from -inf to
    # +inf), element by element.
    grid, d, bq, dtype, g, B, H, beta, mode = random_causal_case(seed)
    w = small_workload(f"crand{seed}", grid, d, bq, dtype=dtype, H=H, B=B, seed=90 + seed)
    print(f"[causal] random {seed}: grid={grid} N={w.N} d={d} bq={bq} {dtype} G={g} B={B} H={H} beta={beta} "
          f"{mode}", flush=True)
    q, k, v = synth.make_qkv(w)
    out, gmask, counts = run_causal(dev, w, g, q, k, v, beta, mode)
    assert bool(torch.isfinite(out).all())
    qn, kn, vn = to_np(q), to_np(k), to_np(v)
    ref = ora.forward(qn, kn, vn, w.block_q, 64, beta, mode, causal_granule=g)
    if mode != "dense":
        flips = assert_mask_matches(gmask, ref["mask"], ref["s_hat"], ref["tau"])
        if flips:
            ref = ora.forward(qn, kn, vn, w.block_q, 64, beta, mode, causal_granule=g, mask=gmask)
        assert np.array_equal(counts, gmask.sum(axis=(2, 3)))
    else:
        assert np.all(counts == routable_pairs(w, g))
    assert_output_close(to_np(out), ref["out"], w.dtype, f"causal random {seed}")


def test_causal_full_selection_is_bitwise_dense(dev):
    w, g, (q, k, v) = inputs("bf16_d128_q128_token")
    dense, _, _ = run_causal(dev, w, g, q, k, v, 0.0, "dense")
    for mode in ("sparse", "sparse_no_correction"):
        out, gmask, _ = run_causal(dev, w, g, q, k, v, -INF, mode)
        r, _ = ora.causal_block_ranges(w.N, w.block_q, 64, g)
        assert np.array_equal(gmask.sum(axis=-1)[0, 0], r)
        assert torch.equal(out, dense)


def test_causal_deterministic(dev):
    w, g, (q, k, v) = inputs("bf16_d128_q128_frame")
    a, _, _ = run_causal(dev, w, g, q, k, v, 0.8, "sparse")
    b, _, _ = run_causal(dev, w, g, q, k, v, 0.8, "sparse")
    assert torch.equal(a, b)


# --------------------------------------------------------------------------- 720p video shape

@pytest.fixture(scope="module")
def video(dev):
    w = configs.WORKLOADS["video720p"]
    print(f"[causal] generating {w.name}", flush=True)
    q, k, v = synth.make_qkv(w, workers=synth.default_workers())
    yield w, (q, k, v)
    del q, k, v


@pytest.mark.parametrize("g", [3600, 1])   # frame-causal (45 x 80 tokens per frame), token-causal
@pytest.mark.parametrize("mode", ["sparse", "dense"])
def test_causal_full_size_sampled(dev, video, g, mode):
    w, (q, k, v) = video
    beta = configs.beta_for(w)
    print(f"[causal] full {w.name} G={g} mode={mode}", flush=True)
    out, gmask, counts = run_causal(dev, w, g, q, k, v, beta, mode)
    mask_for_oracle = None
    if mode != "dense":
        r = ora.routing(q.float().numpy(), k.float().numpy(), w.block_q, 64, beta, causal_granule=g)
        flips = assert_mask_matches(gmask, r["mask"], r["s_hat"], r["tau"])
        print(f"[causal] {w.name} G={g}: kept {float(r['frac'].mean()):.4f} of routable pairs, "
              f"{flips} in-band flips", flush=True)
        assert np.array_equal(counts, gmask.sum(axis=(2, 3)))
        mask_for_oracle = gmask
    heads = [(0, 0), (w.B - 1, w.H - 1)]
    qblocks = sorted({0, 1, w.NQ // 3, w.NQ // 2, w.NQ - 1})
    qs, ks, vs = (x[[b for b, _ in heads], [h for _, h in heads]].float().numpy()[None] for x in (q, k, v))
    sub_mask = None if mask_for_oracle is None else mask_for_oracle[[b for b, _ in heads], [h for _, h in heads]][None]
    ref = ora.forward(qs, ks, vs, w.block_q, 64, beta, mode, query_blocks=qblocks, mask=sub_mask, causal_granule=g)
    got = out[[b for b, _ in heads], [h for _, h in heads]].float().cpu().numpy()[None].astype(np.float64)
    rows = np.concatenate([np.arange(i * w.block_q, min((i + 1) * w.block_q, w.N)) for i in qblocks])
    assert_output_close(got[:, :, rows], ref["out"][:, :, rows], w.dtype, f"causal {w.name}/G={g}/{mode}")
