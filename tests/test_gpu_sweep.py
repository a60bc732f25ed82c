"""GPU parity at the workloads' own cutoffs: the 720p kept-fraction sweep and the tiny workload.

The 720p shape (B=1, H=40, N=75,600, d=128, blocks 128 x 64) runs at each calibrated cutoff of the
sweep (50/25/20/10/5 % kept; 100 % is beta = -inf).  Each point checks, in order:

* the complete selection mask of the GPU against the fp64 oracle's own routing (bit-exact outside
  the 1e-3 band around tau_i; in-band flips are counted and printed), and the per-head counts;
* the kept fraction against the calibration target;
* every row of three whole heads (0, 19 and 39: all 591 query blocks, the ragged last one
  included) against the oracle evaluated on the GPU's selection, in sparse and no-correction
  mode (and dense mode at the 20 % headline), within max-abs 2e-2 and mean-rel 2e-3.

The oracle is given the GPU's mask only after that mask has passed the routing check, so a
difference inside the band is attributed to arithmetic, not routing (Section 4.5 compares the
modes under identical indices the same way).
"""
import math

import numpy as np
import pytest
import torch

from oracle import sol_attn_oracle as ora
from paper_2607_24027_amd import binding as sb
from paper_2607_24027_amd import configs, synth
from tests.parity import assert_mask_matches, assert_output_close, errors, oracle_whole_heads, to_np

pytestmark = pytest.mark.gpu

W720 = configs.WORKLOADS["video720p"]
HEADS = (0, 19, 39)                      # batch 0; first, middle and last head
POINTS = (0.50, 0.25, 0.20, 0.10, 0.05)  # calibrated kept fractions of the 720p sweep


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    sb.lib()
    return torch.device("cuda:0")


_state = {}


def inputs720(dev):
    """720p inputs on the host and the GPU, and the oracle's proxies and row statistics (shared by
    every cutoff: only tau_i = mu_i + beta sigma_i and the selection depend on beta)."""
    if not _state:
        print("[sweep] generating video720p inputs", flush=True)
        q, k, v = synth.make_qkv(W720, workers=synth.default_workers())
        _state["host"] = (q, k, v)
        _state["dev"] = tuple(t.to(dev) for t in (q, k, v))
        print("[sweep] oracle proxies and row statistics", flush=True)
        r = ora.routing(q.float().numpy(), k.float().numpy(), W720.block_q, 64, 0.0)
        _state["s_hat"], _state["mu"], _state["sigma"] = r["s_hat"], r["mu"], r["sigma"]
        _state["runs"] = {}
    return _state


def oracle_mask(st, beta):
    tau = ora.thresholds(st["mu"], st["sigma"], beta)
    return ora.route(st["s_hat"], tau), tau


def gpu_run(dev, kept, mode):
    """One forward of the 720p shape at the cutoff for `kept`; returns the selection mask, counts and
    the outputs of the compared heads (host).  Cached per (kept, mode)."""
    st = inputs720(dev)
    key = (kept, mode)
    if key not in st["runs"]:
        beta = configs.beta_for(W720, kept)
        qd, kd, vd = st["dev"]
        nkr = W720.NK
        mask = torch.zeros((1, W720.H, W720.NQ, sb.mask_words(nkr)), dtype=torch.int32, device=dev)
        counts = torch.full((1, W720.H), -1, dtype=torch.int32, device=dev)
        out = torch.full_like(qd, math.nan)
        sb.forward(qd, kd, vd, W720.block_q, 64, beta, mode, out=out, counts=counts,
                   mask_out=None if mode == "dense" else mask)
        torch.cuda.synchronize()
        assert bool(torch.isfinite(out).all()), f"720p {mode} at {kept}: rows left unwritten"
        gmask = None if mode == "dense" else sb.unpack_mask(mask.cpu().numpy().view(np.uint32), nkr)
        heads = out[0, list(HEADS)].float().cpu().numpy().astype(np.float64)
        st["runs"][key] = (beta, gmask, counts.cpu().numpy().view(np.uint32), heads)
    return st["runs"][key]


@pytest.mark.parametrize("kept", POINTS)
def test_sweep_routing_720p(dev, kept):
    st = inputs720(dev)
    beta, gmask, counts, _ = gpu_run(dev, kept, "sparse")
    ref_mask, tau = oracle_mask(st, beta)
    flips = assert_mask_matches(gmask, ref_mask, st["s_hat"], tau)
    assert np.array_equal(counts, gmask.sum(axis=(2, 3)))
    frac = float(gmask.mean())
    print(f"[sweep] {kept:.2f}: beta {beta:.6f}, kept {frac:.4f} (oracle {float(ref_mask.mean()):.4f}), "
          f"{flips} in-band flips of {gmask.size} pairs", flush=True)
    assert abs(float(ref_mask.mean()) - kept) < 0.005
    # the no-correction kernel routes with the same code: the same selection, bit for bit
    _, gmask_nc, counts_nc, _ = gpu_run(dev, kept, "sparse_no_correction")
    assert np.array_equal(gmask_nc, gmask) and np.array_equal(counts_nc, counts)


def _whole_heads(dev, kept, mode):
    st = inputs720(dev)
    beta, gmask, _, got = gpu_run(dev, kept, mode)
    if gmask is not None:
        ref_mask, tau = oracle_mask(st, beta)
        assert_mask_matches(gmask, ref_mask, st["s_hat"], tau)
        sub_mask = gmask[0, list(HEADS)][None]
    else:
        sub_mask = None
    q, k, v = st["host"]
    qs, ks, vs = (x[0, list(HEADS)].float().numpy() for x in (q, k, v))
    print(f"[sweep] {kept:.2f} {mode}: oracle on heads {HEADS}", flush=True)
    ref = oracle_whole_heads(qs, ks, vs, W720.block_q, 64, beta, mode,
                             mask=None if sub_mask is None else sub_mask[0])
    for n, h in enumerate(HEADS):
        max_abs, mean_rel = errors(got[n], ref[n])
        print(f"[sweep] {kept:.2f} {mode} head {h}: all {W720.N} rows, max-abs {max_abs:.3e}, "
              f"mean-rel {mean_rel:.3e}", flush=True)
        assert_output_close(got[n], ref[n], "bf16", f"720p {mode} kept {kept} head {h}")


@pytest.mark.parametrize("kept", POINTS)
@pytest.mark.parametrize("mode", ["sparse", "sparse_no_correction"])
def test_sweep_whole_heads_720p(dev, kept, mode):
    _whole_heads(dev, kept, mode)


def test_headline_whole_heads_720p_dense(dev):
    _whole_heads(dev, W720.target_kept, "dense")


def test_sweep_full_selection_is_bitwise_dense_720p(dev):
    # The 100 % point: beta = -inf selects every block, and both sparse modes reproduce dense mode
    # bit for bit on every row of every head.
    st = inputs720(dev)
    qd, kd, vd = st["dev"]
    dense = sb.forward(qd, kd, vd, W720.block_q, 64, 0.0, "dense")
    for mode in ("sparse", "sparse_no_correction"):
        out = sb.forward(qd, kd, vd, W720.block_q, 64, -math.inf, mode)
        torch.cuda.synchronize()
        assert torch.equal(out, dense), mode


def test_sweep_release_inputs():
    # frees the 720p tensors before later test modules run
    _state.clear()
    torch.cuda.empty_cache()


# --------------------------------------------------------------------------- the tiny workload
TINY = configs.WORKLOADS["tiny"]


@pytest.mark.parametrize("mode", ["dense", "sparse", "sparse_no_correction"])
def test_tiny_workload_at_its_cutoff(dev, mode):
    # B=1, H=2, d=64, f32, N=2048 (4x16x32 grid), 64x64 blocks, seed 0, beta calibrated for 30 % kept:
    # complete mask and every output element against the oracle.
    beta = configs.beta_for(TINY)
    q, k, v = synth.make_qkv(TINY)
    qd, kd, vd = (t.to(dev) for t in (q, k, v))
    nkr = TINY.NK
    mask = torch.zeros((1, TINY.H, TINY.NQ, sb.mask_words(nkr)), dtype=torch.int32, device=dev)
    counts = torch.full((1, TINY.H), -1, dtype=torch.int32, device=dev)
    out = torch.full_like(qd, math.nan)
    sb.forward(qd, kd, vd, TINY.block_q, 64, beta, mode, out=out, counts=counts,
               mask_out=None if mode == "dense" else mask)
    torch.cuda.synchronize()
    qn, kn, vn = to_np(q), to_np(k), to_np(v)
    ref = ora.forward(qn, kn, vn, TINY.block_q, 64, beta, mode)
    cnt = counts.cpu().numpy().view(np.uint32)
    if mode != "dense":
        gmask = sb.unpack_mask(mask.cpu().numpy().view(np.uint32), nkr)
        flips = assert_mask_matches(gmask, ref["mask"], ref["s_hat"], ref["tau"])
        assert np.array_equal(cnt, gmask.sum(axis=(2, 3)))
        assert abs(float(ref["mask"].mean()) - TINY.target_kept) < 0.01
        if flips:
            ref = ora.forward(qn, kn, vn, TINY.block_q, 64, beta, mode, mask=gmask)
    else:
        assert np.all(cnt == TINY.NQ * nkr)
    max_abs, mean_rel = assert_output_close(to_np(out), ref["out"], "f32", f"tiny/{mode}")
    print(f"[tiny] {mode} beta {beta}: max-abs {max_abs:.3e}, mean-rel {mean_rel:.3e}", flush=True)
