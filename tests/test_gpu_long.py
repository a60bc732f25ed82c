"""GPU parity near the longest sequence the bf16 path supports at d = 128.

At about 1.48M tokens the per-block routing state (selection words, their prefix
counts and the two 16-bit lists) fills most of the on-chip budget, so the fused
kernel runs one workgroup per compute unit instead of two.  This exercises that
launch configuration and the largest list lengths: the complete selection mask
against the oracle's routing (bit-exact outside the 1e-3 band), the counts, and the
outputs of the first, a middle and the ragged last query block against the fp64
oracle evaluated with the GPU's mask.
"""
import math

import numpy as np
import pytest
import torch

from oracle import sol_attn_oracle as ora
from paper_2607_24027_amd import binding as sb
from paper_2607_24027_amd import synth
from paper_2607_24027_amd.configs import Workload
from tests.parity import assert_mask_matches, assert_output_close

pytestmark = pytest.mark.gpu

# 41 x 160 x 225 = 1,476,000 tokens: 23,063 key blocks (ragged by 32 tokens), 11,532 query blocks
LONG = Workload("long_video", B=1, H=1, d=128, dtype="bf16", grid=(41, 160, 225), block_q=128, block_k=64,
                target_kept=0.2, seed=7)
BETA = 1.0   # about a fifth of the routable blocks kept on these inputs


@pytest.mark.timeout(600)   # the fp64 oracle needs about a minute at this length
def test_longest_supported_sequence_sparse():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    sb.lib()
    dev = torch.device("cuda:0")
    w = LONG
    print(f"[long] generating N={w.N}", flush=True)
    q, k, v = synth.make_qkv(w)
    qd, kd, vd = (t.to(dev) for t in (q, k, v))
    nkr = w.NK
    mask = torch.zeros((1, 1, w.NQ, sb.mask_words(nkr)), dtype=torch.int32, device=dev)
    counts = torch.full((1, 1), -1, dtype=torch.int32, device=dev)
    out = torch.full_like(qd, math.nan)
    print("[long] sparse forward", flush=True)
    sb.forward(qd, kd, vd, w.block_q, 64, BETA, "sparse", out=out, counts=counts, mask_out=mask)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(out).all()), "rows left unwritten"
    gmask = sb.unpack_mask(mask.cpu().numpy().view(np.uint32), nkr)
    del mask, qd, kd, vd
    kept = float(gmask.mean())
    print(f"[long] kept {kept:.4f}; oracle routing", flush=True)
    assert 0.05 < kept < 0.5
    qn, kn, vn = (t.float().numpy() for t in (q, k, v))
    r = ora.routing(qn, kn, w.block_q, 64, BETA)
    flips = assert_mask_matches(gmask, r["mask"], r["s_hat"], r["tau"])
    print(f"[long] {flips} in-band mask flips of {gmask.size}", flush=True)
    assert np.array_equal(counts.cpu().numpy().view(np.uint32), gmask.sum(axis=(2, 3)))
    del r
    qblocks = [0, w.NQ // 2, w.NQ - 1]
    print(f"[long] oracle outputs of query blocks {qblocks}", flush=True)
    ref = ora.forward(qn, kn, vn, w.block_q, 64, BETA, "sparse", query_blocks=qblocks, mask=gmask)["out"]
    rows = np.concatenate([np.arange(i * w.block_q, min((i + 1) * w.block_q, w.N)) for i in qblocks])
    got = out.float().cpu().numpy().astype(np.float64)
    max_abs, mean_rel = assert_output_close(got[:, :, rows], ref[:, :, rows], w.dtype, "long/sparse")
    print(f"[long] max-abs {max_abs:.3e} mean-rel {mean_rel:.3e}", flush=True)


# 16 x 120 x 125 = 240,000 tokens, frame-causal with one 15,000-token frame per step: 3,750 key
# blocks, whose row proxies sit in the tile stages during the routing prologue, so two workgroups
# still share a compute unit
LONG_CAUSAL = Workload("long_video_causal", B=1, H=1, d=128, dtype="bf16", grid=(16, 120, 125), block_q=128,
                       block_k=64, target_kept=0.2, seed=8)
GRANULE = 120 * 125


@pytest.mark.timeout(600)
def test_long_causal_sequence_sparse():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    sb.lib()
    dev = torch.device("cuda:0")
    w = LONG_CAUSAL
    print(f"[long] generating N={w.N} (causal, granule {GRANULE})", flush=True)
    q, k, v = synth.make_qkv(w)
    qd, kd, vd = (t.to(dev) for t in (q, k, v))
    mask = torch.zeros((1, 1, w.NQ, sb.mask_words(w.NK)), dtype=torch.int32, device=dev)
    counts = torch.full((1, 1), -1, dtype=torch.int32, device=dev)
    out = torch.full_like(qd, math.nan)
    sb.forward(qd, kd, vd, w.block_q, 64, BETA, "sparse", out=out, counts=counts, mask_out=mask,
               causal_granule=GRANULE)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(out).all()), "rows left unwritten"
    gmask = sb.unpack_mask(mask.cpu().numpy().view(np.uint32), w.NK)
    del mask, qd, kd, vd
    qn, kn, vn = (t.float().numpy() for t in (q, k, v))
    r = ora.routing(qn, kn, w.block_q, 64, BETA, causal_granule=GRANULE)
    flips = assert_mask_matches(gmask, r["mask"], r["s_hat"], r["tau"])
    print(f"[long] causal: kept {float(r['frac'].mean()):.4f} of routable pairs, {flips} in-band flips", flush=True)
    assert np.array_equal(counts.cpu().numpy().view(np.uint32), gmask.sum(axis=(2, 3)))
    del r
    qblocks = [0, w.NQ // 2, w.NQ - 1]
    ref = ora.forward(qn, kn, vn, w.block_q, 64, BETA, "sparse", query_blocks=qblocks, mask=gmask,
                      causal_granule=GRANULE)["out"]
    rows = np.concatenate([np.arange(i * w.block_q, min((i + 1) * w.block_q, w.N)) for i in qblocks])
    got = out.float().cpu().numpy().astype(np.float64)
    max_abs, mean_rel = assert_output_close(got[:, :, rows], ref[:, :, rows], w.dtype, "long causal/sparse")
    print(f"[long] causal max-abs {max_abs:.3e} mean-rel {mean_rel:.3e}", flush=True)
