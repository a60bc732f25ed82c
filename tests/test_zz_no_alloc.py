"""The forward entry point that allocates nothing (sol_attn_forward_noalloc), against the
workspace entry point (sol_attn_forward_ex) on the same inputs: two calls in a row on the same
built-in scratch, the second with a smaller input, each compared element by element (outputs,
counts and selection masks must agree bit for bit: both run the same kernels)."""
import math

import numpy as np
import pytest
import torch

from paper_2607_24027_amd import binding as sb
from paper_2607_24027_amd import synth
from tests.parity import assert_output_close, small_workload, to_np

pytestmark = pytest.mark.gpu

CASES = [
    # (grid, d, block_q, dtype, text tokens, B, H, mode, beta)
    ((6, 10, 150), 128, 128, "bf16", 0, 1, 4, "sparse", 0.7),            # N = 9000, 4 heads
    ((4, 20, 33), 64, 64, "bf16", 512, 1, 2, "sparse_no_correction", 0.4),  # N = 3152, forced text tail
    ((3, 10, 41), 128, 128, "f32", 0, 1, 1, "sparse", 0.5),               # N = 1230, f32 path
    ((5, 13), 128, 128, "bf16", 0, 2, 3, "dense", 0.0),                   # N = 65
]


def _run_pair(dev, case, seed):
    grid, d, bq, dtype, text, B, H, mode, beta = case
    w = small_workload(f"noalloc{seed}", grid, d, bq, dtype=dtype, text_tokens=text, H=H, B=B, seed=seed)
    q, k, v = (t.to(dev) for t in synth.make_qkv(w))
    nkr = w.NK - text // 64
    need = sb.workspace_bytes(B, H, w.N, d, bq, 64, mode, sb.SOL_BF16 if dtype == "bf16" else sb.SOL_F32, text)
    assert 0 < need <= 64 << 20
    outs, counts, masks = [], [], []
    for noalloc in (True, False):
        out = torch.full_like(q, math.nan)
        cnt = torch.full((B, H), -1, dtype=torch.int32, device=dev)
        mask = torch.zeros((B, H, w.NQ, sb.mask_words(nkr)), dtype=torch.int32, device=dev)
        if noalloc:
            sb.forward_noalloc(q, k, v, out, cnt, bq, 64, beta, mode, keep_tail_tokens=text, mask_out=mask)
        else:
            ws = torch.empty(need, dtype=torch.uint8, device=dev)
            sb.forward(q, k, v, bq, 64, beta, mode, keep_tail_tokens=text, out=out, workspace=ws, counts=cnt,
                       mask_out=mask)
        torch.cuda.synchronize()
        outs.append(out)
        counts.append(cnt)
        masks.append(mask)
    assert bool(torch.isfinite(outs[0]).all()), "rows left unwritten"
    assert_output_close(to_np(outs[0]), to_np(outs[1]), dtype, f"noalloc {mode}")
    assert torch.equal(outs[0], outs[1])
    assert torch.equal(counts[0], counts[1])
    assert torch.equal(masks[0], masks[1])
    return w


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    sb.lib()
    return torch.device("cuda:0")


def test_noalloc_matches_workspace_entry_point_two_calls(dev):
    # first a larger input, then a smaller one on the same scratch
    w0 = _run_pair(dev, CASES[0], 71)
    w1 = _run_pair(dev, CASES[1], 72)
    assert w1.B * w1.H * w1.N < w0.B * w0.H * w0.N


def test_noalloc_f32_and_dense_two_calls(dev):
    w0 = _run_pair(dev, CASES[2], 73)
    w1 = _run_pair(dev, CASES[3], 74)
    assert w1.B * w1.H * w1.N < w0.B * w0.H * w0.N


def test_noalloc_rejects_shapes_beyond_the_scratch(dev):
    w = small_workload("noalloc_big", (4, 100, 200), 128, 128, H=8, seed=75)   # 80,000 tokens x 8 heads
    q = torch.zeros((1, 8, w.N, 128), dtype=torch.bfloat16, device=dev)
    out = torch.empty_like(q)
    cnt = torch.zeros((1, 8), dtype=torch.int32, device=dev)
    with pytest.raises(sb.SolAttnError) as ei:
        sb.forward_noalloc(q, q, q, out, cnt, 128, 64, 0.5, "sparse")
    assert ei.value.code == sb.SOL_ERR_WORKSPACE
