"""Routed attention under causal masks at the 720p video shape (B=1, H=40, N=75600, d=128,
bf16): frame-causal (G = 3600, one 45 x 80 frame, autoregressive video) and token-causal
(G = 1).  For each granule: the dense causal kernel, then sparse and sparse-without-correction
at the cutoff calibrated for 20 % kept on the bidirectional shape (the kept fraction of the
routable pairs is reported).

    python tests/causal_bench.py [--steps K] [--warmup W] [--granule G ...]

Per mode: mean step time and fused-kernel time (HIP events), speedup over the dense causal
kernel, and the MFMA rate of the tiles the kernel computes: 4 d x 64 x (rows of the query
block) flops per exact or correction tile, masked parts of partially visible tiles included.
The dense-equivalent work is 4 d x (visible (query, key) pairs).  One JSON line per granule.
"""
from __future__ import annotations

import argparse
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

MFMA_PEAK_TFLOPS = 2500.0


def causal_ranges(n, bq, bk, g):
    """(r_i, e_i) per query block: key blocks [0, r_i) visible to all rows, [r_i, e_i) to some."""
    nq, nk = -(-n // bq), -(-n // bk)
    r = np.empty(nq, dtype=np.int64)
    e = np.empty(nq, dtype=np.int64)
    for i in range(nq):
        lo = min((i * bq // g + 1) * g, n)
        hi = min(((min((i + 1) * bq, n) - 1) // g + 1) * g, n)
        r[i] = nk if lo >= n else lo // bk
        e[i] = -(-hi // bk)
    return r, e


def visible_pairs(n, g):
    t = np.arange(n, dtype=np.int64)
    return int(np.minimum((t // g + 1) * g, n).sum())


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--granule", type=int, nargs="*", default=[3600, 1])
    args = ap.parse_args()

    import torch
    from bench import time_steps
    from paper_2607_24027_amd import binding as sb
    from paper_2607_24027_amd import configs, synth

    sb.lib()
    w = configs.WORKLOADS["video720p"]
    beta = configs.beta_for(w, 0.20)
    print(f"[causal_bench] {w.name} N={w.N} H={w.H}", file=sys.stderr, flush=True)
    q, k, v = synth.make_qkv(w, workers=synth.default_workers())
    qd, kd, vd = (x.cuda() for x in (q, k, v))
    out = torch.empty_like(qd)
    nq_rows = np.full(w.NQ, w.block_q, dtype=np.float64)
    nq_rows[-1] = w.N - (w.NQ - 1) * w.block_q
    tile_flop = 4.0 * w.d * 64 * nq_rows          # one 64-key tile for each query block

    for g in args.granule:
        r, e = causal_ranges(w.N, w.block_q, w.block_k, g)
        dense_equiv = 4.0 * w.d * visible_pairs(w.N, g) * w.B * w.H
        rec = {"workload": w.name, "granule": g, "beta": beta, "routable_pairs_per_head": int(r.sum()),
               "partial_blocks_per_head": int((e - r).sum()), "dense_equiv_flop": dense_equiv}

        def run(mode, mask=None):
            return sb.forward(qd, kd, vd, w.block_q, w.block_k, beta, mode, out=out, mask_out=mask,
                              causal_granule=g)

        dn = time_steps(lambda: run("dense"), args.steps, args.warmup)
        dense_tiles = float((e * tile_flop).sum()) * w.B * w.H
        rec["dense"] = {**dn, "mfma_tflops": dense_tiles / (dn["kernel"] * 1e9)}
        mask = torch.zeros((w.B, w.H, w.NQ, sb.mask_words(w.NK)), dtype=torch.int32, device="cuda")
        run("sparse", mask)
        torch.cuda.synchronize()
        sel = sb.unpack_mask(mask.cpu().numpy().view(np.uint32), w.NK)      # [B,H,NQ,NK]
        nsel = sel.sum(axis=-1).astype(np.float64)                          # [B,H,NQ]
        nuns = r[None, None, :] - nsel
        exact_tiles = float(((nsel + (e - r)[None, None, :]) * tile_flop).sum())
        corr_tiles = float((np.ceil(nuns / 64.0) * tile_flop).sum())
        rec["kept_of_routable"] = float(nsel.sum() / (r.sum() * w.B * w.H))
        for mode in ("sparse", "sparse_no_correction"):
            t = time_steps(lambda: run(mode), args.steps, args.warmup)
            flop = exact_tiles + (corr_tiles if mode == "sparse" else 0.0)
            rec[mode] = {**t, "speedup_kernel": dn["kernel"] / t["kernel"], "speedup_step": dn["mean"] / t["mean"],
                         "mfma_tflops": flop / (t["kernel"] * 1e9),
                         "dense_equiv_tflops": dense_equiv / (t["mean"] * 1e9)}
        rec["target_speedup"] = 0.8 / max(rec["kept_of_routable"], 1e-9)
        rec["mfma_peak_tflops"] = MFMA_PEAK_TFLOPS
        print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
