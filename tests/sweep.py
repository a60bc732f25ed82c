"""Routing-cutoff sweep on the 720p video shape (B=1, H=40, N=75,600, d=128, bf16).

For each kept fraction in configs.SWEEP_KEPT (cutoffs calibrated on the fp64 oracle's
routing): the selected fraction the library reports, the fused kernel and whole-forward
times of the sparse and no-correction modes, the speedup over the library's dense mode, and
the approximation error of both modes against exact dense attention (the fp64 oracle) on a
sample of query blocks, together with the parity of the sparse output against the oracle run
with the library's own mask once that mask has been checked against the oracle's routing
(bit-exact outside the 1e-3 band around tau_i).

    python tests/sweep.py [--steps 10] [--warmup 3] [--out FILE]
    python tests/sweep.py --launch-once    # one launch per (kept, mode), for counter runs

Run on a GPU; prints one JSON object per kept fraction.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

SAMPLE_HEADS = (0, 17, 39)
SAMPLE_BLOCKS = (0, 150, 301, 450, 590)   # 590 is the ragged last query block


def rel_l2(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def cosine(a, b):
    return float((a * b).sum() / (np.linalg.norm(a) * np.linalg.norm(b)))


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--launch-once", action="store_true")
    ap.add_argument("--no-error", action="store_true")
    ap.add_argument("--out", default=None)
    args = ap.parse_args()

    import torch
    from oracle import sol_attn_oracle as ora
    from paper_2607_24027_amd import binding, configs, synth
    from bench import time_steps
    from tests.parity import assert_mask_matches, errors

    binding.lib()
    w = configs.WORKLOADS["video720p"]
    q, k, v = synth.make_qkv(w, workers=synth.default_workers())
    qd, kd, vd = (x.cuda() for x in (q, k, v))
    out = torch.empty_like(qd)
    nkr = w.NK

    def run(mode, beta, o=None, mask=None):
        return binding.forward(qd, kd, vd, w.block_q, w.block_k, beta, mode, 0, out=out if o is None else o,
                               mask_out=mask)

    if args.launch_once:
        order = []
        for kept in configs.SWEEP_KEPT:
            beta = configs.beta_for(w, kept)
            for mode in ("sparse", "sparse_no_correction"):
                run(mode, beta)
                torch.cuda.synchronize()
                order.append({"kept": kept, "mode": mode, "frac": float(np.mean(binding.stats(w.B, w.H)))})
        run("dense", 0.0)
        torch.cuda.synchronize()
        order.append({"kept": 1.0, "mode": "dense"})
        print(json.dumps({"launch_order": order}), flush=True)
        return

    dense = time_steps(lambda: run("dense", 0.0), args.steps, args.warmup)
    print(json.dumps({"dense_ms": dense}), flush=True)

    # fp64 exact attention on the sample rows (shared by every cutoff)
    sample = {}
    if not args.no_error:
        for h in SAMPLE_HEADS:
            qs, ks, vs = (x[0:1, h:h + 1].float().numpy().astype(np.float64) for x in (q, k, v))
            ref = ora.forward(qs, ks, vs, w.block_q, w.block_k, 0.0, "dense", query_blocks=list(SAMPLE_BLOCKS))
            sample[h] = (qs, ks, vs, ref["out"][0, 0])
    rows = np.concatenate([np.arange(i * w.block_q, min((i + 1) * w.block_q, w.N)) for i in SAMPLE_BLOCKS])
    # the oracle's proxies and row statistics: its routing at any cutoff is route(s_hat, mu + beta sigma)
    routing = ora.routing(q.float().numpy(), k.float().numpy(), w.block_q, w.block_k, 0.0)

    results = []
    for kept in configs.SWEEP_KEPT:
        beta = configs.beta_for(w, kept)
        mask = torch.zeros((w.B, w.H, w.NQ, binding.mask_words(nkr)), dtype=torch.int32, device="cuda")
        o_sp = torch.empty_like(qd)
        o_nc = torch.empty_like(qd)
        run("sparse", beta, o_sp, mask)
        run("sparse_no_correction", beta, o_nc)
        torch.cuda.synchronize()
        frac = np.array(binding.stats(w.B, w.H))
        gmask = binding.unpack_mask(mask.cpu().numpy().view(np.uint32), nkr)
        tau = ora.thresholds(routing["mu"], routing["sigma"], beta)
        flips = assert_mask_matches(gmask, ora.route(routing["s_hat"], tau), routing["s_hat"], tau)
        sp = time_steps(lambda: run("sparse", beta), args.steps, args.warmup)
        nc = time_steps(lambda: run("sparse_no_correction", beta), args.steps, args.warmup)
        rec = {"kept_target": kept, "beta": beta, "selected_fraction": {
                   "mean": float(frac.mean()), "min": float(frac.min()), "max": float(frac.max())},
               "sparse_ms": sp, "no_correction_ms": nc,
               "speedup_step": round(dense["mean"] / sp["mean"], 4),
               "speedup_kernel": round(dense["kernel"] / sp["kernel"], 4),
               "speedup_no_correction_kernel": round(dense["kernel"] / nc["kernel"], 4),
               "target_speedup": round(0.8 / max(float(frac.mean()), 1e-9), 4),
               "mask_in_band_flips": flips}
        if sample:
            e_sp, e_nc, cos_sp, cos_nc, parity = [], [], [], [], []
            for h, (qs, ks, vs, ref_dense) in sample.items():
                g_sp = o_sp[0, h].float().cpu().numpy().astype(np.float64)[rows]
                g_nc = o_nc[0, h].float().cpu().numpy().astype(np.float64)[rows]
                rd = ref_dense[rows]
                e_sp.append(rel_l2(g_sp, rd))
                e_nc.append(rel_l2(g_nc, rd))
                cos_sp.append(cosine(g_sp, rd))
                cos_nc.append(cosine(g_nc, rd))
                ref_sp = ora.forward(qs, ks, vs, w.block_q, w.block_k, beta, "sparse", query_blocks=list(SAMPLE_BLOCKS),
                                     mask=gmask[0:1, h:h + 1])["out"][0, 0][rows]
                parity.append(errors(g_sp, ref_sp))
            rec["error_vs_dense"] = {"heads": list(SAMPLE_HEADS), "query_blocks": list(SAMPLE_BLOCKS),
                                     "rel_l2_sparse": float(np.mean(e_sp)), "rel_l2_no_correction": float(np.mean(e_nc)),
                                     "cos_sparse": float(np.mean(cos_sp)), "cos_no_correction": float(np.mean(cos_nc)),
                                     "parity_max_abs_vs_oracle": max(p[0] for p in parity),
                                     "parity_mean_rel_vs_oracle": max(p[1] for p in parity)}
        results.append(rec)
        print(json.dumps(rec), flush=True)
    if args.out:
        with open(args.out, "w") as f:
            json.dump({"dense_ms": dense, "sweep": results}, f, indent=1)


if __name__ == "__main__":
    main()
