"""Routing latency at the 720p video shape (B=1, H=40, N=75600, d=128, bf16): threshold
routing against top-k and top-p routing over a materialised proxy map (the comparison in
the kernel-efficiency evaluation, Fig. routing_latency).

Stages timed (median over `reps` launches, CUDA events on the current stream, inputs
resident in HBM):
  pool        block means Q̄, K̄, V̄ of q, k, v (common to every routing scheme)
  thresholds  pooled-key moments and tau_i = mu_i + beta*sigma_i (Eq. threshold_stats_exact):
              the only routing work outside the fused attention kernel.  Its entry point
              allocates and synchronises, so its kernels are timed by rocprofv3 only
              (moments_partial_block, moments_final_kernel, tau_kernel); it is called here so
              that they appear in the trace.
  fused_route the fused kernel in sparse_no_correction mode at beta = +inf: every key block is
              routed and listed on chip, no tile is computed.  An upper bound of the in-kernel
              routing cost, since it also reads Q and writes O.
  topk, topp  proxy map s_hat = s Q̄ K̄^T written to HBM, then a top-k (radix select) or top-p
              (sort + cumulative mass) pass over every row, producing a key-block mask.

k and p are chosen for about 15 % kept (the figure's operating density is not stated in the
paper; Fig. density_distribution compares the schemes at 15 %).  One JSON line on stdout.
For per-kernel times run it under  rocprofv3 --kernel-trace --stats.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def _median_ms(fn, reps):
    import torch
    times = []
    for _ in range(reps):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        fn()
        b.record()
        b.synchronize()
        times.append(a.elapsed_time(b))
    times.sort()
    return times[len(times) // 2]


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--reps", type=int, default=20)
    ap.add_argument("--kept", type=float, default=0.15)
    ap.add_argument("--top-p", type=float, default=0.30)
    args = ap.parse_args(argv)

    import numpy as np
    import torch
    from paper_2607_24027_amd import binding as sb
    from paper_2607_24027_amd import configs, synth

    sb.lib()
    w = configs.WORKLOADS["video720p"]
    print(f"routing_latency: {w.name} B={w.B} H={w.H} N={w.N} d={w.d}", file=sys.stderr, flush=True)
    q, k, v = synth.make_qkv(w, workers=synth.default_workers())
    q, k, v = (x.cuda() for x in (q, k, v))
    out = torch.empty_like(q)
    kk = int(round(args.kept * w.NK))
    beta = configs.beta_for(w, 0.20)
    st = {}

    qbar, kbar, _ = sb.pool_blocks(q, k, v, w.block_q, w.block_k)
    prox, mask = sb.route_materialized(qbar, kbar, "topk", kk)
    stages = {
        "pool": lambda: sb.pool_blocks(q, k, v, w.block_q, w.block_k),
        "fused_route": lambda: sb.forward(q, k, v, w.block_q, w.block_k, math.inf, "sparse_no_correction",
                                          out=out),
        "topk": lambda: sb.route_materialized(qbar, kbar, "topk", kk, proxies=prox, mask_out=mask),
        "topp": lambda: sb.route_materialized(qbar, kbar, "topp", args.top_p, proxies=prox, mask_out=mask),
    }
    for _ in range(args.reps):
        sb.thresholds(qbar, kbar, beta)
    for name, fn in stages.items():
        fn()
        torch.cuda.synchronize()
        st[name] = round(_median_ms(fn, args.reps), 4)
        print(f"  {name}: {st[name]} ms", file=sys.stderr, flush=True)

    sb.timing_enable(True)
    sb.kernel_timing()
    for _ in range(args.reps):
        stages["fused_route"]()
    torch.cuda.synchronize()
    ms, n = sb.kernel_timing()
    sb.timing_enable(False)
    st["fused_route_kernel"] = round(ms / max(n, 1), 4)

    _, mk = sb.route_materialized(qbar, kbar, "topk", kk, proxies=prox)
    kept_k = float(sb.unpack_mask(mk.cpu().numpy().view(np.uint32), w.NK).mean())
    _, mp = sb.route_materialized(qbar, kbar, "topp", args.top_p, proxies=prox)
    kept_p = float(sb.unpack_mask(mp.cpu().numpy().view(np.uint32), w.NK).mean())
    res = {
        "workload": w.name, "reps": args.reps, "median_ms": st,
        "topk_k": kk, "topk_kept": round(kept_k, 4), "topp_p": args.top_p, "topp_kept": round(kept_p, 4),
        "proxy_map_bytes": int(prox.numel() * 4),
        "threshold_state_bytes": int(w.B * w.H * (w.d * w.d + w.d + 3 * w.NQ) * 4),
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
