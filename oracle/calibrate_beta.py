"""Calibrate the routing cutoff beta of each workload on the CPU oracle.

Bisection on beta until the oracle's kept fraction of routable (query block,
key block) pairs, over all heads, is within 0.25 points of the target.  The
initial bracket is centred on the Gaussian calibration beta = Phi^-1(1 - rho)
(Section 3.1, Gaussian density rho_G(beta) = 1 - Phi(beta)) and widened until it
holds the target.

Each workload is calibrated for its target kept fraction with the exact threshold
statistics (key "<workload>@<kept>") and with the diagonal estimator of the Appendix
(key "<workload>@<kept>/diagonal"); the 720p shape also for the sweep points.

Writes paper_2607_24027_amd/betas.json.  Calls only the oracle and the seeded
input generator.  Run from the repository root:  python -m oracle.calibrate_beta
"""
from __future__ import annotations

import json
import os
import sys
from statistics import NormalDist

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

from oracle import sol_attn_oracle as ora  # noqa: E402
from paper_2607_24027_amd import configs, synth  # noqa: E402


def kept_fraction(r, beta):
    tau = ora.thresholds(r["mu"], r["sigma"], beta)
    return float(ora.route(r["s_hat"], tau).mean())


def proxies(workload, threshold_mode="exact"):
    q, k, _ = synth.make_qkv(workload, workers=synth.default_workers())
    return ora.routing(q.float().numpy(), k.float().numpy(), workload.block_q, workload.block_k,
                       0.0, keep_tail_tokens=workload.text_tokens, threshold_mode=threshold_mode)


def calibrate(r, target, tol=0.0025):
    b0 = NormalDist().inv_cdf(1.0 - target)
    lo, hi = b0 - 2.0, b0 + 2.0
    # widen the bracket until it holds the target (the diagonal estimator's sigma can
    # be far from the proxy rows' spread, and beta with it)
    while kept_fraction(r, hi) > target and hi < 1e3:
        hi = 2.0 * hi + 1.0
    while kept_fraction(r, lo) < target and lo > -1e3:
        lo = 2.0 * lo - 1.0
    for _ in range(60):
        mid = 0.5 * (lo + hi)
        f = kept_fraction(r, mid)
        if abs(f - target) <= tol and hi - lo < 1e-4:
            break
        if f > target:
            lo = mid
        else:
            hi = mid
    beta = round(0.5 * (lo + hi), 6)
    return beta, kept_fraction(r, beta)


def main():
    out = {}
    for w in configs.WORKLOADS.values():
        for tmode in ("exact", "diagonal"):
            r = proxies(w, tmode)
            targets = [w.target_kept]
            if w is configs.VIDEO_720P and tmode == "exact":
                targets += [kp for kp in configs.SWEEP_KEPT if kp < 1.0]
            for kp in sorted(set(targets)):
                beta, f = calibrate(r, kp)
                key = f"{w.name}@{kp:.2f}" + ("" if tmode == "exact" else "/diagonal")
                print(f"{key}: beta={beta:.6f} kept={f:.4f}", flush=True)
                out[key] = beta
            del r
    path = os.path.join(os.path.dirname(configs.__file__), "betas.json")
    with open(path, "w") as fh:
        json.dump(out, fh, indent=1, sort_keys=True)
        fh.write("\n")
    print("wrote", path)


if __name__ == "__main__":
    main()
