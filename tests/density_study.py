"""Density control of threshold routing against top-k and top-p (CPU, fp64 oracle).

Section 3.1 ties the standardised cutoff beta to the Gaussian reference density
rho_G(beta) = 1 - Phi(beta) and argues that threshold routing keeps a query-dependent
budget with a stable density, unlike top-k (fixed count) and top-p (cumulative mass,
from one block up to ceil(pN)).  On the synthetic workloads this script reports:

  * the mean kept fraction of threshold routing against rho_G(beta) over a range of beta;
  * at a common mean density (15 %), the distribution of per-query-block densities
    (p10 / p25 / median / p75 / p90) for threshold routing (beta calibrated), top-k
    (k = round(0.15 * NK_routable)) and top-p (p calibrated; mass = Softmax(s_hat_i) as in
    Eq. block_proxy), both through the oracle's route_topk / route_topp.

    python tests/density_study.py [workload ...]
"""
from __future__ import annotations

import json
import os
import sys
from statistics import NormalDist

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

TARGET = 0.15


def bisect(f, lo, hi, target, iters=60):
    """f decreasing in its argument; returns x with f(x) ~= target."""
    for _ in range(iters):
        mid = 0.5 * (lo + hi)
        if f(mid) > target:
            lo = mid
        else:
            hi = mid
    return 0.5 * (lo + hi)


def pcts(x):
    return {k: float(v) for k, v in zip(("p10", "p25", "median", "p75", "p90"), np.percentile(x, [10, 25, 50, 75, 90]))}


def main():
    from oracle import sol_attn_oracle as ora
    from paper_2607_24027_amd import configs, synth

    names = sys.argv[1:] or ["video480p", "video720p", "image"]
    for name in names:
        w = configs.WORKLOADS[name]
        q, k, _ = synth.make_qkv(w, workers=synth.default_workers())
        r = ora.routing(q.float().numpy(), k.float().numpy(), w.block_q, w.block_k, 0.0,
                        keep_tail_tokens=w.text_tokens)
        s_hat, mu, sigma = r["s_hat"], r["mu"], r["sigma"]        # [B,H,NQ,NKr]
        nkr = s_hat.shape[-1]

        def kept(beta):
            return float(ora.route(s_hat, ora.thresholds(mu, sigma, beta)).mean())

        gauss = [{"beta": b, "rho_G": 1.0 - NormalDist().cdf(b), "kept": kept(b)}
                 for b in (-0.5, 0.0, 0.5, 1.0, 1.5, 2.0)]

        # threshold routing at the common density
        beta = bisect(kept, -5.0, 10.0, TARGET)
        dens_thr = ora.route(s_hat, ora.thresholds(mu, sigma, beta)).mean(axis=-1).ravel()
        # top-k: a fixed count per query block
        kk = int(round(TARGET * nkr))
        dens_topk = ora.route_topk(s_hat, kk).mean(axis=-1).ravel()
        # top-p: p is calibrated on the sorted cumulative mass (computed once), then the
        # densities are taken from the oracle's route_topp at that p
        order = np.argsort(-s_hat, axis=-1, kind="stable")
        srt = np.take_along_axis(s_hat, order, axis=-1)
        prob = np.exp(srt - srt[..., :1])
        prob /= prob.sum(axis=-1, keepdims=True)
        before = np.cumsum(prob, axis=-1) - prob

        def topp_counts(p):
            return (before < p).sum(axis=-1)

        p = bisect(lambda pp: -float(topp_counts(pp).mean() / nkr), 0.0, 1.0, -TARGET)
        dens_topp = ora.route_topp(s_hat, p).mean(axis=-1).ravel()
        rec = {"workload": name, "nk_routable": nkr, "gaussian_reference": gauss,
               "common_density": TARGET,
               "threshold": {"beta": beta, "mean": float(dens_thr.mean()), **pcts(dens_thr)},
               "top_k": {"k": kk, "mean": float(dens_topk.mean()), **pcts(dens_topk)},
               "top_p": {"p": p, "mean": float(dens_topp.mean()), **pcts(dens_topp),
                         "min": float(dens_topp.min()), "max": float(dens_topp.max())}}
        print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
