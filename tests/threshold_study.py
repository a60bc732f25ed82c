"""Exact against diagonal threshold statistics on the synthetic workloads (CPU, fp64 oracle).

For each workload: the kept fraction of the diagonal estimator (Appendix, Eq.
appendix_diagonal_threshold) at the exact estimator's calibrated cutoff, and, at
equal density (each estimator at its own calibrated cutoff), the agreement of the two
masks (Jaccard of the selected sets) and the spread of the per-query-block densities.

    python tests/threshold_study.py [workload ...]
"""
from __future__ import annotations

import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def main():
    from oracle import sol_attn_oracle as ora
    from paper_2607_24027_amd import configs, synth

    names = sys.argv[1:] or ["video480p", "video720p", "image"]
    for name in names:
        w = configs.WORKLOADS[name]
        q, k, _ = synth.make_qkv(w, workers=synth.default_workers())
        qn, kn = q.float().numpy(), k.float().numpy()
        b_ex = configs.beta_for(w)
        b_dg = configs.beta_for(w, threshold_mode="diagonal")
        ex = ora.routing(qn, kn, w.block_q, w.block_k, b_ex, keep_tail_tokens=w.text_tokens)
        dg_same = ora.routing(qn, kn, w.block_q, w.block_k, b_ex, keep_tail_tokens=w.text_tokens,
                              threshold_mode="diagonal")
        dg = ora.routing(qn, kn, w.block_q, w.block_k, b_dg, keep_tail_tokens=w.text_tokens,
                         threshold_mode="diagonal")
        m_ex, m_dg = ex["mask"], dg["mask"]
        jac = float((m_ex & m_dg).sum() / max((m_ex | m_dg).sum(), 1))
        sig_ratio = dg["sigma"] / np.maximum(ex["sigma"], 1e-30)
        dens_ex = m_ex.mean(axis=-1).ravel()
        dens_dg = m_dg.mean(axis=-1).ravel()
        rec = {"workload": name, "beta_exact": b_ex, "beta_diagonal": b_dg,
               "kept_exact": float(m_ex.mean()),
               "kept_diagonal_at_exact_beta": float(dg_same["mask"].mean()),
               "kept_diagonal_at_own_beta": float(m_dg.mean()),
               "sigma_diag_over_exact": {"median": float(np.median(sig_ratio)), "p10": float(np.percentile(sig_ratio, 10)),
                                         "p90": float(np.percentile(sig_ratio, 90))},
               "jaccard_equal_density": jac,
               "pair_agreement_equal_density": float((m_ex == m_dg).mean()),
               "query_block_density_std": {"exact": float(dens_ex.std()), "diagonal": float(dens_dg.std())}}
        print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
