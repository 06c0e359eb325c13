"""Write tests/golden/fit_golden.npz: the fp64 oracle's compact fit after the
full 400 Adam steps, for the targets the GPU test fits -- two heads at
T = 1024 (``fit_target_means(2, 1024, stream_id=43)``) and head 0 of the
benchmarked 12-head layer at T = 4096 (``fit_target_means(1, 4096,
stream_id=44)``, whose single head is that layer's head 0).

Per head it stores the oracle's fitted pattern in gauge-free form: the row
normalisers log Z, the pattern's column sums and diagonal sums, a few whole
rows of the pattern, and the acceptance KL (plus the fitted alpha and rho,
whose gauge is not unique).  Calls only ``oracle.fit_oracle`` and the seeded
generator; about ten minutes of CPU (the T = 4096 fit is dense float64).

Usage: ``python tests/golden/make_fit_golden.py``.
"""

import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import fit_oracle as fo  # noqa: E402
from paper_2609_34650_amd import inputs  # noqa: E402

CASES = {"t1024": (2, 1024, 43), "t4096": (1, 4096, 44)}


def sample_rows(T):
    return np.array(sorted({0, 1, 2, 100, T // 2, T - 2, T - 1}))


def main():
    out = {}
    for name, (H, T, sid) in CASES.items():
        mean = inputs.fit_target_means(H, T, stream_id=sid)
        for h in range(H):
            t = fo.fit_targets(mean[h].astype(np.float64))
            a, r = fo.fit(t["eta_abs"], t["eta_rel"])
            kl = fo.fit_kl(a, r, t["eta_abs"], t["eta_rel"], t["neg_entropy"])
            _, _, _, logz = fo.fit_objective(a, r, t["eta_abs"], t["eta_rel"])
            P = np.exp(fo.compact_logits(a, r) - logz[:, None])
            rows = sample_rows(T)
            key = f"{name}_h{h}"
            out[key + "_a"] = a
            out[key + "_r"] = r
            out[key + "_logz"] = logz
            out[key + "_kl"] = np.float64(kl)
            out[key + "_col"] = P.sum(axis=0)
            out[key + "_diag"] = np.array([np.trace(P, offset=-d) for d in range(T)])
            out[key + "_rows"] = rows
            out[key + "_P_rows"] = P[rows]
            print(key, "kl", kl, flush=True)
    np.savez_compressed(os.path.join(HERE, "fit_golden.npz"), **out)


if __name__ == "__main__":
    main()
