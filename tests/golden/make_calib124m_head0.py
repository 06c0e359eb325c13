"""Write tests/golden/calib124m_4k_head0.npz: the fp64 oracle's calibration
statistics for head 0 of the 124M-style calibration workload (32 inputs,
T = 4096, d = 64, bf16-rounded inputs from the seeded generator), all rows.

Calls only ``oracle.calib_oracle`` and the seeded input generator; the GPU
test ``test_calib_full_size_no_m2`` compares the benchmarked accumulation path
(no per-entry squared deviations) with these values.  About a minute of CPU.

Usage: ``python tests/golden/make_calib124m_head0.py``.
"""

import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import calib_oracle as co  # noqa: E402
from paper_2609_34650_amd import inputs  # noqa: E402

ROWS = np.array([0, 1, 127, 128, 2049, 4000, 4095])


def main():
    w = inputs.CALIB_WORKLOADS["calib124m_4k"]
    inp = inputs.calib_inputs(w.n_cal, w.H, w.T, w.d, w.dtype, stream_id=w.stream_id)
    o = co.calibration_stats(inp["Q"][:, :1], inp["K"][:, :1])
    np.savez_compressed(os.path.join(HERE, "calib124m_4k_head0.npz"),
                        rows=ROWS, A_mean_rows=o["A_mean"][0, ROWS], s_var=o["s_var"][0], s_kl=o["s_kl"][0],
                        eta_abs=o["eta_abs"][0], eta_rel=o["eta_rel"][0])


if __name__ == "__main__":
    main()
