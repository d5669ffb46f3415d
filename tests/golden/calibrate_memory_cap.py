"""Capacity of the tight-memory workload (8 tenants, 10,000 ops, 64 devices).

The workload's resident footprint is drawn so that about 30% of uniform random
placements exceed device capacity: the capacity is the nearest-rank 70th
percentile of max_d peak[d] over 4,096 uniform random placements drawn from
the workload's own calibration stream.  This script computes it with the
oracle only and prints the constant that the input generator holds
(TIGHT_CAP_BYTES); tests/test_synth.py re-runs it and checks the two agree.
"""
import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))

import oracle  # noqa: E402
from paper_2608_15762_amd import synth  # noqa: E402

CID = 3
N_SAMPLES = 4096


def compute(n_samples: int = N_SAMPLES, n_threads: int = 8) -> int:
    g = synth.build_gmg(CID)
    P = synth.uniform_placements(g, synth.calibration_key(CID), 0, n_samples)
    out = oracle.simulate_batch(oracle.OracleGmg(g), P, n_threads=n_threads)
    worst = np.sort(out["peak"].max(axis=1))
    rank = -(-70 * n_samples // 100)  # nearest rank: ceil(0.7 n)
    return int(worst[rank - 1])


if __name__ == "__main__":
    print(compute())
