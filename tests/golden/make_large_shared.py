"""Write the oracle's marginals of the large shared-model workload for every
agent (tests/golden/large_shared_{vmp,mmp}.npz): F = 4 factors of 32 states,
M = 4 modalities of 32 outcomes on all factors, 90% zeros, b = 64, T = 16,
16 iterations.  Calls only the seeded generator and the fp64 oracle;
stored as float32 (the comparison tolerance is 1e-5).

    python tests/golden/make_large_shared.py
"""
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2607_17855_amd import synth  # noqa: E402


def main():
    w = synth.large_shared()
    for algo in ("vmp", "mmp"):
        t0 = time.time()
        q = oracle.infer(algo, w.model, w.obs, w.act, w.iters)
        path = os.path.join(HERE, f"large_shared_{algo}.npz")
        np.savez_compressed(path, q=q.astype(np.float32), obs=w.obs, act=w.act)
        print(f"{path}: {q.shape}, {time.time() - t0:.0f} s", flush=True)


if __name__ == "__main__":
    main()
