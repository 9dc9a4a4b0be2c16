"""The large shared-model workload (F = 4 x 32 states, M = 4 x 32 outcomes on
all factors, 90% zeros, b = 64, T = 16, 16 iterations) on every layout and
precision class the benchmark runs, all 64 agents against the oracle's
marginals stored by tests/golden/make_large_shared.py (fp64 oracle, stored as
float32), 1e-5 max-abs."""
import functools
import os

import numpy as np
import pytest

from paper_2607_17855_amd import bi, synth

pytestmark = pytest.mark.gpu
TOL = 1e-5
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

PACKINGS = {
    "dense_f16_pairs": (bi.BI_DENSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS, "stream"),
    "sparse_f16_pairs": (bi.BI_SPARSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS, "sparse"),
    "dense_f32": (bi.BI_DENSE_A | bi.BI_FAST_F32, "stream"),
    "sparse_f64": (bi.BI_SPARSE_A, "sparse"),
}


@functools.lru_cache(maxsize=None)
def _workload():
    return synth.large_shared()


@functools.lru_cache(maxsize=None)
def _golden(algo):
    with np.load(os.path.join(GOLDEN, f"large_shared_{algo}.npz")) as z:
        return z["q"].astype(np.float64), z["obs"], z["act"]


@pytest.mark.parametrize("packing", sorted(PACKINGS))
def test_large_shared_all_agents(packing):
    import torch
    w = _workload()
    flags, family = PACKINGS[packing]
    print(f"[gpu] large shared model, {packing}: packing", flush=True)
    pm = bi.PackedModel(w.model, flags=flags, device="cuda")
    obs = torch.from_numpy(w.obs).cuda()
    act = torch.from_numpy(w.act).cuda()
    for algo in ("vmp", "mmp"):
        ref, gobs, gact = _golden(algo)
        assert np.array_equal(gobs, w.obs) and np.array_equal(gact, w.act), "generator differs from the golden inputs"
        assert pm.path(w.b, w.T, algo) == family
        print(f"[gpu]   {packing} {algo} ({family} kernels), 64 agents", flush=True)
        q = pm.infer(algo, obs, act, w.iters)
        torch.cuda.synchronize()
        q = q.cpu().numpy()
        err = np.abs(q - ref).max(axis=(1, 2))
        print(f"[gpu]     max|gpu - oracle| = {err.max():.2e} (worst agent {int(err.argmax())})", flush=True)
        assert err.max() <= TOL
    pm.close()
