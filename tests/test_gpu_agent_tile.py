"""Tile form of the agent kernels' Z/V phase (slices read from global memory):
shapes chosen to reach each of its cases, against the oracle, with the
library's profile showing that the tile form ran.

  - a row side longer than one block of 12 rows (20, 15 and 16 rows), with
    one and with two row factors (block boundaries inside the second factor);
  - several 32-column chunks per context (42 columns) and a ragged last chunk;
  - an odd column count (the pair's second column is the padding column);
  - a rank-0 row side (V only) and two column factors;
  - soft observations (the per-context log-likelihood tensors);
  - a window longer than one context chunk of the Z/V scratch (T = 100);
  - FPI on steps whose slices exceed one step's LDS staging, with a slice of
    598 rows taking one dot product per thread beside tiled ones.
"""
import numpy as np
import pytest

from paper_2607_17855_amd import bi, synth
import oracle
from test_gpu_parity import check_invariants

pytestmark = pytest.mark.gpu
TOL = 1e-5

CASES = [
    # (n, U, K, deps, b, T, per_agent): the slices of one context exceed what
    # the window's LDS staging takes, so the window kernel reads them from
    # global memory
    ([20, 6, 7], [2, 1, 3], [5, 3, 4], [[0, 1, 2], [1], [0, 2]], 6, 12, True),
    ([3, 5, 4, 6], [1, 2, 2, 1], [4, 3], [[0, 1, 2, 3], [2, 3]], 5, 30, True),
    ([4, 4, 30], [2, 2, 1], [6], [[0, 1, 2]], 4, 20, False),
    ([20, 6, 7], [2, 1, 3], [5, 3, 4], [[0, 1, 2], [1], [0, 2]], 3, 100, True),
]


def _torch():
    import torch
    return torch


def _workload(case, iters):
    n, U, K, deps, b, T, per_agent = CASES[case]
    rng = np.random.Generator(np.random.PCG64(1300 + case))
    model = synth.make_model(rng, n, U, K, deps, b if per_agent else 1, 0.7, 1.0, uniform_D=False)
    obs, act = synth.sample_sequences(rng, model, b, T)
    return synth.Workload(f"tile{case}", ["vmp", "mmp"], model, obs, act, iters)


def _dev(x):
    return _torch().from_numpy(np.ascontiguousarray(x)).cuda()


@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("algo", ["vmp", "mmp"])
def test_tile_vs_oracle(case, algo):
    torch = _torch()
    w = _workload(case, 16 if case == 0 else 3)
    print(f"[gpu] {w.name} {algo} b={w.b} T={w.T} iters={w.iters}", flush=True)
    pm = bi.PackedModel(w.model, bi.BI_DENSE_A)
    try:
        assert pm.path(w.b, w.T, algo) == "agent"
        bi.bi_profile_begin()
        q = pm.infer(algo, _dev(w.obs), _dev(w.act), w.iters)
        torch.cuda.synchronize()
        names = set(bi.bi_profile_end())
        assert "agent_window_tile" in names, names
        q = q.cpu().numpy()
        check_invariants(w, q)
        ref = oracle.infer(algo, w.model, w.obs, w.act, w.iters)
        err = float(np.abs(q - ref).max())
        print(f"[gpu]   tile vs oracle {err:.3e}", flush=True)
        assert err <= TOL
        # fixed summation order: the same call gives the same bits
        q2 = pm.infer(algo, _dev(w.obs), _dev(w.act), w.iters)
        torch.cuda.synchronize()
        assert np.array_equal(q, q2.cpu().numpy())
    finally:
        pm.close()


# FPI reads a step's slices from global memory when they exceed what one
# step's LDS staging takes: the tile form then serves the modalities of at
# most 96 rows, one dot product per thread the taller ones (mixed).
FPI_CASES = [
    # (n, K, deps, b, T): every modality tiled (a 30 x 700 slice)
    ([30, 25, 28], [3, 4], [[0, 1, 2], [2]], 3, 4),
    # a 598 x 31 slice (one dot product per thread) beside tiled ones
    ([23, 26, 31], [3, 4, 5], [[0, 1, 2], [0, 2], [1]], 3, 4),
]


@pytest.mark.parametrize("case", range(len(FPI_CASES)))
@pytest.mark.parametrize("algo", ["fpi", "vmp", "mmp"])
def test_tile_large_slices(case, algo):
    torch = _torch()
    n, K, deps, b, T = FPI_CASES[case]
    rng = np.random.Generator(np.random.PCG64(1360 + case))
    model = synth.make_model(rng, n, [2] * len(n), K, deps, b, 0.7, 1.0, uniform_D=False)
    obs, act = synth.sample_sequences(rng, model, b, T)
    w = synth.Workload(f"tile_large{case}", [algo], model, obs, act, 4)
    print(f"[gpu] {w.name} {algo} b={w.b} T={w.T}", flush=True)
    pm = bi.PackedModel(w.model, bi.BI_DENSE_A)
    try:
        bi.bi_profile_begin()
        q = pm.infer(algo, _dev(w.obs), _dev(w.act), w.iters)
        torch.cuda.synchronize()
        names = set(bi.bi_profile_end())
        assert ("agent_filter_tile" if algo == "fpi" else "agent_window_tile") in names, names
        q = q.cpu().numpy()
        check_invariants(w, q)
        ref = oracle.infer(algo, w.model, w.obs, w.act, w.iters)
        err = float(np.abs(q - ref).max())
        print(f"[gpu]   tile vs oracle {err:.3e}", flush=True)
        assert err <= TOL
    finally:
        pm.close()


@pytest.mark.parametrize("algo", ["vmp", "mmp"])
def test_tile_soft_observations(algo):
    torch = _torch()
    w = _workload(0, 3)
    so = synth.soft_obs(np.random.Generator(np.random.PCG64(1350)), w.obs, w.model.K, confidence=0.5)
    print(f"[gpu] {w.name} soft {algo} b={w.b} T={w.T}", flush=True)
    pm = bi.PackedModel(w.model, bi.BI_DENSE_A)
    try:
        bi.bi_profile_begin()
        q = pm.infer_soft(algo, _dev(so), _dev(w.act), w.iters)
        torch.cuda.synchronize()
        names = set(bi.bi_profile_end())
        assert "agent_window_tile" in names, names
        q = q.cpu().numpy()
        check_invariants(w, q)
        ref = oracle.infer_soft(algo, w.model, so.astype(np.float64), w.act, w.iters)
        err = float(np.abs(q - ref).max())
        print(f"[gpu]   tile soft vs oracle {err:.3e}", flush=True)
        assert err <= TOL
        # one-hot vectors reproduce the integer call bit for bit
        qs = pm.infer_soft(algo, _dev(synth.one_hot_obs(w.obs, w.model.K)), _dev(w.act), w.iters)
        qi = pm.infer(algo, _dev(w.obs), _dev(w.act), w.iters)
        torch.cuda.synchronize()
        assert np.array_equal(qs.cpu().numpy(), qi.cpu().numpy())
    finally:
        pm.close()
