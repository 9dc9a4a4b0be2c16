"""Soft observations on the GPU (bi_infer_soft): the expected log-likelihood
tensors of every context, then the agent-resident iterations, against the
oracle; one-hot vectors against the integer-outcome call."""
import numpy as np
import pytest

from paper_2607_17855_amd import bi, synth
import oracle
from test_gpu_parity import check_invariants

pytestmark = pytest.mark.gpu
TOL = 1e-5


def _torch():
    import torch
    return torch


def _dev(x):
    return _torch().from_numpy(np.ascontiguousarray(x)).cuda()


def _soft(seed, w, confidence=0.6, p_hard=0.2):
    rng = np.random.Generator(np.random.PCG64(seed))
    return synth.soft_obs(rng, w.obs, w.model.K, confidence=confidence, p_hard=p_hard)


def _run_soft(pm, w, algo, so, prior=None, damping=1.0):
    torch = _torch()
    print(f"[gpu] {w.name} soft {algo} b={w.b} T={w.T} iters={w.iters} flags={pm.flags} damping={damping} "
          f"prior={prior is not None}", flush=True)
    q = pm.infer_soft(algo, _dev(so), _dev(w.act), w.iters, prior=None if prior is None else _dev(prior),
                      damping=damping)
    torch.cuda.synchronize()
    return q.cpu().numpy()


def _check_vs_oracle(w, so, algos, flags=bi.BI_DENSE_A, agents=None):
    pm = bi.PackedModel(w.model, flags)
    try:
        for algo in algos:
            q = _run_soft(pm, w, algo, so)
            check_invariants(w, q)
            ref = oracle.infer_soft(algo, w.model, so.astype(np.float64), w.act, w.iters, agents=agents)
            got = q if agents is None else q[list(agents)]
            err = float(np.abs(got - ref).max())
            print(f"[gpu]   soft {algo} vs oracle {err:.3e}", flush=True)
            assert err <= TOL
    finally:
        pm.close()


@pytest.mark.parametrize("seed", range(6))
def test_soft_small_vs_oracle(seed):
    w = synth.random_small(440 + seed, F_max=4, n_max=6, M_max=4, K_max=5, T_max=6, b=5,
                           per_agent=bool(seed % 2))
    _check_vs_oracle(w, _soft(840 + seed, w), ("fpi", "vmp", "mmp"))


@pytest.mark.parametrize("seed", range(3))
def test_soft_one_hot_equals_integer_observations(seed):
    torch = _torch()
    w = synth.random_small(460 + seed, F_max=3, n_max=6, M_max=3, K_max=5, T_max=5, b=4,
                           per_agent=bool(seed % 2))
    pm = bi.PackedModel(w.model)
    try:
        oh = synth.one_hot_obs(w.obs, w.model.K)
        for algo in ("fpi", "vmp", "mmp"):
            qs = _run_soft(pm, w, algo, oh)
            qi = pm.infer(algo, _dev(w.obs), _dev(w.act), w.iters)
            torch.cuda.synchronize()
            # sum_o w[o] X[o] with one weight 1 and the rest 0 is X exactly, and
            # the iterations then run the same code on the same values
            assert np.array_equal(qs, qi.cpu().numpy())
    finally:
        pm.close()


# larger slices: the window no longer fits in LDS (per-step staging, or the
# slices read from the workspace), rank-3 and rank-4 modalities, many steps
LARGE = [
    # (n, U, K, deps, b, T, per_agent)
    ([24, 20, 16], [2, 1, 3], [6, 3], [[0, 1, 2], [1, 2]], 6, 7, True),
    ([10, 9, 8, 7], [1, 2, 1, 2], [4, 3, 5], [[0, 1, 2, 3], [0, 2], [3]], 4, 3, False),
    ([8, 6], [3, 1], [5, 7, 4], [[0, 1]] * 3, 16, 10, True),
]


@pytest.mark.parametrize("case", range(len(LARGE)))
def test_soft_larger_slices_vs_oracle(case):
    n, U, K, deps, b, T, per_agent = LARGE[case]
    rng = np.random.Generator(np.random.PCG64(880 + case))
    model = synth.make_model(rng, n, U, K, deps, b if per_agent else 1, 1.0, 1.0, uniform_D=False)
    obs, act = synth.sample_sequences(rng, model, b, T)
    w = synth.Workload(f"soft_large{case}", ["fpi", "vmp", "mmp"], model, obs, act, 3)
    _check_vs_oracle(w, _soft(900 + case, w, confidence=0.5), ("fpi", "vmp", "mmp"))


def test_soft_with_prior_and_damping():
    w = synth.random_small(480, F_max=3, n_max=5, M_max=3, K_max=4, T_max=5, b=4, per_agent=True)
    so = _soft(920, w)
    prior = synth.random_prior(np.random.Generator(np.random.PCG64(921)), w.model.n, w.b, alpha=0.7, p_zero=0.3)
    pm = bi.PackedModel(w.model)
    try:
        for algo in ("fpi", "vmp", "mmp"):
            q = _run_soft(pm, w, algo, so, prior=prior, damping=0.6)
            ref = oracle.infer_soft(algo, w.model, so.astype(np.float64), w.act, w.iters,
                                    prior=prior.astype(np.float64), damping=0.6)
            err = float(np.abs(q - ref).max())
            print(f"[gpu]   soft {algo} prior+damping vs oracle {err:.3e}", flush=True)
            assert err <= TOL
    finally:
        pm.close()


def test_soft_on_sparse_packed_model():
    """A model packed with the sparse layout keeps its dense planes, which the
    soft path reads."""
    rng = np.random.Generator(np.random.PCG64(940))
    model = synth.make_model(rng, [9, 7, 5], [2, 1, 3], [3, 2, 4], [[0, 1, 2], [1], [0, 2]], 1, 1.0, 1.0,
                             sparsity=0.6, uniform_D=False)
    obs, act = synth.sample_sequences(rng, model, 12, 4)
    w = synth.Workload("soft_sparse", ["vmp", "mmp"], model, obs, act, 2)
    _check_vs_oracle(w, _soft(941, w), ("vmp", "mmp"), flags=bi.BI_SPARSE_A)
