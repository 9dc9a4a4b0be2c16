"""HIP path (through the C-ABI) against the fp64 oracle, element by element.

Tolerance: 1e-5 max-abs per marginal entry, the fp32 target.  Every case
prints its name before touching the GPU so that a failure names its case.
"""
import functools

import numpy as np
import pytest

from paper_2607_17855_amd import bi, synth
import oracle

pytestmark = pytest.mark.gpu
TOL = 1e-5


def _torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return torch


def run_gpu(w, algo, flags=bi.BI_DENSE_A, pm=None):
    torch = _torch()
    print(f"[gpu] {w.name} {algo} b={w.b} T={w.T} iters={w.iters} flags={flags}", flush=True)
    if pm is None:
        pm = bi.PackedModel(w.model, flags)
    obs = torch.from_numpy(np.ascontiguousarray(w.obs)).cuda()
    act = torch.from_numpy(np.ascontiguousarray(w.act)).cuda()
    q = pm.infer(algo, obs, act, w.iters)
    torch.cuda.synchronize()
    return q.cpu().numpy(), pm


def check_invariants(w, q):
    assert np.all(np.isfinite(q))
    assert q.min() >= 0.0
    offs = np.cumsum([0] + list(w.model.n))
    for f in range(w.model.F):
        assert np.abs(q[..., offs[f]:offs[f + 1]].sum(-1) - 1.0).max() < 1e-5


def check(w, algo, agents=None, flags=bi.BI_DENSE_A):
    q, pm = run_gpu(w, algo, flags)
    check_invariants(w, q)
    ref = oracle.infer(algo, w.model, w.obs, w.act, w.iters, agents=agents)
    got = q if agents is None else q[list(agents)]
    err = float(np.abs(got - ref).max())
    print(f"[gpu]   max|gpu - oracle| = {err:.3e}", flush=True)
    assert err <= TOL, f"{w.name} {algo}: max abs error {err:.3e} > {TOL}"
    pm.close()
    return q


@functools.lru_cache(maxsize=None)
def cfg(i, **kw):
    return {1: synth.hmm_small, 2: synth.two_factor_agents, 3: synth.three_factor_agents}[i](**kw)


@pytest.mark.parametrize("algo", ["fpi", "vmp", "mmp"])
def test_hmm_small(algo):
    check(cfg(1), algo)


@pytest.mark.parametrize("algo", ["vmp", "fpi", "mmp"])
def test_two_factor_agents(algo):
    w = cfg(2)
    check(w, algo, agents=None if algo == "vmp" else range(0, w.b, 7))


@pytest.mark.parametrize("algo", ["mmp", "vmp", "fpi"])
def test_three_factor_agents(algo):
    w = cfg(3)
    check(w, algo, agents=None if algo == "mmp" else range(0, w.b, 31))


@pytest.mark.parametrize("seed", range(24))
def test_random_small(seed):
    w = synth.random_small(1000 + seed, F_max=4, n_max=7, M_max=4, K_max=6, T_max=6, b=5,
                           sparsity=0.5 if seed % 3 == 0 else 0.0)
    for algo in ("fpi", "vmp", "mmp"):
        check(w, algo)


def test_single_step_window_and_single_state():
    # T = 1 (no transitions), and a factor with a single state (q = 1 exactly)
    rng = np.random.Generator(np.random.PCG64(5))
    model = synth.make_model(rng, [1, 3, 2], [1, 2, 1], [3, 2], [[0, 1], [1, 2]], 4, 1.0, 1.0)
    for T in (1, 2):
        obs, act = synth.sample_sequences(rng, model, 4, T)
        w = synth.Workload(f"n1_T{T}", ["fpi", "vmp", "mmp"], model, obs, act, 5)
        for algo in w.algos:
            check(w, algo)


def test_rank4_and_ragged_columns():
    # rank-4 dependency (2 x 2 split) with column counts that are not multiples of 4
    rng = np.random.Generator(np.random.PCG64(9))
    model = synth.make_model(rng, [3, 5, 2, 7], [2, 1, 3, 1], [4, 3, 5], [[0, 1, 2, 3], [1, 3], [0, 2, 3]], 1,
                             1.0, 1.0, sparsity=0.6)
    obs, act = synth.sample_sequences(rng, model, 6, 7)
    w = synth.Workload("rank4_ragged", ["fpi", "vmp", "mmp"], model, obs, act, 8)
    for algo in w.algos:
        check(w, algo)


def test_deterministic_and_agent_equivariant():
    w = cfg(2)
    q1, pm = run_gpu(w, "vmp")
    q2, _ = run_gpu(w, "vmp", pm=pm)
    assert np.array_equal(q1, q2), "two identical calls differ"
    perm = np.random.Generator(np.random.PCG64(1)).permutation(w.b)
    wp = synth.Workload("F2_perm", w.algos, w.model.agent_slice(perm), w.obs[perm], w.act[perm], w.iters)
    qp, _ = run_gpu(wp, "vmp")
    assert np.array_equal(qp, q1[perm])
    pm.close()


def test_shared_equals_replicated():
    w = synth.random_small(77, F_max=3, n_max=6, b=6, per_agent=False)
    m = w.model
    rep = synth.Model(m.n, m.U, m.K, m.deps, w.b, [np.repeat(a, w.b, axis=0) for a in m.A],
                      [np.repeat(a, w.b, axis=0) for a in m.B], [np.repeat(a, w.b, axis=0) for a in m.D])
    wr = synth.Workload("replicated", w.algos, rep, w.obs, w.act, w.iters)
    for algo in ("fpi", "vmp", "mmp"):
        qs, _ = run_gpu(w, algo)
        qr, _ = run_gpu(wr, algo)
        assert np.abs(qs - qr).max() <= 1e-6


def _sweep_sample(regime, count, seed):
    """A seeded sample of sweep models whose oracle cost stays small."""
    rng = np.random.Generator(np.random.PCG64(seed))
    out = []
    for case in rng.permutation(synth.N_SWEEP):
        if synth.sweep_spec(int(case), regime).a_floats() <= 400_000:
            out.append(int(case))
        if len(out) == count:
            break
    return sorted(out)


SWEEP = [("uniform", c) for c in _sweep_sample("uniform", 24, 4)] + \
        [("skewed", c) for c in _sweep_sample("skewed", 24, 46)]


@pytest.mark.parametrize("regime,case", SWEEP)
def test_sweep_sample(regime, case):
    """Sweep models of both dimension regimes (one model shared by 256
    agents): every algorithm on the family the selector picks, and VMP / MMP
    on the sparse kernels, against the oracle on four agents."""
    import os
    w = synth.sweep_model(case, regime=regime)
    agents = [0, 1, 128, 255]
    for algo in ("fpi", "vmp", "mmp"):
        check(w, algo, agents=agents)
    old = os.environ.get("BI_FORCE_PATH")
    os.environ["BI_FORCE_PATH"] = "sparse"
    try:
        for algo in ("vmp", "mmp"):
            q, pm = run_gpu(w, algo, flags=bi.BI_SPARSE_A)
            assert pm.path(w.b, w.T, algo) == "sparse"
            ref = oracle.infer(algo, w.model, w.obs, w.act, w.iters, agents=agents)
            err = float(np.abs(q[agents] - ref).max())
            print(f"[gpu]   sweep {regime} {case} {algo} sparse vs oracle {err:.3e}", flush=True)
            assert err <= TOL
            pm.close()
    finally:
        if old is None:
            os.environ.pop("BI_FORCE_PATH", None)
        else:
            os.environ["BI_FORCE_PATH"] = old
