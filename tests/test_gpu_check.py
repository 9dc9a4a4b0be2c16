"""BI_CHECK: out-of-range observations and actions are reported by the input
check (a device scan plus a stream sync) before any inference kernel runs;
valid inputs give the same marginals as a model packed without the flag."""
import os

import numpy as np
import pytest

from paper_2607_17855_amd import bi, synth

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    return torch


def _dev(x):
    return _torch().from_numpy(np.ascontiguousarray(x)).cuda()


def _shared_big(seed, b=8, T=4):
    rng = np.random.Generator(np.random.PCG64(seed))
    model = synth.make_model(rng, [32, 32, 16], [2, 1, 3], [3, 2], [[0, 1, 2], [1]], 1, 1.0, 1.0, sparsity=0.5,
                             uniform_D=False)
    obs, act = synth.sample_sequences(rng, model, b, T)
    return synth.Workload(f"check{seed}", ["vmp", "mmp"], model, obs, act, 2)


CASES = [
    # (workload maker, flags, algos, family): agent-resident, dense streaming, sparse streaming
    (lambda: synth.random_small(610, b=4, T_max=5, per_agent=True), bi.BI_DENSE_A, ("fpi", "vmp", "mmp"), "agent"),
    (lambda: _shared_big(611), bi.BI_DENSE_A | bi.BI_FAST_F32, ("vmp", "mmp"), "stream"),
    (lambda: _shared_big(613), bi.BI_DENSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS, ("vmp", "mmp"), "stream"),
    (lambda: _shared_big(612), bi.BI_SPARSE_A, ("vmp", "mmp"), "sparse"),
]


@pytest.fixture
def family(request):
    """Force the case's kernel family (the selector would pick by size)."""
    fam = CASES[request.node.callspec.params["case"]][3]
    old = os.environ.get("BI_FORCE_PATH")
    os.environ["BI_FORCE_PATH"] = fam
    yield fam
    if old is None:
        os.environ.pop("BI_FORCE_PATH", None)
    else:
        os.environ["BI_FORCE_PATH"] = old


@pytest.mark.parametrize("case", range(len(CASES)))
def test_check_passes_valid_inputs_unchanged(case, family):
    torch = _torch()
    make, flags, algos, _ = CASES[case]
    w = make()
    p0 = bi.PackedModel(w.model, flags)
    p1 = bi.PackedModel(w.model, flags | bi.BI_CHECK)
    try:
        obs, act = _dev(w.obs), _dev(w.act)
        for algo in algos:
            print(f"[gpu] {w.name} {algo} flags={flags} check", flush=True)
            assert p1.path(w.b, w.T, algo) == family
            q0 = p0.infer(algo, obs, act, w.iters)
            q1 = p1.infer(algo, obs, act, w.iters)
            torch.cuda.synchronize()
            assert np.array_equal(q0.cpu().numpy(), q1.cpu().numpy())
    finally:
        p0.close()
        p1.close()


@pytest.mark.parametrize("case", range(len(CASES)))
def test_check_reports_the_first_bad_entry(case, family):
    torch = _torch()
    make, flags, algos, _ = CASES[case]
    w = make()
    if w.T < 2:
        pytest.skip("needs actions")
    pm = bi.PackedModel(w.model, flags | bi.BI_CHECK)
    try:
        algo = algos[-1]
        # an outcome equal to K_m, then a negative one before it
        obs = w.obs.copy()
        b, T, M = obs.shape
        a, t, m = b - 1, T - 1, M - 1
        obs[a, t, m] = w.model.K[m]
        print(f"[gpu] {w.name} {algo} bad obs[{a},{t},{m}]", flush=True)
        q = torch.full((b, T, w.model.n_total), -7.0, dtype=torch.float32, device="cuda")
        with pytest.raises(bi.BiError) as ei:
            pm.infer(algo, _dev(obs), _dev(w.act), w.iters, q=q)
        assert ei.value.code == bi.BI_ERR_INVALID_ARG
        assert f"obs[{(a * T + t) * M + m}] (agent {a}, step {t}, modality {m})" in str(ei.value)
        torch.cuda.synchronize()
        assert bool((q == -7.0).all()), "no inference kernel may run after a failed check"
        obs[0, 0, 0] = -1
        with pytest.raises(bi.BiError) as ei:
            pm.infer(algo, _dev(obs), _dev(w.act), w.iters, q=q)
        assert "2 out-of-range inputs; first: obs[0]" in str(ei.value)
        # an action equal to U_f
        act = w.act.copy()
        F = act.shape[2]
        act[1, T - 2, F - 1] = w.model.U[F - 1]
        print(f"[gpu] {w.name} {algo} bad act[1,{T - 2},{F - 1}]", flush=True)
        with pytest.raises(bi.BiError) as ei:
            pm.infer(algo, _dev(w.obs), _dev(act), w.iters, q=q)
        assert f"act[{(1 * (T - 1) + T - 2) * F + F - 1}] (agent 1, step {T - 2}, factor {F - 1})" in str(ei.value)
        # soft observations: the actions are checked
        so = synth.one_hot_obs(w.obs, w.model.K)
        with pytest.raises(bi.BiError):
            pm.infer_soft(algo, _dev(so), _dev(act), w.iters, q=q)
        torch.cuda.synchronize()
        assert bool((q == -7.0).all())
        qs = pm.infer_soft(algo, _dev(so), _dev(w.act), w.iters)
        torch.cuda.synchronize()
        assert np.all(np.isfinite(qs.cpu().numpy()))
    finally:
        pm.close()
