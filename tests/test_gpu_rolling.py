"""Rolling inference on the GPU: the first-step prior entry points
(bi_vfilter_prior / bi_vmp_prior / bi_mmp_prior) on every path, and
bi_predict, against the oracle; and filtering run one step at a time through
predict + a one-step window, against the full window."""
import os

import numpy as np
import pytest

from paper_2607_17855_amd import bi, synth
import oracle
from test_gpu_parity import check_invariants, run_gpu

pytestmark = pytest.mark.gpu
TOL = 1e-5


def _torch():
    import torch
    return torch


def _dev(x):
    return _torch().from_numpy(np.ascontiguousarray(x)).cuda()


def _infer(pm, w, algo, prior):
    torch = _torch()
    print(f"[gpu] {w.name} {algo} b={w.b} T={w.T} iters={w.iters} flags={pm.flags} prior={prior is not None}",
          flush=True)
    q = pm.infer(algo, _dev(w.obs), _dev(w.act), w.iters, prior=None if prior is None else _dev(prior))
    torch.cuda.synchronize()
    return q.cpu().numpy()


def _prior(seed, w, p_zero=0.3):
    rng = np.random.Generator(np.random.PCG64(seed))
    return synth.random_prior(rng, w.model.n, w.b, alpha=0.7, p_zero=p_zero)


def _d_as_prior(w):
    """D of every agent, stacked [b][sum n] (float32 like the model)."""
    ai = np.zeros(w.b, dtype=np.int64) if w.model.mb == 1 else np.arange(w.b)
    return np.concatenate([d[ai] for d in w.model.D], axis=1).astype(np.float32)


class _ForcePath:
    def __init__(self, path):
        self.path = path

    def __enter__(self):
        self.old = os.environ.get("BI_FORCE_PATH")
        if self.path is None:
            os.environ.pop("BI_FORCE_PATH", None)
        else:
            os.environ["BI_FORCE_PATH"] = self.path

    def __exit__(self, *exc):
        if self.old is None:
            os.environ.pop("BI_FORCE_PATH", None)
        else:
            os.environ["BI_FORCE_PATH"] = self.old


def _check_prior(w, algo, flags, path, seed):
    """prior entry point vs the oracle; prior = D reproduces the call without a
    prior (the packed log D is taken on the host, the prior's log on the
    device: equal up to the last bit of the fp64 logarithm)."""
    pm = bi.PackedModel(w.model, flags)
    try:
        with _ForcePath(path):
            prior = _prior(seed, w)
            q = _infer(pm, w, algo, prior)
            check_invariants(w, q)
            ref = oracle.infer(algo, w.model, w.obs, w.act, w.iters, prior=prior.astype(np.float64))
            err = float(np.abs(q - ref).max())
            print(f"[gpu]   {algo} prior vs oracle {err:.3e}", flush=True)
            assert err <= TOL
            q_d = _infer(pm, w, algo, _d_as_prior(w))
            q_0 = _infer(pm, w, algo, None)
            assert float(np.abs(q_d - q_0).max()) <= 1e-6, "prior = D must match the call without a prior"
    finally:
        pm.close()


@pytest.mark.parametrize("seed", range(6))
def test_prior_agent_path(seed):
    w = synth.random_small(300 + seed, b=5, T_max=5, per_agent=bool(seed % 2))
    for algo in ("fpi", "vmp", "mmp"):
        _check_prior(w, algo, bi.BI_DENSE_A, "agent", 500 + seed)


def _shared_model(seed, n, U, K, deps, b, T, sparsity=0.0, iters=2):
    rng = np.random.Generator(np.random.PCG64(seed))
    model = synth.make_model(rng, n, U, K, deps, 1, 1.0, 1.0, sparsity=sparsity, uniform_D=False)
    obs, act = synth.sample_sequences(rng, model, b, T)
    return synth.Workload(f"roll{seed}", ["vmp", "mmp"], model, obs, act, iters)


SHARED = [
    # (n, U, K, deps, b, T): general streaming kernel (ragged tiles, rank 1..3),
    # the one-contraction-per-workgroup kernel (two factors per side, second
    # factors of 16 / 32 states), and a window of one step
    ([9, 7, 5], [2, 1, 3], [3, 2, 4], [[0, 1, 2], [1], [0, 2]], 24, 5),
    ([6, 16, 4, 32], [2, 1, 2, 1], [3], [[0, 1, 2, 3]], 24, 5),
    ([13, 11, 6, 3], [1, 2, 2, 1], [5, 3], [[0, 1, 2, 3], [1, 3]], 40, 1),
    ([4, 32, 6, 32], [2, 1, 2, 1], [3, 2], [[0, 1, 2, 3], [0, 1, 2, 3]], 30, 4),
]
# dense streaming packings: fp32 copy, and fp16 pairs (the matrix-core shapes
# then run on fp16 matrix cores)
DENSE_FAST = [bi.BI_DENSE_A | bi.BI_FAST_F32, bi.BI_DENSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS]


@pytest.mark.parametrize("case", range(len(SHARED)))
@pytest.mark.parametrize("flags", DENSE_FAST)
def test_prior_stream_path(case, flags):
    w = _shared_model(600 + case, *SHARED[case])
    for algo in ("vmp", "mmp"):
        _check_prior(w, algo, flags, "stream", 700 + case)


@pytest.mark.parametrize("case", range(len(SHARED)))
def test_prior_sparse_path(case):
    w = _shared_model(620 + case, *SHARED[case], sparsity=0.6)
    for algo in ("vmp", "mmp"):
        _check_prior(w, algo, bi.BI_SPARSE_A, "sparse", 720 + case)


@pytest.mark.parametrize("seed", range(4))
def test_predict_vs_oracle(seed):
    torch = _torch()
    w = synth.random_small(330 + seed, b=6, T_max=4, n_max=70 if seed == 3 else 5, per_agent=bool(seed % 2))
    q, pm = run_gpu(w, "fpi")
    rng = np.random.Generator(np.random.PCG64(800 + seed))
    act = np.stack([rng.integers(0, u, size=w.b) for u in w.model.U], axis=1).astype(np.int32)
    try:
        qd = _dev(q.astype(np.float32))
        for t in range(w.T):
            # one step of a [b][T][sum n] output: rows T * sum n apart
            out = pm.predict(qd[:, t], _dev(act))
            torch.cuda.synchronize()
            got = out.cpu().numpy()
            ref = oracle.predict(w.model, q[:, t].astype(np.float64), act)
            err = float(np.abs(got - ref).max())
            print(f"[gpu]   predict t={t} vs oracle {err:.3e}", flush=True)
            assert err <= TOL
    finally:
        pm.close()


@pytest.mark.parametrize("seed", range(4))
def test_online_filter_matches_full_window(seed):
    """FPI over T steps == T one-step windows, each carrying the predictive
    prior of the previous step's marginal (the first one D)."""
    torch = _torch()
    w = synth.random_small(360 + seed, b=4, T_max=6, per_agent=bool(seed % 2))
    pm = bi.PackedModel(w.model)
    try:
        full = _infer(pm, w, "fpi", None)
        ref = oracle.infer("fpi", w.model, w.obs, w.act, w.iters)
        assert float(np.abs(full - ref).max()) <= TOL
        prior = _dev(_d_as_prior(w))
        steps = []
        for t in range(w.T):
            obs_t = _dev(w.obs[:, t:t + 1])
            q_t = pm.infer("fpi", obs_t, None, w.iters, prior=prior)
            steps.append(q_t[:, 0])
            if t + 1 < w.T:
                prior = pm.predict(q_t[:, 0], _dev(w.act[:, t]))
        torch.cuda.synchronize()
        online = torch.stack(steps, dim=1).cpu().numpy()
        err = float(np.abs(online - full).max())
        print(f"[gpu]   online vs full-window FPI {err:.3e}", flush=True)
        assert err <= TOL
    finally:
        pm.close()


def _check_damped(w, algo, flags, path, seed, tau, with_prior):
    """bi_infer with damping (and optionally a prior) vs the oracle."""
    torch = _torch()
    pm = bi.PackedModel(w.model, flags)
    try:
        with _ForcePath(path):
            prior = _prior(seed, w) if with_prior else None
            print(f"[gpu] {w.name} {algo} b={w.b} T={w.T} iters={w.iters} flags={flags} damping={tau} "
                  f"prior={with_prior}", flush=True)
            q = pm.infer(algo, _dev(w.obs), _dev(w.act), w.iters, prior=None if prior is None else _dev(prior),
                         damping=tau)
            torch.cuda.synchronize()
            q = q.cpu().numpy()
            check_invariants(w, q)
            ref = oracle.infer(algo, w.model, w.obs, w.act, w.iters,
                               prior=None if prior is None else prior.astype(np.float64), damping=tau)
            err = float(np.abs(q - ref).max())
            print(f"[gpu]   {algo} damped vs oracle {err:.3e}", flush=True)
            assert err <= TOL
    finally:
        pm.close()


@pytest.mark.parametrize("seed", range(4))
def test_damping_agent_path(seed):
    w = synth.random_small(340 + seed, b=4, T_max=5, per_agent=bool(seed % 2))
    for algo in ("fpi", "vmp", "mmp"):
        _check_damped(w, algo, bi.BI_DENSE_A, "agent", 540 + seed, (0.3, 0.5, 0.8, 0.65)[seed], seed >= 2)


@pytest.mark.parametrize("case", range(len(SHARED)))
def test_damping_stream_and_sparse_paths(case):
    w = _shared_model(640 + case, *SHARED[case], iters=3)
    ws = _shared_model(660 + case, *SHARED[case], sparsity=0.6, iters=3)
    for algo in ("vmp", "mmp"):
        for flags in DENSE_FAST:
            _check_damped(w, algo, flags, "stream", 740 + case, 0.45, case % 2 == 1)
        _check_damped(ws, algo, bi.BI_SPARSE_A, "sparse", 760 + case, 0.7, case % 2 == 0)
