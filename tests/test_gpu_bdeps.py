"""B-dependency lists (the general transition model of Sec. III-B) on the
GPU: the agent-resident kernels and bi_predict against the oracle."""
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


def _workload(seed, n, U, K, deps, lists, b, T, per_agent, iters=4):
    rng = np.random.Generator(np.random.PCG64(seed))
    model = synth.make_model(rng, n, U, K, deps, b if per_agent else 1, 1.0, 1.0, uniform_D=False, bdeps=lists)
    obs, act = synth.sample_sequences(rng, model, b, T)
    return synth.Workload(f"bdeps{seed}", ["fpi", "vmp", "mmp"], model, obs, act, iters)


CASES = [
    # (n, U, K, deps, B-dependency lists, b, T, per_agent)
    ([3, 4, 2], [2, 1, 3], [3, 2], [[0, 1], [2]], [[0, 2], [1], [0, 1, 2]], 6, 5, True),
    ([5, 3], [2, 2], [4, 3, 2], [[0], [1], [0, 1]], [[1], [0, 1]], 8, 6, False),
    ([4, 3, 2, 3], [1, 2, 2, 1], [3, 3], [[0, 1, 2, 3], [1, 3]], [[0, 1], [0, 1, 2, 3], [2], [1, 3]], 5, 4, True),
    ([2, 6], [3, 1], [5], [[0, 1]], [[0, 1], [0]], 7, 1, True),
    # transition tables beyond the LDS staging limit (read from global memory)
    ([12, 10, 8], [2, 2, 1], [4, 3], [[0, 1, 2], [1]], [[0, 1, 2], [0, 1], [1, 2]], 4, 4, True),
]


def _run(pm, w, algo, soft=None, prior=None, damping=1.0):
    torch = _torch()
    print(f"[gpu] {w.name} {algo} b={w.b} T={w.T} iters={w.iters} soft={soft is not None} "
          f"prior={prior is not None} damping={damping}", flush=True)
    if soft is None:
        q = pm.infer(algo, _dev(w.obs), _dev(w.act), w.iters, prior=None if prior is None else _dev(prior),
                     damping=damping)
    else:
        q = pm.infer_soft(algo, _dev(soft), _dev(w.act), w.iters, prior=None if prior is None else _dev(prior),
                          damping=damping)
    torch.cuda.synchronize()
    return q.cpu().numpy()


@pytest.mark.parametrize("case", range(len(CASES)))
def test_bdeps_vs_oracle(case):
    w = _workload(960 + case, *CASES[case])
    pm = bi.PackedModel(w.model)
    try:
        for algo in ("fpi", "vmp", "mmp"):
            assert pm.path(w.b, w.T, algo) == "agent"
            q = _run(pm, w, algo)
            check_invariants(w, q)
            ref = oracle.infer(algo, w.model, w.obs, w.act, w.iters)
            err = float(np.abs(q - ref).max())
            print(f"[gpu]   bdeps {algo} vs oracle {err:.3e}", flush=True)
            assert err <= TOL
    finally:
        pm.close()


def test_bdeps_soft_prior_damping():
    w = _workload(980, *CASES[0])
    rng = np.random.Generator(np.random.PCG64(981))
    so = synth.soft_obs(rng, w.obs, w.model.K, confidence=0.6)
    prior = synth.random_prior(rng, w.model.n, w.b, alpha=0.7, p_zero=0.2)
    pm = bi.PackedModel(w.model)
    try:
        for algo in ("fpi", "vmp", "mmp"):
            q = _run(pm, w, algo, soft=so, prior=prior, damping=0.7)
            ref = oracle.infer_soft(algo, w.model, so.astype(np.float64), w.act, w.iters,
                                    prior=prior.astype(np.float64), damping=0.7)
            err = float(np.abs(q - ref).max())
            print(f"[gpu]   bdeps soft+prior+damping {algo} vs oracle {err:.3e}", flush=True)
            assert err <= TOL
    finally:
        pm.close()


@pytest.mark.parametrize("case", [0, 2, 4])
def test_bdeps_predict_vs_oracle(case):
    torch = _torch()
    w = _workload(990 + case, *CASES[case])
    pm = bi.PackedModel(w.model)
    try:
        q = _run(pm, w, "fpi")
        rng = np.random.Generator(np.random.PCG64(995 + case))
        act = np.stack([rng.integers(0, u, size=w.b) for u in w.model.U], axis=1).astype(np.int32)
        qd = _dev(q.astype(np.float32))
        for t in range(w.T):
            out = pm.predict(qd[:, t], _dev(act))
            torch.cuda.synchronize()
            ref = oracle.predict(w.model, q[:, t].astype(np.float64), act)
            err = float(np.abs(out.cpu().numpy() - ref).max())
            print(f"[gpu]   bdeps predict t={t} vs oracle {err:.3e}", flush=True)
            assert err <= TOL
    finally:
        pm.close()


# shared models with B-dependency lists on the streaming kernels: the
# general transition messages of the update kernel (one lane per state)
STREAM_CASES = [
    # (n, U, K, deps, lists, b, T, packing flags, family, damping, prior)
    ([5, 3], [2, 2], [4, 3, 2], [[0], [1], [0, 1]], [[1], [0, 1]], 8, 6,
     bi.BI_DENSE_A | bi.BI_FAST_F32, "stream", 1.0, False),
    ([4, 3, 2, 3], [1, 2, 2, 1], [3, 3], [[0, 1, 2, 3], [1, 3]], [[0, 1], [0, 1, 2, 3], [2], [1, 3]], 12, 5,
     bi.BI_SPARSE_A, "sparse", 1.0, True),
    ([12, 10, 8], [2, 2, 1], [4, 3], [[0, 1, 2], [1]], [[0, 1, 2], [0, 1], [1, 2]], 16, 4,
     bi.BI_DENSE_A | bi.BI_FAST_F32, "stream", 0.6, True),
    # matrix-core shapes: the fp16-pair single-read kernel and the sparse pair tiles
    ([4, 32, 2, 32], [2, 1, 2, 1], [3], [[0, 1, 2, 3]], [[0, 1], [1], [1, 2], [3]], 24, 4,
     bi.BI_DENSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS, "stream", 1.0, False),
    ([4, 32, 6, 16], [2, 1, 2, 1], [3], [[0, 1, 2, 3]], [[0, 3], [1], [2], [0, 3]], 24, 4,
     bi.BI_SPARSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS, "sparse", 1.0, False),
]


@pytest.mark.parametrize("case", range(len(STREAM_CASES)))
def test_bdeps_streaming_vs_oracle_and_agent(case):
    import os
    n, U, K, deps, lists, b, T, flags, family, tau, with_prior = STREAM_CASES[case]
    sp = 0.7 if flags & bi.BI_SPARSE_A else 0.0
    rng = np.random.Generator(np.random.PCG64(1960 + case))
    model = synth.make_model(rng, n, U, K, deps, 1, 1.0, 1.0, sparsity=sp, uniform_D=False, bdeps=lists)
    obs, act = synth.sample_sequences(rng, model, b, T)
    w = synth.Workload(f"bdeps_stream{case}", ["vmp", "mmp"], model, obs, act, 3)
    prior = synth.random_prior(rng, model.n, b, alpha=0.7) if with_prior else None
    old = os.environ.get("BI_FORCE_PATH")
    pm = bi.PackedModel(model, flags=flags)
    try:
        for algo in ("vmp", "mmp"):
            os.environ["BI_FORCE_PATH"] = family
            assert pm.path(b, T, algo) == family
            q = _run(pm, w, algo, prior=prior, damping=tau)
            check_invariants(w, q)
            ref = oracle.infer(algo, model, obs, act, w.iters, prior=None if prior is None else prior.astype(np.float64),
                               damping=tau)
            err = float(np.abs(q - ref).max())
            print(f"[gpu]   bdeps {family} {algo} vs oracle {err:.3e}", flush=True)
            assert err <= TOL
            os.environ["BI_FORCE_PATH"] = "agent"
            qa = _run(pm, w, algo, prior=prior, damping=tau)
            assert float(np.abs(q - qa).max()) <= TOL
    finally:
        if old is None:
            os.environ.pop("BI_FORCE_PATH", None)
        else:
            os.environ["BI_FORCE_PATH"] = old
        pm.close()
