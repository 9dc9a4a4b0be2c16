"""Soft observations (Sec. III-C, the log-likelihood as the contraction of
log A_m with an observation vector) on the streaming kernels of shared
models: each context's slot o observes outcome o wherever its vectors give o
a nonzero weight, the likelihood kernels run over the slots, and the update
sums a context's slots weighted by its vectors.  Against the oracle, with
the library's profile showing that the streaming family ran; one-hot vectors
against the integer-outcome call (the same bits); vectors with all-zero
blocks (no evidence from that modality) and vectors mixing one-hot and
spread blocks."""
import os

import numpy as np
import pytest

from paper_2607_17855_amd import bi, synth
import oracle
from test_gpu_parity import check_invariants

pytestmark = pytest.mark.gpu
TOL = 1e-5

F32 = bi.BI_DENSE_A | bi.BI_FAST_F32
PAIRS = bi.BI_DENSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS
SPARSE64 = bi.BI_SPARSE_A
SPARSE16 = bi.BI_SPARSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS

# (name, n, U, K, deps, b, T, sparsity, flags, family, likelihood kernel)
CASES = [
    ("general", [9, 7, 5], [2, 1, 3], [3, 2, 4], [[0, 1, 2], [1], [0, 2]], 24, 5, 0.0, F32, "stream", "lik"),
    ("general4", [13, 11, 6, 3], [1, 2, 2, 1], [5, 3], [[0, 1, 2, 3], [1, 3]], 20, 4, 0.0, F32, "stream", "lik"),
    ("split", [6, 16, 4, 32], [2, 1, 2, 1], [3], [[0, 1, 2, 3]], 24, 5, 0.0, F32, "stream", "lik_split"),
    ("split16", [2, 32, 10, 16], [1, 2, 1, 2], [4, 2], [[0, 1, 2, 3], [0, 1, 2, 3]], 20, 4, 0.0, PAIRS,
     "stream", "lik_split16"),
    ("rowcol", [12, 32, 2, 32], [1, 2, 1, 2], [4, 2], [[0, 1, 2, 3], [0, 1, 2, 3]], 20, 4, 0.0, PAIRS,
     "stream", "lik_rowcol16"),
    ("sparse", [9, 7, 5], [2, 1, 3], [3, 2, 4], [[0, 1, 2], [1], [0, 2]], 24, 5, 0.6, SPARSE64, "sparse",
     "lik_sparse"),
    ("sparse16", [6, 16, 4, 32], [2, 1, 2, 1], [3, 2], [[0, 1, 2, 3], [0, 1, 2, 3]], 24, 4, 0.8, SPARSE16,
     "sparse", "lik_sparse16"),
]


def _torch():
    import torch
    return torch


def _dev(x):
    return _torch().from_numpy(np.ascontiguousarray(x)).cuda()


@pytest.fixture
def family_env():
    old = os.environ.get("BI_FORCE_PATH")
    yield
    if old is None:
        os.environ.pop("BI_FORCE_PATH", None)
    else:
        os.environ["BI_FORCE_PATH"] = old


def _workload(case, iters=2):
    name, n, U, K, deps, b, T, sp, flags, fam, kern = CASES[case]
    rng = np.random.Generator(np.random.PCG64(2100 + case))
    model = synth.make_model(rng, n, U, K, deps, 1, 1.0, 1.0, sparsity=sp, uniform_D=False)
    obs, act = synth.sample_sequences(rng, model, b, T)
    return synth.Workload(f"soft_{name}", ["vmp", "mmp"], model, obs, act, iters), flags, fam, kern


def _vectors(seed, w, zero_blocks=True):
    """Spread and one-hot blocks mixed; with zero_blocks, some blocks all zero
    (no evidence from that modality at that step)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    so = synth.soft_obs(rng, w.obs, w.model.K, confidence=0.6, p_hard=0.3)
    if zero_blocks:
        k0 = 0
        for km in w.model.K:
            mask = rng.random((w.b, w.T)) < 0.15
            so[:, :, k0:k0 + km][mask] = 0.0
            k0 += km
    return so


def _soft_call(pm, algo, so, w):
    torch = _torch()
    bi.bi_profile_begin()
    q = pm.infer_soft(algo, _dev(so), _dev(w.act), w.iters)
    torch.cuda.synchronize()
    names = set(bi.bi_profile_end())
    return q.cpu().numpy(), names


@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("algo", ["vmp", "mmp"])
def test_soft_streaming_vs_oracle(case, algo, family_env):
    w, flags, fam, kern = _workload(case)
    so = _vectors(2200 + case, w)
    os.environ["BI_FORCE_PATH"] = fam
    print(f"[gpu] {w.name} soft {algo} on {fam} ({kern}) b={w.b} T={w.T}", flush=True)
    pm = bi.PackedModel(w.model, flags)
    try:
        assert pm.path(w.b, w.T, algo) == fam
        q, names = _soft_call(pm, algo, so, w)
        assert kern in names and "agent_window" not in names, names
        check_invariants(w, q)
        ref = oracle.infer_soft(algo, w.model, so.astype(np.float64), w.act, w.iters)
        err = float(np.abs(q - ref).max())
        print(f"[gpu]   soft {fam} vs oracle {err:.3e}", flush=True)
        assert err <= TOL
        # fixed summation order: the same call gives the same bits
        q2, _ = _soft_call(pm, algo, so, w)
        assert np.array_equal(q, q2)
    finally:
        pm.close()


@pytest.mark.parametrize("case", range(len(CASES)))
def test_soft_streaming_one_hot_equals_integer(case, family_env):
    w, flags, fam, kern = _workload(case)
    os.environ["BI_FORCE_PATH"] = fam
    torch = _torch()
    pm = bi.PackedModel(w.model, flags)
    try:
        for algo in ("vmp", "mmp"):
            print(f"[gpu] {w.name} one-hot {algo} on {fam}", flush=True)
            qs, names = _soft_call(pm, algo, synth.one_hot_obs(w.obs, w.model.K), w)
            assert kern in names, names
            qi = pm.infer(algo, _dev(w.obs), _dev(w.act), w.iters)
            torch.cuda.synchronize()
            assert np.array_equal(qs, qi.cpu().numpy())
    finally:
        pm.close()


def test_soft_streaming_matches_agent_path(family_env):
    """The streaming and agent-resident soft calls on the same model and
    vectors (the agent path forms the log-likelihood tensors instead)."""
    w, flags, fam, kern = _workload(4, iters=3)
    so = _vectors(2300, w, zero_blocks=False)
    pm = bi.PackedModel(w.model, flags)
    try:
        for algo in ("vmp", "mmp"):
            os.environ["BI_FORCE_PATH"] = fam
            qs, names = _soft_call(pm, algo, so, w)
            assert kern in names, names
            os.environ["BI_FORCE_PATH"] = "agent"
            qa, names = _soft_call(pm, algo, so, w)
            assert "agent_window" in "".join(names), names
            err = float(np.abs(qs - qa).max())
            print(f"[gpu]   soft {algo} stream vs agent {err:.3e}", flush=True)
            assert err <= TOL
    finally:
        pm.close()


@pytest.mark.parametrize("case", [4, 6])
def test_soft_streaming_prior_and_damping(case, family_env):
    """A prior over the first step and a damping step on the soft streaming
    call, against the oracle with the same options."""
    w, flags, fam, kern = _workload(case, iters=3)
    so = _vectors(2500 + case, w)
    prior = synth.random_prior(np.random.Generator(np.random.PCG64(2510 + case)), w.model.n, w.b, alpha=0.7,
                               p_zero=0.3)
    os.environ["BI_FORCE_PATH"] = fam
    torch = _torch()
    pm = bi.PackedModel(w.model, flags)
    try:
        for algo in ("vmp", "mmp"):
            print(f"[gpu] {w.name} soft {algo} on {fam} prior + damping 0.7", flush=True)
            bi.bi_profile_begin()
            q = pm.infer_soft(algo, _dev(so), _dev(w.act), w.iters, prior=_dev(prior), damping=0.7)
            torch.cuda.synchronize()
            names = set(bi.bi_profile_end())
            assert kern in names, names
            q = q.cpu().numpy()
            check_invariants(w, q)
            ref = oracle.infer_soft(algo, w.model, so.astype(np.float64), w.act, w.iters, prior=prior,
                                    damping=0.7)
            err = float(np.abs(q - ref).max())
            print(f"[gpu]   soft prior+damping vs oracle {err:.3e}", flush=True)
            assert err <= TOL
    finally:
        pm.close()


@pytest.mark.parametrize("case", [4, 6])
def test_soft_streaming_graph_replay(case, family_env):
    """The soft streaming call captured in a HIP graph replays the eager
    call's bits, with eager calls on the same workspace between replays."""
    torch = _torch()
    w, flags, fam, kern = _workload(case)
    so = _dev(_vectors(2600 + case, w))
    act = _dev(w.act)
    os.environ["BI_FORCE_PATH"] = fam
    pm = bi.PackedModel(w.model, flags)
    try:
        for algo in ("vmp", "mmp"):
            print(f"[gpu] {w.name} soft {algo} on {fam} graph capture", flush=True)
            ws = pm.workspace_soft(w.b, w.T, algo)
            shape = (w.b, w.T, w.model.n_total)
            q_eager = torch.empty(shape, dtype=torch.float32, device="cuda")
            pm.infer_soft(algo, so, act, w.iters, q=q_eager, ws=ws)
            torch.cuda.synchronize()
            ref = q_eager.cpu().numpy()
            q_g = torch.empty(shape, dtype=torch.float32, device="cuda")
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                pm.infer_soft(algo, so, act, w.iters, q=q_g, ws=ws)
            torch.cuda.current_stream().wait_stream(side)
            torch.cuda.synchronize()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                pm.infer_soft(algo, so, act, w.iters, q=q_g, ws=ws)
            for rep in range(3):
                q_g.fill_(-1.0)
                pm.infer_soft(algo, so, act, w.iters, q=q_eager, ws=ws)
                torch.cuda.synchronize()
                graph.replay()
                torch.cuda.synchronize()
                got = q_g.cpu().numpy()
                assert np.array_equal(got, ref), f"replay {rep}: max diff {np.abs(got - ref).max()}"
            del graph
    finally:
        pm.close()


def test_soft_streaming_with_input_check(family_env):
    """BI_CHECK on a soft streaming call: the status words after the slots'
    workspace; the result equals the unchecked call's."""
    torch = _torch()
    w, flags, fam, kern = _workload(4)
    so = _vectors(2700, w)
    os.environ["BI_FORCE_PATH"] = fam
    pm0 = bi.PackedModel(w.model, flags)
    pm1 = bi.PackedModel(w.model, flags | bi.BI_CHECK)
    try:
        for algo in ("vmp", "mmp"):
            q0, _ = _soft_call(pm0, algo, so, w)
            q1, names = _soft_call(pm1, algo, so, w)
            assert kern in names, names
            assert np.array_equal(q0, q1)
    finally:
        pm0.close()
        pm1.close()
