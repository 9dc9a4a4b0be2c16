"""Sparse path (BI_SPARSE_A, shared model: fp64 gathers over the nonzero
entries; with BI_FAST_F32 | BI_F16_PAIRS, fp16-pair matrix-core tiles fed
from the nonzeros) against the oracle, the agent-resident path and the dense
layout."""
import functools
import os

import numpy as np
import pytest

from paper_2607_17855_amd import bi, synth
import oracle
from test_gpu_parity import check_invariants, run_gpu

pytestmark = pytest.mark.gpu
TOL = 1e-5


def _shared_model(seed, n, U, K, deps, b, T, sparsity, iters=2):
    rng = np.random.Generator(np.random.PCG64(seed))
    model = synth.make_model(rng, n, U, K, deps, 1, 1.0, 1.0, sparsity=sparsity, uniform_D=False)
    obs, act = synth.sample_sequences(rng, model, b, T)
    return synth.Workload(f"sparse{seed}", ["vmp", "mmp"], model, obs, act, iters)


CASES = [
    # (n, U, K, deps, b, T, sparsity)
    # rank 1 (no row factors: one side only), rank 2 / 3 / 4 with one or two
    # factors per side, several tiles of two-factor lines (13 x 11 rows), a
    # bucket of more than 64 contexts (200 contexts, 2 outcomes), single-state
    # factors, dense A (sparsity 0) and very sparse A
    ([9, 7, 5], [2, 1, 3], [3, 2, 4], [[0, 1, 2], [1], [0, 2]], 24, 5, 0.5),
    ([13, 11, 6, 3], [1, 2, 2, 1], [5, 3], [[0, 1, 2, 3], [1, 3]], 40, 4, 0.7),
    ([70], [2], [3], [[0]], 30, 3, 0.3),
    ([33, 5], [2, 2], [2, 2, 3], [[0, 1], [0], [1]], 64, 6, 0.0),
    ([4, 4, 4, 4], [1, 1, 1, 1], [2], [[0, 1, 2, 3]], 100, 2, 0.9),
    ([1, 6, 1], [1, 2, 1], [3, 2], [[0, 1, 2], [1, 2]], 12, 3, 0.5),
    ([40, 40], [3, 2], [4], [[0, 1]], 20, 4, 0.95),
]


@pytest.fixture
def force_sparse():
    # small models would run agent-resident under the selector: force the
    # sparse kernels, which are what these cases test
    old = os.environ.get("BI_FORCE_PATH")
    os.environ["BI_FORCE_PATH"] = "sparse"
    yield
    if old is None:
        os.environ.pop("BI_FORCE_PATH", None)
    else:
        os.environ["BI_FORCE_PATH"] = old


@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("iters", [1, 3])
def test_sparse_small_vs_oracle_and_agent(case, iters, force_sparse):
    n, U, K, deps, b, T, sp = CASES[case]
    w = _shared_model(70 + case, n, U, K, deps, b, T, sp, iters=iters)
    for algo in ("vmp", "mmp"):
        q, pm = run_gpu(w, algo, flags=bi.BI_SPARSE_A)
        assert pm.path(w.b, w.T, algo) == "sparse", "the forced sparse kernels must run"
        check_invariants(w, q)
        ref = oracle.infer(algo, w.model, w.obs, w.act, w.iters)
        err = float(np.abs(q - ref).max())
        print(f"[gpu]   sparse vs oracle {err:.3e}", flush=True)
        assert err <= TOL
        old = os.environ.get("BI_FORCE_PATH")
        os.environ["BI_FORCE_PATH"] = "agent"
        try:
            qa, _ = run_gpu(w, algo, pm=pm)
        finally:
            os.environ["BI_FORCE_PATH"] = old
        assert float(np.abs(q - qa).max()) <= TOL
        # FPI has no sparse kernel: the same packed model runs it agent-resident
        if algo == "vmp":
            assert pm.path(w.b, w.T, "fpi") == "agent"
        pm.close()


def test_sparse_fpi_uses_dense_planes():
    n, U, K, deps, b, T, sp = CASES[0]
    w = _shared_model(90, n, U, K, deps, b, T, sp, iters=3)
    q, pm = run_gpu(w, "fpi", flags=bi.BI_SPARSE_A)
    ref = oracle.infer("fpi", w.model, w.obs, w.act, w.iters)
    assert float(np.abs(q - ref).max()) <= TOL
    pm.close()


@functools.lru_cache(maxsize=None)
def large_shared():
    return synth.large_shared()


LARGE_AGENTS = [0, 21, 42, 63]


@pytest.mark.parametrize("algo", ["vmp", "mmp"])
def test_large_shared_sparse(algo):
    w = large_shared()
    q, pm = run_gpu(w, algo, flags=bi.BI_SPARSE_A)
    assert pm.path(w.b, w.T, algo) == "sparse", "the selector must send the large model to the sparse kernels"
    st = pm.stats()
    print(f"[gpu]   large shared model sparse: nnz {st['a_nnz']} device bytes {st['device_bytes']}", flush=True)
    check_invariants(w, q)
    q2, _ = run_gpu(w, algo, pm=pm)
    assert np.array_equal(q, q2), "sparse path is not reproducible"
    ref = oracle.infer(algo, w.model, w.obs, w.act, w.iters, agents=LARGE_AGENTS)
    err = float(np.abs(q[LARGE_AGENTS] - ref).max())
    print(f"[gpu]   large shared model {algo} sparse vs oracle (agents {LARGE_AGENTS}): {err:.3e}", flush=True)
    assert err <= TOL
    pm.close()


# shapes of the sparse fp16-pair tiles (two factors per side, second factors
# of 16 or 32 states, even first factors): 96 lines (a partial 64-line block),
# 1024 lines (four tiles), 16 and 32 entry states, a bucket of more than 48
# contexts (two context passes), dense A (runs longer than the 256 entries a
# wave holds in flight) and very sparse A (empty runs)
SQ_CASES = [
    # (n, U, K, deps, b, T, sparsity)
    ([6, 16, 4, 32], [2, 1, 2, 1], [3], [[0, 1, 2, 3]], 24, 5, 0.9),
    ([2, 32, 10, 16], [1, 2, 1, 2], [4, 2], [[0, 1, 2, 3], [0, 1, 2, 3]], 40, 4, 0.5),
    ([4, 32, 32, 16], [2, 2, 1, 1], [2], [[0, 1, 2, 3]], 60, 2, 0.0),
    ([32, 32, 2, 32], [1, 1, 2, 2], [3], [[0, 1, 2, 3]], 30, 3, 0.97),
    ([2, 16, 2, 16], [2, 2, 2, 2], [2, 3], [[0, 1, 2, 3], [0, 1, 2, 3]], 50, 3, 0.7),
]
SQ_FLAGS = bi.BI_SPARSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS
# (case, iterations).  The fp16-pair precision class is for models whose
# marginals are insensitive to rounding of the log-likelihoods; cases 1 and 4
# are not beyond one sweep: a perturbation of log A at the pair error scale
# ((ln A - ln eps) 2^-20) moves the fp64 oracle's marginals by 3-5e-6 after
# two sweeps and 1e-5-4e-4 after three, and even the fp32 dense path is 4e-5
# off after three.  The others stay below 2e-6 through three sweeps.
SQ_RUNS = [(c, 1) for c in range(len(SQ_CASES))] + [(0, 2), (2, 3), (3, 3)]


@pytest.mark.parametrize("case,iters", SQ_RUNS)
def test_sparse_pairs_vs_oracle_agent_and_dense_pairs(case, iters, force_sparse):
    n, U, K, deps, b, T, sp = SQ_CASES[case]
    w = _shared_model(1400 + case, n, U, K, deps, b, T, sp, iters=iters)
    for algo in ("vmp", "mmp"):
        print(f"[gpu] sparse pairs case {case} iters {iters} {algo}", flush=True)
        bi.bi_profile_begin()
        q, pm = run_gpu(w, algo, flags=SQ_FLAGS)
        names = set(bi.bi_profile_end())
        assert pm.path(w.b, w.T, algo) == "sparse"
        assert "lik_sparse16" in names, names
        check_invariants(w, q)
        ref = oracle.infer(algo, w.model, w.obs, w.act, w.iters)
        err = float(np.abs(q - ref).max())
        print(f"[gpu]   sparse pairs vs oracle {err:.3e}", flush=True)
        assert err <= TOL
        q2, _ = run_gpu(w, algo, pm=pm)
        assert np.array_equal(q, q2), "sparse pair path is not reproducible"
        old = os.environ.get("BI_FORCE_PATH")
        os.environ["BI_FORCE_PATH"] = "agent"
        try:
            qa, _ = run_gpu(w, algo, pm=pm)
        finally:
            os.environ["BI_FORCE_PATH"] = old
        assert float(np.abs(q - qa).max()) <= TOL
        pm.close()
        # the dense fp16-pair tiles on the same model
        os.environ["BI_FORCE_PATH"] = "stream"
        try:
            qd, pmd = run_gpu(w, algo, flags=bi.BI_DENSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS)
        finally:
            os.environ["BI_FORCE_PATH"] = old
        pmd.close()
        assert float(np.abs(q - qd).max()) <= TOL


@pytest.mark.parametrize("algo", ["vmp", "mmp"])
def test_large_shared_sparse_pairs(algo):
    w = large_shared()
    print(f"[gpu] large shared model {algo} sparse pairs", flush=True)
    bi.bi_profile_begin()
    q, pm = run_gpu(w, algo, flags=SQ_FLAGS)
    names = set(bi.bi_profile_end())
    assert pm.path(w.b, w.T, algo) == "sparse", "the selector must send the large model to the sparse kernels"
    assert "lik_sparse16" in names, names
    check_invariants(w, q)
    q2, _ = run_gpu(w, algo, pm=pm)
    assert np.array_equal(q, q2), "sparse pair path is not reproducible"
    ref = oracle.infer(algo, w.model, w.obs, w.act, w.iters, agents=LARGE_AGENTS)
    err = float(np.abs(q[LARGE_AGENTS] - ref).max())
    print(f"[gpu]   large shared model {algo} sparse pairs vs oracle (agents {LARGE_AGENTS}): {err:.3e}", flush=True)
    assert err <= TOL
    pm.close()
