"""Streaming path (shared model, BI_FAST_F32: fp32 matrix-core contractions,
fp64 updates) against the oracle and against the fp64 agent-resident path."""
import functools
import os

import numpy as np
import pytest

from paper_2607_17855_amd import bi, synth
import oracle
from test_gpu_parity import check_invariants, run_gpu

pytestmark = pytest.mark.gpu
TOL = 1e-5


@pytest.fixture
def force_stream():
    old = os.environ.get("BI_FORCE_PATH")
    os.environ["BI_FORCE_PATH"] = "stream"
    yield
    if old is None:
        os.environ.pop("BI_FORCE_PATH", None)
    else:
        os.environ["BI_FORCE_PATH"] = old


def _shared_model(seed, n, U, K, deps, b, T, alpha=1.0, sparsity=0.0, iters=2):
    rng = np.random.Generator(np.random.PCG64(seed))
    model = synth.make_model(rng, n, U, K, deps, 1, alpha, alpha, sparsity=sparsity, uniform_D=False)
    obs, act = synth.sample_sequences(rng, model, b, T)
    return synth.Workload(f"shared{seed}", ["vmp", "mmp"], model, obs, act, iters)


CASES = [
    # (n, U, K, deps, b, T): ragged row tiles (R % 64 != 0), ragged column blocks,
    # every rank 1..4, buckets of more than 32 contexts (few outcomes)
    ([9, 7, 5], [2, 1, 3], [3, 2, 4], [[0, 1, 2], [1], [0, 2]], 24, 5),
    ([13, 11, 6, 3], [1, 2, 2, 1], [5, 3], [[0, 1, 2, 3], [1, 3]], 40, 4),
    ([70], [2], [3], [[0]], 30, 3),
    ([33, 5], [2, 2], [2, 2, 3], [[0, 1], [0], [1]], 64, 6),
    ([4, 4, 4, 4], [1, 1, 1, 1], [2], [[0, 1, 2, 3]], 100, 2),
    # 19 factors: the update kernel's waves take several factors each, the
    # factors past the 16 whose fields are kernel arguments read their
    # descriptors, and factor 18 is in no dependency list (no likelihood)
    ([3, 2, 2, 3, 2, 2, 3, 2, 2, 3, 2, 2, 3, 2, 2, 3, 2, 3, 2], [2, 1, 2, 1, 2, 1, 2, 1, 2, 1, 2, 1, 2, 1, 2, 1, 3, 2, 2],
     [3, 4, 2, 3, 3], [[0, 1, 2, 3], [4, 5, 16], [6, 7, 8, 17], [9, 10, 11, 12], [13, 14, 15]], 20, 4),
    # a one-step window (no actions)
    ([5, 4], [2, 1], [3, 2], [[0, 1], [1]], 16, 1),
]


@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("iters", [1, 2])
def test_stream_small_vs_oracle_and_agent(case, iters, force_stream):
    n, U, K, deps, b, T = CASES[case]
    w = _shared_model(50 + case, n, U, K, deps, b, T, iters=iters)
    for algo in ("vmp", "mmp"):
        q, pm = run_gpu(w, algo, flags=bi.BI_DENSE_A | bi.BI_FAST_F32)
        check_invariants(w, q)
        ref = oracle.infer(algo, w.model, w.obs, w.act, w.iters)
        err = float(np.abs(q - ref).max())
        print(f"[gpu]   stream vs oracle {err:.3e}", flush=True)
        assert err <= TOL
        os.environ["BI_FORCE_PATH"] = "agent"
        qa, _ = run_gpu(w, algo, pm=pm)
        os.environ["BI_FORCE_PATH"] = "stream"
        assert float(np.abs(q - qa).max()) <= TOL
        pm.close()


# shapes taken by the split matrix-core kernel (two factors per side, second
# factors of 16 or 32 states, even first factors): ragged row and column
# tiles, 4 and 8 k-steps per state, two modalities, several column tiles and
# a bucket of more than 48 contexts
SPLIT_CASES = [
    ([6, 16, 4, 32], [2, 1, 2, 1], [3], [[0, 1, 2, 3]], 24, 5),
    ([2, 32, 10, 16], [1, 2, 1, 2], [4, 2], [[0, 1, 2, 3], [0, 1, 2, 3]], 40, 4),
    ([4, 32, 32, 16], [2, 2, 1, 1], [2], [[0, 1, 2, 3]], 60, 2),
]


FAST = {"f32": bi.BI_DENSE_A | bi.BI_FAST_F32, "f16pairs": bi.BI_DENSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS}


@pytest.mark.parametrize("case", range(len(SPLIT_CASES)))
@pytest.mark.parametrize("prec", list(FAST))
def test_split_kernel_vs_oracle_and_agent(case, prec, force_stream):
    n, U, K, deps, b, T = SPLIT_CASES[case]
    w = _shared_model(80 + case, n, U, K, deps, b, T, iters=2)
    for algo in ("vmp", "mmp"):
        q, pm = run_gpu(w, algo, flags=FAST[prec])
        check_invariants(w, q)
        ref = oracle.infer(algo, w.model, w.obs, w.act, w.iters)
        err = float(np.abs(q - ref).max())
        print(f"[gpu]   split ({prec}) stream vs oracle {err:.3e}", flush=True)
        bi.bi_profile_begin()
        run_gpu(w, algo, pm=pm)
        names = set(bi.bi_profile_end())
        assert ("lik_split16" if prec == "f16pairs" else "lik_split") in names, names
        assert err <= TOL
        os.environ["BI_FORCE_PATH"] = "agent"
        qa, _ = run_gpu(w, algo, pm=pm)
        os.environ["BI_FORCE_PATH"] = "stream"
        assert float(np.abs(q - qa).max()) <= TOL
        pm.close()


# shapes taken by the single-read fp16-pair kernel (two factors per side,
# both second factors of 32 states): a row tile of 6 of its 8 row states, two
# modalities over two row tiles (the second one half full), and buckets of
# more than 48 contexts (a second pass of 1 context block)
ROWCOL_CASES = [
    ([6, 32, 4, 32], [2, 1, 2, 1], [3], [[0, 1, 2, 3]], 24, 5),
    ([12, 32, 2, 32], [1, 2, 1, 2], [4, 2], [[0, 1, 2, 3], [0, 1, 2, 3]], 40, 4),
    ([8, 32, 8, 32], [2, 2, 1, 1], [2], [[0, 1, 2, 3]], 60, 2),
]


@pytest.mark.parametrize("case", range(len(ROWCOL_CASES)))
def test_rowcol_kernel_vs_oracle_and_agent(case, force_stream):
    n, U, K, deps, b, T = ROWCOL_CASES[case]
    w = _shared_model(90 + case, n, U, K, deps, b, T, iters=2)
    for algo in ("vmp", "mmp"):
        q, pm = run_gpu(w, algo, flags=FAST["f16pairs"])
        check_invariants(w, q)
        ref = oracle.infer(algo, w.model, w.obs, w.act, w.iters)
        err = float(np.abs(q - ref).max())
        print(f"[gpu]   rowcol stream vs oracle {err:.3e}", flush=True)
        bi.bi_profile_begin()
        q2, _ = run_gpu(w, algo, pm=pm)
        names = set(bi.bi_profile_end())
        assert "lik_rowcol16" in names, names
        assert err <= TOL
        # the same call again gives the same bits (fixed summation order)
        assert np.array_equal(q, q2)
        os.environ["BI_FORCE_PATH"] = "agent"
        qa, _ = run_gpu(w, algo, pm=pm)
        os.environ["BI_FORCE_PATH"] = "stream"
        assert float(np.abs(q - qa).max()) <= TOL
        pm.close()


@functools.lru_cache(maxsize=None)
def large_shared():
    return synth.large_shared()


LARGE_AGENTS = [0, 21, 42, 63]


@pytest.mark.parametrize("algo", ["vmp", "mmp"])
@pytest.mark.parametrize("prec", list(FAST))
def test_large_shared_stream(algo, prec):
    w = large_shared()
    print(f"[gpu] large shared model {algo} {prec}", flush=True)
    q, pm = run_gpu(w, algo, flags=FAST[prec])
    assert pm.path(w.b, w.T, algo) == "stream", "the selector must send the large model to the streaming kernels"
    assert pm.workspace(w.b, w.T, algo) is not None, "the large shared model must take the streaming path"
    check_invariants(w, q)
    q2, _ = run_gpu(w, algo, pm=pm)
    assert np.array_equal(q, q2), "streaming path is not reproducible"
    ref = oracle.infer(algo, w.model, w.obs, w.act, w.iters, agents=LARGE_AGENTS)
    err = float(np.abs(q[LARGE_AGENTS] - ref).max())
    print(f"[gpu]   large shared model {algo} stream ({prec}) vs oracle (agents {LARGE_AGENTS}): {err:.3e}", flush=True)
    assert err <= TOL
    pm.close()
