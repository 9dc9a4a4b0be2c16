"""HIP graph capture of inference calls.  With the output and the workspace
allocated beforehand, bi_vfilter / bi_vmp / bi_mmp only enqueue kernels on the
caller's stream (no allocation, copy or synchronisation), so a call can be
captured once and replayed.  Every replay, with eager calls and
synchronisations in between, must reproduce the eager result bit for bit (the
kernels are deterministic), on every kernel family."""
import os

import numpy as np
import pytest

from paper_2607_17855_amd import bi, synth

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    return torch


def _shared(seed, n, U, K, deps, b, T, sparsity=0.0):
    rng = np.random.Generator(np.random.PCG64(seed))
    model = synth.make_model(rng, n, U, K, deps, 1, 1.0, 1.0, sparsity=sparsity, uniform_D=False)
    obs, act = synth.sample_sequences(rng, model, b, T)
    return synth.Workload(f"graph{seed}", ["vmp", "mmp"], model, obs, act, 3)


def _agents(seed, n, K, deps, b, T, algos):
    rng = np.random.Generator(np.random.PCG64(seed))
    model = synth.make_model(rng, n, [2] * len(n), K, deps, b, 0.7, 1.0, uniform_D=False)
    obs, act = synth.sample_sequences(rng, model, b, T)
    return synth.Workload(f"graph{seed}", list(algos), model, obs, act, 3)


CASES = [
    # (workload maker, packing flags, algorithms, kernel family)
    (lambda: synth.two_factor_agents(b=32), bi.BI_DENSE_A, ("fpi", "vmp", "mmp"), "agent"),
    # windows read from global memory (tile form), and FPI steps in the tile form
    (lambda: _agents(1204, [20, 6, 7], [5, 3, 4], [[0, 1, 2], [1], [0, 2]], 6, 12, ("vmp", "mmp")),
     bi.BI_DENSE_A, ("vmp", "mmp"), "agent"),
    (lambda: _agents(1205, [30, 25, 28], [3, 4], [[0, 1, 2], [2]], 3, 4, ("fpi",)), bi.BI_DENSE_A, ("fpi",), "agent"),
    (lambda: _shared(1200, [9, 7, 5], [2, 1, 3], [3, 2, 4], [[0, 1, 2], [1], [0, 2]], 24, 5),
     bi.BI_DENSE_A | bi.BI_FAST_F32, ("vmp", "mmp"), "stream"),
    (lambda: _shared(1201, [4, 32, 6, 32], [2, 1, 2, 1], [3], [[0, 1, 2, 3]], 30, 4),
     bi.BI_DENSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS, ("vmp", "mmp"), "stream"),
    (lambda: _shared(1202, [9, 7, 5], [2, 1, 3], [3, 2, 4], [[0, 1, 2], [1], [0, 2]], 24, 5, sparsity=0.6),
     bi.BI_SPARSE_A, ("vmp", "mmp"), "sparse"),
    (lambda: _shared(1203, [4, 32, 6, 16], [2, 1, 2, 1], [3], [[0, 1, 2, 3]], 30, 4, sparsity=0.8),
     bi.BI_SPARSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS, ("vmp", "mmp"), "sparse"),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_captured_call_replays_exactly(case):
    torch = _torch()
    make, flags, algos, family = CASES[case]
    w = make()
    old = os.environ.get("BI_FORCE_PATH")
    os.environ["BI_FORCE_PATH"] = family
    pm = bi.PackedModel(w.model, flags)
    try:
        obs = torch.from_numpy(np.ascontiguousarray(w.obs)).cuda()
        act = torch.from_numpy(np.ascontiguousarray(w.act)).cuda()
        for algo in algos:
            print(f"[gpu] {w.name} {algo} {family} graph capture", flush=True)
            assert pm.path(w.b, w.T, algo) == family
            ws = pm.workspace(w.b, w.T, algo)
            shape = (w.b, w.T, w.model.n_total)
            q_eager = torch.empty(shape, dtype=torch.float32, device="cuda")
            pm.infer(algo, obs, act, w.iters, q=q_eager, ws=ws)
            torch.cuda.synchronize()
            ref = q_eager.cpu().numpy()
            q_g = torch.empty(shape, dtype=torch.float32, device="cuda")
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):   # warm-up on a side stream before capture
                pm.infer(algo, obs, act, w.iters, q=q_g, ws=ws)
            torch.cuda.current_stream().wait_stream(side)
            torch.cuda.synchronize()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                pm.infer(algo, obs, act, w.iters, q=q_g, ws=ws)
            for rep in range(3):
                q_g.fill_(-1.0)
                # eager work between the replays, on the same workspace
                pm.infer(algo, obs, act, w.iters, q=q_eager, ws=ws)
                torch.cuda.synchronize()
                graph.replay()
                torch.cuda.synchronize()
                got = q_g.cpu().numpy()
                assert np.array_equal(got, ref), f"replay {rep}: max diff {np.abs(got - ref).max()}"
            del graph
    finally:
        pm.close()
        if old is None:
            os.environ.pop("BI_FORCE_PATH", None)
        else:
            os.environ["BI_FORCE_PATH"] = old
