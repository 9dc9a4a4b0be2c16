"""bi_infer_static (no allocation: the library's static device scratch)
against bi_infer with a caller workspace, through the C-ABI, on every kernel
family: two calls in a row, the second with a smaller batch and window, each
equal bit for bit to bi_infer on the same input and within 1e-5 of the
oracle."""
import os

import numpy as np
import pytest

from paper_2607_17855_amd import bi, synth
import oracle

pytestmark = pytest.mark.gpu
TOL = 1e-5


def _torch():
    import torch
    return torch


def _shared(seed, n, U, K, deps, b, T, sparsity=0.0):
    rng = np.random.Generator(np.random.PCG64(seed))
    model = synth.make_model(rng, n, U, K, deps, 1, 1.0, 1.0, sparsity=sparsity, uniform_D=False)
    obs, act = synth.sample_sequences(rng, model, b, T)
    return model, obs, act


# (name, family forced, packing flags, model maker, (b, T) of the first call, (b, T) of the second)
CASES = [
    ("rowcol", "stream", bi.BI_DENSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS,
     lambda b, T: _shared(71, [4, 32, 2, 32], [2, 1, 2, 1], [3], [[0, 1, 2, 3]], b, T), (24, 4), (9, 3)),
    ("dense_general", "stream", bi.BI_DENSE_A | bi.BI_FAST_F32,
     lambda b, T: _shared(72, [9, 7, 5], [2, 1, 3], [3, 2, 4], [[0, 1, 2], [1], [0, 2]], b, T), (24, 5), (7, 2)),
    ("sparse_f64", "sparse", bi.BI_SPARSE_A,
     lambda b, T: _shared(73, [9, 7, 5], [2, 1, 3], [3, 2, 4], [[0, 1, 2], [1], [0, 2]], b, T, 0.6), (20, 4), (5, 3)),
    ("sparse_pairs", "sparse", bi.BI_SPARSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS,
     lambda b, T: _shared(74, [4, 32, 6, 16], [2, 1, 2, 1], [3], [[0, 1, 2, 3]], b, T, 0.8), (24, 4), (6, 2)),
    ("agent", "agent", bi.BI_DENSE_A,
     lambda b, T: _shared(75, [6, 5], [2, 3], [4, 3], [[0, 1], [1]], b, T), (16, 5), (4, 2)),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_static_scratch_matches_workspace_call(case):
    torch = _torch()
    name, family, flags, make, first, second = CASES[case]
    model, obs_all, act_all = make(*first)
    old = os.environ.get("BI_FORCE_PATH")
    os.environ["BI_FORCE_PATH"] = family
    try:
        pm = bi.PackedModel(model, flags=flags, device="cuda")
        for algo in ("vmp", "mmp", "fpi"):
            for b, T in (first, second):   # the second call is smaller and runs on what the first left
                obs, act = np.ascontiguousarray(obs_all[:b, :T]), np.ascontiguousarray(act_all[:b, :T - 1])
                print(f"[gpu] no-alloc {name} {algo} b={b} T={T} path={pm.path(b, T, algo)}", flush=True)
                if algo != "fpi":
                    assert pm.path(b, T, algo) == family
                od, ad = torch.from_numpy(obs).cuda(), torch.from_numpy(act).cuda()
                q_s = torch.full((b, T, model.n_total), -3.0, dtype=torch.float32, device="cuda")
                bi.bi_infer_static(pm.handle, bi.ALGO_IDS[algo], b, T, od, ad, 3, q_s)
                q_w = pm.infer(algo, od, ad, 3)
                torch.cuda.synchronize()
                qs, qw = q_s.cpu().numpy(), q_w.cpu().numpy()
                assert np.array_equal(qs, qw), f"{name} {algo}: static scratch differs from the workspace call"
                ref = oracle.infer(algo, model, obs, act, 3)
                err = float(np.abs(qs - ref).max())
                print(f"[gpu]   max|static - oracle| = {err:.2e}", flush=True)
                assert err <= TOL
        pm.close()
    finally:
        if old is None:
            os.environ.pop("BI_FORCE_PATH", None)
        else:
            os.environ["BI_FORCE_PATH"] = old
