"""The largest models of the seeded POMDP sweeps (every spec above 400 000 A
entries, both dimension regimes: 29 models, one model shared by 256 agents)
against the oracle on two agents:
  - the default packing (agent-resident fp64 kernels), FPI / VMP / MMP;
  - the fp64 sparse kernels (BI_SPARSE_A, forced), VMP / MMP;
  - every family allowed (BI_SPARSE_A | BI_FAST_F32 | BI_F16_PAIRS), VMP /
    MMP, as the selector routes the call: the kernels that actually ran
    (library profiling) must be the family bi_query_path reports.
The fast classes round the log-likelihoods to fp32 or fp16 pairs; on these
models (Dirichlet(1) columns, no zeros) the marginals stay within 1e-5 of
the oracle through the 16 sweeps."""
import os

import numpy as np
import pytest

from paper_2607_17855_amd import bi, synth
import oracle

pytestmark = pytest.mark.gpu
TOL = 1e-5
AGENTS = [0, 255]
LARGE = [(r, c) for r in ("uniform", "skewed") for c in range(synth.N_SWEEP)
         if synth.sweep_spec(c, r).a_floats() > 400_000]
ALL_FAMILIES = bi.BI_SPARSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS
FAMILY_OF = {"agent_window": "agent", "agent_window_tile": "agent", "agent_filter": "agent", "agent_filter_tile": "agent", "lik_sparse": "sparse", "lik_sparse16": "sparse",
             "lik": "stream", "lik_split": "stream", "lik_split16": "stream", "lik_rowcol16": "stream"}


def _torch():
    import torch
    return torch


class _Force:
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


_REF = {}


def _ref(regime, case, w, algo):
    key = (regime, case, algo)
    if key not in _REF:
        _REF[key] = oracle.infer(algo, w.model, w.obs, w.act, w.iters, agents=AGENTS)
    return _REF[key]


def _run(pm, w, algo, profile=False):
    torch = _torch()
    obs = torch.from_numpy(np.ascontiguousarray(w.obs)).cuda()
    act = torch.from_numpy(np.ascontiguousarray(w.act)).cuda()
    if profile:
        bi.bi_profile_begin()
    q = pm.infer(algo, obs, act, w.iters)
    torch.cuda.synchronize()
    prof = bi.bi_profile_end() if profile else {}
    return q.cpu().numpy(), prof


@pytest.mark.parametrize("regime,case", LARGE)
def test_large_sweep_model(regime, case):
    w = synth.sweep_model(case, regime=regime)
    print(f"[gpu] sweep {regime} {case}: {synth.sweep_spec(case, regime).a_floats()} A entries, T={w.T}", flush=True)
    with _Force(None):
        pm = bi.PackedModel(w.model, flags=bi.BI_DENSE_A)
        for algo in ("fpi", "vmp", "mmp"):
            print(f"[gpu]   default packing {algo} ({pm.path(w.b, w.T, algo)})", flush=True)
            q, _ = _run(pm, w, algo)
            err = float(np.abs(q[AGENTS] - _ref(regime, case, w, algo)).max())
            print(f"[gpu]     max|gpu - oracle| = {err:.2e}", flush=True)
            assert err <= TOL
        pm.close()
    pm = bi.PackedModel(w.model, flags=bi.BI_SPARSE_A)
    with _Force("sparse"):
        for algo in ("vmp", "mmp"):
            if pm.path(w.b, w.T, algo) != "sparse":
                continue   # beyond the sparse kernels' limits: the agent path above covers it
            print(f"[gpu]   fp64 sparse kernels {algo}", flush=True)
            q, _ = _run(pm, w, algo)
            err = float(np.abs(q[AGENTS] - _ref(regime, case, w, algo)).max())
            print(f"[gpu]     max|gpu - oracle| = {err:.2e}", flush=True)
            assert err <= TOL
    pm.close()


@pytest.mark.parametrize("regime,case", LARGE)
@pytest.mark.parametrize("algo", ["vmp", "mmp"])
def test_large_sweep_selector_routed(regime, case, algo):
    w = synth.sweep_model(case, regime=regime)
    with _Force(None):
        pm = bi.PackedModel(w.model, flags=ALL_FAMILIES)
        family = pm.path(w.b, w.T, algo)
        print(f"[gpu] sweep {regime} {case} {algo}: selector -> {family} ({pm.explain_path(w.b, w.T, algo)})",
              flush=True)
        q, prof = _run(pm, w, algo, profile=True)
        pm.close()
    ran = {FAMILY_OF[k] for k in prof if k in FAMILY_OF}
    assert ran == {family}, f"selector reported {family}, kernels of {ran} ran ({sorted(prof)})"
    err = float(np.abs(q[AGENTS] - _ref(regime, case, w, algo)).max())
    print(f"[gpu]   max|gpu - oracle| = {err:.2e}", flush=True)
    assert err <= TOL
