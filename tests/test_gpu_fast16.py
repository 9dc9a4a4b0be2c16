"""The opt-in fast precision classes (BI_FAST_F32: fp32 matrix cores;
BI_F16_PAIRS: fp16 (high, residual) pairs) on every kernel shape of the
streaming tests, at the workloads' 16 iterations, against the fp64 oracle.

The classes round the log-likelihoods (relative 2^-24 for fp32, about 2^-21
for the pairs).  Whether 16 Jacobi sweeps keep such a rounding small is a
property of the model, not of the kernels: each case also measures how far
the fp64 oracle itself moves when every nonzero log A is perturbed at the
class's rounding scale (two seeded draws).  A case must be within 1e-5 of the
oracle unless that sensitivity already exceeds 1e-5; then no computation at
the class's precision can meet the bar and the case is an expected failure
whose reason gives both numbers."""
import os

import numpy as np
import pytest

from paper_2607_17855_amd import bi, synth
import oracle
import test_gpu_sparse as tsp
import test_gpu_stream as tst

pytestmark = pytest.mark.gpu
TOL = 1e-5
ITERS = 16
SCALE = {"f32": 2.0 ** -24, "f16pairs": 2.0 ** -21}

# (name, family, flags, precision, workload maker)
CASES = []
for i, (n, U, K, deps, b, T) in enumerate(tst.CASES):
    CASES.append((f"stream_general_{i}", "stream", bi.BI_DENSE_A | bi.BI_FAST_F32, "f32",
                  (tst._shared_model, (50 + i, n, U, K, deps, b, T), {})))
for i, (n, U, K, deps, b, T) in enumerate(tst.SPLIT_CASES):
    for prec, fl in tst.FAST.items():
        CASES.append((f"split_{prec}_{i}", "stream", fl, prec, (tst._shared_model, (80 + i, n, U, K, deps, b, T), {})))
for i, (n, U, K, deps, b, T) in enumerate(tst.ROWCOL_CASES):
    CASES.append((f"rowcol_{i}", "stream", tst.FAST["f16pairs"], "f16pairs",
                  (tst._shared_model, (90 + i, n, U, K, deps, b, T), {})))
for i, (n, U, K, deps, b, T, sp) in enumerate(tsp.SQ_CASES):
    CASES.append((f"sparse_pairs_{i}", "sparse", tsp.SQ_FLAGS, "f16pairs",
                  (tsp._shared_model, (1400 + i, n, U, K, deps, b, T, sp), {})))


def _perturbed(model, scale, seed):
    """The model with every nonzero log A moved by a relative u * scale,
    u uniform in [-1, 1] (zeros stay exact: their log is the clamp)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    A2 = []
    for a in model.A:
        a64 = a.astype(np.float64)
        la = np.log(np.maximum(a64, 1e-16)) - np.log(1e-16)
        la = la * (1.0 + rng.uniform(-1.0, 1.0, la.shape) * scale)
        A2.append(np.where(a64 > 1e-16, np.exp(la + np.log(1e-16)), 0.0))
    return synth.Model(model.n, model.U, model.K, model.deps, model.mb, A2,
                       [x.astype(np.float64) for x in model.B], [x.astype(np.float64) for x in model.D])


@pytest.mark.parametrize("case", range(len(CASES)), ids=[c[0] for c in CASES])
@pytest.mark.parametrize("algo", ["vmp", "mmp"])
def test_fast_class_at_16_iterations(case, algo):
    import torch
    name, family, flags, prec, (make, args, kw) = CASES[case]
    w = make(*args, iters=ITERS, **kw)
    old = os.environ.get("BI_FORCE_PATH")
    os.environ["BI_FORCE_PATH"] = family
    try:
        print(f"[gpu] {name} {algo} ({family}, {prec}) b={w.b} T={w.T} iters={ITERS}", flush=True)
        pm = bi.PackedModel(w.model, flags=flags)
        assert pm.path(w.b, w.T, algo) == family
        q = pm.infer(algo, torch.from_numpy(np.ascontiguousarray(w.obs)).cuda(),
                     torch.from_numpy(np.ascontiguousarray(w.act)).cuda(), ITERS)
        torch.cuda.synchronize()
        q = q.cpu().numpy()
        pm.close()
    finally:
        if old is None:
            os.environ.pop("BI_FORCE_PATH", None)
        else:
            os.environ["BI_FORCE_PATH"] = old
    tst.check_invariants(w, q)
    ref = oracle.infer(algo, w.model, w.obs, w.act, ITERS)
    err = float(np.abs(q - ref).max())
    print(f"[gpu]   max|gpu - oracle| = {err:.2e}", flush=True)
    if err <= TOL:
        return
    sens = max(float(np.abs(oracle.infer(algo, _perturbed(w.model, SCALE[prec], s), w.obs, w.act, ITERS) - ref).max())
               for s in (1, 2))
    print(f"[gpu]   the oracle moves {sens:.2e} under a {SCALE[prec]:.1e} relative perturbation of log A", flush=True)
    assert sens > TOL, f"{name} {algo}: error {err:.2e} although the model is insensitive ({sens:.2e})"
    pytest.xfail(f"ill-conditioned at 16 sweeps: max error {err:.1e}; the fp64 oracle itself moves {sens:.1e} "
                 f"under a {prec} rounding-scale perturbation of log A")
