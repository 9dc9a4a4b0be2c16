"""ctypes front end of ``bi_oracle.c`` (test infrastructure only).

``infer(algo, model, obs, act, iters)`` converts the float32 model arrays of a
:class:`paper_2607_17855_amd.synth.Model` to float64 and runs the C oracle;
``prior=`` replaces p(s_1) = D by the caller's prior (rolling inference), and
``predict(model, q, act)`` gives the predictive prior B q of the next step.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "bi_oracle.c")
_LIB = os.path.join(_HERE, "libbi_oracle.so")
ALGOS = {"fpi": 0, "vmp": 1, "mmp": 2}
_lib = None


def lib_path() -> str:
    return _LIB


def build() -> str:
    """Compile the oracle with gcc (plain C11 + OpenMP, no fast-math)."""
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fopenmp", "-fPIC", "-shared", "-o", _LIB + ".tmp",
           _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


def load_library(path: str):
    """Open an oracle shared library (the built one, or a test's mutant copy)."""
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    lib.orc_infer.restype = ctypes.c_int
    lib.orc_infer.argtypes = [ctypes.c_int, ctypes.c_int, P(ctypes.c_int), P(ctypes.c_int), ctypes.c_int,
                              P(ctypes.c_int), P(ctypes.c_int), P(ctypes.c_int), ctypes.c_int,
                              P(ctypes.c_void_p), P(ctypes.c_void_p), P(ctypes.c_void_p), ctypes.c_int,
                              ctypes.c_int, P(ctypes.c_int), P(ctypes.c_int), ctypes.c_int,
                              P(ctypes.c_double), ctypes.c_int]
    lib.orc_infer_prior.restype = ctypes.c_int
    lib.orc_infer_prior.argtypes = [ctypes.c_int, ctypes.c_int, P(ctypes.c_int), P(ctypes.c_int), ctypes.c_int,
                                    P(ctypes.c_int), P(ctypes.c_int), P(ctypes.c_int), ctypes.c_int,
                                    P(ctypes.c_void_p), P(ctypes.c_void_p), P(ctypes.c_void_p), ctypes.c_int,
                                    ctypes.c_int, P(ctypes.c_int), P(ctypes.c_int), P(ctypes.c_double),
                                    ctypes.c_int, P(ctypes.c_double), ctypes.c_int]
    lib.orc_infer_ex.restype = ctypes.c_int
    lib.orc_infer_ex.argtypes = [ctypes.c_int, ctypes.c_int, P(ctypes.c_int), P(ctypes.c_int), ctypes.c_int,
                                 P(ctypes.c_int), P(ctypes.c_int), P(ctypes.c_int), ctypes.c_int,
                                 P(ctypes.c_void_p), P(ctypes.c_void_p), P(ctypes.c_void_p), ctypes.c_int,
                                 ctypes.c_int, P(ctypes.c_int), P(ctypes.c_int), P(ctypes.c_double),
                                 ctypes.c_double, ctypes.c_int, P(ctypes.c_double), ctypes.c_int]
    lib.orc_infer_soft.restype = ctypes.c_int
    lib.orc_infer_soft.argtypes = [ctypes.c_int, ctypes.c_int, P(ctypes.c_int), P(ctypes.c_int), ctypes.c_int,
                                   P(ctypes.c_int), P(ctypes.c_int), P(ctypes.c_int), ctypes.c_int,
                                   P(ctypes.c_void_p), P(ctypes.c_void_p), P(ctypes.c_void_p), ctypes.c_int,
                                   ctypes.c_int, P(ctypes.c_double), P(ctypes.c_int), P(ctypes.c_double),
                                   ctypes.c_double, ctypes.c_int, P(ctypes.c_double), ctypes.c_int]
    lib.orc_infer_general.restype = ctypes.c_int
    lib.orc_infer_general.argtypes = [ctypes.c_int, ctypes.c_int, P(ctypes.c_int), P(ctypes.c_int), ctypes.c_int,
                                      P(ctypes.c_int), P(ctypes.c_int), P(ctypes.c_int), ctypes.c_int,
                                      P(ctypes.c_void_p), P(ctypes.c_void_p), P(ctypes.c_void_p),
                                      P(ctypes.c_int), P(ctypes.c_int), ctypes.c_int, ctypes.c_int,
                                      P(ctypes.c_int), P(ctypes.c_double), P(ctypes.c_int), P(ctypes.c_double),
                                      ctypes.c_double, ctypes.c_int, P(ctypes.c_double), ctypes.c_int]
    lib.orc_predict_general.restype = ctypes.c_int
    lib.orc_predict_general.argtypes = [ctypes.c_int, P(ctypes.c_int), P(ctypes.c_int), ctypes.c_int,
                                        P(ctypes.c_void_p), P(ctypes.c_int), P(ctypes.c_int), ctypes.c_int,
                                        P(ctypes.c_double), P(ctypes.c_int), P(ctypes.c_double)]
    lib.orc_predict.restype = ctypes.c_int
    lib.orc_predict.argtypes = [ctypes.c_int, P(ctypes.c_int), P(ctypes.c_int), ctypes.c_int, P(ctypes.c_void_p),
                                ctypes.c_int, P(ctypes.c_double), P(ctypes.c_int), P(ctypes.c_double)]
    lib.orc_default_threads.restype = ctypes.c_int
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = load_library(_LIB)
    return _lib


def default_threads() -> int:
    return int(_load().orc_default_threads())


def _i32(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.int32))


def infer(algo: str, model, obs: np.ndarray, act: np.ndarray, iters: int,
          agents: Optional[Sequence[int]] = None, threads: int = 0, lib=None,
          prior: Optional[np.ndarray] = None, damping: float = 1.0) -> np.ndarray:
    """Posterior marginals q [b][T][sum n] (float64) of ``algo`` for every agent,
    or for the listed ``agents`` only (agents are independent).  ``obs``: int
    outcomes [b][T][M].  ``prior``: [b][sum n] distributions over the first
    step, replacing D.  ``damping``: step tau in (0, 1] of
    q <- (1 - tau) q + tau q_new (1 = plain update)."""
    return _run(algo, model, obs, None, act, iters, agents, threads, lib, prior, damping)


def infer_soft(algo: str, model, obs_soft: np.ndarray, act: np.ndarray, iters: int,
               agents: Optional[Sequence[int]] = None, threads: int = 0, lib=None,
               prior: Optional[np.ndarray] = None, damping: float = 1.0) -> np.ndarray:
    """As ``infer`` with soft observations ``obs_soft`` [b][T][sum K]: modality
    m's observation vector (a distribution over its outcomes) at offset
    sum_{m' < m} K_m'."""
    return _run(algo, model, None, obs_soft, act, iters, agents, threads, lib, prior, damping)


def _run(algo, model, obs, obs_soft, act, iters, agents, threads, lib, prior, damping):
    if lib is None:
        lib = _load()
    if agents is not None:
        agents = list(agents)
        model = model.agent_slice(agents)
        if obs is not None:
            obs = obs[agents]
        else:
            obs_soft = obs_soft[agents]
        act = act[agents]
        if prior is not None:
            prior = np.asarray(prior)[agents]
    b, T = (obs if obs is not None else obs_soft).shape[:2]
    M = len(model.K)
    F = len(model.n)
    n, U, K = _i32(model.n), _i32(model.U), _i32(model.K)
    dep_off = _i32(np.cumsum([0] + [len(d) for d in model.deps]))
    dep = _i32([f for d in model.deps for f in d])
    A = [np.ascontiguousarray(a, dtype=np.float64) for a in model.A]
    B = [np.ascontiguousarray(x, dtype=np.float64) for x in model.B]
    D = [np.ascontiguousarray(x, dtype=np.float64) for x in model.D]
    ptrs = lambda arrs: (ctypes.c_void_p * len(arrs))(*[a.ctypes.data for a in arrs])  # noqa: E731
    act_c = _i32(act) if T > 1 else _i32(np.zeros((b, 1, F)))
    q = np.zeros((b, T, int(sum(model.n))), dtype=np.float64)
    ip = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_int))  # noqa: E731
    dp = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))  # noqa: E731
    pr = None if prior is None else np.ascontiguousarray(prior, dtype=np.float64).reshape(b, int(sum(model.n)))
    bdeps = getattr(model, "bdeps", None)
    if bdeps is not None:
        # B-dependency lists (general transition model)
        bd_off = _i32(np.cumsum([0] + [len(d) for d in bdeps]))
        bd = _i32([g for d in bdeps for g in d])
        os_c = None if obs_soft is None else np.ascontiguousarray(obs_soft, dtype=np.float64)
        obs_c = None if obs is None else _i32(obs)
        if os_c is not None and os_c.shape != (b, T, int(sum(model.K))):
            raise ValueError(f"soft observations of shape {os_c.shape}, expected {(b, T, int(sum(model.K)))}")
        rc = lib.orc_infer_general(ALGOS[algo], F, ip(n), ip(U), M, ip(K), ip(dep_off), ip(dep), int(model.mb),
                                   ptrs(A), ptrs(B), ptrs(D), ip(bd_off), ip(bd), b, T,
                                   None if obs_c is None else ip(obs_c), None if os_c is None else dp(os_c),
                                   ip(act_c), None if pr is None else dp(pr), float(damping), int(iters), dp(q),
                                   int(threads))
    elif obs_soft is not None:
        os_c = np.ascontiguousarray(obs_soft, dtype=np.float64)
        if os_c.shape != (b, T, int(sum(model.K))):
            raise ValueError(f"soft observations of shape {os_c.shape}, expected {(b, T, int(sum(model.K)))}")
        rc = lib.orc_infer_soft(ALGOS[algo], F, ip(n), ip(U), M, ip(K), ip(dep_off), ip(dep), int(model.mb),
                                ptrs(A), ptrs(B), ptrs(D), b, T, dp(os_c), ip(act_c),
                                None if pr is None else dp(pr), float(damping), int(iters), dp(q), int(threads))
    elif prior is None and damping == 1.0:
        obs_c = _i32(obs)
        rc = lib.orc_infer(ALGOS[algo], F, ip(n), ip(U), M, ip(K), ip(dep_off), ip(dep), int(model.mb),
                           ptrs(A), ptrs(B), ptrs(D), b, T, ip(obs_c), ip(act_c), int(iters), dp(q), int(threads))
    else:
        obs_c = _i32(obs)
        rc = lib.orc_infer_ex(ALGOS[algo], F, ip(n), ip(U), M, ip(K), ip(dep_off), ip(dep), int(model.mb),
                              ptrs(A), ptrs(B), ptrs(D), b, T, ip(obs_c), ip(act_c),
                              None if pr is None else dp(pr), float(damping), int(iters), dp(q), int(threads))
    if rc != 0:
        raise ValueError(f"oracle rejected the arguments (rc={rc})")
    return q


def predict(model, q: np.ndarray, act: np.ndarray, lib=None) -> np.ndarray:
    """Predictive prior [b][sum n] (float64) of the next step: for every agent
    and factor f, B_f[:, :, u_f] q_f, with q [b][sum n] and act [b][F] (with
    B-dependency lists: B_f contracted with the marginals of its list)."""
    if lib is None:
        lib = _load()
    q = np.ascontiguousarray(q, dtype=np.float64)
    b = q.shape[0]
    F = len(model.n)
    n, U = _i32(model.n), _i32(model.U)
    B = [np.ascontiguousarray(x, dtype=np.float64) for x in model.B]
    ptrs = lambda arrs: (ctypes.c_void_p * len(arrs))(*[a.ctypes.data for a in arrs])  # noqa: E731
    ip = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_int))  # noqa: E731
    act_c = _i32(np.asarray(act).reshape(b, F))
    out = np.zeros((b, int(sum(model.n))), dtype=np.float64)
    bdeps = getattr(model, "bdeps", None)
    if bdeps is not None:
        bd_off = _i32(np.cumsum([0] + [len(d) for d in bdeps]))
        bd = _i32([g for d in bdeps for g in d])
        rc = lib.orc_predict_general(F, ip(n), ip(U), int(model.mb), ptrs(B), ip(bd_off), ip(bd), b,
                                     q.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), ip(act_c),
                                     out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    else:
        rc = lib.orc_predict(F, ip(n), ip(U), int(model.mb), ptrs(B), b,
                             q.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), ip(act_c),
                             out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    if rc != 0:
        raise ValueError(f"oracle rejected the arguments (rc={rc})")
    return out
