"""Seeded synthetic POMDP workloads (generative models, actions, observations).

This module only *draws* inputs; it holds none of the inference arithmetic.
Both the HIP path (through the C-ABI) and the fp64 oracle consume exactly the
arrays produced here.

Model conventions (the factorised POMDP of Sec. III-B, "Terminology and
notation"):

* ``A[m]``: float32 ``[mb][K_m][n_{d_1}]...[n_{d_k}]`` with ``dep(m) = (d_1 < ...
  < d_k)``; ``A[m][a, o, s...] = P(o^m = o | s^{d_1}, ..., s^{d_k})`` (the outcome
  axis first, then the dependency axes in list order).
* ``B[f]``: float32 ``[mb][n_f][n_f][U_f]``; ``B[f][a, i, j, u] = P(s_{t+1}^f = i |
  s_t^f = j, u_t^f = u)`` (trivial B-dependencies, the case the paper's
  layouts support, Sec. III-B).  With B-dependency lists ``bdeps[f] =
  (g_1 < ... < g_k)`` (the general transition model of Sec. III-B),
  ``B[f]`` is ``[mb][n_f][n_{g_1}]...[n_{g_k}][U_f]`` with
  ``B[f][a, i, j_1, ..., j_k, u] = P(s_{t+1}^f = i | s_t^{g_1} = j_1, ..., u_t^f = u)``;
  ``bdeps = None`` means ``bdeps[f] = [f]``.
* ``D[f]``: float32 ``[mb][n_f]``, the prior ``p(s_1^f)``.
* ``mb`` is 1 for a model shared by every agent, else the number of agents.

Sequences are drawn from the generative process: ``s_0 ~ D``, ``u_t`` uniform,
``s_{t+1} ~ B[:, s_t, u_t]``, ``o_t^m ~ A_m[:, s_t^{dep(m)}]``.

Seeds: ``SeedSequence([17855, config, case, stream])`` with stream 0 for the
model parameters, 1 for the sequences and 2 for the structure (dimensions and
dependency lists), so that every draw is reproducible on any machine.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence

import numpy as np

SEED_ROOT = 17855


def _rng(cfg: int, case: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_ROOT, cfg, case, stream])))


@dataclasses.dataclass
class Model:
    n: List[int]                 # states per factor
    U: List[int]                 # actions per factor
    K: List[int]                 # outcomes per modality
    deps: List[List[int]]        # ascending factor list per modality
    mb: int                      # 1 = shared by all agents
    A: List[np.ndarray]          # see module docstring
    B: List[np.ndarray]
    D: List[np.ndarray]
    bdeps: Optional[List[List[int]]] = None   # B-dependency lists (None: trivial)

    def bdep(self, f: int) -> List[int]:
        """Factors whose current states condition the next state of f."""
        return list(self.bdeps[f]) if self.bdeps is not None else [f]

    @property
    def trivial_bdeps(self) -> bool:
        return self.bdeps is None or all(list(d) == [f] for f, d in enumerate(self.bdeps))

    @property
    def F(self) -> int:
        return len(self.n)

    @property
    def M(self) -> int:
        return len(self.K)

    @property
    def n_total(self) -> int:
        return int(sum(self.n))

    def agent_slice(self, agents: Sequence[int]) -> "Model":
        """The models of a subset of agents (identity for a shared model)."""
        if self.mb == 1:
            return self
        idx = np.asarray(agents, dtype=np.int64)
        return Model(list(self.n), list(self.U), list(self.K), [list(d) for d in self.deps], len(idx),
                     [np.ascontiguousarray(a[idx]) for a in self.A],
                     [np.ascontiguousarray(b[idx]) for b in self.B],
                     [np.ascontiguousarray(d[idx]) for d in self.D],
                     None if self.bdeps is None else [list(d) for d in self.bdeps])


@dataclasses.dataclass
class Workload:
    name: str
    algos: List[str]             # subset of {"fpi", "vmp", "mmp"}
    model: Model
    obs: np.ndarray              # int32 [b][T][M]
    act: np.ndarray              # int32 [b][max(T-1,0)][F]
    iters: int
    sparse_A: bool = False       # the sparse A layout is also exercised

    @property
    def b(self) -> int:
        return int(self.obs.shape[0])

    @property
    def T(self) -> int:
        return int(self.obs.shape[1])


# ---------------------------------------------------------------------------
# parameter draws
# ---------------------------------------------------------------------------

def _dirichlet_columns(rng: np.random.Generator, alpha: float, shape_outer, k: int, shape_inner) -> np.ndarray:
    """Draw Dirichlet(alpha) vectors of length k along axis len(shape_outer)."""
    g = rng.standard_gamma(alpha, size=tuple(shape_outer) + (k,) + tuple(shape_inner))
    ax = len(shape_outer)
    s = g.sum(axis=ax, keepdims=True)
    # a column of all-zero gammas (possible for small alpha in float64 underflow)
    # becomes uniform
    bad = s <= 0
    if np.any(bad):
        g = np.where(bad, 1.0, g)
        s = g.sum(axis=ax, keepdims=True)
    return g / s


def _sparsify_columns(rng: np.random.Generator, a: np.ndarray, axis: int, p_zero: float) -> np.ndarray:
    """Impose random zeros with probability p_zero, keep one random entry of any
    column that became all-zero, then renormalise the columns (the large shared model)."""
    keep = rng.random(a.shape) >= p_zero
    col_any = keep.any(axis=axis, keepdims=True)
    if not np.all(col_any):
        k = a.shape[axis]
        pick = rng.integers(0, k, size=col_any.shape)
        onehot = np.arange(k).reshape([-1 if i == axis else 1 for i in range(a.ndim)]) == pick
        keep = np.where(col_any, keep, onehot)
    a = np.where(keep, a, 0.0)
    return a / a.sum(axis=axis, keepdims=True)


def make_model(rng: np.random.Generator, n, U, K, deps, mb: int, alpha_A: float = 1.0, alpha_B: float = 1.0,
               sparsity: float = 0.0, uniform_D: bool = True, bdeps=None) -> Model:
    n = [int(x) for x in n]
    U = [int(x) for x in U]
    K = [int(x) for x in K]
    deps = [sorted(int(f) for f in d) for d in deps]
    A = []
    for m, d in enumerate(deps):
        inner = [n[f] for f in d]
        a = _dirichlet_columns(rng, alpha_A, (mb,), K[m], inner)
        if sparsity > 0:
            a = _sparsify_columns(rng, a, 1, sparsity)
        A.append(np.ascontiguousarray(a, dtype=np.float32))
    if bdeps is not None:
        bdeps = [sorted(int(g) for g in d) for d in bdeps]
    B = []
    for f in range(len(n)):
        cond = [n[g] for g in bdeps[f]] if bdeps is not None else [n[f]]
        b = _dirichlet_columns(rng, alpha_B, (mb,), n[f], tuple(cond) + (U[f],))
        B.append(np.ascontiguousarray(b, dtype=np.float32))
    D = []
    for f in range(len(n)):
        if uniform_D:
            d = np.full((mb, n[f]), 1.0 / n[f])
        else:
            d = _dirichlet_columns(rng, 1.0, (mb,), n[f], ())
        D.append(np.ascontiguousarray(d, dtype=np.float32))
    return Model(n, U, K, deps, mb, A, B, D, bdeps)


def _sample_cat(rng: np.random.Generator, p: np.ndarray) -> np.ndarray:
    """One categorical draw per row of p ([b][k], rows sum to ~1)."""
    c = np.cumsum(p.astype(np.float64), axis=1)
    u = rng.random(p.shape[0]) * c[:, -1]
    idx = (c > u[:, None]).argmax(axis=1)
    return idx.astype(np.int32)


def sample_sequences(rng: np.random.Generator, model: Model, b: int, T: int):
    """Actions and observations from the generative process, for b agents."""
    F, M = model.F, model.M
    ai = np.zeros(b, dtype=np.int64) if model.mb == 1 else np.arange(b, dtype=np.int64)
    assert model.mb in (1, b)
    s = np.zeros((b, F), dtype=np.int64)
    for f in range(F):
        s[:, f] = _sample_cat(rng, model.D[f][ai])
    obs = np.zeros((b, T, M), dtype=np.int32)
    act = np.zeros((b, max(T - 1, 0), F), dtype=np.int32)
    for t in range(T):
        for m in range(M):
            # column A_m[a, :, s_dep] of every agent
            col = _gather_col(model.A[m], ai, [s[:, f] for f in model.deps[m]])
            obs[:, t, m] = _sample_cat(rng, col)
        if t + 1 < T:
            prev = s.copy()                                  # every factor moves from the same s_t
            for f in range(F):
                u = rng.integers(0, model.U[f], size=b)
                act[:, t, f] = u
                col = model.B[f][(ai, slice(None)) + tuple(prev[:, g] for g in model.bdep(f)) + (u,)]   # [b][n_f]
                s[:, f] = _sample_cat(rng, col)
    return obs, act


def random_prior(rng: np.random.Generator, n: Sequence[int], b: int, alpha: float = 1.0,
                 p_zero: float = 0.0) -> np.ndarray:
    """A first-step belief per agent, float32 [b][sum n]: each factor's block a
    Dirichlet(alpha) draw, with states set to zero at rate p_zero (one state
    of every block kept) and the block renormalised."""
    out = np.zeros((b, int(sum(n))), dtype=np.float32)
    off = 0
    for nf in n:
        p = rng.dirichlet(np.full(nf, alpha), size=b)
        if p_zero > 0.0:
            zero = rng.random((b, nf)) < p_zero
            zero[np.arange(b), rng.integers(0, nf, size=b)] = False
            p = np.where(zero, 0.0, p)
            p /= p.sum(axis=1, keepdims=True)
        out[:, off:off + nf] = p.astype(np.float32)
        off += nf
    return out


def one_hot_obs(obs: np.ndarray, K: Sequence[int]) -> np.ndarray:
    """Integer outcomes [b][T][M] as soft observation vectors, float32
    [b][T][sum K] (modality m's one-hot block at sum_{m' < m} K_m')."""
    b, T, M = obs.shape
    out = np.zeros((b, T, int(sum(K))), dtype=np.float32)
    k0 = 0
    for m in range(M):
        np.put_along_axis(out[:, :, k0:k0 + K[m]], obs[:, :, m:m + 1].astype(np.int64), 1.0, axis=2)
        k0 += K[m]
    return out


def soft_obs(rng: np.random.Generator, obs: np.ndarray, K: Sequence[int], confidence: float = 0.7,
             alpha: float = 1.0, p_hard: float = 0.0) -> np.ndarray:
    """Soft observation vectors float32 [b][T][sum K] around integer outcomes:
    each block puts `confidence` on the drawn outcome and spreads the rest as a
    Dirichlet(alpha) draw over all outcomes (a noisy sensor's output); blocks
    are one-hot at rate p_hard."""
    b, T, M = obs.shape
    hard = one_hot_obs(obs, K).astype(np.float64)
    out = np.zeros_like(hard)
    k0 = 0
    for m in range(M):
        km = K[m]
        noise = rng.dirichlet(np.full(km, alpha), size=(b, T))
        blk = confidence * hard[:, :, k0:k0 + km] + (1.0 - confidence) * noise
        keep = rng.random((b, T, 1)) < p_hard
        out[:, :, k0:k0 + km] = np.where(keep, hard[:, :, k0:k0 + km], blk)
        k0 += km
    return out.astype(np.float32)


def _gather_col(a: np.ndarray, ai: np.ndarray, coords) -> np.ndarray:
    """a[ai[i], :, coords[0][i], coords[1][i], ...] for every i -> [b][K]."""
    k = a.shape[1]
    inner = a.shape[2:]
    flat = np.zeros(len(ai), dtype=np.int64)
    for c, dim in zip(coords, inner):
        flat = flat * dim + c
    a2 = a.reshape(a.shape[0], k, -1)
    return a2[ai, :, flat]


# ---------------------------------------------------------------------------
# the five workload families
# ---------------------------------------------------------------------------

def _random_subset(rng: np.random.Generator, F: int) -> List[int]:
    while True:
        mask = rng.random(F) < 0.5
        if mask.any():
            return [int(f) for f in np.nonzero(mask)[0]]


def hmm_small(case: int = 0) -> Workload:
    """Single-factor HMM: 4 states, 3 outcomes, 2 actions, T=8, b=1, FPI x16."""
    rm, rs = _rng(1, case, 0), _rng(1, case, 1)
    model = make_model(rm, [4], [2], [3], [[0]], 1, 1.0, 1.0)
    obs, act = sample_sequences(rs, model, 1, 8)
    return Workload("hmm_n4_T8_b1", ["fpi"], model, obs, act, 16)


def two_factor_agents(case: int = 0, b: int = 1024) -> Workload:
    """F=2 (8,6; U=3,1), M=3 (5,7,4) all on both factors, T=10, per-agent models."""
    rm, rs = _rng(2, case, 0), _rng(2, case, 1)
    model = make_model(rm, [8, 6], [3, 1], [5, 7, 4], [[0, 1]] * 3, b, 1.0, 1.0)
    obs, act = sample_sequences(rs, model, b, 10)
    return Workload(f"F2_M3_T10_b{b}", ["vmp"], model, obs, act, 16)


def three_factor_structure(case: int = 0) -> List[List[int]]:
    rd = _rng(3, case, 2)
    return [_random_subset(rd, 3) for _ in range(4)]


# B-dependency lists of the coupled-transition variant of the F=3 workload:
# every factor moves conditioned on itself and on one other factor
THREE_FACTOR_BDEPS = [[0, 1], [1, 2], [0, 2]]


def three_factor_agents(case: int = 0, b: int = 4096, bdeps=None) -> Workload:
    """F=3 (12,10,8; U=4,2,1), M=4 x 16 outcomes on random factor subsets, T=20,
    per-agent Dirichlet(0.5) models.  bdeps: optional B-dependency lists (the
    general transition model; None: each factor on its own previous state)."""
    deps = three_factor_structure(case)
    rm, rs = _rng(3, case, 0), _rng(3, case, 1)
    model = make_model(rm, [12, 10, 8], [4, 2, 1], [16] * 4, deps, b, 0.5, 0.5, bdeps=bdeps)
    obs, act = sample_sequences(rs, model, b, 20)
    tag = "" if bdeps is None else "_bdeps"
    return Workload(f"F3_M4_T20_b{b}{tag}", ["mmp"], model, obs, act, 16)


@dataclasses.dataclass
class SweepSpec:
    n: List[int]
    U: List[int]
    K: List[int]
    deps: List[List[int]]
    T: int

    def a_floats(self) -> int:
        return int(sum(k * int(np.prod([self.n[f] for f in d])) for k, d in zip(self.K, self.deps)))


# seed family of the skewed-regime sweep (the uniform sweep uses 4)
SKEWED_CFG = 46


def _skewed_dims(rd: np.random.Generator, count: int, lo: int = 2, hi: int = 32) -> List[int]:
    """Sizes of the skewed regime (Sec. V-A, fine-grained dimensionality
    sampling): each size comes from the top 10% of [lo, hi] with probability
    1/5, otherwise from the bottom 10%, giving strongly imbalanced shapes."""
    band = max(1, int(round(0.1 * (hi - lo))))
    top = rd.random(count) < 0.2
    high = rd.integers(hi - band, hi + 1, size=count)
    low = rd.integers(lo, lo + band + 1, size=count)
    return [int(h) if t else int(x) for t, h, x in zip(top, high, low)]


def sweep_spec(case: int, regime: str = "uniform") -> SweepSpec:
    """One of the sweep POMDP specifications (case = 0..769).  regime
    "uniform" draws every state and outcome count uniformly from 2..32;
    "skewed" draws them from the extremes of that range (_skewed_dims)."""
    if regime not in ("uniform", "skewed"):
        raise ValueError(f"unknown regime {regime!r}")
    rd = _rng(4 if regime == "uniform" else SKEWED_CFG, case, 2)
    F = int(rd.integers(1, 5))
    if regime == "uniform":
        n = [int(x) for x in rd.integers(2, 33, size=F)]
    else:
        n = _skewed_dims(rd, F)
    U = [int(x) for x in rd.integers(1, 6, size=F)]
    M = int(rd.integers(1, 6))
    if regime == "uniform":
        K = [int(x) for x in rd.integers(2, 33, size=M)]
    else:
        K = _skewed_dims(rd, M)
    deps = [_random_subset(rd, F) for _ in range(M)]
    T = int(rd.integers(1, 21))
    return SweepSpec(n, U, K, deps, T)


N_SWEEP = 770


def sweep_model(case: int, b: int = 256, regime: str = "uniform") -> Workload:
    """Sweep POMDP ``case``: one generative model shared by the b agents."""
    sp = sweep_spec(case, regime)
    cfg = 4 if regime == "uniform" else SKEWED_CFG
    rm, rs = _rng(cfg, case, 0), _rng(cfg, case, 1)
    model = make_model(rm, sp.n, sp.U, sp.K, sp.deps, 1, 1.0, 1.0)
    obs, act = sample_sequences(rs, model, b, sp.T)
    tag = "sweep" if regime == "uniform" else "sweep_skewed"
    return Workload(f"{tag}_case{case}_b{b}", ["fpi", "vmp", "mmp"], model, obs, act, 16)


def large_shared(case: int = 0, b: int = 64, n: int = 32, F: int = 4, M: int = 4, K: int = 32, T: int = 16) -> Workload:
    """Large shared model: F=4 x 32 states (4 actions), M=4 x 32 outcomes, every
    A_m on all factors, 90% random zeros then renormalised columns, T=16."""
    rm, rs = _rng(5, case, 0), _rng(5, case, 1)
    model = make_model(rm, [n] * F, [4] * F, [K] * M, [list(range(F))] * M, 1, 1.0, 1.0, sparsity=0.9)
    obs, act = sample_sequences(rs, model, b, T)
    return Workload(f"shared_F{F}x{n}_M{M}x{K}_T{T}_b{b}", ["vmp", "mmp"], model, obs, act, 16, sparse_A=True)


def random_small(seed: int, F_max: int = 3, n_max: int = 5, M_max: int = 3, K_max: int = 4, T_max: int = 4,
                 b: int = 3, per_agent: Optional[bool] = None, alpha: float = 1.0, sparsity: float = 0.0) -> Workload:
    """Tiny random POMDPs for property tests and brute-force pins."""
    rd = _rng(99, seed, 2)
    F = int(rd.integers(1, F_max + 1))
    n = [int(x) for x in rd.integers(2, n_max + 1, size=F)]
    U = [int(x) for x in rd.integers(1, 4, size=F)]
    M = int(rd.integers(1, M_max + 1))
    K = [int(x) for x in rd.integers(2, K_max + 1, size=M)]
    deps = [_random_subset(rd, F) for _ in range(M)]
    T = int(rd.integers(1, T_max + 1))
    if per_agent is None:
        per_agent = bool(rd.integers(0, 2))
    mb = b if per_agent else 1
    model = make_model(_rng(99, seed, 0), n, U, K, deps, mb, alpha, alpha, sparsity=sparsity,
                       uniform_D=bool(rd.integers(0, 2)))
    obs, act = sample_sequences(_rng(99, seed, 1), model, b, T)
    return Workload(f"small{seed}", ["fpi", "vmp", "mmp"], model, obs, act, int(rd.integers(1, 6)))
