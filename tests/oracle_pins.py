"""Pins of the oracle against results fixed by the paper and by mathematics.

Each ``pin_*`` takes an ``infer(algo, model, obs, act, iters)`` callable (the
oracle, or a deliberately broken copy of it in the mutation tests) and returns
the largest absolute deviation from the independently computed expectation.
Pins of the rolling-inference entry points also use the predictive prior of
the same oracle library (``_predict_of(infer)``).
"""
from __future__ import annotations

import os
from fractions import Fraction

import numpy as np

from paper_2607_17855_amd import synth
import bruteforce as bf

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _hmm(seed, n=4, K=(3,), U=2, T=6, b=2, alpha=1.0, mb=None, uniform_D=False):
    rng = np.random.Generator(np.random.PCG64(seed))
    model = synth.make_model(rng, [n], [U], list(K), [[0]] * len(K), b if mb is None else mb, alpha, alpha,
                             uniform_D=uniform_D)
    obs, act = synth.sample_sequences(rng, model, b, T)
    return model, obs, act


def pin_bayes_filter(infer):
    """F = 1: variational filtering is exact filtering (Sec. III-A update with a
    single factor has no mean-field approximation), so FPI must equal the
    textbook forward algorithm, for any iteration count."""
    err = 0.0
    for seed, K, iters in [(1, (3,), 1), (2, (5, 2), 3), (3, (2, 2, 4), 16)]:
        model, obs, act = _hmm(seed, n=5, K=K, T=7, b=3)
        q = infer("fpi", model, obs, act, iters)
        for a in range(obs.shape[0]):
            alpha = bf.forward_filter([np.float64(A[a]) for A in model.A], np.float64(model.B[0][a]),
                                      np.float64(model.D[0][a]), obs[a], act[a, :, 0])
            err = max(err, float(np.abs(q[a] - alpha).max()))
    return err


def pin_golden_hmm2(infer):
    """Hand-derived two-state filter (tests/golden/hmm2_filter.txt)."""
    vals = {}
    with open(os.path.join(GOLDEN, "hmm2_filter.txt")) as fh:
        for line in fh:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            key, rhs = line.split("=", 1)
            vals[key.strip()] = [float(Fraction(x)) for x in rhs.split()]
    A = np.array([vals["A0"], vals["A1"]], dtype=np.float32)          # A[o][s]
    B = np.array(vals["B"], dtype=np.float32).reshape(2, 2, 1)         # B[i][j][u]
    D = np.array(vals["D"], dtype=np.float32)
    model = synth.Model([2], [1], [2], [[0]], 1, [A[None]], [B[None]], [D[None]])
    obs = np.array(vals["obs"], dtype=np.int32).reshape(1, -1, 1)
    act = np.zeros((1, obs.shape[1] - 1, 1), dtype=np.int32)
    q = infer("fpi", model, obs, act, 4)
    want = np.array([vals["q0"], vals["q1"]])
    # inputs were rounded to float32, so compare at float32 input precision
    return float(np.abs(q[0] - want).max())


def pin_vmp_bruteforce(infer, seeds=range(12)):
    """VMP = the coordinate update of Sec. III-A on the window joint of Sec.
    III-B under a fully factorised q, evaluated by enumerating the joint."""
    err = 0.0
    for seed in seeds:
        # odd seeds carry exact zeros in A and B (the clamped-log reading)
        w = synth.random_small(seed, F_max=3, n_max=3, M_max=3, K_max=3, T_max=3, b=2,
                               sparsity=0.4 if seed % 2 else 0.0)
        ref = bf.vmp_bruteforce(w.model, w.obs, w.act, w.iters)
        q = infer("vmp", w.model, w.obs, w.act, w.iters)
        err = max(err, float(np.abs(q - ref).max()))
    return err


def pin_fpi_bruteforce(infer, seeds=range(12)):
    """FPI = per-step coordinate updates over the enumerated single-step joint."""
    err = 0.0
    for seed in seeds:
        w = synth.random_small(100 + seed, F_max=3, n_max=4, M_max=3, K_max=3, T_max=4, b=2,
                               sparsity=0.4 if seed % 2 else 0.0)
        ref = bf.fpi_bruteforce(w.model, w.obs, w.act, w.iters)
        q = infer("fpi", w.model, w.obs, w.act, w.iters)
        err = max(err, float(np.abs(q - ref).max()))
    return err


def pin_long_dependency_lists(infer):
    """Dependency lists of 5 to 7 factors (the paper's random population draws
    list lengths up to 10, Sec. V-A; any A-dependencies, Sec. III-B): FPI
    against the enumerated single-step joint."""
    err = 0.0
    cases = [
        # (n, deps, K)
        ([2, 2, 3, 2, 2, 2], [[0, 1, 2, 3, 4], [2, 5]], [3, 2]),
        ([2, 3, 2, 2, 2, 2], [[0, 1, 2, 3, 4, 5], [1], [0, 3, 5]], [2, 3, 4]),
        ([2, 2, 2, 2, 2, 2, 3], [[0, 1, 2, 3, 4, 5, 6]], [4]),
    ]
    for i, (n, deps, K) in enumerate(cases):
        rng = np.random.Generator(np.random.PCG64(1700 + i))
        F = len(n)
        model = synth.make_model(rng, n, [2] * F, K, deps, 2, 0.8, 1.0, uniform_D=False)
        obs, act = synth.sample_sequences(rng, model, 2, 3)
        for iters in (1, 4):
            ref = bf.fpi_bruteforce(model, obs, act, iters)
            q = infer("fpi", model, obs, act, iters)
            err = max(err, float(np.abs(q - ref).max()))
    return err


def pin_factorised_exact(infer):
    """Every dependency list a singleton: the joint factorises over factors, so
    filtering is exact per factor and FPI equals a forward filter per factor."""
    rng = np.random.Generator(np.random.PCG64(7))
    n, U, K = [3, 4, 2], [2, 1, 3], [3, 2, 4, 3]
    deps = [[0], [1], [2], [0]]
    b, T = 2, 5
    model = synth.make_model(rng, n, U, K, deps, b, 1.0, 1.0, uniform_D=False)
    obs, act = synth.sample_sequences(rng, model, b, T)
    q = infer("fpi", model, obs, act, 2)
    offs = np.cumsum([0] + n)
    err = 0.0
    for a in range(b):
        for f in range(len(n)):
            ms = [m for m, d in enumerate(deps) if d == [f]]
            alpha = bf.forward_filter([np.float64(model.A[m][a]) for m in ms], np.float64(model.B[f][a]),
                                      np.float64(model.D[f][a]), obs[a][:, ms], act[a, :, f])
            err = max(err, float(np.abs(q[a, :, offs[f]:offs[f + 1]] - alpha).max()))
    return err


def pin_t1_identity(infer):
    """T = 1: no temporal messages, the three schemes coincide and equal the
    single-step mean-field fixed-point iteration (checked by enumeration)."""
    err = 0.0
    for seed in range(6):
        w = synth.random_small(200 + seed, F_max=3, n_max=4, T_max=1, b=2)
        ref = bf.vmp_bruteforce(w.model, w.obs, w.act, w.iters)
        for algo in ("fpi", "vmp", "mmp"):
            err = max(err, float(np.abs(infer(algo, w.model, w.obs, w.act, w.iters) - ref).max()))
    return err


def _iid_model(seed, n=4, U=3, K=(3, 2), T=5, b=2):
    """Single factor whose transition ignores the previous state:
    B[:, j, u] = p_u for every j."""
    rng = np.random.Generator(np.random.PCG64(seed))
    model = synth.make_model(rng, [n], [U], list(K), [[0]] * len(K), b, 1.0, 1.0, uniform_D=False)
    p = rng.dirichlet(np.ones(n), size=(b, U))                   # [b][U][n]
    B = np.repeat(np.transpose(p, (0, 2, 1))[:, :, None, :], n, axis=2)   # [b][i][j][u] = p_u(i)
    model.B[0] = np.ascontiguousarray(B, dtype=np.float32)
    obs, act = synth.sample_sequences(rng, model, b, T)
    return model, obs, act


def pin_iid_closed_forms(infer):
    """Transitions that ignore the previous state: the backward message is
    constant in s and cancels, the forward message is log p_u; hence the closed
    forms  VMP: q_0 ~ L_0 D, q_t ~ L_t p;  MMP: q_0 ~ L_0 D^(1/2), q_t ~ L_t p^(1/2)
    inside the window and L_{T-1} p at its end (L_t = prod_m A_m[o_t])."""
    err = 0.0
    for seed, T in [(11, 5), (12, 2), (13, 6)]:
        model, obs, act = _iid_model(seed, T=T)
        b = obs.shape[0]
        qv = infer("vmp", model, obs, act, 3)
        qm = infer("mmp", model, obs, act, 3)
        for a in range(b):
            B = np.float64(model.B[0][a])
            D = np.float64(model.D[0][a])
            for t in range(T):
                L = np.ones(model.n[0])
                for m in range(model.M):
                    L = L * np.float64(model.A[m][a][obs[a, t, m]])
                prior = D if t == 0 else B[:, 0, act[a, t - 1, 0]]
                v = L * prior
                err = max(err, float(np.abs(qv[a, t] - v / v.sum()).max()))
                w = L * (prior if t == T - 1 else np.sqrt(prior))
                err = max(err, float(np.abs(qm[a, t] - w / w.sum()).max()))
    return err


def pin_mmp_permutation_smoothing(infer):
    """Deterministic cyclic transition s' = pi(s), uniform D, an uninformative
    first outcome and an informative second one (T = 2).  The backward message
    of MMP is the likelihood of the future marginal under the transition, so at
    the fixed point q_0(s) equals the exact smoothing posterior
    p(s_0 = s | o_0, o_1) ~ A[o_1][pi(s)]."""
    n = 3
    pi = np.array([1, 2, 0])                       # a 3-cycle: pi != pi^-1
    B = np.zeros((1, n, n, 1), dtype=np.float32)
    for j in range(n):
        B[0, pi[j], j, 0] = 1.0
    A = np.array([[0.2, 0.2, 0.2],                 # outcome 0: uninformative
                  [0.7, 0.1, 0.3],
                  [0.1, 0.7, 0.5]], dtype=np.float32)
    A /= A.sum(axis=0, keepdims=True)
    D = np.full((1, n), 1.0 / n, dtype=np.float32)
    model = synth.Model([n], [1], [3], [[0]], 1, [A[None]], [B], [D])
    err = 0.0
    for o1 in (1, 2):
        obs = np.array([[[0], [o1]]], dtype=np.int32)
        act = np.zeros((1, 1, 1), dtype=np.int32)
        q = infer("mmp", model, obs, act, 200)
        exact = bf.exact_window_marginals(model, obs[0], act[0], 0)[0]
        want = np.float64(A[o1][pi])
        want /= want.sum()
        err = max(err, float(np.abs(exact - want).max()), float(np.abs(q[0, 0] - want).max()))
    return err


def _relabel_states(model, f, perm):
    """New label i' of factor f's state perm[i'] (state perm[i'] is renamed i')."""
    A = []
    for m, d in enumerate(model.deps):
        a = model.A[m]
        if f in d:
            a = np.take(a, perm, axis=2 + d.index(f))
        A.append(np.ascontiguousarray(a))
    B = list(model.B)
    B[f] = np.ascontiguousarray(np.take(np.take(model.B[f], perm, axis=1), perm, axis=2))
    D = list(model.D)
    D[f] = np.ascontiguousarray(np.take(model.D[f], perm, axis=1))
    return synth.Model(list(model.n), list(model.U), list(model.K), [list(d) for d in model.deps], model.mb, A, B, D)


def _reorder_factors(model, order, act):
    """Factor g of the new model is factor order[g] of the old one."""
    inv = np.argsort(order)
    deps, A = [], []
    for m, d in enumerate(model.deps):
        nd = sorted(int(inv[f]) for f in d)
        # axis of new factor g comes from old factor order[g]
        src = [d.index(int(order[g])) for g in nd]
        A.append(np.ascontiguousarray(np.transpose(model.A[m], [0, 1] + [2 + s for s in src])))
        deps.append(nd)
    nm = synth.Model([model.n[o] for o in order], [model.U[o] for o in order], list(model.K), deps, model.mb, A,
                     [model.B[o] for o in order], [model.D[o] for o in order])
    return nm, np.ascontiguousarray(act[:, :, order])


def pin_invariants(infer):
    """Normalisation, non-negativity, agent-permutation, state-relabelling,
    factor- and modality-reorder equivariance, shared == replicated model, and
    finiteness with exact zeros in A and B."""
    worst = 0.0
    for seed in range(4):
        w = synth.random_small(300 + seed, F_max=3, n_max=5, M_max=3, K_max=4, T_max=5, b=4, per_agent=True,
                               sparsity=0.3 if seed % 2 else 0.0)
        mdl, obs, act = w.model, w.obs, w.act
        offs = np.cumsum([0] + mdl.n)
        for algo in ("fpi", "vmp", "mmp"):
            q = infer(algo, mdl, obs, act, w.iters)
            if not np.all(np.isfinite(q)) or q.min() < 0:
                return np.inf
            for f in range(mdl.F):
                worst = max(worst, float(np.abs(q[..., offs[f]:offs[f + 1]].sum(-1) - 1).max()))
            perm = np.array([3, 1, 0, 2])
            qp = infer(algo, mdl.agent_slice(perm), obs[perm], act[perm], w.iters)
            worst = max(worst, float(np.abs(qp - q[perm]).max()))
            f = int(np.argmax(mdl.n))
            sp = np.random.Generator(np.random.PCG64(seed)).permutation(mdl.n[f])
            qr = infer(algo, _relabel_states(mdl, f, sp), obs, act, w.iters)
            worst = max(worst, float(np.abs(qr[..., offs[f] + np.arange(mdl.n[f])] - q[..., offs[f] + sp]).max()))
            if mdl.F > 1:
                order = np.arange(mdl.F)[::-1].copy()
                m2, act2 = _reorder_factors(mdl, order, act)
                q2 = infer(algo, m2, obs, act2, w.iters)
                offs2 = np.cumsum([0] + m2.n)
                for g, o in enumerate(order):
                    worst = max(worst, float(np.abs(q2[..., offs2[g]:offs2[g + 1]] -
                                                    q[..., offs[o]:offs[o + 1]]).max()))
            if mdl.M > 1:
                mo = np.arange(mdl.M)[::-1].copy()
                m3 = synth.Model(mdl.n, mdl.U, [mdl.K[i] for i in mo], [mdl.deps[i] for i in mo], mdl.mb,
                                 [mdl.A[i] for i in mo], mdl.B, mdl.D)
                q3 = infer(algo, m3, np.ascontiguousarray(obs[:, :, mo]), act, w.iters)
                worst = max(worst, float(np.abs(q3 - q).max()))
    # shared == replicated
    w = synth.random_small(400, F_max=3, n_max=4, b=3, per_agent=False)
    rep = synth.Model(w.model.n, w.model.U, w.model.K, w.model.deps, w.b,
                      [np.repeat(a, w.b, axis=0) for a in w.model.A], [np.repeat(a, w.b, axis=0) for a in w.model.B],
                      [np.repeat(a, w.b, axis=0) for a in w.model.D])
    for algo in ("fpi", "vmp", "mmp"):
        worst = max(worst, float(np.abs(infer(algo, w.model, w.obs, w.act, w.iters) -
                                        infer(algo, rep, w.obs, w.act, w.iters)).max()))
    return worst


def _predict_of(infer):
    """The oracle's predict() on the library that ``infer`` runs."""
    import oracle
    lib = getattr(infer, "keywords", {}).get("lib")
    return lambda model, q, act: oracle.predict(model, q, act, lib=lib)


def pin_online_filter(infer):
    """Rolling inference: FPI is causal, so filtering a window in one call must
    equal filtering it one step per call, each step's prior being the
    predictive prior B q of the previous step's posterior (Sec. III-B: the
    window is the current step plus the steps before it).  The first call
    passes D explicitly as the prior."""
    predict = _predict_of(infer)
    err = 0.0
    for seed in range(4):
        w = synth.random_small(300 + seed, F_max=3, n_max=5, M_max=3, K_max=4, T_max=5, b=3)
        full = infer("fpi", w.model, w.obs, w.act, w.iters)
        offs = np.cumsum([0] + list(w.model.n))
        prior = np.concatenate([np.broadcast_to(np.float64(d[0] if w.model.mb == 1 else d), (w.b, len(d[0])))
                                if w.model.mb == 1 else np.float64(d) for d in w.model.D], axis=1)
        for t in range(w.T):
            step = infer("fpi", w.model, w.obs[:, t:t + 1], w.act[:, :0], w.iters, prior=prior)
            err = max(err, float(np.abs(step[:, 0] - full[:, t]).max()))
            if t + 1 < w.T:
                prior = predict(w.model, step[:, 0], w.act[:, t])
        assert offs[-1] == full.shape[-1]
    return err


def pin_prior_t1(infer):
    """A caller's prior p over a single step: the three schemes coincide (no
    temporal messages besides the prior) and, with one factor, equal Bayes'
    rule A[o] * p / Z for any p."""
    err = 0.0
    for seed in range(3):
        w = synth.random_small(320 + seed, F_max=3, n_max=5, M_max=3, K_max=4, T_max=1, b=3)
        rng = np.random.Generator(np.random.PCG64(seed))
        prior = np.concatenate([rng.dirichlet(np.ones(n), size=w.b) for n in w.model.n], axis=1)
        ref = infer("fpi", w.model, w.obs[:, :1], w.act[:, :0], w.iters, prior=prior)
        for algo in ("vmp", "mmp"):
            q = infer(algo, w.model, w.obs[:, :1], w.act[:, :0], w.iters, prior=prior)
            err = max(err, float(np.abs(q - ref).max()))
    for seed, K in [(11, (3,)), (12, (4, 2))]:
        model, obs, act = _hmm(seed, n=5, K=K, T=1, b=3)
        rng = np.random.Generator(np.random.PCG64(seed))
        prior = rng.dirichlet(np.ones(5), size=3)
        prior[0, 1] = 0.0   # a zero prior state stays at zero
        prior[0] /= prior[0].sum()
        q = infer("fpi", model, obs, act, 2, prior=prior)
        for a in range(3):
            post = prior[a].copy()
            for m, A in enumerate(model.A):
                post = post * np.float64(A[a][obs[a, 0, m]])
            err = max(err, float(np.abs(q[a, 0] - post / post.sum()).max()))
    return err


def pin_damped_filter(infer):
    """Damping q <- (1 - tau) q + tau q_new with one factor: FPI's target at
    step t, Bayes' rule A[o_t] * prior_t / Z, does not depend on the current
    iterate, so K sweeps from the uniform start leave
    q_t = target + (1 - tau)^K (uniform - target) exactly, and the next
    step's prior is B q_t of that (not yet converged) marginal."""
    err = 0.0
    for seed, K, iters, tau in [(21, (3,), 1, 0.3), (22, (5, 2), 4, 0.7), (23, (2, 2, 4), 3, 0.5)]:
        model, obs, act = _hmm(seed, n=5, K=K, T=6, b=3)
        q = infer("fpi", model, obs, act, iters, damping=tau)
        n = model.n[0]
        for a in range(obs.shape[0]):
            B = np.float64(model.B[0][a])
            pred = np.float64(model.D[0][a])
            for t in range(obs.shape[1]):
                lik = np.ones(n)
                for m, A in enumerate(model.A):
                    lik = lik * np.float64(A[a][obs[a, t, m]])
                target = lik * pred / (lik * pred).sum()
                want = target + (1.0 - tau) ** iters * (np.full(n, 1.0 / n) - target)
                err = max(err, float(np.abs(q[a, t] - want).max()))
                if t + 1 < obs.shape[1]:
                    pred = B[:, :, act[a, t, 0]] @ want
    return err


def pin_damped_iid(infer):
    """Damping with transitions that ignore the previous state: the VMP and
    MMP targets (the closed forms of pin_iid_closed_forms) do not depend on
    the iterate, so K damped sweeps give target + (1 - tau)^K (uniform - target)."""
    err = 0.0
    for seed, T, iters, tau in [(31, 5, 3, 0.4), (32, 2, 1, 0.8), (33, 4, 6, 0.25)]:
        model, obs, act = _iid_model(seed, T=T)
        b, n = obs.shape[0], model.n[0]
        qv = infer("vmp", model, obs, act, iters, damping=tau)
        qm = infer("mmp", model, obs, act, iters, damping=tau)
        shrink = (1.0 - tau) ** iters
        for a in range(b):
            B = np.float64(model.B[0][a])
            D = np.float64(model.D[0][a])
            for t in range(T):
                L = np.ones(n)
                for m in range(model.M):
                    L = L * np.float64(model.A[m][a][obs[a, t, m]])
                prior = D if t == 0 else B[:, 0, act[a, t - 1, 0]]
                for q, tgt in ((qv, L * prior), (qm, L * (prior if t == T - 1 else np.sqrt(prior)))):
                    tgt = tgt / tgt.sum()
                    err = max(err, float(np.abs(q[a, t] - (tgt + shrink * (1.0 / n - tgt))).max()))
    return err


def pin_damped_fixed_point(infer):
    """A fixed point of the plain update is a fixed point of the damped one:
    on models where the plain Jacobi iteration converges, the damped
    iteration converges to the same marginals (VMP and MMP, several factors,
    a window of several steps).  Convergence of each run is checked too."""
    err = 0.0
    for seed in (41, 42, 43):
        w = synth.random_small(seed, F_max=3, n_max=4, M_max=3, K_max=3, T_max=4, b=2)
        for algo in ("vmp", "mmp"):
            plain = infer(algo, w.model, w.obs, w.act, 300)
            plain1 = infer(algo, w.model, w.obs, w.act, 301)
            damped = infer(algo, w.model, w.obs, w.act, 600, damping=0.5)
            damped1 = infer(algo, w.model, w.obs, w.act, 601, damping=0.5)
            err = max(err, float(np.abs(plain - plain1).max()), float(np.abs(damped - damped1).max()),
                      float(np.abs(plain - damped).max()))
    return err


def _soft_of(infer):
    """The oracle's infer_soft() on the library that ``infer`` runs."""
    import oracle
    lib = getattr(infer, "keywords", {}).get("lib")
    return lambda *args, **kw: oracle.infer_soft(*args, lib=lib, **kw)


def pin_soft_onehot(infer):
    """One-hot observation vectors are integer observations: the merged
    log-likelihood sum_o o[o] log A[o] picks one slice (Sec. III-C, the
    observation vector of the running example), so every algorithm must give
    the integer-observation result exactly, on the same oracle."""
    infer_soft = _soft_of(infer)
    err = 0.0
    for seed in range(4):
        w = synth.random_small(400 + seed, F_max=3, n_max=4, M_max=3, K_max=4, T_max=4, b=3)
        oh = synth.one_hot_obs(w.obs, w.model.K)
        for algo in ("fpi", "vmp", "mmp"):
            err = max(err, float(np.abs(infer_soft(algo, w.model, oh, w.act, w.iters) -
                                        infer(algo, w.model, w.obs, w.act, w.iters)).max()))
    return err


def pin_soft_bruteforce(infer):
    """Soft observations against enumeration: the observation term of the
    joint becomes the expected log-likelihood sum_o w[o] log A[o, s_dep]
    (computed by tensordot in the checker), and VMP / FPI are the mean-field
    updates over that enumerated joint; MMP equals them for a single step."""
    infer_soft = _soft_of(infer)
    err = 0.0
    for seed in range(6):
        w = synth.random_small(420 + seed, F_max=3, n_max=4, M_max=3, K_max=4, T_max=3, b=2)
        rng = np.random.Generator(np.random.PCG64(seed))
        so = synth.soft_obs(rng, w.obs, w.model.K, confidence=0.5, p_hard=0.2).astype(np.float64)
        err = max(err, float(np.abs(infer_soft("vmp", w.model, so, w.act, w.iters) -
                                    bf.vmp_bruteforce(w.model, so, w.act, w.iters, soft=True)).max()))
        err = max(err, float(np.abs(infer_soft("fpi", w.model, so, w.act, w.iters) -
                                    bf.fpi_bruteforce(w.model, so, w.act, w.iters, soft=True)).max()))
        ref1 = bf.vmp_bruteforce(w.model, so[:, :1], w.act[:, :0], w.iters, soft=True)
        err = max(err, float(np.abs(infer_soft("mmp", w.model, so[:, :1], w.act[:, :0], w.iters) - ref1).max()))
    return err


def pin_soft_filter(infer):
    """One factor with soft evidence: FPI is exact filtering with the
    geometric likelihood L_t(s) = prod_m prod_o A_m[o, s]^(w_{t,m}[o])
    (the exponential of the expected log-likelihood)."""
    infer_soft = _soft_of(infer)
    err = 0.0
    for seed, K in [(51, (3,)), (52, (4, 2)), (53, (2, 5, 3))]:
        model, obs, act = _hmm(seed, n=5, K=K, T=6, b=3)
        rng = np.random.Generator(np.random.PCG64(seed))
        so = synth.soft_obs(rng, obs, model.K, confidence=0.4).astype(np.float64)
        q = infer_soft("fpi", model, so, act, 2)
        for a in range(obs.shape[0]):
            B = np.float64(model.B[0][a])
            pred = np.float64(model.D[0][a])
            for t in range(obs.shape[1]):
                lik = np.ones(5)
                k0 = 0
                for m, A in enumerate(model.A):
                    Aa = np.float64(A[a])                        # [K][n]
                    wv = so[a, t, k0:k0 + model.K[m]]
                    lik = lik * np.prod(Aa ** wv[:, None], axis=0)
                    k0 += model.K[m]
                post = lik * pred / (lik * pred).sum()
                err = max(err, float(np.abs(q[a, t] - post).max()))
                if t + 1 < obs.shape[1]:
                    pred = B[:, :, act[a, t, 0]] @ post
    return err


def _bdep_model(seed, F, n_max=4, M_max=3, K_max=3, T=4, b=2, singleton_A=False, lists=None):
    """Small model with random B-dependency lists (random non-empty subsets)."""
    rd = np.random.Generator(np.random.PCG64(seed))
    n = [int(x) for x in rd.integers(2, n_max + 1, size=F)]
    U = [int(x) for x in rd.integers(1, 3, size=F)]
    if singleton_A:
        deps = [[f] for f in range(F)]
    else:
        deps = [sorted(set(int(g) for g in rd.choice(F, size=int(rd.integers(1, F + 1)), replace=False)))
                for _ in range(int(rd.integers(1, M_max + 1)))]
    K = [int(x) for x in rd.integers(2, K_max + 1, size=len(deps))]
    if lists is None:
        lists = [sorted(set(int(g) for g in rd.choice(F, size=int(rd.integers(1, F + 1)), replace=False)))
                 for _ in range(F)]
    model = synth.make_model(rd, n, U, K, deps, b, 1.0, 1.0, uniform_D=False, bdeps=lists)
    obs, act = synth.sample_sequences(rd, model, b, T)
    return model, obs, act


def pin_bdeps_trivial_lists(infer):
    """Listing every factor's own previous state ({f}) through the general
    B-dependency path is the trivial model, result for result."""
    err = 0.0
    for seed in range(4):
        w = synth.random_small(500 + seed, F_max=3, n_max=4, T_max=5, b=3)
        m = w.model
        mg = synth.Model(m.n, m.U, m.K, m.deps, m.mb, m.A, m.B, m.D, [[f] for f in range(m.F)])
        for algo in ("fpi", "vmp", "mmp"):
            err = max(err, float(np.abs(infer(algo, mg, w.obs, w.act, w.iters) -
                                        infer(algo, m, w.obs, w.act, w.iters)).max()))
    return err


def pin_bdeps_bruteforce(infer):
    """General B-dependencies against enumeration: the transition terms of
    the joint become log B_f[s_t^f][s_{t-1}^{dep(f)}] (Sec. III-B), VMP is the
    mean-field update over that joint, and FPI uses the predictive marginal
    of the enumerated previous-step posterior."""
    err = 0.0
    for seed in range(8):
        model, obs, act = _bdep_model(600 + seed, F=2 + seed % 2, T=3 if seed % 2 else 4)
        err = max(err, float(np.abs(infer("vmp", model, obs, act, 5) -
                                    bf.vmp_bruteforce(model, obs, act, 5)).max()))
        err = max(err, float(np.abs(infer("fpi", model, obs, act, 4) -
                                    bf.fpi_bruteforce(model, obs, act, 4)).max()))
    return err


def pin_bdeps_uninformative_transitions(infer):
    """Transitions that ignore every dependency (B_f[s][s_dep][u] = p_u(s))
    with a factorised likelihood (one modality per factor): every backward
    message is constant in s and cancels, so
      VMP: q_{t,f} ~ L_{t,f} p_f  (D_f at t = 0);
      MMP: q_{t,f} ~ L_{t,f} p_f^(1 / (1 + c_f)) inside the window, with c_f
           the number of factors whose B-dependency list holds f (the mean
           of the forward message and the c_f backward ones), L p at t = T-1."""
    err = 0.0
    for seed, lists in [(31, [[0, 1], [0, 1], [1, 2]]), (32, [[1], [0, 1, 2], [0, 1]]), (33, [[0, 1], [0]])]:
        F = len(lists)
        model, obs, act = _bdep_model(seed, F=F, T=5, b=2, singleton_A=True, lists=lists)
        rd = np.random.Generator(np.random.PCG64(seed + 100))
        for f in range(F):   # B_f constant over the dependency states
            shp = model.B[f].shape
            p = rd.dirichlet(np.ones(shp[1]), size=(shp[0], shp[-1]))       # [mb][U][n_f]
            p = np.transpose(p, (0, 2, 1)).reshape(shp[0], shp[1], *([1] * (len(shp) - 3)), shp[-1])
            model.B[f] = np.ascontiguousarray(np.broadcast_to(p, shp), dtype=np.float32)
        obs, act = synth.sample_sequences(rd, model, 2, 5)
        children = [sum(f in d for d in lists) for f in range(F)]
        qv = infer("vmp", model, obs, act, 3)
        qm = infer("mmp", model, obs, act, 3)
        offs = np.cumsum([0] + list(model.n))
        T = obs.shape[1]
        for a in range(obs.shape[0]):
            for t in range(T):
                for f in range(F):
                    L = np.float64(model.A[f][a][obs[a, t, f]])
                    if t == 0:
                        prior = np.float64(model.D[f][a])
                    else:
                        prior = np.float64(model.B[f][a][(slice(None),) + (0,) * (model.B[f].ndim - 3) +
                                                        (act[a, t - 1, f],)])
                    v = L * prior
                    err = max(err, float(np.abs(qv[a, t, offs[f]:offs[f + 1]] - v / v.sum()).max()))
                    c = children[f] if t + 1 < T else 0
                    wm = L * prior ** (1.0 / (1 + c))
                    err = max(err, float(np.abs(qm[a, t, offs[f]:offs[f + 1]] - wm / wm.sum()).max()))
    return err


def pin_predict_bruteforce(infer):
    """Predictive prior with B-dependency lists (and trivial ones) against
    enumeration of the full joint of the current states under the factorised
    marginals; per-agent and shared models, several agents with different
    marginals and actions."""
    predict = _predict_of(infer)
    err = 0.0
    for seed in range(6):
        F = 2 + seed % 2
        lists = [[f] for f in range(F)] if seed == 5 else None   # explicit trivial lists too
        model, obs, act = _bdep_model(640 + seed, F=F, T=2, b=3, lists=lists)
        if seed % 3 == 2:   # one model shared by the agents
            model = synth.Model(model.n, model.U, model.K, model.deps, 1, [x[:1] for x in model.A],
                                [x[:1] for x in model.B], [x[:1] for x in model.D], model.bdeps)
        rd = np.random.Generator(np.random.PCG64(seed + 900))
        q = np.concatenate([rd.dirichlet(np.ones(n), size=3) for n in model.n], axis=1)
        u = np.stack([rd.integers(0, U, size=3) for U in model.U], axis=1).astype(np.int32)
        err = max(err, float(np.abs(predict(model, q, u) - bf.predictive_bruteforce(model, q, u)).max()))
    return err


def pin_online_filter_bdeps(infer):
    """Rolling inference with B-dependency lists: FPI stays causal, so the
    window filtered in one call equals one-step calls chained through the
    predictive prior of the previous step's posterior (whose factors are
    coupled through the lists)."""
    predict = _predict_of(infer)
    err = 0.0
    for seed in range(4):
        model, obs, act = _bdep_model(660 + seed, F=2 + seed % 2, T=4, b=3)
        full = infer("fpi", model, obs, act, 4)
        prior = np.concatenate([np.float64(d) for d in model.D], axis=1)
        for t in range(obs.shape[1]):
            step = infer("fpi", model, obs[:, t:t + 1], act[:, :0], 4, prior=prior)
            err = max(err, float(np.abs(step[:, 0] - full[:, t]).max()))
            if t + 1 < obs.shape[1]:
                prior = predict(model, step[:, 0], act[:, t])
    return err


ALL_PINS = {
    "bayes_filter": (pin_bayes_filter, 1e-12),
    "golden_hmm2": (pin_golden_hmm2, 1e-7),
    "vmp_bruteforce": (pin_vmp_bruteforce, 1e-12),
    "fpi_bruteforce": (pin_fpi_bruteforce, 1e-12),
    "factorised_exact": (pin_factorised_exact, 1e-12),
    "long_dependency_lists": (pin_long_dependency_lists, 1e-12),
    "t1_identity": (pin_t1_identity, 1e-12),
    "iid_closed_forms": (pin_iid_closed_forms, 1e-12),
    "mmp_permutation_smoothing": (pin_mmp_permutation_smoothing, 1e-10),
    "invariants": (pin_invariants, 1e-12),
    "online_filter": (pin_online_filter, 1e-12),
    "prior_t1": (pin_prior_t1, 1e-12),
    "damped_filter": (pin_damped_filter, 1e-12),
    "damped_iid": (pin_damped_iid, 1e-12),
    "damped_fixed_point": (pin_damped_fixed_point, 1e-10),
    "soft_onehot": (pin_soft_onehot, 0.0),
    "soft_bruteforce": (pin_soft_bruteforce, 1e-12),
    "soft_filter": (pin_soft_filter, 1e-12),
    "bdeps_trivial_lists": (pin_bdeps_trivial_lists, 0.0),
    "bdeps_bruteforce": (pin_bdeps_bruteforce, 1e-12),
    "bdeps_uninformative_transitions": (pin_bdeps_uninformative_transitions, 1e-12),
    "predict_bruteforce": (pin_predict_bruteforce, 1e-12),
    "online_filter_bdeps": (pin_online_filter_bdeps, 1e-12),
}
