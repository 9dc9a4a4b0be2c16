"""Independent NumPy checkers used to pin the oracle (tiny inputs only).

Nothing here shares code with the oracle: the joint distribution of Sec. III-B
is enumerated explicitly over every hidden variable, and the mean-field update
of Sec. III-A (log q(s^f) = E_{q(s^{\\f})}[log p(o, s)] + const) is evaluated by
brute-force expectation over that enumerated joint.  The textbook forward
algorithm (exact HMM filtering) is written out separately.
"""
from __future__ import annotations

import itertools
import string

import numpy as np

EPS = 1e-16


def LN(x):
    """Clamped log: the reading that a zero probability contributes log(1e-16)."""
    return np.log(np.maximum(np.asarray(x, dtype=np.float64), EPS))


def _bdep(model, f):
    bd = getattr(model, "bdeps", None)
    return list(bd[f]) if bd is not None else [f]


def _agent(arr, mb, a):
    return np.asarray(arr[0 if mb == 1 else a], dtype=np.float64)


def obs_loglik(model, a, m, obs_t, soft=False):
    """Observation term of modality m at one step, an array over s_dep:
    log A_m[o] for an integer outcome, or for a soft observation (obs_t the
    concatenated vectors [sum K]) its expectation sum_o w[o] log A_m[o]."""
    LA = LN(_agent(model.A[m], model.mb, a))                   # [K][s_d1]..[s_dk]
    if not soft:
        return LA[obs_t[m]]
    k0 = int(sum(model.K[:m]))
    w = np.asarray(obs_t[k0:k0 + model.K[m]], dtype=np.float64)
    return np.tensordot(w, LA, axes=(0, 0))


def window_log_joint(model, obs_a, act_a, a, soft=False):
    """log p(o_{0:T-1}, s_{0:T-1} | u) of one agent as a dense array with one
    axis per hidden variable (t, f), ordered t-major (with soft observations
    obs_a is [T][sum K] and each observation term is obs_loglik's expectation)."""
    T = obs_a.shape[0]
    F = len(model.n)
    shape = [model.n[f] for t in range(T) for f in range(F)]
    lp = np.zeros(shape)

    def ax(t, f):
        return t * F + f

    def add(term, axes):
        # broadcast `term` (whose axes are `axes`, in that order) into lp
        order = np.argsort(axes)
        term = np.transpose(term, order)
        axes_sorted = [axes[i] for i in order]
        view = [1] * len(shape)
        for i, x in enumerate(axes_sorted):
            view[x] = shape[x]
        return lp + term.reshape(view)

    for f in range(F):
        lp = add(LN(_agent(model.D[f], model.mb, a)), [ax(0, f)])
    for t in range(1, T):
        for f in range(F):
            # B_f[s_t^f][s_{t-1}^{g_1}]..[s_{t-1}^{g_k}] (g: B-dependency list, {f} if trivial)
            Bf = _agent(model.B[f], model.mb, a)[..., act_a[t - 1, f]]
            lp = add(LN(Bf), [ax(t, f)] + [ax(t - 1, g) for g in _bdep(model, f)])
    for t in range(T):
        for m, d in enumerate(model.deps):
            lp = add(obs_loglik(model, a, m, obs_a[t], soft), [ax(t, f) for f in d])
    return lp


def expected_given(lp, q_list, v):
    """E_{prod_{w != v} q_w}[lp | x_v] for every value of variable v."""
    nv = lp.ndim
    letters = string.ascii_letters[:nv]
    operands = [lp]
    subs = [letters]
    for w in range(nv):
        if w == v:
            continue
        operands.append(q_list[w])
        subs.append(letters[w])
    expr = ",".join(subs) + "->" + letters[v]
    return np.einsum(expr, *operands, optimize=True)


def softmax(v):
    v = v - v.max()
    e = np.exp(v)
    return e / e.sum()


def vmp_bruteforce(model, obs, act, iters, soft=False):
    """Mean-field (Jacobi) coordinate updates over the enumerated window joint."""
    b, T, _ = obs.shape
    F = len(model.n)
    out = np.zeros((b, T, sum(model.n)))
    offs = np.cumsum([0] + list(model.n))
    for a in range(b):
        lp = window_log_joint(model, obs[a], act[a] if T > 1 else None, a, soft)
        q = [np.full(model.n[f], 1.0 / model.n[f]) for t in range(T) for f in range(F)]
        for _ in range(iters):
            q = [softmax(expected_given(lp, q, v)) for v in range(T * F)]
        for t in range(T):
            for f in range(F):
                out[a, t, offs[f]:offs[f + 1]] = q[t * F + f]
    return out


def fpi_bruteforce(model, obs, act, iters, soft=False):
    """Variational filtering: per time step, mean-field updates over the
    enumerated single-step joint  p(o_t | s_t) prod_f p_{t,f}(s_t^f), with the
    predictive prior p_{t,f} = B_f[u_{t-1}] q_{t-1,f} (D at t = 0)."""
    b, T, _ = obs.shape
    F = len(model.n)
    out = np.zeros((b, T, sum(model.n)))
    offs = np.cumsum([0] + list(model.n))
    for a in range(b):
        prev = None
        for t in range(T):
            lp = np.zeros(model.n)
            for f in range(F):
                if t == 0:
                    prior = _agent(model.D[f], model.mb, a)
                else:
                    # predictive marginal: B_f contracted with the previous step's
                    # marginals of its B-dependencies
                    Bf = _agent(model.B[f], model.mb, a)[..., act[a, t - 1, f]]
                    dl = _bdep(model, f)
                    letters = string.ascii_letters[1:1 + len(dl)]
                    prior = np.einsum("a" + letters + "," + ",".join(letters) + "->a", Bf,
                                      *[prev[g] for g in dl])
                view = [1] * F
                view[f] = model.n[f]
                lp = lp + LN(prior).reshape(view)
            for m, d in enumerate(model.deps):
                Am = obs_loglik(model, a, m, obs[a, t], soft)
                view = [1] * F
                for f in d:
                    view[f] = model.n[f]
                lp = lp + Am.reshape(view)
            q = [np.full(model.n[f], 1.0 / model.n[f]) for f in range(F)]
            for _ in range(iters):
                q = [softmax(expected_given(lp, q, f)) for f in range(F)]
            for f in range(F):
                out[a, t, offs[f]:offs[f + 1]] = q[f]
            prev = q
    return out


def forward_filter(A_list, B, D, obs, act):
    """Textbook HMM forward algorithm (single hidden factor): normalised
    filtering marginals alpha_t = p(s_t | o_{0:t}, u_{0:t-1}).
    A_list: list of [K_m][n]; B: [n][n][U] with B[i][j][u] = P(i | j, u); D: [n]."""
    T = obs.shape[0]
    n = D.shape[0]
    alpha = np.zeros((T, n))
    pred = np.asarray(D, dtype=np.float64)
    for t in range(T):
        if t > 0:
            pred = B[:, :, act[t - 1]] @ alpha[t - 1]
        lik = np.ones(n)
        for m, A in enumerate(A_list):
            lik = lik * A[obs[t, m]]
        post = lik * pred
        alpha[t] = post / post.sum()
    return alpha


def exact_window_marginals(model, obs_a, act_a, a):
    """Exact posterior marginals p(s_{t,f} | o_{0:T-1}, u) of one agent."""
    lp = window_log_joint(model, obs_a, act_a, a)
    p = np.exp(lp - lp.max())
    p /= p.sum()
    T = obs_a.shape[0]
    F = len(model.n)
    res = []
    for t in range(T):
        for f in range(F):
            v = t * F + f
            res.append(p.sum(axis=tuple(w for w in range(p.ndim) if w != v)))
    return res


def all_assignments(shape):
    return itertools.product(*[range(s) for s in shape])


def predictive_bruteforce(model, q, act):
    """Predictive marginal of every factor at the next step, by enumerating
    the joint of ALL current states under the factorised q (Sec. III-B
    transition model: s_{t+1}^f ~ B_f[:, s_t^{list(f)}, u_f]):
      p_f(i) = sum_{s_0..s_{F-1}} prod_g q_g(s_g) B_f[i][s_{list(f)}][u_f].
    q: [b][sum n], act: [b][F]; returns [b][sum n] (float64)."""
    F = len(model.n)
    offs = np.cumsum([0] + list(model.n))
    b = q.shape[0]
    out = np.zeros((b, int(offs[-1])))
    for a in range(b):
        for joint in itertools.product(*[range(n) for n in model.n]):
            w = 1.0
            for g in range(F):
                w *= float(q[a, offs[g] + joint[g]])
            for f in range(F):
                Bf = _agent(model.B[f], model.mb, a)
                cond = tuple(joint[g] for g in _bdep(model, f))
                out[a, offs[f]:offs[f + 1]] += w * Bf[(slice(None),) + cond + (int(act[a, f]),)]
    return out
