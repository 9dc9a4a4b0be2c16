/*
 * Reference ("oracle") implementation of the discrete HMM/POMDP belief updates
 * of "A Hardware-oriented Approach for Efficient Bayesian Inference
 * Computation and Deployment": variational filtering (FPI), variational
 * message passing (VMP) and marginal message passing (MMP).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
 * CPU definition that the GPU library is checked against.  It is compiled by
 * the build step, called only from the tests, the smoke check and the CPU
 * baseline leg of the benchmark, and it shares no code, header or table with
 * the GPU library (neither includes nor links the other).
 *
 * Everything is computed in double precision, in the looped per-modality
 * form (Sec. III-C, the "original" loop of contractions that the merged
 * layouts reproduce), one agent at a time (OpenMP over agents only).
 *
 * Model (Sec. III-B, the factorised joint over o_{1:T}, s_{1:T} given u):
 *   A[m] : [mb][K_m][n_{d1}]..[n_{dk}]   P(o^m | s^{d1..dk}), dep list ascending
 *   B[f] : [mb][n_f][n_f][U_f]           B[i][j][u] = P(s_{t+1}=i | s_t=j, u)
 *   D[f] : [mb][n_f]                     p(s_1)
 *   mb = 1 (shared by all agents) or the number of agents.
 *   obs  : [b][T][M] int,  act : [b][T-1][F] int,  q : [b][T][sum n_f].
 *
 * Readings of points the paper leaves open (the paper gives only the generic
 * coordinate update of Sec. III-A and the joint of Sec. III-B):
 *   LN(x) = log(max(x, 1e-16))  (log of zero is clamped, never -inf)
 *   q initialised uniform; fixed iteration count; Jacobi schedule (every
 *   marginal of iteration k is computed from the marginals of iteration k-1);
 *   no damping unless asked for (below).
 *   Likelihood message (Sec. IV: marginalisation of the log-likelihood under
 *   the other factors' marginals, summed over the Markov blanket):
 *     lam_{t,f}(s) = sum_{m: f in dep(m)} sum_{s_dep: s_f = s}
 *                    LN(A_m[o_{t,m}, s_dep]) * prod_{g in dep(m), g != f} q_{t,g}(s_g)
 *   FPI: for t = 0..T-1 in order, prior p_{t,f} = D_f (t = 0) or
 *        B_f[:,:,u_{t-1,f}] q_{t-1,f} (final marginal of step t-1);
 *        q_t <- uniform, then iters times q_{t,f} = softmax(lam_{t,f} + LN(p_{t,f})).
 *   VMP: the generic update of Sec. III-A applied to the joint of Sec. III-B
 *        under q = prod_{t,f} q_{t,f}:
 *        q_{t,f} = softmax(lam + fwd + bwd),
 *        fwd = LN(D_f) (t = 0) else sum_{s'} LN(B_f[s, s', u_{t-1}]) q_{t-1,f}(s'),
 *        bwd = 0 (t = T-1) else sum_{s''} q_{t+1,f}(s'') LN(B_f[s'', s, u_t]).
 *   MMP: fwd = LN(D_f) (t = 0) else LN(B_f[:,:,u_{t-1}] q_{t-1,f}),
 *        bwd = LN(B_f[:,:,u_t]^T q_{t+1,f}) (t < T-1),
 *        q_{t,f} = softmax(lam + mean of the temporal messages present at t):
 *        (fwd + bwd)/2 for t < T-1, fwd alone at t = T-1.
 *   Rolling inference (the window of Sec. III-B is the current step and the
 *   h steps before it): a caller may replace D_f by its own prior over the
 *   window's first step (every LN(D_f) above becomes LN(prior_f)), typically
 *   the predictive prior B_f[:,:,u] q_f of an earlier marginal (orc_predict).
 *   B-dependencies (orc_infer_general): B_f may condition s_{t+1}^f on a
 *   list of factors g_1 < .. < g_k at t (the general transition model of
 *   Sec. III-B; the list {f} is the trivial case above).  Then, with
 *   E[.] the expectation under the factorised q of the step named,
 *     VMP fwd_{t,f}(s) = E_{q_{t-1}}[LN B_f[s][s_dep]],
 *         bwd_{t,f}(s) = sum over the factors j whose list holds f of
 *                        E_{q_{t+1,j}, q_{t,dep(j) \ f}}[LN B_j[s''][s_dep, s_f = s]];
 *     MMP uses the logs of the same expectations of B (not of LN B) and the
 *         mean of the forward message and of the backward messages present;
 *     FPI's prior is the predictive marginal E_{q_{t-1}}[B_f[s][s_dep]].
 *   Soft observations (orc_infer_soft): o_{t,m} is a vector over the K_m
 *   outcomes and every LN(A_m[o_{t,m}, s_dep]) above becomes the expected
 *   log-likelihood sum_o o_{t,m}[o] LN(A_m[o, s_dep]) (the log(A) . o
 *   contraction of Sec. III-C); an integer outcome is the one-hot vector.
 *   Damping (optional, step size tau in (0, 1]): every sweep mixes the new
 *   marginal with the current one, q <- (1 - tau) q + tau q_new, where q_new
 *   is the softmax above computed from the current q; tau = 1 is the plain
 *   update.  A fixed point of the plain update is one of the damped update.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_EPS 1e-16
#define ORC_MAX_RANK 32

enum { ORC_FPI = 0, ORC_VMP = 1, ORC_MMP = 2 };

typedef struct {
    int F, M, mb;
    const int *n, *U, *K, *dep_off, *dep;
    const double *const *A;
    const double *const *B;
    const double *const *D;
    const int *bdep_off, *bdep;   /* B-dependency lists; NULL: bdep(f) = {f} */
} orc_model;

/* B-dependency list of factor f: *k entries */
static const int *bdeps_of(const orc_model *md, int f, int *k)
{
    if (md->bdep_off) {
        *k = md->bdep_off[f + 1] - md->bdep_off[f];
        return md->bdep + md->bdep_off[f];
    }
    *k = 1;
    return NULL;   /* trivial: the list is {f} */
}

static double LN(double x) { return log(x > ORC_EPS ? x : ORC_EPS); }

/* In-place softmax over v[0..n-1]. */
static void softmax(double *v, int n)
{
    double mx = v[0];
    for (int i = 1; i < n; ++i)
        if (v[i] > mx) mx = v[i];
    double s = 0.0;
    for (int i = 0; i < n; ++i) {
        v[i] = exp(v[i] - mx);
        s += v[i];
    }
    for (int i = 0; i < n; ++i) v[i] /= s;
}

static size_t slice_size(const orc_model *md, int m)
{
    size_t p = 1;
    for (int i = md->dep_off[m]; i < md->dep_off[m + 1]; ++i) p *= (size_t)md->n[md->dep[i]];
    return p;
}

/* Observations of one agent: integer outcomes hard[T][M], or soft ones,
 * soft[T][sum K] (a distribution over modality m's outcomes at koff[m]). */
typedef struct {
    const int *hard;
    const double *soft;
    const int *koff;
    int ksum;
} orc_obs;

/* Log-likelihood tensors of context t, concatenated over the modalities
 * (modality m's values at poff[m], row-major over s_dep like A):
 *   integer outcome o:    ll_m(s_dep) = LN(A_m[o, s_dep]);
 *   soft observation o_m: ll_m(s_dep) = sum_o o_m[o] LN(A_m[o, s_dep]),
 * i.e. the product log(A_block) . o_concat of the block-diagonal merge
 * (Sec. III-C and Appendix: each A_m reshaped to p_m x K_m, the blocks on
 * the diagonal, the observation vectors concatenated). */
static void context_loglik(const orc_model *md, int a, const orc_obs *ob, int t, const size_t *poff, double *ll)
{
    int am = md->mb == 1 ? 0 : a;
    for (int m = 0; m < md->M; ++m) {
        const size_t P = slice_size(md, m);
        const double *Am = md->A[m] + (size_t)am * md->K[m] * P;   /* [K_m][P] */
        double *out = ll + poff[m];
        if (ob->hard) {
            const double *slice = Am + (size_t)ob->hard[(size_t)t * md->M + m] * P;
            for (size_t e = 0; e < P; ++e) out[e] = LN(slice[e]);
        } else {
            const double *om = ob->soft + (size_t)t * ob->ksum + ob->koff[m];
            for (size_t e = 0; e < P; ++e) {
                double v = 0.0;
                for (int o = 0; o < md->K[m]; ++o) v += om[o] * LN(Am[(size_t)o * P + e]);
                out[e] = v;
            }
        }
    }
}

/* Likelihood messages of one context from its log-likelihood tensors ll
 * (context_loglik).  q: [sum n] marginals of the context; lam: [sum n]
 * output.  qoff[f] is the offset of factor f in q / lam. */
static void likelihood_messages(const orc_model *md, const double *lls, const size_t *poff, const double *q,
                                const int *qoff, int ntot, double *lam)
{
    for (int i = 0; i < ntot; ++i) lam[i] = 0.0;
    for (int m = 0; m < md->M; ++m) {
        const int k = md->dep_off[m + 1] - md->dep_off[m];
        const int *d = md->dep + md->dep_off[m];
        const size_t P = slice_size(md, m);
        const double *llm = lls + poff[m];
        int idx[ORC_MAX_RANK];
        for (int i = 0; i < k; ++i) idx[i] = 0;
        for (size_t e = 0; e < P; ++e) {
            const double ll = llm[e];
            for (int i = 0; i < k; ++i) {
                double w = 1.0;
                for (int j = 0; j < k; ++j)
                    if (j != i) w *= q[qoff[d[j]] + idx[j]];
                lam[qoff[d[i]] + idx[i]] += ll * w;
            }
            /* odometer over s_dep, last axis fastest (row-major A) */
            for (int i = k - 1; i >= 0; --i) {
                if (++idx[i] < md->n[d[i]]) break;
                idx[i] = 0;
            }
        }
    }
}

/* states of the B-dependencies of f taken together (prod of their n) */
static size_t bdep_states(const orc_model *md, int f)
{
    int k;
    const int *d = bdeps_of(md, f, &k);
    if (!d) return (size_t)md->n[f];
    size_t p = 1;
    for (int i = 0; i < k; ++i) p *= (size_t)md->n[d[i]];
    return p;
}

static const double *B_at(const orc_model *md, int f, int a)
{
    int am = md->mb == 1 ? 0 : a;
    return md->B[f] + (size_t)am * (size_t)md->n[f] * bdep_states(md, f) * (size_t)md->U[f];
}

/*
 * Contraction of B_f over its B-dependencies (Sec. III-B transition model,
 * B_f[i][s_{g_1}]..[s_{g_k}][u], row-major over the list):
 *   sum_{s_dep} val(B_f[i][s_dep][u]) prod_{g in dep, g != skip} q[qoff[g] + s_g]
 * with val = LN when logB, the identity otherwise; the dependency at list
 * position `skip` (-1: none) is held at state `fixv` and not weighted.
 * q holds the marginals of one step of one agent ([sum n]).
 */
static double b_contract(const orc_model *md, const double *Bf, int f, int i, int u, const double *q,
                         const int *qoff, int skip, int fixv, int logB)
{
    int k;
    const int *d = bdeps_of(md, f, &k);
    int dl[ORC_MAX_RANK], idx[ORC_MAX_RANK];
    for (int j = 0; j < k; ++j) {
        dl[j] = d ? d[j] : f;
        idx[j] = j == skip ? fixv : 0;
    }
    const size_t P = bdep_states(md, f);
    const int U = md->U[f];
    double acc = 0.0;
    for (;;) {
        size_t flat = 0;
        double w = 1.0;
        for (int j = 0; j < k; ++j) {
            flat = flat * (size_t)md->n[dl[j]] + (size_t)idx[j];
            if (j != skip) w *= q[qoff[dl[j]] + idx[j]];
        }
        const double b = Bf[((size_t)i * P + flat) * U + u];
        acc += (logB ? LN(b) : b) * w;
        /* odometer over the free positions, last fastest */
        int j = k - 1;
        for (; j >= 0; --j) {
            if (j == skip) continue;
            if (++idx[j] < md->n[dl[j]]) break;
            idx[j] = 0;
        }
        if (j < 0) break;
    }
    return acc;
}

/* Position of factor f in the B-dependency list of j, or -1. */
static int bdep_pos(const orc_model *md, int j, int f)
{
    int k;
    const int *d = bdeps_of(md, j, &k);
    if (!d) return j == f ? 0 : -1;
    for (int i = 0; i < k; ++i)
        if (d[i] == f) return i;
    return -1;
}

/* p(s_1) of agent a: the caller's prior (prior: [b][ntot]) or D_f */
static const double *first_prior(const orc_model *md, const double *prior, int f, int a, const int *qoff, int ntot)
{
    if (prior) return prior + (size_t)a * ntot + qoff[f];
    return md->D[f] + (size_t)(md->mb == 1 ? 0 : a) * md->n[f];
}

/* q <- (1 - tau) q + tau q_new over n values (tau = 1: plain replacement). */
static void damp(double *q, const double *q_new, int n, double tau)
{
    for (int s = 0; s < n; ++s) q[s] = tau == 1.0 ? q_new[s] : (1.0 - tau) * q[s] + tau * q_new[s];
}

static void run_fpi(const orc_model *md, int a, int T, const orc_obs *obs, const int *act, int iters, double *q,
                    const int *qoff, int ntot, double *work, const double *prior, double tau, const size_t *poff,
                    double *lls)
{
    double *cur = work, *lam = work + ntot, *logp = work + 2 * ntot, *v = work + 3 * ntot;
    for (int t = 0; t < T; ++t) {
        for (int f = 0; f < md->F; ++f) {
            const int nf = md->n[f];
            if (t == 0) {
                const double *p0 = first_prior(md, prior, f, a, qoff, ntot);
                for (int s = 0; s < nf; ++s) logp[qoff[f] + s] = LN(p0[s]);
            } else {
                /* predictive marginal of s_t^f under the factorised q_{t-1} */
                const double *Bf = B_at(md, f, a);
                const int u = act[(size_t)(t - 1) * md->F + f];
                const double *qp = q + (size_t)(t - 1) * ntot;
                for (int i = 0; i < nf; ++i) logp[qoff[f] + i] = LN(b_contract(md, Bf, f, i, u, qp, qoff, -1, 0, 0));
            }
            for (int s = 0; s < nf; ++s) cur[qoff[f] + s] = 1.0 / nf;
        }
        for (int k = 0; k < iters; ++k) {
            context_loglik(md, a, obs, t, poff, lls);
            likelihood_messages(md, lls, poff, cur, qoff, ntot, lam);
            for (int f = 0; f < md->F; ++f) {
                for (int s = 0; s < md->n[f]; ++s) v[s] = lam[qoff[f] + s] + logp[qoff[f] + s];
                softmax(v, md->n[f]);
                damp(cur + qoff[f], v, md->n[f], tau);
            }
        }
        memcpy(q + (size_t)t * ntot, cur, sizeof(double) * (size_t)ntot);
    }
}

static void run_window(const orc_model *md, int algo, int a, int T, const orc_obs *obs, const int *act, int iters,
                       double *q, const int *qoff, int ntot, double *work, const double *prior, double tau,
                       const size_t *poff, double *lls)
{
    double *qn = work;                               /* [T][ntot] next iterate */
    double *lam = work + (size_t)T * ntot;            /* [T][ntot] */
    for (int t = 0; t < T; ++t)
        for (int f = 0; f < md->F; ++f)
            for (int s = 0; s < md->n[f]; ++s) q[(size_t)t * ntot + qoff[f] + s] = 1.0 / md->n[f];
    for (int k = 0; k < iters; ++k) {
        for (int t = 0; t < T; ++t)
        {
            context_loglik(md, a, obs, t, poff, lls);
            likelihood_messages(md, lls, poff, q + (size_t)t * ntot, qoff, ntot, lam + (size_t)t * ntot);
        }
        for (int t = 0; t < T; ++t) {
            /* Transition messages (Sec. III-B joint): the forward one from
             * B_f given the factors it depends on at t-1, and one backward
             * message from every factor j whose B-dependencies contain f
             * (its "children"), given s_{t+1}^j and the other dependencies
             * of j at t.  With trivial lists: B_f[s][s'] q_{t-1,f}(s') and
             * q_{t+1,f}(s'') B_f[s''][s]. */
            const double *qprev = t > 0 ? q + (size_t)(t - 1) * ntot : NULL;
            const double *qcur = q + (size_t)t * ntot;
            const double *qnext = t + 1 < T ? q + (size_t)(t + 1) * ntot : NULL;
            for (int f = 0; f < md->F; ++f) {
                const int nf = md->n[f];
                const double *Bf = B_at(md, f, a);
                const double *p0 = first_prior(md, prior, f, a, qoff, ntot);
                const int uprev = t > 0 ? act[(size_t)(t - 1) * md->F + f] : 0;
                double *v = qn + (size_t)t * ntot + qoff[f];
                for (int s = 0; s < nf; ++s) {
                    double fwd;
                    if (t == 0)
                        fwd = LN(p0[s]);
                    else if (algo == ORC_VMP)
                        fwd = b_contract(md, Bf, f, s, uprev, qprev, qoff, -1, 0, 1);
                    else
                        fwd = LN(b_contract(md, Bf, f, s, uprev, qprev, qoff, -1, 0, 0));
                    double bwd = 0.0;   /* VMP: sum of the backward messages; MMP: sum of their logs */
                    int children = 0;
                    if (qnext) {
                        for (int j = 0; j < md->F; ++j) {
                            const int pos = bdep_pos(md, j, f);
                            if (pos < 0) continue;
                            const double *Bj = B_at(md, j, a);
                            const int unext = act[(size_t)t * md->F + j];
                            double m = 0.0;
                            for (int sn = 0; sn < md->n[j]; ++sn)
                                m += qnext[qoff[j] + sn] *
                                     b_contract(md, Bj, j, sn, unext, qcur, qoff, pos, s, algo == ORC_VMP);
                            bwd += algo == ORC_VMP ? m : LN(m);
                            ++children;
                        }
                    }
                    if (algo == ORC_VMP)
                        v[s] = lam[(size_t)t * ntot + qoff[f] + s] + fwd + bwd;
                    else if (children > 0)   /* mean of the messages present */
                        v[s] = lam[(size_t)t * ntot + qoff[f] + s] + (fwd + bwd) / (double)(1 + children);
                    else
                        v[s] = lam[(size_t)t * ntot + qoff[f] + s] + fwd;
                }
                softmax(v, nf);
            }
        }
        damp(q, qn, T * ntot, tau);
    }
}

/* Shared driver of orc_infer_ex and orc_infer_soft: exactly one of hard
 * ([b][T][M] outcomes) and soft ([b][T][sum K] observation vectors) is set. */
/* Checks B-dependency lists (NULL: trivial): non-empty, ascending, in range. */
static int bdeps_ok(int F, const int *bdep_off, const int *bdep)
{
    if (!bdep_off) return 1;
    if (!bdep || bdep_off[0] != 0) return 0;
    for (int f = 0; f < F; ++f) {
        const int k = bdep_off[f + 1] - bdep_off[f];
        if (k < 1 || k > ORC_MAX_RANK) return 0;
        for (int i = bdep_off[f]; i < bdep_off[f + 1]; ++i) {
            if (bdep[i] < 0 || bdep[i] >= F) return 0;
            if (i > bdep_off[f] && bdep[i] <= bdep[i - 1]) return 0;
        }
    }
    return 1;
}

static int run_all(int algo, int F, const int *n, const int *U, int M, const int *K, const int *dep_off,
                   const int *dep, int mb, const double *const *A, const double *const *B, const double *const *D,
                   const int *bdep_off, const int *bdep, int b, int T, const int *hard, const double *soft,
                   const int *act, const double *prior, double tau, int iters, double *q, int nthreads)
{
    if (F < 1 || !bdeps_ok(F, bdep_off, bdep)) return -1;
    if (algo < 0 || algo > 2 || F < 1 || M < 1 || b < 1 || T < 1 || iters < 1) return -1;
    if (!(tau > 0.0 && tau <= 1.0)) return -1;
    if (mb != 1 && mb != b) return -1;
    if (!n || !U || !K || !dep_off || !dep || !A || !B || !D || !(hard || soft) || !q) return -1;
    if (T > 1 && !act) return -1;
    int ntot = 0;
    int *qoff = (int *)malloc(sizeof(int) * (size_t)F);
    int *koff = (int *)malloc(sizeof(int) * (size_t)M);
    size_t *poff = (size_t *)malloc(sizeof(size_t) * (size_t)(M + 1));
    if (!qoff || !koff || !poff) { free(qoff); free(koff); free(poff); return -1; }
    int bad = 0, ksum = 0;
    for (int f = 0; f < F; ++f) {
        if (n[f] < 1 || U[f] < 1) bad = 1;
        qoff[f] = ntot;
        ntot += n[f];
    }
    orc_model md = {F, M, mb, n, U, K, dep_off, dep, A, B, D, bdep_off, bdep};
    poff[0] = 0;
    for (int m = 0; m < M && !bad; ++m) {
        int k = dep_off[m + 1] - dep_off[m];
        if (k < 1 || k > ORC_MAX_RANK || K[m] < 1) { bad = 1; break; }
        for (int i = dep_off[m]; i < dep_off[m + 1]; ++i)
            if (dep[i] < 0 || dep[i] >= F) bad = 1;
        if (bad) break;
        koff[m] = ksum;
        ksum += K[m];
        poff[m + 1] = poff[m] + slice_size(&md, m);
    }
    if (bad) { free(qoff); free(koff); free(poff); return -1; }
    const size_t work_per = (size_t)(4 + 2 * T) * (size_t)ntot + poff[M];
    const int nt = nthreads > 0 ? nthreads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 1) num_threads(nt) reduction(| : bad)
    for (int a = 0; a < b; ++a) {
        double *work = (double *)malloc(sizeof(double) * work_per);
        if (!work) { bad = 1; continue; }
        double *lls = work + (size_t)(4 + 2 * T) * (size_t)ntot;
        orc_obs ob = {hard ? hard + (size_t)a * T * M : NULL, soft ? soft + (size_t)a * T * ksum : NULL, koff, ksum};
        const int *ua = T > 1 ? act + (size_t)a * (T - 1) * F : NULL;
        double *qa = q + (size_t)a * T * ntot;
        if (algo == ORC_FPI)
            run_fpi(&md, a, T, &ob, ua, iters, qa, qoff, ntot, work, prior, tau, poff, lls);
        else
            run_window(&md, algo, a, T, &ob, ua, iters, qa, qoff, ntot, work, prior, tau, poff, lls);
        free(work);
    }
    free(qoff);
    free(koff);
    free(poff);
    return bad ? -1 : 0;
}

/*
 * Run `algo` (0 FPI, 1 VMP, 2 MMP) for b agents.  prior: NULL (p(s_1) = D)
 * or [b][sum n_f], each factor's block a distribution over its states; tau:
 * damping step in (0, 1].  Returns 0, or -1 on an invalid argument.
 * nthreads <= 0 uses the OpenMP default.
 */
int orc_infer_ex(int algo, int F, const int *n, const int *U, int M, const int *K, const int *dep_off,
                 const int *dep, int mb, const double *const *A, const double *const *B, const double *const *D,
                 int b, int T, const int *obs, const int *act, const double *prior, double tau, int iters,
                 double *q, int nthreads)
{
    if (!obs) return -1;
    return run_all(algo, F, n, U, M, K, dep_off, dep, mb, A, B, D, NULL, NULL, b, T, obs, NULL, act, prior, tau,
                   iters, q, nthreads);
}

/*
 * As orc_infer_ex with soft observations: obs_soft [b][T][sum K], the
 * observation vector of modality m (a distribution over its K_m outcomes,
 * one-hot for an integer outcome) at offset sum_{m' < m} K_m'.
 */
int orc_infer_soft(int algo, int F, const int *n, const int *U, int M, const int *K, const int *dep_off,
                   const int *dep, int mb, const double *const *A, const double *const *B, const double *const *D,
                   int b, int T, const double *obs_soft, const int *act, const double *prior, double tau,
                   int iters, double *q, int nthreads)
{
    if (!obs_soft) return -1;
    return run_all(algo, F, n, U, M, K, dep_off, dep, mb, A, B, D, NULL, NULL, b, T, NULL, obs_soft, act, prior, tau,
                   iters, q, nthreads);
}

/*
 * The general entry point: B-dependency lists bdep_off [F+1] / bdep (B_f of
 * shape [mb][n_f][n_{g_1}]..[n_{g_k}][U_f]; NULL: every list is {f}), and
 * either integer observations (obs) or soft ones (obs_soft), the other NULL.
 */
int orc_infer_general(int algo, int F, const int *n, const int *U, int M, const int *K, const int *dep_off,
                      const int *dep, int mb, const double *const *A, const double *const *B,
                      const double *const *D, const int *bdep_off, const int *bdep, int b, int T, const int *obs,
                      const double *obs_soft, const int *act, const double *prior, double tau, int iters, double *q,
                      int nthreads)
{
    if ((obs == NULL) == (obs_soft == NULL)) return -1;
    return run_all(algo, F, n, U, M, K, dep_off, dep, mb, A, B, D, bdep_off, bdep, b, T, obs, obs_soft, act, prior,
                   tau, iters, q, nthreads);
}

int orc_infer_prior(int algo, int F, const int *n, const int *U, int M, const int *K, const int *dep_off,
                    const int *dep, int mb, const double *const *A, const double *const *B, const double *const *D,
                    int b, int T, const int *obs, const int *act, const double *prior, int iters, double *q,
                    int nthreads)
{
    return orc_infer_ex(algo, F, n, U, M, K, dep_off, dep, mb, A, B, D, b, T, obs, act, prior, 1.0, iters, q,
                        nthreads);
}

int orc_infer(int algo, int F, const int *n, const int *U, int M, const int *K, const int *dep_off,
              const int *dep, int mb, const double *const *A, const double *const *B, const double *const *D,
              int b, int T, const int *obs, const int *act, int iters, double *q, int nthreads)
{
    return orc_infer_prior(algo, F, n, U, M, K, dep_off, dep, mb, A, B, D, b, T, obs, act, NULL, iters, q,
                           nthreads);
}

/*
 * Predictive prior of the next step (the same product as FPI's prior):
 *   out[a][f](i) = sum_j B_f[i][j][u_{a,f}] q[a][f](j)
 * q: [b][sum n_f] marginals, act: [b][F], out: [b][sum n_f].  Returns 0 or -1.
 */
int orc_predict(int F, const int *n, const int *U, int mb, const double *const *B, int b, const double *q,
                const int *act, double *out)
{
    if (F < 1 || b < 1 || (mb != 1 && mb != b) || !n || !U || !B || !q || !act || !out) return -1;
    int ntot = 0;
    for (int f = 0; f < F; ++f) {
        if (n[f] < 1 || U[f] < 1) return -1;
        ntot += n[f];
    }
    for (int a = 0; a < b; ++a) {
        int off = 0;
        for (int f = 0; f < F; ++f) {
            const int nf = n[f], u = act[(size_t)a * F + f];
            if (u < 0 || u >= U[f]) return -1;
            const double *Bf = B[f] + (size_t)(mb == 1 ? 0 : a) * nf * nf * U[f];
            for (int i = 0; i < nf; ++i) {
                double p = 0.0;
                for (int j = 0; j < nf; ++j) p += Bf[((size_t)i * nf + j) * U[f] + u] * q[(size_t)a * ntot + off + j];
                out[(size_t)a * ntot + off + i] = p;
            }
            off += nf;
        }
    }
    return 0;
}

/*
 * Predictive prior with B-dependency lists (NULL: trivial, as orc_predict):
 *   out[a][f](i) = sum_{s_dep} B_f[i][s_dep][u_{a,f}] prod_{g in dep(f)} q[a][g](s_g)
 * the predictive marginal of s_{t+1}^f under the factorised q.
 */
int orc_predict_general(int F, const int *n, const int *U, int mb, const double *const *B, const int *bdep_off,
                        const int *bdep, int b, const double *q, const int *act, double *out)
{
    if (F < 1 || b < 1 || (mb != 1 && mb != b) || !n || !U || !B || !q || !act || !out) return -1;
    if (!bdeps_ok(F, bdep_off, bdep)) return -1;
    int *qoff = (int *)malloc(sizeof(int) * (size_t)F);
    if (!qoff) return -1;
    int ntot = 0;
    for (int f = 0; f < F; ++f) {
        if (n[f] < 1 || U[f] < 1) { free(qoff); return -1; }
        qoff[f] = ntot;
        ntot += n[f];
    }
    orc_model md = {F, 0, mb, n, U, NULL, NULL, NULL, NULL, B, NULL, bdep_off, bdep};
    int bad = 0;
    for (int a = 0; a < b && !bad; ++a) {
        for (int f = 0; f < F; ++f) {
            const int u = act[(size_t)a * F + f];
            if (u < 0 || u >= U[f]) { bad = 1; break; }
            const double *Bf = B_at(&md, f, a);
            for (int i = 0; i < n[f]; ++i)
                out[(size_t)a * ntot + qoff[f] + i] = b_contract(&md, Bf, f, i, u, q + (size_t)a * ntot, qoff, -1, 0, 0);
        }
    }
    free(qoff);
    return bad ? -1 : 0;
}

/* Number of OpenMP threads orc_infer uses when nthreads <= 0. */
int orc_default_threads(void) { return omp_get_max_threads(); }
