// Agent-resident kernels: one workgroup (256 threads, 4 waves) per agent runs
// every iteration of FPI, VMP or MMP without leaving the kernel.  Marginals,
// likelihood messages and the Z/V scratch of the two-sided slice view live in
// LDS; the emission slices, B and D are read from the packed buffer (L2 /
// MALL resident for the per-agent models this path serves).
//
// One iteration of VMP / MMP (Jacobi over every (t, f), Sec. IV):
//   1. Z/V: for every context t and modality m, Z = X t and V = s X over the
//      observed slice X = LA_m[o_{t,m}] (layout.h), each output a dot product
//      owned by one thread;
//   2. lam_{t,f}: small contractions of Z (row factors of m) or V (column
//      factors), summed over the modalities that depend on f;
//   3. update: one wave per (t, f) forms the transition messages from the
//      neighbouring marginals and applies the masked softmax with wave
//      shuffles, writing the other half of the double-buffered marginals.
// FPI runs the same three phases on a single context t at a time, after
// forming the predictive prior from the final marginals of step t-1.
//
// All arithmetic is fp64 (the updates are ill-conditioned for some models,
// see layout.h); on gfx950 an fp64 FMA issues at the rate of an unpacked
// fp32 FMA, so this path pays only in LDS footprint.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "internal.h"
#include "profile.h"

namespace bi {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kStageMaxM = 16;

// Observed slices staged in LDS: a context's block holds modality m's slice at
// po[m] with rows padded to Cp + 1 values (conflict-free row and column
// reads); pr[m] is the slice's offset in the unpadded concatenation.
enum StageMode { kStageNone = 0, kStageChunk = 1, kStageWindow = 2 };

struct AgentArgs {
    const char *base;      // packed buffer
    const ModDesc *mods;   // device descriptor tables (inside the packed buffer)
    const FacDesc *facs;
    int F, M, shared;      // shared: one model for every agent
    int T, iters, ntot, zvpc, nc;  // nc: contexts per Z/V chunk
    int stage;             // StageMode
    int sctx, sraw;        // staged values per context (padded), unpadded values per context
    int po[kStageMaxM + 1], pr[kStageMaxM + 1];
    const int32_t *obs;    // integer outcomes [agent][T][M], or NULL with ll
    const double *ll;      // soft observations: log-likelihood tensors [agent][T][llpc] (soft.hip)
    int64_t llpc;
    const int32_t *act;
    const float *prior;    // optional [agent][ntot] prior of the first step (replaces D)
    double tau;            // damping step: q <- (1 - tau) q + tau q_new (1: plain update)
    float *q;
};

template <class T>
__device__ inline const T *at(const char *base, int64_t byte_off)
{
    return reinterpret_cast<const T *>(base + byte_off);
}

__device__ inline double ln_clamped(double x) { return log(fmax(x, kEps)); }

__device__ inline double wave_max(double v)
{
    for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, 64));
    return v;
}

__device__ inline double wave_sum(double v)
{
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// One Z or V output of an observed slice X (row stride xs) for the marginals
// qt: j < R gives Z[j], j = R + col gives V[col].
__device__ inline double zv_one(const AgentArgs &a, const ModDesc &md, const double *X, int64_t xs,
                                const double *qt, int j)
{
    const int R = md.R;
    double acc = 0.0;
    if (j < R) {  // Z[r] = sum_c X[r][c] t[c]
        if (md.nrow > 0) {  // (Z of a rank-0 row side feeds no message)
            const double *row = X + (int64_t)j * xs;
            const double *q0 = qt + a.facs[md.cf[0]].q_off;
            if (md.ncol == 1) {
                for (int cc = 0; cc < md.C; ++cc) acc = fma(row[cc], q0[cc], acc);
            } else {
                const double *q1 = qt + a.facs[md.cf[1]].q_off;
                const int n0 = md.cn[0], n1 = md.cn[1];
                for (int c0 = 0; c0 < n0; ++c0) {
                    double in = 0.0;
                    const double *rr = row + c0 * n1;
                    for (int c1 = 0; c1 < n1; ++c1) in = fma(rr[c1], q1[c1], in);
                    acc = fma(q0[c0], in, acc);
                }
            }
        }
    } else {  // V[c] = sum_r s[r] X[r][c]
        const int col = j - R;
        if (md.nrow == 0) {
            acc = X[col];
        } else if (md.nrow == 1) {
            const double *q0 = qt + a.facs[md.rf[0]].q_off;
            for (int r = 0; r < R; ++r) acc = fma(q0[r], X[(int64_t)r * xs + col], acc);
        } else {
            const double *q0 = qt + a.facs[md.rf[0]].q_off;
            const double *q1 = qt + a.facs[md.rf[1]].q_off;
            const int n0 = md.rn[0], n1 = md.rn[1];
            for (int r0 = 0; r0 < n0; ++r0) {
                double in = 0.0;
                const double *xc = X + (int64_t)r0 * n1 * xs + col;
                for (int r1 = 0; r1 < n1; ++r1) in = fma(q1[r1], xc[(int64_t)r1 * xs], in);
                acc = fma(q0[r0], in, acc);
            }
        }
    }
    return acc;
}

// Copy the observed slices of contexts [t0, t0 + nc) into stg (one block of
// sctx values per context): every thread issues its loads before any store,
// so the workgroup pays one memory round trip for the whole chunk.
__device__ void stage_slices(const AgentArgs &a, int agent, int t0, int nc, double *stg)
{
    const int total = nc * a.sraw;
    for (int i0 = 0; i0 < total; i0 += 8 * kThreads) {
        double v[8];
        int dst[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int i = i0 + u * kThreads + (int)threadIdx.x;
            dst[u] = -1;
            v[u] = 0.0;
            if (i < total) {
                const int c = i / a.sraw, rem = i - c * a.sraw;
                int m = 0;
                while (m + 1 < a.M && a.pr[m + 1] <= rem) ++m;
                const ModDesc &md = a.mods[m];
                const int e = rem - a.pr[m], r = e / md.Cp, col = e - r * md.Cp;
                const int64_t ctx = (int64_t)agent * a.T + t0 + c;
                const double *X;
                if (a.ll) {
                    X = a.ll + ctx * a.llpc + a.pr[m];
                } else {
                    const int o = a.obs[ctx * a.M + m];
                    X = at<double>(a.base, md.la_off) + (a.shared ? 0 : (int64_t)agent * md.la_agent) +
                        (int64_t)o * md.slice;
                }
                v[u] = X[e];
                dst[u] = c * a.sctx + a.po[m] + r * (md.Cp + 1) + col;
            }
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (dst[u] >= 0) stg[dst[u]] = v[u];
    }
}

// Phase 1: Z/V of contexts [t0, t0 + nc) into zv[c][zvpc].
// q: marginals of context t at q + t * ntot.  With staged slices, X of
// context t0 + c comes from stg + (sc0 + c) * sctx (LDS); otherwise from the
// packed buffer.
__device__ void phase_zv(const AgentArgs &a, int agent, int t0, int nc, const double *q, double *zv,
                         const double *stg, int sc0)
{
    const int tid = threadIdx.x;
    int base = 0;
    int64_t llo = 0;   // offset of modality m in a context's log-likelihood tensors
    for (int m = 0; m < a.M; ++m) {
        const ModDesc &md = a.mods[m];
        const int R = md.R, C = md.C, Cp = md.Cp;
        const int per = R + C;
        const int cnt = nc * per;
        const double *la = at<double>(a.base, md.la_off) + (a.shared ? 0 : (int64_t)agent * md.la_agent);
        int i = tid - (base % kThreads);
        if (i < 0) i += kThreads;
        for (; i < cnt; i += kThreads) {
            const int c = i / per, j = i - c * per;
            const int t = t0 + c;
            const double *qt = q + t * a.ntot;
            double acc;
            if (stg) {
                acc = zv_one(a, md, stg + (int64_t)(sc0 + c) * a.sctx + a.po[m], Cp + 1, qt, j);
            } else if (a.ll) {
                acc = zv_one(a, md, a.ll + ((int64_t)agent * a.T + t) * a.llpc + llo, Cp, qt, j);
            } else {
                const int o = a.obs[((int64_t)agent * a.T + t) * a.M + m];
                acc = zv_one(a, md, la + (int64_t)o * md.slice, Cp, qt, j);
            }
            zv[c * a.zvpc + md.zv_off + j] = acc;
        }
        base += cnt;
        llo += md.slice;
    }
}

// Phase 2: lam of contexts [t0, t0 + nc) into lam[t][ntot].
__device__ void phase_lam(const AgentArgs &a, int t0, int nc, const double *q, const double *zv, const int *sfac,
                          double *lam)
{
    for (int i = threadIdx.x; i < nc * a.ntot; i += kThreads) {
        const int c = i / a.ntot, j = i - c * a.ntot;
        const int f = sfac[j];
        const int s = j - a.facs[f].q_off;
        const double *qt = q + (t0 + c) * a.ntot;
        double acc = 0.0;
        for (int m = 0; m < a.M; ++m) {
            const ModDesc &md = a.mods[m];
            const double *Z = zv + c * a.zvpc + md.zv_off;
            const double *V = Z + md.R;
            if (md.nrow >= 1 && md.rf[0] == f) {
                if (md.nrow == 1) {
                    acc += Z[s];
                } else {
                    const double *q1 = qt + a.facs[md.rf[1]].q_off;
                    const int n1 = md.rn[1];
                    double in = 0.0;
                    for (int r1 = 0; r1 < n1; ++r1) in = fma(Z[s * n1 + r1], q1[r1], in);
                    acc += in;
                }
            } else if (md.nrow == 2 && md.rf[1] == f) {
                const double *q0 = qt + a.facs[md.rf[0]].q_off;
                const int n0 = md.rn[0], n1 = md.rn[1];
                double in = 0.0;
                for (int r0 = 0; r0 < n0; ++r0) in = fma(Z[r0 * n1 + s], q0[r0], in);
                acc += in;
            } else if (md.cf[0] == f) {
                if (md.ncol == 1) {
                    acc += V[s];
                } else {
                    const double *q1 = qt + a.facs[md.cf[1]].q_off;
                    const int n1 = md.cn[1];
                    double in = 0.0;
                    for (int c1 = 0; c1 < n1; ++c1) in = fma(V[s * n1 + c1], q1[c1], in);
                    acc += in;
                }
            } else if (md.ncol == 2 && md.cf[1] == f) {
                const double *q0 = qt + a.facs[md.cf[0]].q_off;
                const int n0 = md.cn[0], n1 = md.cn[1];
                double in = 0.0;
                for (int c0 = 0; c0 < n0; ++c0) in = fma(V[c0 * n1 + s], q0[c0], in);
                acc += in;
            }
        }
        lam[(t0 + c) * a.ntot + j] = acc;
    }
}

// Masked softmax of the values already stored in v[0..n) by this wave.
__device__ void wave_softmax(double *v, int n, int lane)
{
    double mx = -INFINITY;
    for (int s = lane; s < n; s += 64) mx = fmax(mx, v[s]);
    mx = wave_max(mx);
    double sum = 0.0;
    for (int s = lane; s < n; s += 64) {
        const double e = exp(v[s] - mx);
        v[s] = e;
        sum += e;
    }
    sum = wave_sum(sum);
    for (int s = lane; s < n; s += 64) v[s] = v[s] / sum;
}

// lam for every context of the window (phases 1 and 2 over context chunks;
// staged chunks are copied to LDS first unless the whole window is resident).
__device__ void window_lam(const AgentArgs &a, int agent, const double *q, double *zv, double *stg, const int *sfac,
                           double *lam)
{
    for (int t0 = 0; t0 < a.T; t0 += a.nc) {
        const int nc = min(a.nc, a.T - t0);
        if (a.stage == kStageChunk) {
            stage_slices(a, agent, t0, nc, stg);
            __syncthreads();
        }
        phase_zv(a, agent, t0, nc, q, zv, a.stage == kStageNone ? nullptr : stg,
                 a.stage == kStageWindow ? t0 : 0);
        __syncthreads();
        phase_lam(a, t0, nc, q, zv, sfac, lam);
        __syncthreads();
    }
}

__device__ void init_tables(const AgentArgs &a, int *sfac)
{
    for (int j = threadIdx.x; j < a.ntot; j += kThreads) {
        int f = 0;
        while (f + 1 < a.F && a.facs[f + 1].q_off <= j) ++f;
        sfac[j] = f;
    }
}

template <int ALGO>  // BI_ALGO_VMP or BI_ALGO_MMP
__global__ __launch_bounds__(kThreads) void agent_window_kernel(AgentArgs a)
{
    extern __shared__ double smem[];
    const int agent = blockIdx.x;
    const int TN = a.T * a.ntot;
    double *qa = smem, *qb = qa + TN, *lam = qb + TN, *zv = lam + TN, *stg = zv + a.nc * a.zvpc;
    const int nstg = a.stage == kStageWindow ? a.T : a.stage == kStageChunk ? a.nc : 0;
    int *sfac = reinterpret_cast<int *>(stg + (int64_t)nstg * a.sctx);
    init_tables(a, sfac);
    if (a.stage == kStageWindow) stage_slices(a, agent, 0, a.T, stg);   // every iteration reads them from LDS
    __syncthreads();
    for (int i = threadIdx.x; i < TN; i += kThreads) qa[i] = 1.0 / a.facs[sfac[i % a.ntot]].n;
    __syncthreads();
    const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
    const int64_t am = a.shared ? 0 : agent;
    double *cur = qa, *nxt = qb;
    for (int k = 0; k < a.iters; ++k) {
        window_lam(a, agent, cur, zv, stg, sfac, lam);
        for (int p = wave; p < a.T * a.F; p += kWaves) {
            const int t = p / a.F, f = p - t * a.F;
            const FacDesc &fd = a.facs[f];
            const int n = fd.n;
            const double *qprev = t > 0 ? cur + (t - 1) * a.ntot + fd.q_off : nullptr;
            const double *qnext = t + 1 < a.T ? cur + (t + 1) * a.ntot + fd.q_off : nullptr;
            const int up = t > 0 ? a.act[((int64_t)agent * (a.T - 1) + t - 1) * a.F + f] : 0;
            const int un = t + 1 < a.T ? a.act[((int64_t)agent * (a.T - 1) + t) * a.F + f] : 0;
            // VMP uses log B, MMP the linear B (log taken after the product)
            const double *LBp = at<double>(a.base, fd.lb_off) + am * fd.b_agent + (int64_t)up * n * n;  // [i][j]
            const double *LBn = at<double>(a.base, fd.lb_off) + am * fd.b_agent + (int64_t)un * n * n;
            const float *Bp = at<float>(a.base, fd.b_off) + am * fd.b_agent + (int64_t)up * n * n;
            const float *Bn = at<float>(a.base, fd.b_off) + am * fd.b_agent + (int64_t)un * n * n;
            const double *ld = at<double>(a.base, fd.ld_off) + am * fd.ld_agent;
            double *v = nxt + t * a.ntot + fd.q_off;
            const double *lm = lam + t * a.ntot + fd.q_off;
            for (int s = lane; s < n; s += 64) {
                double fwd, bwd = 0.0;
                if (t == 0) {
                    fwd = a.prior ? ln_clamped((double)a.prior[(int64_t)agent * a.ntot + fd.q_off + s]) : ld[s];
                } else if (ALGO == BI_ALGO_VMP) {
                    double acc = 0.0;
                    for (int j = 0; j < n; ++j) acc = fma(LBp[s * n + j], qprev[j], acc);
                    fwd = acc;
                } else {
                    double acc = 0.0;
                    for (int j = 0; j < n; ++j) acc = fma((double)Bp[s * n + j], qprev[j], acc);
                    fwd = ln_clamped(acc);
                }
                if (qnext) {
                    double acc = 0.0;
                    if (ALGO == BI_ALGO_VMP) {
                        for (int i = 0; i < n; ++i) acc = fma(qnext[i], LBn[i * n + s], acc);
                        bwd = acc;
                    } else {
                        for (int i = 0; i < n; ++i) acc = fma(qnext[i], (double)Bn[i * n + s], acc);
                        bwd = ln_clamped(acc);
                    }
                }
                double val;
                if (ALGO == BI_ALGO_VMP)
                    val = lm[s] + fwd + bwd;
                else
                    val = qnext ? lm[s] + 0.5 * (fwd + bwd) : lm[s] + fwd;
                v[s] = val;
            }
            wave_softmax(v, n, lane);
            if (a.tau != 1.0) {
                const double *old = cur + t * a.ntot + fd.q_off;
                for (int s = lane; s < n; s += 64) v[s] = (1.0 - a.tau) * old[s] + a.tau * v[s];
            }
        }
        __syncthreads();
        double *tmp = cur;
        cur = nxt;
        nxt = tmp;
    }
    float *out = a.q + (int64_t)agent * TN;
    for (int i = threadIdx.x; i < TN; i += kThreads) out[i] = (float)cur[i];
}

__global__ __launch_bounds__(kThreads) void agent_filter_kernel(AgentArgs a)
{
    extern __shared__ double smem[];
    const int agent = blockIdx.x;
    const int TN = a.T * a.ntot;
    // qfin: final marginals of every step; cur: current iterate of step t,
    // placed at row t of a [T][ntot] view so phase_zv / phase_lam index it
    // like the window kernel
    double *qfin = smem, *cur = qfin + TN, *lam = cur + TN, *zv = lam + TN, *logp = zv + a.zvpc;
    double *stg = logp + a.ntot;
    const int nstg = a.stage == kStageWindow ? a.T : a.stage == kStageChunk ? 1 : 0;
    int *sfac = reinterpret_cast<int *>(stg + (int64_t)nstg * a.sctx);
    init_tables(a, sfac);
    if (a.stage == kStageWindow) stage_slices(a, agent, 0, a.T, stg);
    __syncthreads();
    const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
    const int64_t am = a.shared ? 0 : agent;
    for (int t = 0; t < a.T; ++t) {
        // predictive prior of step t and uniform start
        for (int f = wave; f < a.F; f += kWaves) {
            const FacDesc &fd = a.facs[f];
            const int n = fd.n;
            double *lp = logp + fd.q_off;
            if (t == 0) {
                const double *ld = at<double>(a.base, fd.ld_off) + am * fd.ld_agent;
                if (a.prior) {
                    const float *pr = a.prior + (int64_t)agent * a.ntot + fd.q_off;
                    for (int s = lane; s < n; s += 64) lp[s] = ln_clamped((double)pr[s]);
                } else {
                    for (int s = lane; s < n; s += 64) lp[s] = ld[s];
                }
            } else {
                const int u = a.act[((int64_t)agent * (a.T - 1) + t - 1) * a.F + f];
                const float *Bp = at<float>(a.base, fd.b_off) + am * fd.b_agent + (int64_t)u * n * n;
                const double *qp = qfin + (t - 1) * a.ntot + fd.q_off;
                for (int s = lane; s < n; s += 64) {
                    double acc = 0.0;
                    for (int j = 0; j < n; ++j) acc = fma((double)Bp[s * n + j], qp[j], acc);
                    lp[s] = ln_clamped(acc);
                }
            }
        }
        double *qt = cur + t * a.ntot;
        for (int j = threadIdx.x; j < a.ntot; j += kThreads) qt[j] = 1.0 / a.facs[sfac[j]].n;
        if (a.stage == kStageChunk) stage_slices(a, agent, t, 1, stg);   // step t's slices, for all its iterations
        __syncthreads();
        for (int k = 0; k < a.iters; ++k) {
            phase_zv(a, agent, t, 1, cur, zv, a.stage == kStageNone ? nullptr : stg,
                     a.stage == kStageWindow ? t : 0);
            __syncthreads();
            phase_lam(a, t, 1, cur, zv, sfac, lam);
            __syncthreads();
            // Jacobi: lam holds every factor's message from the previous iterate
            // (damped: the new marginal is formed in lam's row, then mixed
            // into the current one; each lane owns the same states throughout)
            for (int f = wave; f < a.F; f += kWaves) {
                const FacDesc &fd = a.facs[f];
                double *lm = lam + t * a.ntot + fd.q_off;
                double *v = a.tau != 1.0 ? lm : qt + fd.q_off;
                const double *lp = logp + fd.q_off;
                for (int s = lane; s < fd.n; s += 64) v[s] = lm[s] + lp[s];
                wave_softmax(v, fd.n, lane);
                if (a.tau != 1.0) {
                    double *qf = qt + fd.q_off;
                    for (int s = lane; s < fd.n; s += 64) qf[s] = (1.0 - a.tau) * qf[s] + a.tau * v[s];
                }
            }
            __syncthreads();
        }
        for (int j = threadIdx.x; j < a.ntot; j += kThreads) qfin[t * a.ntot + j] = qt[j];
        __syncthreads();
    }
    float *out = a.q + (int64_t)agent * TN;
    for (int i = threadIdx.x; i < TN; i += kThreads) out[i] = (float)qfin[i];
}

constexpr size_t kLdsMax = 160 * 1024;

}  // namespace

int launch_agent(const bi_model *m, int algo, int b, int T, const int32_t *obs, const double *ll,
                 const int32_t *act, const float *prior, double tau, int iters, float *q, hipStream_t stream)
{
    AgentArgs a;
    a.base = m->dev;
    a.mods = reinterpret_cast<const ModDesc *>(m->dev);
    a.facs = reinterpret_cast<const FacDesc *>(m->dev + align_up((int64_t)sizeof(ModDesc) * m->M, kAlign));
    a.F = m->F;
    a.M = m->M;
    a.shared = m->mb == 1;
    a.T = T;
    a.iters = iters;
    a.ntot = m->ntot;
    a.zvpc = m->zvpc;
    a.obs = obs;
    a.ll = ll;
    a.llpc = 0;
    for (const ModDesc &md : m->mods) a.llpc += md.slice;
    a.act = act;
    a.prior = prior;
    a.tau = tau;
    a.q = q;
    const size_t TN = (size_t)T * m->ntot;
    // staged slice layout (see AgentArgs)
    int64_t sctx = 0, sraw = 0;
    bool can_stage = m->M <= kStageMaxM;
    for (int i = 0; i < m->M && can_stage; ++i) {
        const ModDesc &md = m->mods[i];
        a.po[i] = (int)sctx;
        a.pr[i] = (int)sraw;
        sctx += (int64_t)md.R * (md.Cp + 1);
        sraw += (int64_t)md.R * md.Cp;
        if (sctx > (int64_t)kLdsMax / 8) can_stage = false;
    }
    if (can_stage) {
        a.po[m->M] = (int)sctx;
        a.pr[m->M] = (int)sraw;
    }
    a.sctx = (int)sctx;
    a.sraw = (int)sraw;
    const size_t sb = 8 * (size_t)sctx;   // staged bytes per context
    const size_t budget2 = 80 * 1024;    // two workgroups per CU
    size_t fixed, per_ctx = (size_t)m->zvpc * 8, lds;
    a.stage = kStageNone;
    if (algo == BI_ALGO_FPI) {
        fixed = (3 * TN + m->ntot) * 8 + (size_t)m->ntot * 4 + per_ctx;
        a.nc = 1;
        if (can_stage && fixed + T * sb <= budget2)
            a.stage = kStageWindow;
        else if (can_stage && fixed + sb <= kLdsMax)
            a.stage = kStageChunk;
        lds = fixed + (a.stage == kStageWindow ? T * sb : a.stage == kStageChunk ? sb : 0);
    } else {
        fixed = 3 * TN * 8 + (size_t)m->ntot * 4;
        if (can_stage && fixed + T * (per_ctx + sb) <= budget2) {
            // the whole window's slices stay in LDS for every iteration
            a.stage = kStageWindow;
            a.nc = T;
            lds = fixed + T * (per_ctx + sb);
        } else {
            // slices read from the packed buffer: whole window in one chunk
            // when it fits in 80 KB, otherwise as many contexts as 160 KB allow.
            // (Copying each chunk's slices to LDS first measured slower here:
            // the extra barriers per chunk cost more than the saved reads.)
            size_t nc = T;
            if (fixed + nc * per_ctx > budget2) nc = fixed < kLdsMax ? (kLdsMax - fixed) / per_ctx : 0;
            if (nc > (size_t)T) nc = T;
            a.nc = (int)nc;
            lds = fixed + (size_t)a.nc * per_ctx;
        }
    }
    if (a.nc < 1 || lds > kLdsMax)
        return fail(BI_ERR_UNSUPPORTED, "agent working set (%zu bytes of LDS) exceeds the 160 KB budget", lds);
    hipError_t e;
    if (algo == BI_ALGO_FPI) {
        e = hipFuncSetAttribute((const void *)agent_filter_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)kLdsMax);
        if (e == hipSuccess) {
            ProfScope p("agent_filter", stream);
            hipLaunchKernelGGL(agent_filter_kernel, dim3(b), dim3(kThreads), lds, stream, a);
            e = hipGetLastError();
        }
    } else if (algo == BI_ALGO_VMP) {
        e = hipFuncSetAttribute((const void *)agent_window_kernel<BI_ALGO_VMP>,
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsMax);
        if (e == hipSuccess) {
            ProfScope p("agent_window", stream);
            hipLaunchKernelGGL(agent_window_kernel<BI_ALGO_VMP>, dim3(b), dim3(kThreads), lds, stream, a);
            e = hipGetLastError();
        }
    } else {
        e = hipFuncSetAttribute((const void *)agent_window_kernel<BI_ALGO_MMP>,
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsMax);
        if (e == hipSuccess) {
            ProfScope p("agent_window", stream);
            hipLaunchKernelGGL(agent_window_kernel<BI_ALGO_MMP>, dim3(b), dim3(kThreads), lds, stream, a);
            e = hipGetLastError();
        }
    }
    if (e != hipSuccess) return fail(BI_ERR_DEVICE, "kernel launch failed: %s", hipGetErrorString(e));
    return BI_OK;
}

}  // namespace bi
