// Streaming kernels for a model shared by every agent (BI_FAST_F32): VMP and
// MMP over b*T contexts, one iteration = one likelihood launch + one update
// launch, marginals double-buffered in the workspace.
//
// Likelihood messages (Sec. IV marginalisation, two-sided slice view of
// layout.h).  Contexts are first bucketed by their observed outcome, per
// modality; every slice X = LA_m[o] is then read from HBM once per iteration
// and applied to all J contexts that observed o, which makes the work two
// dense contractions with the slice as the shared operand:
//   Z[c][r] = sum_col X[r][col] t_c[col]      (rows x contexts, K = columns)
//   V[c][col] = sum_r s_c[r] X[r][col]        (contexts x columns, K = rows)
// both on fp32 matrix cores (v_mfma_f32_16x16x4f32).  A workgroup (8 waves,
// one per CU) owns 256 slice rows of one (m, o) bucket and streams the row
// tile through LDS in 32-column blocks (register prefetch two blocks ahead):
// Z accumulates in registers across the blocks (each wave owns 32 rows), V of
// each block is computed as four row-quarter partials (each wave one column
// group and one quarter), summed and folded at once into the column factors'
// messages.  The tile height sets the ratio of matrix-core work to the
// per-block folding and operand building.  Each workgroup writes one partial
// message vector per context and tile; the update kernel sums the partials in
// fp64 (fixed order, no atomics, bitwise reproducible), adds the transition
// messages and applies the softmax.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "internal.h"
#include "profile.h"
#include "stream.h"
#include "transition.h"

namespace bi {
namespace {

constexpr int kRT = 256;       // slice rows per workgroup tile
constexpr int kCB = 32;        // columns per staged block
constexpr int kNKB = 3;        // 16-wide MFMA context blocks per pass
constexpr int kJG = 16 * kNKB; // contexts per pass over the tile
constexpr int kThreads = 512;  // 8 waves, one workgroup per CU
constexpr int kQuarters = 4;   // row quarters of the V contraction
constexpr int kXS = kCB + 4;   // padded LDS row strides (floats)
constexpr int kSS = kRT + 4;
constexpr int kTS = kCB + 4;
constexpr int kVS = kCB + 4;   // 4 rows apart land 16 banks apart

typedef float f4 __attribute__((ext_vector_type(4)));

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

// ---------------------------------------------------------------------------
// Set-up of a call, one launch: workgroups 0 .. M-1 sort the contexts by
// observed outcome, one per modality (bucketing); the others write the
// uniform start of the marginals.  Slot order inside a bucket is not fixed
// (atomics) but results do not depend on it: every context's outputs come
// from its own MFMA column.
// ---------------------------------------------------------------------------
template <typename QT>
__global__ __launch_bounds__(1024) void prep_kernel(StreamArgs a, QT *q)
{
    if ((int)blockIdx.x >= a.M) {   // uniform start
        const int64_t total = (int64_t)a.nctx * a.ntot;
        const int64_t nthr = (int64_t)(gridDim.x - a.M) * blockDim.x;
        for (int64_t i = (blockIdx.x - a.M) * (int64_t)blockDim.x + threadIdx.x; i < total; i += nthr) {
            const int j = (int)(i % a.ntot);
            int f = 0;
            while (f + 1 < a.F && a.facs[f + 1].q_off <= j) ++f;
            q[i] = QT(1) / QT(a.facs[f].n);
        }
        return;
    }
    extern __shared__ int cnt[];   // [K + 1] counts, then starts; [K] fill counters
    const int m = blockIdx.x;
    const StreamMod &sm = a.sm[m];
    int *fil = cnt + sm.K + 1;
    int32_t *list = a.bctx + (int64_t)m * a.nlist;
    // the outcome list entry i observes in this modality (-1: none): the
    // context's outcome, or for soft vectors the slot's outcome when the
    // context's vector gives it a nonzero weight
    auto outcome = [&](int i) -> int {
        if (!a.soft) return a.obs[(int64_t)i * a.M + m];
        const int c = i >> a.vshift, o = i & ((1 << a.vshift) - 1);
        return o < sm.K && a.soft[(int64_t)c * a.ksum + sm.fofs + o] != 0.0f ? o : -1;
    };
    for (int o = threadIdx.x; o < 2 * sm.K + 1; o += blockDim.x) cnt[o] = 0;
    __syncthreads();
    for (int i = threadIdx.x; i < a.nlist; i += blockDim.x) {
        const int o = outcome(i);
        if (o >= 0) atomicAdd(&cnt[o], 1);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        int run = 0;
        for (int o = 0; o < sm.K; ++o) {
            const int c = cnt[o];
            cnt[o] = run;
            run += c;
        }
        cnt[sm.K] = run;
    }
    __syncthreads();
    int32_t *start = a.bstart + sm.bofs;
    for (int o = threadIdx.x; o <= sm.K; o += blockDim.x) start[o] = cnt[o];
    for (int i = threadIdx.x; i < a.nlist; i += blockDim.x) {
        const int o = outcome(i);
        if (o >= 0) list[cnt[o] + atomicAdd(&fil[o], 1)] = i;
    }
}

// ---------------------------------------------------------------------------
// likelihood partials
// ---------------------------------------------------------------------------
struct LikShared {
    float xs[kRT][kXS];            // staged slice block; row-factor marginals at the end
    float ss[kJG][kSS];            // s_c[r] for the tile's rows; Z at the end
    float ts[kJG][kTS];            // t_c[col] for the current block
    float vs[kQuarters][kJG][kVS]; // V row-quarter partials of the current block; partial vectors at the end
};

__device__ inline const float *qrow(const StreamArgs &a, const float *q, int ctx, int f)
{
    return q + (int64_t)(ctx >> a.vshift) * a.ntot + a.facs[f].q_off;
}

// Fold a block of one side's values W[c][k] (k = index lo..hi-1 along that
// side, stored at W[c][k - base]) into the messages of the side's factors:
//   two == 0:  out[c][k] += W[c][k]
//   two == 1:  k = (i0, i1) with i1 fastest (n1 states),
//              out[c][n0 + i1] += sum_{i0} W[c][k] * q[c][i0]
//              out[c][i0]      += sum_{i1} W[c][k] * q[c][n0 + i1]
// q: [ctx][qs] marginals of the side's factors (first factor, then second).
// Every output entry is owned by one thread or one 4-lane group (fixed
// summation order, no atomics); loops carry no integer division.
template <int NP>  // number of partial planes of W summed on the fly
__device__ inline float wv(const float *Wf, int pstride, int idx)
{
    float v = Wf[idx];
#pragma unroll
    for (int p = 1; p < NP; ++p) v += Wf[p * pstride + idx];
    return v;
}

template <int NP>
__device__ inline void fold_block(const float *Wf, int pstride, int ws, int lo, int hi, int jl, int two, int n0,
                                  int n1, const float *q, int qs, int base, float *out, int os)
{
    if (lo >= hi) return;
    const int tid = threadIdx.x;
    const int width = hi - lo;
    if (!two) {
        // items (c, k): tid -> k = lo + t % width ...  (width <= kCB or kRT)
        for (int i = tid; i < jl * width; i += kThreads) {
            const int c = i / width, k = i - c * width;
            out[c * os + lo + k] += wv<NP>(Wf, pstride, c * ws + lo + k - base);
        }
        return;
    }
    const int i0lo = lo / n1, i0hi = (hi - 1) / n1;
    const int ni0 = i0hi - i0lo + 1;
    // second factor: items (c, i1), summed over the i0 of the block
    {
        int c = tid / n1, i1 = tid - c * n1;
        const int dc = kThreads / n1, di = kThreads - dc * n1;
        for (; c < jl;) {
            float acc = 0.0f;
            const int wo = c * ws - base;
            const float *qc = q + c * qs;
            int k = i0lo * n1 + i1;
            for (int i0 = i0lo; i0 <= i0hi; ++i0, k += n1)
                if (k >= lo && k < hi) acc = fmaf(wv<NP>(Wf, pstride, wo + k), qc[i0], acc);
            out[c * os + n0 + i1] += acc;
            c += dc;
            i1 += di;
            if (i1 >= n1) {
                i1 -= n1;
                ++c;
            }
        }
    }
    // first factor: items (c, i0) split over 4 lanes (i1 quarters) + shuffles
    {
        const int part = tid & 3;
        const int ngroups = jl * ni0;
        for (int g0 = 0; g0 < ngroups; g0 += kThreads / 4) {
            const int g = g0 + (tid >> 2);
            float acc = 0.0f;
            int c = 0, i0 = 0;
            if (g < ngroups) {
                c = g / ni0;
                i0 = i0lo + (g - c * ni0);
                const int wo = c * ws - base;
                const float *qc = q + c * qs + n0;
                // lane `part` takes every fourth state (interleaved: neighbouring
                // lanes hit neighbouring banks)
                const int a0 = max(lo, i0 * n1), a1 = min(hi, (i0 + 1) * n1);
                for (int k = a0 + part; k < a1; k += 4) acc = fmaf(wv<NP>(Wf, pstride, wo + k), qc[k - i0 * n1], acc);
            }
            acc += __shfl_xor(acc, 1, 64);
            acc += __shfl_xor(acc, 2, 64);
            if (g < ngroups && part == 0) out[c * os + i0] += acc;
        }
    }
}

__global__ __launch_bounds__(kThreads, 1) void lik_kernel(StreamArgs a, const float *q, float *part)
{
    extern __shared__ float dyn[];
    LikShared &sh = *reinterpret_cast<LikShared *>(dyn);
    __shared__ int ctxs[kJG];

    // decode (modality, outcome, row tile)
    const int wg = a.flip ? (int)gridDim.x - 1 - (int)blockIdx.x : (int)blockIdx.x;   // grid = a.nwg
    int m = 0;
    while (m + 1 < a.M && a.sm[m + 1].wg0 <= wg) ++m;
    const StreamMod &sm = a.sm[m];
    const int local = wg - sm.wg0;
    const int o = local / sm.ntiles, tile = local - o * sm.ntiles;
    const int32_t *start = a.bstart + sm.bofs;
    const int b0 = start[o], J = start[o + 1] - b0;
    if (J == 0) return;
    const ModDesc &md = a.mods[m];
    const int R = md.R, C = md.C, Cp = md.Cp;
    const int r0 = tile * kRT;
    const int rows = min(kRT, R - r0);
    const int two = md.ncol == 2;
    const int n0 = md.cn[0], n1 = two ? md.cn[1] : 1;
    const int ncs = two ? n0 + n1 : n0;
    const int qcs = ncs | 1;                                  // odd row stride: contexts spread over banks
    float *lamc = dyn + sizeof(LikShared) / sizeof(float);   // [kJG][qcs] column-factor messages
    float *qc = lamc + kJG * qcs;                             // [kJG][qcs] column-factor marginals
    const float *X = reinterpret_cast<const float *>(a.base + md.la32_off) + (int64_t)o * md.slice +
                     (int64_t)r0 * Cp;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int li = lane & 15, lk = lane >> 4;
    const int nblocks = (Cp + kCB - 1) / kCB;

    // a thread's fixed column inside every block (for t_c), and its split
    const int my_cc = tid & (kCB - 1);

    constexpr int kSlots = kRT * kCB / 4 / kThreads;   // float4 slots of a block per thread
    auto load_block = [&](int cb, f4 (&reg)[kSlots]) {
#pragma unroll
        for (int u = 0; u < kSlots; ++u) {
            const int slot = tid + u * kThreads;
            const int rr = slot / (kCB / 4), c4 = slot - rr * (kCB / 4);
            const int col = cb * kCB + c4 * 4;
            f4 v = {0.f, 0.f, 0.f, 0.f};
            if (rr < rows && col < Cp) v = *reinterpret_cast<const f4 *>(X + (int64_t)rr * Cp + col);
            reg[u] = v;
        }
    };
    auto store_block = [&](const f4 (&reg)[kSlots]) {
#pragma unroll
        for (int u = 0; u < kSlots; ++u) {
            const int slot = tid + u * kThreads;
            const int rr = slot / (kCB / 4), c4 = slot - rr * (kCB / 4);
            *reinterpret_cast<f4 *>(&sh.xs[rr][c4 * 4]) = reg[u];
        }
    };
    auto build_t = [&](int cb) {
        const int col = cb * kCB + my_cc;
        const bool ok = col < C;
        const int c0 = two ? col / n1 : col, c1 = two ? col - c0 * n1 : 0;
        for (int c = tid / kCB; c < kJG; c += kThreads / kCB) {
            float v = 0.0f;
            if (ok) v = two ? qc[c * qcs + c0] * qc[c * qcs + n0 + c1] : qc[c * qcs + c0];
            sh.ts[c][my_cc] = v;
        }
    };

    for (int g0 = 0; g0 < J; g0 += kJG) {
        const int jg = min(kJG, J - g0);
        const int nkb = (jg + 15) >> 4;
        if (tid < kJG) ctxs[tid] = tid < jg ? a.bctx[(int64_t)m * a.nlist + b0 + g0 + tid] : -1;
        __syncthreads();
        for (int i = tid; i < kJG * ncs; i += kThreads) {
            const int c = i / ncs, e = i - c * ncs;
            const int ctx = ctxs[c];
            float v = 0.0f;
            if (ctx >= 0) v = e < n0 ? qrow(a, q, ctx, md.cf[0])[e] : qrow(a, q, ctx, md.cf[1])[e - n0];
            qc[c * qcs + e] = v;
            lamc[c * qcs + e] = 0.0f;
        }
        for (int i = tid; i < kJG * kRT; i += kThreads) {
            const int c = i / kRT, rr = i - c * kRT;
            float v = 0.0f;
            const int ctx = ctxs[c];
            if (ctx >= 0 && rr < rows) {
                const int r = r0 + rr;
                if (md.nrow == 0) {
                    v = 1.0f;
                } else if (md.nrow == 1) {
                    v = qrow(a, q, ctx, md.rf[0])[r];
                } else {
                    const int rn1 = md.rn[1];
                    v = qrow(a, q, ctx, md.rf[0])[r / rn1] * qrow(a, q, ctx, md.rf[1])[r % rn1];
                }
            }
            sh.ss[c][rr] = v;
        }
        f4 zacc[2][kNKB];
#pragma unroll
        for (int zb = 0; zb < 2; ++zb)
#pragma unroll
            for (int kb = 0; kb < kNKB; ++kb) zacc[zb][kb] = f4{0.f, 0.f, 0.f, 0.f};

        f4 preA[kSlots], preB[kSlots];
        load_block(0, preB);
        store_block(preB);
        if (nblocks > 1) load_block(1, preA);
        __syncthreads();   // qc, ss, block 0 visible
        build_t(0);
        // the V operand s_c[r] of this wave's row quarter is the same for every
        // column block: keep it in registers for the whole tile
        const int vg = wave & 1, vh = wave >> 1;
        f4 sreg[kRT / kQuarters / 16][kNKB];
#pragma unroll
        for (int k4 = 0; k4 < kRT / kQuarters / 16; ++k4)
#pragma unroll
            for (int kb = 0; kb < kNKB; ++kb)
                sreg[k4][kb] = *reinterpret_cast<const f4 *>(
                    &sh.ss[16 * kb + li][(kRT / kQuarters) * vh + 16 * k4 + 4 * lk]);
        __syncthreads();

        // one column block: MFMAs on block cb (in LDS), block cb+1 in `have`,
        // block cb+2 fetched into `fetch`
        auto body = [&](int cb, f4 (&have)[kSlots], f4 (&fetch)[kSlots]) {
            if (cb + 2 < nblocks) load_block(cb + 2, fetch);
            // Z: tile rows 32*wave.. (two 16-row blocks), K = block columns
#pragma unroll
            for (int k4 = 0; k4 < kCB / 16; ++k4) {
                f4 xa[2], tb[kNKB];
#pragma unroll
                for (int zb = 0; zb < 2; ++zb)
                    xa[zb] = *reinterpret_cast<const f4 *>(&sh.xs[32 * wave + 16 * zb + li][16 * k4 + 4 * lk]);
#pragma unroll
                for (int kb = 0; kb < kNKB; ++kb)
                    if (kb < nkb) tb[kb] = *reinterpret_cast<const f4 *>(&sh.ts[16 * kb + li][16 * k4 + 4 * lk]);
#pragma unroll
                for (int jj = 0; jj < 4; ++jj)
#pragma unroll
                    for (int zb = 0; zb < 2; ++zb)
#pragma unroll
                        for (int kb = 0; kb < kNKB; ++kb)
                            if (kb < nkb)
                                zacc[zb][kb] =
                                    __builtin_amdgcn_mfma_f32_16x16x4f32(xa[zb][jj], tb[kb][jj], zacc[zb][kb], 0, 0, 0);
            }
            // V: column group (wave & 1) of the block, row quarter (wave >> 1)
            f4 vacc[kNKB];
#pragma unroll
            for (int kb = 0; kb < kNKB; ++kb) vacc[kb] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int k4 = 0; k4 < kRT / kQuarters / 16; ++k4) {
                const int rb = (kRT / kQuarters) * vh + 16 * k4 + 4 * lk;
                float xb[4];
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) xb[jj] = sh.xs[rb + jj][16 * vg + li];
#pragma unroll
                for (int jj = 0; jj < 4; ++jj)
#pragma unroll
                    for (int kb = 0; kb < kNKB; ++kb)
                        if (kb < nkb)
                            vacc[kb] =
                                __builtin_amdgcn_mfma_f32_16x16x4f32(sreg[k4][kb][jj], xb[jj], vacc[kb], 0, 0, 0);
            }
#pragma unroll
            for (int kb = 0; kb < kNKB; ++kb)
                if (kb < nkb)
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr) sh.vs[vh][16 * kb + 4 * lk + rr][16 * vg + li] = vacc[kb][rr];
            __syncthreads();
            if (cb + 1 < nblocks) store_block(have);
            // fold V of this block into the column factors' messages
            fold_block<kQuarters>(&sh.vs[0][0][0], kJG * kVS, kVS, cb * kCB, min(cb * kCB + kCB, C), nkb * 16, two,
                                  n0, n1, qc, qcs, cb * kCB, lamc, qcs);
            if (cb + 1 < nblocks) build_t(cb + 1);
            __syncthreads();
        };
        for (int cb = 0; cb < nblocks; cb += 2) {
            body(cb, preA, preB);
            if (cb + 1 < nblocks) body(cb + 1, preB, preA);
        }

        // Z of the tile rows -> row factors' messages, staged with the column
        // factors' messages into one partial vector per context
        float(*zs)[kSS] = sh.ss;            // [kJG][kRT]
        float *qr = &sh.xs[0][0];           // [kJG][nrs] row-factor marginals
        float *pv = &sh.vs[0][0][0];        // [kJG][dsum] partial vectors
        const int dsum = md.dsum;
        const int nr0 = md.nrow >= 1 ? md.rn[0] : 0;
        const int nr1 = md.nrow == 2 ? md.rn[1] : 1;
        const int nrs = md.nrow == 2 ? nr0 + nr1 : nr0;
        const int qrs = nrs | 1, pvs = dsum | 1;   // odd strides
#pragma unroll
        for (int zb = 0; zb < 2; ++zb)
#pragma unroll
            for (int kb = 0; kb < kNKB; ++kb)
                if (kb < nkb)
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr) zs[16 * kb + li][32 * wave + 16 * zb + 4 * lk + rr] = zacc[zb][kb][rr];
        for (int i = tid; i < kJG * nrs; i += kThreads) {
            const int c = i / nrs, e = i - c * nrs;
            const int ctx = ctxs[c];
            float v = 0.0f;
            if (ctx >= 0) v = e < nr0 ? qrow(a, q, ctx, md.rf[0])[e] : qrow(a, q, ctx, md.rf[1])[e - nr0];
            qr[c * qrs + e] = v;
        }
        for (int i = tid; i < kJG * dsum; i += kThreads) {
            const int c = i / dsum, e = i - c * dsum;
            pv[c * pvs + e] = e >= nrs ? lamc[c * qcs + (e - nrs)] : 0.0f;
        }
        __syncthreads();
        if (md.nrow >= 1)
            fold_block<1>(&zs[0][0], 0, kSS, r0, r0 + rows, nkb * 16, md.nrow == 2, nr0, nr1, qr, qrs, r0, pv, pvs);
        __syncthreads();
        for (int i = tid; i < jg * dsum; i += kThreads) {
            const int c = i / dsum, e = i - c * dsum;
            part[(int64_t)ctxs[c] * a.pstride + sm.poff + (int64_t)tile * dsum + e] = pv[c * pvs + e];
        }
        __syncthreads();
    }
}

// sum_j M[j * ms] * x[j] over j < n in order (fp64), loads issued 8 at a time
// Two dot products of one state's transition messages over j in [j0, j1):
// The update of one context under B-dependency lists (Sec. III-B transition
// model): factor f's next state depends on the current states of the factors
// of its list, so its forward message contracts B_f (log B_f for VMP) with
// the marginals of the listed factors at t - 1, and every factor j whose list
// holds f sends a backward message, B_j contracted with q_{t+1, j} and the
// marginals at t of j's other listed factors, f held at each state.  MMP
// averages the forward message with the backward ones present.  One lane per
// state; the messages are the agent path's (transition.h).  pc: the
// context's partial messages; qp / qn: full marginal vectors of the
// neighbouring steps (null at the window's ends); the context's own
// marginals come from qin.
template <int ALGO, typename QT, typename PT, typename OT>
__device__ void update_general(const StreamArgs &a, const PT *pc, const QT *qp, const QT *qn, const QT *qin,
                               OT *qout, int ctx, double *vals, int wave, int lane)
{
    const int agent = ctx / a.T, t = ctx - agent * a.T;
    const QT *qself = qin + (int64_t)ctx * a.ntot;
    for (int f = wave; f < a.F; f += 4) {
        const FacDesc &fd = a.facs[f];
        const int n = fd.n;
        double *v = vals + fd.q_off;
        const BDep df = bdep_of(a.facs, fd);
        const int up = t > 0 ? a.act[((int64_t)agent * (a.T - 1) + t - 1) * a.F + f] : 0;
        for (int s = lane; s < n; s += 64) {
            double lam = 0.0;
            for (int i = 0; i < a.nmsg; ++i) {
                const MsgSrc src = a.msg[i];
                if (src.f != f) continue;
                for (int k = 0; k < src.copies; ++k) lam += (double)pc[src.off + s + (int64_t)k * src.stride];
            }
            double fwd;
            if (t == 0)
                fwd = a.prior ? ln_clamped((double)a.prior[(int64_t)agent * a.ntot + fd.q_off + s])
                              : reinterpret_cast<const double *>(a.base + fd.ld_off)[s];
            else if (ALGO == BI_ALGO_VMP)
                fwd = bdep_row(df, reinterpret_cast<const double *>(a.base + fd.lb_off) + ((int64_t)up * n + s) * df.bs,
                               qp, -1, 0);
            else
                fwd = ln_clamped(bdep_row(df, reinterpret_cast<const float *>(a.base + fd.b_off) +
                                                  ((int64_t)up * n + s) * df.bs, qp, -1, 0));
            double bwd = 0.0;
            int children = 0;
            if (qn) {
                for (int c = 0; c < fd.nch; ++c) {
                    const int jf = fd.ch[c], pos = fd.chpos[c];
                    const FacDesc &fj = a.facs[jf];
                    const BDep dj = bdep_of(a.facs, fj);
                    const int nj = fj.n;
                    const int uj = a.act[((int64_t)agent * (a.T - 1) + t) * a.F + jf];
                    const QT *qj = qn + fj.q_off;
                    double msg = 0.0;
                    if (ALGO == BI_ALGO_VMP) {
                        const double *LBj = reinterpret_cast<const double *>(a.base + fj.lb_off) + (int64_t)uj * nj * dj.bs;
                        for (int sn = 0; sn < nj; ++sn)
                            msg = fma((double)qj[sn], bdep_row(dj, LBj + (int64_t)sn * dj.bs, qself, pos, s), msg);
                        bwd += msg;
                    } else {
                        const float *Bj = reinterpret_cast<const float *>(a.base + fj.b_off) + (int64_t)uj * nj * dj.bs;
                        for (int sn = 0; sn < nj; ++sn)
                            msg = fma((double)qj[sn], bdep_row(dj, Bj + (int64_t)sn * dj.bs, qself, pos, s), msg);
                        bwd += ln_clamped(msg);
                    }
                    ++children;
                }
            }
            if (ALGO == BI_ALGO_VMP)
                v[s] = lam + fwd + bwd;
            else
                v[s] = children > 0 ? lam + (fwd + bwd) / (double)(1 + children) : lam + fwd;
        }
        __builtin_amdgcn_wave_barrier();   // v[s] came from lane s (one wave: LDS in program order)
        double mx = -INFINITY;
        for (int s = lane; s < n; s += 64) mx = fmax(mx, v[s]);
        mx = wave_max(mx);
        double sum = 0.0;
        for (int s = lane; s < n; s += 64) {
            const double ev = exp(v[s] - mx);
            v[s] = ev;
            sum += ev;
        }
        sum = wave_sum(sum);
        OT *out = qout + (int64_t)ctx * a.ntot + fd.q_off;
        for (int s = lane; s < n; s += 64)
            out[s] = a.tau != 1.0 ? (OT)((1.0 - a.tau) * (double)qself[fd.q_off + s] + a.tau * (v[s] / sum))
                                  : (OT)(v[s] / sum);
    }
}

// ---------------------------------------------------------------------------
// update: messages summed over their partial vectors (fp64, fixed order),
// transition messages, masked softmax; one workgroup per context, one wave
// per factor.  When they fit (a.stage), the context's partial messages and
// the marginals of its neighbours in time are first copied to LDS by the
// whole workgroup (independent loads, one memory round trip), so the sums
// read LDS.  For factors of up to 32 states two lanes share a state: each
// takes half of its partial vectors and half of the terms of its transition
// dots, and one shuffle adds the halves (the same in both lanes).  QT =
// marginals between iterations, PT = partial messages, OT = this launch's
// output marginals.
// ---------------------------------------------------------------------------
// The actions of factor f before and after step t, both loads at once
// (indices clamped into the window; unused at its ends; none when T = 1).
__device__ inline void trans_actions(const StreamArgs &a, int f, int agent, int t, int &up, int &un)
{
    up = 0;
    un = 0;
    if (a.T > 1) {
        const int32_t *ar = a.act + (int64_t)agent * (a.T - 1) * a.F + f;
        up = ar[(int64_t)max(t - 1, 0) * a.F];
        un = ar[(int64_t)min(t, a.T - 2) * a.F];
    }
}

// Update of one context under trivial B-dependency lists, for the factors
// of this wave (wave-uniform f, so the factor descriptors, the actions and the
// message-source table come in by scalar loads).  PP / QP: pointers to the
// context's partial messages and to the neighbouring steps' marginals, typed
// for LDS when they were staged (no generic-address loads); hp / hn: whether
// the steps t - 1 / t + 1 exist; up0 / un0: the actions before and after t
// of factor `wave`, loaded before the staging.  Every read of a transition
// product is issued before the partial sums, and the products take their
// operands 8 terms at a time (4 for fp64 log B with fp64 marginals; in j
// order, so the sums are those of one term at a time).
template <int ALGO, typename QT, typename OT, typename PP, typename QP>
__device__ inline void update_trivial(const StreamArgs &a, PP pc, QP qp, QP qn, bool hp, bool hn, const QT *qin,
                                      OT *qout, int ctx, double *vals, int wave, int lane, int up0, int un0)
{
    // log B (VMP) or B (MMP); with fp32 marginals (the fp32-contraction
    // class) VMP reads log B rounded to fp32, like MMP's fp32 B, so both take
    // 8 terms per batch (fp64 log B: 4, and 14.9 against 11.5 us per launch)
    using MT = std::conditional_t<ALGO == BI_ALGO_VMP && sizeof(QT) == 8, double, float>;
    constexpr int W = sizeof(MT) + sizeof(QT) > 8 ? 4 : 8;   // terms per batch (registers: every workgroup resident)
    const int agent = ctx / a.T, t = ctx - agent * a.T;
    for (int f = wave; f < a.F; f += 4) {
        StreamFac sf;
        if (f < kStreamFacs) {
            sf = a.fac[f];
        } else {
            const FacDesc &fd = a.facs[f];
            sf = StreamFac{fd.lb_off, fd.b_off, fd.ld_off, fd.n, fd.q_off, fd.lb32_off};
        }
        const int n = sf.n, qo = sf.q_off;
        int up = up0, un = un0;
        if (f != wave) trans_actions(a, f, agent, t, up, un);
        const MT *M = reinterpret_cast<const MT *>(
            a.base + (ALGO != BI_ALGO_VMP ? sf.b_off : sizeof(QT) == 8 ? sf.lb_off : sf.lb32_off));
        const MT *Mp = M + (int64_t)up * n * n, *Mn = M + (int64_t)un * n * n;
        double *v = vals + qo;
        const int L = n <= 32 ? 2 : 1;          // lanes per state
        const int half = lane & (L - 1);        // which share of the terms this lane takes
        const int h = (n + L - 1) / L;          // transition terms per share
        const int j0 = min(n, half * h), j1 = min(n, j0 + h);
        for (int s0 = 0; s0 < n; s0 += 64 / L) {
            const int s = s0 + lane / L;
            const int sc = min(s, n - 1);       // lanes past the last state compute a copy, unused
            // fwd = sum_j M[u_{t-1}][sc][j] q_{t-1}[j] (a row), bwd = sum_j M[u_t][j][sc] q_{t+1}[j] (a column)
            // (both products are formed at the window's ends too, from valid
            // operands, and dropped: no branch around a load)
            double fwd = 0.0, bwd = 0.0;
            int j = j0;
            for (; j + W <= j1; j += W) {
                MT mf[W], mb[W];
                QT xf[W], xb[W];
#pragma unroll
                for (int u = 0; u < W; ++u) {
                    mf[u] = Mp[(int64_t)sc * n + j + u];
                    mb[u] = Mn[(int64_t)(j + u) * n + sc];
                    xf[u] = qp[qo + j + u];
                    xb[u] = qn[qo + j + u];
                }
#pragma unroll
                for (int u = 0; u < W; ++u) {
                    fwd = fma((double)mf[u], (double)xf[u], fwd);
                    bwd = fma((double)mb[u], (double)xb[u], bwd);
                }
            }
            for (; j < j1; ++j) {
                fwd = fma((double)Mp[(int64_t)sc * n + j], (double)qp[qo + j], fwd);
                bwd = fma((double)Mn[(int64_t)j * n + sc], (double)qn[qo + j], bwd);
            }
            if (!hn) bwd = 0.0;
            double lam = 0.0;
            for (int i = 0; i < a.nmsg; ++i) {
                const MsgSrc src = a.msg[i];
                if (src.f != f) continue;
                for (int k = half; k < src.copies; k += L) lam += (double)pc[src.off + sc + (int64_t)k * src.stride];
            }
            if (L == 2) {
                lam += __shfl_xor(lam, 1, 64);
                fwd += __shfl_xor(fwd, 1, 64);
                bwd += __shfl_xor(bwd, 1, 64);
            }
            if (t == 0)
                fwd = a.prior ? ln_clamped((double)a.prior[(int64_t)agent * a.ntot + qo + sc])
                              : reinterpret_cast<const double *>(a.base + sf.ld_off)[sc];
            else if (ALGO != BI_ALGO_VMP)
                fwd = ln_clamped(fwd);
            if (hn && ALGO != BI_ALGO_VMP) bwd = ln_clamped(bwd);
            if (s < n && half == 0) {
                if (ALGO == BI_ALGO_VMP)
                    v[s] = lam + fwd + bwd;
                else
                    v[s] = hn ? lam + 0.5 * (fwd + bwd) : lam + fwd;
            }
        }
        __builtin_amdgcn_wave_barrier();   // v[s] came from lane L s (one wave: LDS in program order)
        double mx = -INFINITY;
        for (int s = lane; s < n; s += 64) mx = fmax(mx, v[s]);
        mx = wave_max(mx);
        double sum = 0.0;
        for (int s = lane; s < n; s += 64) {
            const double ev = exp(v[s] - mx);
            v[s] = ev;
            sum += ev;
        }
        sum = wave_sum(sum);
        OT *out = qout + (int64_t)ctx * a.ntot + qo;
        if (a.tau != 1.0) {
            const QT *old = qin + (int64_t)ctx * a.ntot + qo;
            for (int s = lane; s < n; s += 64) out[s] = (OT)((1.0 - a.tau) * (double)old[s] + a.tau * (v[s] / sum));
        } else {
            for (int s = lane; s < n; s += 64) out[s] = (OT)(v[s] / sum);
        }
    }
}

template <typename T>
using lds_cptr = const __attribute__((address_space(3))) T *;

template <int ALGO, typename QT, typename PT, typename OT, bool TB>   // TB: every B-dependency list is {f}
__global__ __launch_bounds__(256, 4) void update_kernel(StreamArgs a, const PT *part, const QT *qin, OT *qout)
{
    extern __shared__ double vals[];   // [ntot], then (staged) partials [pstride] and two marginal vectors [ntot]
    const int ctx = blockIdx.x;
    const int agent = ctx / a.T, t = ctx - agent * a.T;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)), lane = threadIdx.x & 63;
    const PT *pc = part + (int64_t)ctx * a.pstride;
    const bool hp = t > 0, hn = t + 1 < a.T;
    const QT *qp = hp ? qin + (int64_t)(ctx - 1) * a.ntot : qin;
    const QT *qn = hn ? qin + (int64_t)(ctx + 1) * a.ntot : qin;
    int up0 = 0, un0 = 0;   // trivial lists: this wave's first factor's actions, in flight during the staging
    if (TB && wave < a.F) trans_actions(a, wave, agent, t, up0, un0);
    if (a.stage) {
        PT *sp = reinterpret_cast<PT *>(vals + a.ntot);
        QT *sq = reinterpret_cast<QT *>(vals + a.ntot + (a.pstride * sizeof(PT) + 7) / 8);
        const int tid = threadIdx.x;
        const int np = (int)a.pstride, nq = a.ntot;
        if (a.soft) {
            // soft vectors: value i of modality m's range is sum_o w_m[o]
            // x (value i of slot o), in fp64 and in o order, over the slots
            // of nonzero weight (the others were not computed: their values
            // are loaded, from inside the buffer, and not used)
            const float *wc = a.soft + (int64_t)ctx * a.ksum;
            const PT *p0 = part + ((int64_t)ctx << a.vshift) * a.pstride;
            for (int i = tid; i < np; i += 256) {
                int mm = 0;
                while (mm + 1 < a.M && a.sm[mm + 1].pbeg <= i) ++mm;
                const float *w = wc + a.sm[mm].fofs;
                const int K = a.sm[mm].K;
                double acc = 0.0;
                for (int o0 = 0; o0 < K; o0 += 8) {
                    float wv[8];
                    PT pv[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        const int o = min(o0 + u, K - 1);
                        wv[u] = o0 + u < K ? w[o] : 0.0f;
                        pv[u] = p0[(int64_t)o * a.pstride + i];
                    }
#pragma unroll
                    for (int u = 0; u < 8; ++u)
                        if (wv[u] != 0.0f) acc = fma((double)wv[u], (double)pv[u], acc);
                }
                sp[i] = (PT)acc;
            }
        } else {
            for (int i0 = tid; i0 < np; i0 += 8 * 256) {   // 8 independent loads per thread, then the stores
                PT v[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) v[u] = pc[min(i0 + 256 * u, np - 1)];
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    if (i0 + 256 * u < np) sp[i0 + 256 * u] = v[u];
            }
        }
        for (int i = tid; i < nq; i += 256) {
            const QT a0 = qp[i], a1 = qn[i];
            sq[i] = a0;
            sq[nq + i] = a1;
        }
        __syncthreads();
        if constexpr (!TB) {
            update_general<ALGO, QT, PT, OT>(a, sp, hp ? sq : nullptr, hn ? sq + nq : nullptr, qin, qout, ctx, vals,
                                             wave, lane);
        } else {
            update_trivial<ALGO, QT, OT>(a, (lds_cptr<PT>)sp, (lds_cptr<QT>)sq, (lds_cptr<QT>)(sq + nq), hp, hn,
                                         qin, qout, ctx, vals, wave, lane, up0, un0);
        }
        return;
    }
    if constexpr (!TB)
        update_general<ALGO, QT, PT, OT>(a, pc, hp ? qp : nullptr, hn ? qn : nullptr, qin, qout, ctx, vals, wave,
                                         lane);
    else
        update_trivial<ALGO, QT, OT>(a, pc, qp, qn, hp, hn, qin, qout, ctx, vals, wave, lane, up0, un0);
}

template <typename QT, typename PT, typename OT>
void launch_update(int algo, const StreamArgs &a, size_t lds, hipStream_t stream, const PT *part, const QT *qin,
                   OT *qout)
{
    // trivial B-dependency lists get a kernel without the general transition
    // code (its registers would cost the common case occupancy)
    if (a.trivb) {
        if (algo == BI_ALGO_VMP)
            hipLaunchKernelGGL((update_kernel<BI_ALGO_VMP, QT, PT, OT, true>), dim3(a.nctx), dim3(256), lds, stream,
                               a, part, qin, qout);
        else
            hipLaunchKernelGGL((update_kernel<BI_ALGO_MMP, QT, PT, OT, true>), dim3(a.nctx), dim3(256), lds, stream,
                               a, part, qin, qout);
    } else {
        if (algo == BI_ALGO_VMP)
            hipLaunchKernelGGL((update_kernel<BI_ALGO_VMP, QT, PT, OT, false>), dim3(a.nctx), dim3(256), lds, stream,
                               a, part, qin, qout);
        else
            hipLaunchKernelGGL((update_kernel<BI_ALGO_MMP, QT, PT, OT, false>), dim3(a.nctx), dim3(256), lds, stream,
                               a, part, qin, qout);
    }
}

}  // namespace

bool stream_eligible(const bi_model *m, int algo)
{
    if (!(m->flags & BI_FAST_F32) || m->mb != 1 || algo == BI_ALGO_FPI) return false;
    if (m->M > kStreamMaxM) return false;
    for (const ModDesc &md : m->mods) {
        if (md.la32_off < 0) return false;
        const int ncs = md.ncol == 2 ? md.cn[0] + md.cn[1] : md.cn[0];
        const int nrs = md.nrow == 2 ? md.rn[0] + md.rn[1] : (md.nrow == 1 ? md.rn[0] : 0);
        // LDS staging limits of the likelihood kernel
        if (sizeof(LikShared) + 2 * sizeof(float) * kJG * (ncs | 1) > 160 * 1024 || kJG * (nrs | 1) > kRT * kXS ||
            kJG * (md.dsum | 1) > kQuarters * kJG * kVS)
            return false;
        if (md.K > kStreamMaxK) return false;
    }
    return true;
}

// Dense-path partial layout: per modality, one dsum vector per row tile
// (row factors' messages, then column factors'), summed over the tiles.
static int64_t dense_plan(const bi_model *m, StreamArgs *a)
{
    int wg = 0;
    int64_t poff = 0;
    a->nmsg = 0;
    for (int i = 0; i < m->M; ++i) {
        const ModDesc &md = m->mods[i];
        StreamMod &sm = a->sm[i];
        sm.ntiles = (md.R + kRT - 1) / kRT;
        sm.wg0 = wg;
        wg += md.K * sm.ntiles;
        sm.poff = poff;
        int e = 0;
        for (int side = 0; side < 2; ++side) {
            const int nf = side == 0 ? md.nrow : md.ncol;
            for (int j = 0; j < nf; ++j) {
                MsgSrc &src = a->msg[a->nmsg++];
                src.f = side == 0 ? md.rf[j] : md.cf[j];
                src.copies = sm.ntiles;
                src.stride = md.dsum;
                src.off = (int32_t)(poff + e);
                e += side == 0 ? md.rn[j] : md.cn[j];
            }
        }
        poff += (int64_t)sm.ntiles * md.dsum;
    }
    a->nwg = wg;
    return poff;
}

// The likelihood kernel a streaming call runs: general dense, dense
// matrix-core tiles (one contraction per workgroup), dense fp16-pair tiles
// reading every slice once, sparse fp64 gathers, sparse fp16-pair
// matrix-core tiles.
enum class Lik { Dense, Split, RowCol, Sparse, Sparse16 };

static Lik lik_kind(const bi_model *m, bool sparse)
{
    if (sparse) return sq_eligible(m) ? Lik::Sparse16 : Lik::Sparse;
    if (rc_eligible(m)) return Lik::RowCol;
    return split_eligible(m) ? Lik::Split : Lik::Dense;
}

// Plan of the workspace: bucket starts / fill counters / sorted contexts /
// partial messages / two marginal buffers (fp32, or fp64 for the sparse fp64
// kernel).
static void plan_ws(const bi_model *m, int b, int T, bool sparse, bool soft, StreamArgs *a, int64_t *offs,
                    int64_t *total)
{
    const int nctx = b * T;
    int kmax = 1;
    for (const ModDesc &md : m->mods) kmax = std::max(kmax, md.K);
    a->vshift = 0;
    while (soft && (1 << a->vshift) < kmax) ++a->vshift;
    const int64_t nlist = (int64_t)nctx << a->vshift;
    a->nlist = (int)std::min<int64_t>(nlist, INT32_MAX);
    int bofs = 0, fofs = 0;
    for (int i = 0; i < m->M; ++i) {
        StreamMod &sm = a->sm[i];
        sm.K = m->mods[i].K;
        sm.bofs = bofs;
        bofs += sm.K + 1;
        sm.fofs = fofs;
        fofs += sm.K;
    }
    const Lik lik = lik_kind(m, sparse);
    a->pstride = lik == Lik::Sparse   ? sparse_plan(m, a)
                 : lik == Lik::Dense  ? dense_plan(m, a)
                 : lik == Lik::RowCol ? rc_plan(m, a)
                                      : split_plan(m, a);
    // where each modality's partial messages start (the plans lay them out in
    // modality order)
    for (int i = 0; i < m->M; ++i) a->sm[i].pbeg = lik == Lik::Dense ? (int)a->sm[i].poff : INT32_MAX;
    if (lik != Lik::Dense)
        for (int k = 0; k < a->ntask; ++k) a->sm[a->task[k].m].pbeg = std::min(a->sm[a->task[k].m].pbeg, a->task[k].so);
    a->ksum = fofs;
    const int64_t es = lik == Lik::Sparse ? 8 : 4;
    int64_t off = 0;
    offs[0] = off;  off = align_up(off + 4 * (int64_t)bofs, kAlign);
    offs[1] = off;  off = align_up(off + 4 * (int64_t)fofs, kAlign);
    offs[2] = off;  off = align_up(off + 4 * (int64_t)m->M * nlist, kAlign);
    offs[3] = off;  off = align_up(off + es * nlist * a->pstride, kAlign);
    offs[4] = off;  off = align_up(off + es * (int64_t)nctx * m->ntot, kAlign);
    offs[5] = off;  off = align_up(off + es * (int64_t)nctx * m->ntot, kAlign);
    *total = off;
}

size_t stream_workspace(const bi_model *m, int b, int T, bool sparse, bool soft)
{
    StreamArgs a{};
    int64_t offs[6], total;
    plan_ws(m, b, T, sparse, soft, &a, offs, &total);
    return (size_t)total;
}

// LDS bytes of the update's staging: the softmax values, the partial messages
// and the two neighbour marginal vectors
static size_t staged_bytes(const bi_model *m, const StreamArgs &a, Lik lik)
{
    const size_t es_p = lik == Lik::Sparse ? sizeof(double) : sizeof(float);   // partials and marginals
    return sizeof(double) * m->ntot + (a.pstride * es_p + 7) / 8 * 8 + 2 * es_p * m->ntot;
}
constexpr size_t kStagedMax = 48 * 1024;
constexpr int kSoftMaxShift = 8;   // soft vectors on the streaming kernels: at most 256 outcomes per modality

bool stream_soft_ok(const bi_model *m, int b, int T, bool sparse)
{
    StreamArgs a{};
    int64_t offs[6], total;
    plan_ws(m, b, T, sparse, true, &a, offs, &total);
    return a.vshift <= kSoftMaxShift && ((int64_t)b * T << a.vshift) < INT32_MAX &&
           staged_bytes(m, a, lik_kind(m, sparse)) <= kStagedMax;
}

template <typename QT>
static void run_iterations(const bi_model *m, int algo, int iters, const StreamArgs &a, char *part, QT *qa, QT *qb,
                           float *q, size_t lik_lds, size_t upd_lds, hipStream_t stream, Lik lik)
{
    QT *cur = qa, *nxt = qb;
    using PT = QT;
    const char *name = lik == Lik::Sparse     ? "lik_sparse"
                       : lik == Lik::Sparse16 ? "lik_sparse16"
                       : lik == Lik::Split    ? (split_pairs(m) ? "lik_split16" : "lik_split")
                       : lik == Lik::RowCol   ? "lik_rowcol16"
                                              : "lik";
    // Odd iterations walk the likelihood work items backwards, so an iteration
    // starts on the slices the previous one read last: those still sit in the
    // memory-side last-level cache (256 MB, shared by all dies) when the
    // observed slices do not all fit in it.
    StreamArgs ab = a;
    for (int k = 0; k < iters; ++k) {
        ab.flip = k & 1;
        {
            ProfScope p(name, stream);
            if (lik == Lik::Sparse)
                sparse_lik_launch(m, ab, reinterpret_cast<const double *>(cur), reinterpret_cast<double *>(part),
                                  stream);
            else if (lik == Lik::RowCol)
                rc_lik_launch(ab, reinterpret_cast<const float *>(cur), reinterpret_cast<float *>(part), stream);
            else if (lik != Lik::Dense)
                split_lik_launch(m, ab, reinterpret_cast<const float *>(cur), reinterpret_cast<float *>(part), stream,
                                 lik == Lik::Sparse16);
            else
                hipLaunchKernelGGL(lik_kernel, dim3(a.nwg), dim3(kThreads), lik_lds, stream, a,
                                   reinterpret_cast<const float *>(cur), reinterpret_cast<float *>(part));
        }
        {
            ProfScope p("update", stream);
            const PT *pp = reinterpret_cast<const PT *>(part);
            if (k + 1 == iters)
                launch_update<QT, PT, float>(algo, a, upd_lds, stream, pp, cur, q);
            else
                launch_update<QT, PT, QT>(algo, a, upd_lds, stream, pp, cur, nxt);
        }
        QT *tmp = cur;
        cur = nxt;
        nxt = tmp;
    }
}

int launch_stream(const bi_model *m, int algo, int b, int T, const int32_t *obs, const int32_t *act,
                  const float *prior, double tau, int iters, float *q, void *ws, hipStream_t stream, bool sparse,
                  const float *soft)
{
    StreamArgs a{};
    int64_t offs[6], total;
    plan_ws(m, b, T, sparse, soft != nullptr, &a, offs, &total);
    if (soft && !stream_soft_ok(m, b, T, sparse))
        return fail(BI_ERR_UNSUPPORTED, "soft observations exceed the streaming kernels' limits");
    char *w = reinterpret_cast<char *>(ws);
    a.base = m->dev;
    a.mods = reinterpret_cast<const ModDesc *>(m->dev);
    a.facs = reinterpret_cast<const FacDesc *>(m->dev + align_up((int64_t)sizeof(ModDesc) * m->M, kAlign));
    a.F = m->F;
    a.M = m->M;
    a.T = T;
    a.nctx = b * T;
    a.ntot = m->ntot;
    a.obs = obs;
    a.soft = soft;
    a.act = act;
    a.prior = prior;
    a.tau = tau;
    a.trivb = m->trivial_b ? 1 : 0;
    for (int f = 0; f < std::min(m->F, kStreamFacs); ++f) {
        const FacDesc &fd = m->facs[f];
        a.fac[f] = StreamFac{fd.lb_off, fd.b_off, fd.ld_off, fd.n, fd.q_off, fd.lb32_off};
    }
    a.bstart = reinterpret_cast<int32_t *>(w + offs[0]);
    a.bctx = reinterpret_cast<int32_t *>(w + offs[2]);
    char *part = w + offs[3];
    const Lik lik = lik_kind(m, sparse);
    if (lik != Lik::Sparse && algo == BI_ALGO_VMP)   // fp32 marginals: the update reads log B in fp32
        for (const FacDesc &fd : m->facs)
            if (fd.lb32_off < 0) return fail(BI_ERR_INVALID_ARG, "fp32 log B missing (pack with BI_FAST_F32)");
    // update: the softmax values, plus (when they fit in 48 KB) the staged
    // partial messages and the two neighbour marginal vectors
    const size_t staged = staged_bytes(m, a, lik);
    a.stage = staged <= kStagedMax ? 1 : 0;
    const size_t upd_lds = a.stage ? staged : sizeof(double) * m->ntot;
    size_t lik_lds = 0;
    if (lik == Lik::Sparse) {
        lik_lds = sparse_lds_bytes(m);
    } else if (lik == Lik::RowCol) {
        lik_lds = rc_lds_bytes();
    } else if (lik != Lik::Dense) {
        lik_lds = split_lds_bytes(m, lik == Lik::Sparse16);
    } else {
        int ncs_max = 1;
        for (const ModDesc &md : m->mods)
            ncs_max = std::max(ncs_max, (md.ncol == 2 ? md.cn[0] + md.cn[1] : md.cn[0]) | 1);
        lik_lds = sizeof(LikShared) + 2 * sizeof(float) * kJG * ncs_max;
    }
    if (lik_lds > 160 * 1024 || upd_lds > 64 * 1024)
        return fail(BI_ERR_UNSUPPORTED, "streaming working set exceeds LDS");
    if (lik == Lik::Sparse) {
        const int rc = sparse_prepare(m);
        if (rc != BI_OK) return rc;
    } else if (lik == Lik::RowCol) {
        const int rc = rc_prepare();
        if (rc != BI_OK) return rc;
    } else if (lik != Lik::Dense) {
        const int rc = split_prepare(m, lik == Lik::Sparse16);
        if (rc != BI_OK) return rc;
    } else {
        const hipError_t e = func_max_lds((const void *)lik_kernel, (int)lik_lds);
        if (e != hipSuccess) return fail(BI_ERR_DEVICE, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    }
    int kmax = 1;
    for (const ModDesc &md : m->mods) kmax = std::max(kmax, md.K);
    // set-up: bucketing and the uniform start in one launch
    const int init_grid = (int)std::min<int64_t>(256, ((int64_t)a.nctx * a.ntot + 1023) / 1024);
    const size_t prep_lds = sizeof(int) * (2 * kmax + 1);
    if (lik == Lik::Sparse) {
        double *qa = reinterpret_cast<double *>(w + offs[4]);
        double *qb = reinterpret_cast<double *>(w + offs[5]);
        {
            ProfScope p("prep", stream);
            hipLaunchKernelGGL(prep_kernel<double>, dim3(m->M + init_grid), dim3(1024), prep_lds, stream, a, qa);
        }
        run_iterations<double>(m, algo, iters, a, part, qa, qb, q, lik_lds, upd_lds, stream, lik);
    } else {
        float *qa = reinterpret_cast<float *>(w + offs[4]);
        float *qb = reinterpret_cast<float *>(w + offs[5]);
        {
            ProfScope p("prep", stream);
            hipLaunchKernelGGL(prep_kernel<float>, dim3(m->M + init_grid), dim3(1024), prep_lds, stream, a, qa);
        }
        run_iterations<float>(m, algo, iters, a, part, qa, qb, q, lik_lds, upd_lds, stream, lik);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(BI_ERR_DEVICE, "kernel launch failed: %s", hipGetErrorString(e));
    return BI_OK;
}

}  // namespace bi
