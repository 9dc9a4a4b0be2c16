// Agent-resident kernels: one workgroup (256 threads, 4 waves) per agent runs
// every iteration of FPI, VMP or MMP without leaving the kernel.  Marginals,
// likelihood messages and the Z/V scratch of the two-sided slice view live in
// LDS; the emission slices, B and D are read from the packed buffer (L2 /
// MALL resident for the per-agent models this path serves).
//
// One iteration of VMP / MMP (Jacobi over every (t, f), Sec. IV):
//   1. Z/V: for every context t and modality m, Z = X t and V = s X over the
//      observed slice X = LA_m[o_{t,m}] (layout.h): one dot product per
//      thread when the window's slices are staged in LDS; from global memory
//      in the tile form (16-lane segments reading each slice once, coalesced;
//      phase_zv_tile);
//   2. lam_{t,f}: small contractions of Z (row factors of m) or V (column
//      factors), summed over the modalities that depend on f;
//   3. update: one lane segment per (t, f) forms the transition messages from
//      the neighbouring marginals and applies the masked softmax with lane
//      exchanges (window_update_seg), writing the other half of the
//      double-buffered marginals (general B-dependency lists: a thread per
//      state, then a segmented softmax through LDS).
// FPI runs phase 1 on a single context t at a time, then one segment per
// factor forms lam, adds the predictive prior of step t (from the final
// marginals of step t-1) and takes the softmax.
//
// All arithmetic is fp64 (the updates are ill-conditioned for some models,
// see layout.h); on gfx950 an fp64 FMA issues at the rate of an unpacked
// fp32 FMA, so this path pays only in LDS footprint.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "internal.h"
#include "profile.h"
#include "transition.h"

namespace bi {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kStageMaxM = 16;
constexpr int kStageMaxF = 16;
constexpr size_t kBStageMax = 64 * 1024;   // bytes of B / log B staged per workgroup

// Observed slices staged in LDS: a context's block holds modality m's slice at
// po[m] with rows padded to Cp + 1 values (conflict-free row and column
// reads); pr[m] is the slice's offset in the unpadded concatenation.
enum StageMode { kStageNone = 0, kStageChunk = 1, kStageWindow = 2 };

// Where phase 1 reads the observed slices: staged in LDS, from global memory
// one dot product per thread, or from global memory in the tile form;
// kSrcLdsShort: staged in LDS, every dot product of at most 8 terms (plain
// loops, see dot8).
enum SliceSrc { kSrcLds = 0, kSrcGlobal = 1, kSrcTile = 2, kSrcLdsShort = 3 };

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
    // The agent's transition tables staged in LDS once per launch when they
    // fit (bst): log B (fp64) for VMP, B (fp32) for MMP and FPI; factor f's
    // [u][i][j] block at element bo[f].  bdoubles: LDS doubles of the table.
    int bst, bdoubles;
    int bo[kStageMaxF + 1];
    // Tile form of the Z/V phase (slices from global memory, M <= kStageMaxM):
    // modality m's block in a context's Z/V scratch starts at zt[m] and holds
    // the Z partial sums of its column chunks, [chunk][R] (row side of rank
    // >= 1 only), then V [C].  The window's outcomes are copied to LDS.
    int tile;
    unsigned tilemask;   // bit m: modality m in the tile form (else one dot product per thread, Z [R] then V [C])
    int zt[kStageMaxM + 1];
    double tau;            // damping step: q <- (1 - tau) q + tau q_new (1: plain update)
    int sw;                // lanes per (step, factor) segment of the update (0: one thread per state)
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

// acc + sum_{i < n} x(i) w(i) as one chain of fma in index order.  The
// operands of up to 8 terms are read before any is used, so a dot product
// over LDS pays one read latency per batch instead of one per term (the
// compiler waits for each read of a plain loop with a run-time trip count).
template <int B, class XF, class WF>
__device__ inline double dot_batch(int &i, XF x, WF w, double acc)
{
    double xv[B], wv[B];
#pragma unroll
    for (int u = 0; u < B; ++u) {
        xv[u] = x(i + u);
        wv[u] = w(i + u);
    }
#pragma unroll
    for (int u = 0; u < B; ++u) acc = fma(xv[u], wv[u], acc);
    i += B;
    return acc;
}

// BT = 1: the plain loop (the LDS-staged window kernel with dot products of
// at most 8 terms, two workgroups per CU, measured 8% faster with it)
template <int BT, class XF, class WF>
__device__ inline double dot8(int n, XF x, WF w, double acc = 0.0)
{
    int i = 0;
    if (BT == 1) {
        while (i < n) acc = dot_batch<1>(i, x, w, acc);
        return acc;
    }
    while (i + 8 <= n) acc = dot_batch<8>(i, x, w, acc);
    if (i + 4 <= n) acc = dot_batch<4>(i, x, w, acc);
    if (i + 2 <= n) acc = dot_batch<2>(i, x, w, acc);
    if (i < n) acc = dot_batch<1>(i, x, w, acc);
    return acc;
}

// max and sum of v[0..n) (n >= 1) in index order, reads batched the same way
template <int BT>
__device__ inline double seg_max(const double *v, int n)
{
    double mx = v[0];
    int i = 1;
    for (; BT > 1 && i + 8 <= n; i += 8) {
        double t[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) t[u] = v[i + u];
#pragma unroll
        for (int u = 0; u < 8; ++u) mx = fmax(mx, t[u]);
    }
    for (; i < n; ++i) mx = fmax(mx, v[i]);
    return mx;
}

template <int BT>
__device__ inline double seg_sum(const double *v, int n)
{
    double sum = 0.0;
    int i = 0;
    for (; BT > 1 && i + 8 <= n; i += 8) {
        double t[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) t[u] = v[i + u];
#pragma unroll
        for (int u = 0; u < 8; ++u) sum += t[u];
    }
    for (; i < n; ++i) sum += v[i];
    return sum;
}

// sum_{i < len} x[i * stride] w(i) with the outer-product weight
// w(i) = q0[i / n1] q1[i % n1] (q1 == nullptr, n1 == 1: w(i) = q0[i]); the
// values of x are loaded 8 at a time, so a long dot product costs one
// memory round trip per 8 terms.
__device__ inline double outer_dot(const double *x, int64_t stride, int len, const double *q0, const double *q1,
                                   int n1)
{
    double acc = 0.0;
    int i0 = 0, i1 = 0;   // i = i0 * n1 + i1
    int i = 0;
    for (; i + 8 <= len; i += 8) {
        double xv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) xv[u] = x[(int64_t)(i + u) * stride];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const double w = q1 ? q0[i0] * q1[i1] : q0[i0];
            acc = fma(xv[u], w, acc);
            if (++i1 == n1) {
                i1 = 0;
                ++i0;
            }
        }
    }
    for (; i < len; ++i) {
        const double w = q1 ? q0[i0] * q1[i1] : q0[i0];
        acc = fma(x[(int64_t)i * stride], w, acc);
        if (++i1 == n1) {
            i1 = 0;
            ++i0;
        }
    }
    return acc;
}

// Weight of line i of a side with k factors f[0..k) of sizes n[0..k) (the
// last factor fastest, as in the slice layout): the product of the factors'
// marginals at i's digits, factor position skip (-1: none) left out.  Used
// for sides of more than two factors (dependency lists of 5 to 10 factors).
__device__ inline double side_weight(const AgentArgs &a, const double *qt, const int32_t *f, const int32_t *n, int k,
                                     int i, int skip = -1)
{
    double w = 1.0;
    for (int g = k - 1; g >= 0; --g) {
        const int d = i % n[g];
        i /= n[g];
        if (g != skip) w *= qt[a.facs[f[g]].q_off + d];
    }
    return w;
}

// One Z or V output of an observed slice X (row stride xs) for the marginals
// qt: j < R gives Z[j] = sum_c X[j][c] t[c], j = R + col gives
// V[col] = sum_r s[r] X[r][col] (t, s: outer products of the column and row
// factors' marginals).
template <bool WIDE>
__device__ inline double zv_one(const AgentArgs &a, const ModDesc &md, const double *X, int64_t xs,
                                const double *qt, int j)
{
    const int R = md.R;
    if (j < R) {
        if (md.nrow == 0) return 0.0;   // Z of a rank-0 row side feeds no message
        if (WIDE && md.ncol > 2)
            return dot8<8>(md.C, [&](int c) { return X[(int64_t)j * xs + c]; },
                           [&](int c) { return side_weight(a, qt, md.cf, md.cn, md.ncol, c); });
        const double *q1 = md.ncol == 2 ? qt + a.facs[md.cf[1]].q_off : nullptr;
        return outer_dot(X + (int64_t)j * xs, 1, md.C, qt + a.facs[md.cf[0]].q_off, q1,
                         md.ncol == 2 ? md.cn[1] : 1);
    }
    const int col = j - R;
    if (md.nrow == 0) return X[col];
    if (WIDE && md.nrow > 2)
        return dot8<8>(R, [&](int r) { return X[(int64_t)r * xs + col]; },
                       [&](int r) { return side_weight(a, qt, md.rf, md.rn, md.nrow, r); });
    const double *q1 = md.nrow == 2 ? qt + a.facs[md.rf[1]].q_off : nullptr;
    return outer_dot(X + col, xs, R, qt + a.facs[md.rf[0]].q_off, q1, md.nrow == 2 ? md.rn[1] : 1);
}

// The same output with the nested loops of the two-sided view, for slices
// staged in LDS (short latency: no batching, fewer registers).
template <int BT, bool WIDE>
__device__ inline double zv_one_lds(const AgentArgs &a, const ModDesc &md, const double *X, int64_t xs,
                                    const double *qt, int j)
{
    const int R = md.R;
    double acc = 0.0;
    if (j < R) {  // Z[r] = sum_c X[r][c] t[c]
        if (md.nrow > 0) {  // (Z of a rank-0 row side feeds no message)
            const double *row = X + (int64_t)j * xs;
            const double *q0 = qt + a.facs[md.cf[0]].q_off;
            if (WIDE && md.ncol > 2) {
                acc = dot8<BT>(md.C, [&](int cc) { return row[cc]; },
                               [&](int cc) { return side_weight(a, qt, md.cf, md.cn, md.ncol, cc); });
            } else if (md.ncol == 1) {
                acc = dot8<BT>(md.C, [&](int cc) { return row[cc]; }, [&](int cc) { return q0[cc]; });
            } else {
                const double *q1 = qt + a.facs[md.cf[1]].q_off;
                const int n0 = md.cn[0], n1 = md.cn[1];
                for (int c0 = 0; c0 < n0; ++c0) {
                    const double *rr = row + c0 * n1;
                    const double in = dot8<BT>(n1, [&](int c1) { return rr[c1]; }, [&](int c1) { return q1[c1]; });
                    acc = fma(q0[c0], in, acc);
                }
            }
        }
    } else {  // V[c] = sum_r s[r] X[r][c]
        const int col = j - R;
        if (md.nrow == 0) {
            acc = X[col];
        } else if (WIDE && md.nrow > 2) {
            acc = dot8<BT>(R, [&](int r) { return X[(int64_t)r * xs + col]; },
                           [&](int r) { return side_weight(a, qt, md.rf, md.rn, md.nrow, r); });
        } else if (md.nrow == 1) {
            const double *q0 = qt + a.facs[md.rf[0]].q_off;
            acc = dot8<BT>(R, [&](int r) { return q0[r]; }, [&](int r) { return X[(int64_t)r * xs + col]; });
        } else {
            const double *q0 = qt + a.facs[md.rf[0]].q_off;
            const double *q1 = qt + a.facs[md.rf[1]].q_off;
            const int n0 = md.rn[0], n1 = md.rn[1];
            for (int r0 = 0; r0 < n0; ++r0) {
                const double *xc = X + (int64_t)r0 * n1 * xs + col;
                const double in =
                    dot8<BT>(n1, [&](int r1) { return q1[r1]; }, [&](int r1) { return xc[(int64_t)r1 * xs]; });
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
// WIDE: some modality has a side of more than two factors
template <bool GX, int BT, bool WIDE>   // GX: slices read from global memory (batched loads); else staged in LDS
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
            if (!GX) {
                acc = zv_one_lds<BT, WIDE>(a, md, stg + (int64_t)(sc0 + c) * a.sctx + a.po[m], Cp + 1, qt, j);
            } else if (a.ll) {
                acc = zv_one<WIDE>(a, md, a.ll + ((int64_t)agent * a.T + t) * a.llpc + llo, Cp, qt, j);
            } else {
                const int o = a.obs[((int64_t)agent * a.T + t) * a.M + m];
                acc = zv_one<WIDE>(a, md, la + (int64_t)o * md.slice, Cp, qt, j);
            }
            zv[c * a.zvpc + md.zv_off + j] = acc;
        }
        base += cnt;
        llo += md.slice;
    }
}

// ---------------------------------------------------------------------------
// Tile form of phase 1 for slices read from global memory.  A unit is
// (context, modality, chunk of 32 columns) and runs on a segment of 16 lanes,
// two adjacent columns per lane: each lane loads its two columns of every row
// (16-byte loads; the lanes of a segment cover 256 contiguous bytes of a row),
// so a slice is read once, coalesced, for both of its sides:
//   V[col]  = sum_r s[r] X[r][col]         in the lane (rows in blocks of RB,
//                                           all loads of a block in flight);
//   Z[r]   += sum_{col in chunk} X[r][col] t[col]
//                                          lane partial products, reduced over
//                                          the segment by DPP exchanges.
// Z of a modality with nch chunks is left as nch partial sums per row; phase
// 2 adds them.  Every sum runs in a fixed order (results are reproducible).
constexpr int kSeg = 16;                 // lanes per unit (one DPP row)
constexpr int kSegs = kThreads / kSeg;   // units in flight per workgroup
constexpr int kTileCols = 2 * kSeg;      // columns per unit

__host__ __device__ constexpr int tile_nch(int C) { return (C + kTileCols - 1) / kTileCols; }

// FPI (one context per step): a slice with more rows than this (a tall one)
// has too few tile units, each walking its row blocks one after another, and
// takes one dot product per thread instead (up to 3x faster on such calls;
// the window kernels, with a chunk of contexts per phase, are faster with
// every modality in the tile form)
constexpr int kTileMaxRows = 96;

// doubles of modality md's block in the tile layout (tiled: in the tile form)
__host__ __device__ inline int tile_block(const ModDesc &md, bool tiled)
{
    return tiled ? (md.nrow > 0 ? tile_nch(md.C) * md.R : 0) + md.C : md.R + md.C;
}

// DPP lane pairings inside a row of 16 lanes: lane i with i ^ 15 (row_mirror),
// i ^ 7 (row_half_mirror), i ^ 3 and i ^ 1 (quad permutations).  Partners of
// pairing k differ in lane bit 3 - k and in no higher bit, so the four of them
// in this order halve a set of values per lane like a butterfly over bits
// 3, 2, 1, 0.
template <int K> struct SegPair;
template <> struct SegPair<0> { static constexpr int ctrl = 0x140; };
template <> struct SegPair<1> { static constexpr int ctrl = 0x141; };
template <> struct SegPair<2> { static constexpr int ctrl = 0x1B; };
template <> struct SegPair<3> { static constexpr int ctrl = 0xB1; };

template <int K>
__device__ inline double seg_swap(double v)
{
    const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), SegPair<K>::ctrl, 0xF, 0xF, true);
    const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), SegPair<K>::ctrl, 0xF, 0xF, true);
    return __hiloint2double(hi, lo);
}

// Sum of z[0..P) over the 16 lanes of the segment, one value per lane left
// in z[0]: P halving steps and 4 - log2 P plain exchanges; the lane then holds
// value index sl >> (4 - log2 P) (lanes that differ only in the low bits hold
// the same sum).  Every lane of the segment must take part.
template <int K, int N>
__device__ inline void seg_halve(double *z, int sl)
{
    if constexpr (N > 1) {
        const bool up = (sl >> (3 - K)) & 1;
#pragma unroll
        for (int i = 0; i < N / 2; ++i) {
            const double lo = z[i], hi = z[i + N / 2];
            z[i] = (up ? hi : lo) + seg_swap<K>(up ? lo : hi);
        }
        seg_halve<K + 1, N / 2>(z, sl);
    } else if constexpr (K < 4) {
        z[0] += seg_swap<K>(z[0]);
        seg_halve<K + 1, 1>(z, sl);
    }
}

constexpr int log2_floor(int x) { return x <= 1 ? 0 : 1 + log2_floor(x / 2); }

// Maximum (MAX) or sum of v over an aligned segment of SW lanes (a power of
// two up to 64), left in every lane: the pairings above within rows of 16,
// lane shuffles beyond.  Every lane gets the same bits (the exchanges are
// symmetric).
template <bool MAX>
__device__ inline double seg_allreduce(double v, int SW)
{
    auto op = [](double x, double y) { return MAX ? fmax(x, y) : x + y; };
    if (SW >= 16) v = op(v, seg_swap<0>(v));
    if (SW >= 8) v = op(v, seg_swap<1>(v));
    if (SW >= 4) v = op(v, seg_swap<2>(v));
    if (SW >= 2) v = op(v, seg_swap<3>(v));
    if (SW >= 32) v = op(v, __shfl_xor(v, 16, 64));
    if (SW >= 64) v = op(v, __shfl_xor(v, 32, 64));
    return v;
}

// One modality's units of contexts [t0, t0 + nc): RB rows per block (every
// row of a block loaded before any is used), P >= RB the power of two the
// segment reduction works on.
template <int RB, bool WIDE>
__device__ void zv_tile_modality(const AgentArgs &a, const ModDesc &md, int agent, int m, int t0, int nc,
                                 const double *q, double *zv, const int *sobs, int64_t llo, int first)
{
    constexpr int P = RB <= 1 ? 1 : RB <= 2 ? 2 : RB <= 4 ? 4 : RB <= 8 ? 8 : 16;
    constexpr int LP = log2_floor(P);
    const int R = md.R, C = md.C, Cp = md.Cp;
    const int nch = tile_nch(C), units = nc * nch;
    const int seg = (int)threadIdx.x / kSeg, sl = (int)threadIdx.x % kSeg;
    const double *la = at<double>(a.base, md.la_off) + (a.shared ? 0 : (int64_t)agent * md.la_agent);
    const bool zrow = md.nrow > 0;
    const int zlen = zrow ? nch * R : 0;
    const int rn1 = md.nrow == 2 ? md.rn[1] : 1, cn1 = md.ncol == 2 ? md.cn[1] : 1;
    int u = seg - first % kSegs;
    if (u < 0) u += kSegs;
    for (; u < units; u += kSegs) {
        const int c = u / nch, cb = u - c * nch;
        const int t = t0 + c;
        const double *qt = q + t * a.ntot;
        const double *X = a.ll ? a.ll + ((int64_t)agent * a.T + t) * a.llpc + llo
                               : la + (int64_t)sobs[t * a.M + m] * md.slice;
        double *blk = zv + c * a.zvpc + a.zt[m];
        // this lane's columns col, col + 1 (col even; Cp is a multiple of 4,
        // so the pair is one aligned 16-byte load and col + 1 < Cp)
        const int col = cb * kTileCols + 2 * sl;
        const int colc = min(col, (C - 1) & ~1);
        double w0 = 0.0, w1 = 0.0;
        if (zrow) {
            const int ca = min(col, C - 1), cbb = min(col + 1, C - 1);
            if (WIDE && md.ncol > 2) {
                w0 = side_weight(a, qt, md.cf, md.cn, md.ncol, ca);
                w1 = side_weight(a, qt, md.cf, md.cn, md.ncol, cbb);
            } else {
                const double *qc0 = qt + a.facs[md.cf[0]].q_off;
                const double *qc1 = md.ncol == 2 ? qt + a.facs[md.cf[1]].q_off : nullptr;
                const int a0 = ca / cn1, a1 = ca - a0 * cn1, b0 = cbb / cn1, b1 = cbb - b0 * cn1;
                w0 = qc1 ? qc0[a0] * qc1[a1] : qc0[a0];
                w1 = qc1 ? qc0[b0] * qc1[b1] : qc0[b0];
            }
            w0 = col < C ? w0 : 0.0;
            w1 = col + 1 < C ? w1 : 0.0;
        }
        const double *qr0 = md.nrow > 0 ? qt + a.facs[md.rf[0]].q_off : nullptr;
        const double *qr1 = md.nrow == 2 ? qt + a.facs[md.rf[1]].q_off : nullptr;
        double v0 = 0.0, v1 = 0.0;
        for (int r0 = 0; r0 < R; r0 += RB) {
            double2 x[RB];
#pragma unroll
            for (int i = 0; i < RB; ++i)
                x[i] = *reinterpret_cast<const double2 *>(X + (int64_t)min(r0 + i, R - 1) * Cp + colc);
            // row weights s[r] (1 for a rank-0 row side)
            int i0 = r0 / rn1, i1 = r0 - i0 * rn1;
            double z[P];
#pragma unroll
            for (int i = 0; i < RB; ++i) {
                double sw = 1.0;
                if (WIDE && md.nrow > 2)
                    sw = side_weight(a, qt, md.rf, md.rn, md.nrow, min(r0 + i, R - 1));
                else if (md.nrow > 0)
                    sw = qr1 ? qr0[min(i0, md.rn[0] - 1)] * qr1[i1] : qr0[min(r0 + i, R - 1)];
                sw = r0 + i < R ? sw : 0.0;
                if (++i1 == rn1) {
                    i1 = 0;
                    ++i0;
                }
                const double x1 = col + 1 < C ? x[i].y : 0.0;   // (column C is padding)
                v0 = fma(sw, x[i].x, v0);
                v1 = fma(sw, x1, v1);
                z[i] = fma(x1, w1, x[i].x * w0);
            }
            if (zrow) {
#pragma unroll
                for (int i = RB; i < P; ++i) z[i] = 0.0;
                seg_halve<0, P>(z, sl);
                const int row = r0 + (sl >> (4 - LP));
                if ((sl & ((1 << (4 - LP)) - 1)) == 0 && row < R) blk[cb * R + row] = z[0];
            }
        }
        double *V = blk + zlen;
        if (col < C) V[col] = v0;
        if (col + 1 < C) V[col + 1] = v1;
    }
}

// A modality of the tile layout outside the tile form: one Z or V output per
// thread (as phase_zv reads from global memory), written to its block.
template <bool WIDE>
__device__ void zv_thread_modality(const AgentArgs &a, const ModDesc &md, int agent, int m, int t0, int nc,
                                   const double *q, double *zv, const int *sobs, int64_t llo, int first)
{
    const int per = md.R + md.C, cnt = nc * per;
    const double *la = at<double>(a.base, md.la_off) + (a.shared ? 0 : (int64_t)agent * md.la_agent);
    int i = (int)threadIdx.x - first % kThreads;
    if (i < 0) i += kThreads;
    for (; i < cnt; i += kThreads) {
        const int c = i / per, j = i - c * per;
        const int t = t0 + c;
        const double *X = a.ll ? a.ll + ((int64_t)agent * a.T + t) * a.llpc + llo
                               : la + (int64_t)sobs[t * a.M + m] * md.slice;
        zv[c * a.zvpc + a.zt[m] + j] = zv_one<WIDE>(a, md, X, md.Cp, q + t * a.ntot, j);
    }
}

// MIXED: modalities outside a.tilemask take one dot product per thread
template <bool WIDE, bool MIXED>
__device__ void phase_zv_tile(const AgentArgs &a, int agent, int t0, int nc, const double *q, double *zv,
                              const int *sobs)
{
    int first = 0, tfirst = 0;
    int64_t llo = 0;
    for (int m = 0; m < a.M; ++m) {
        const ModDesc &md = a.mods[m];
        const int R = md.R;
        if (MIXED && !((a.tilemask >> m) & 1)) {
            zv_thread_modality<WIDE>(a, md, agent, m, t0, nc, q, zv, sobs, llo, tfirst);
            tfirst += nc * (md.R + md.C);
            llo += md.slice;
            continue;
        }
        if (R <= 1)
            zv_tile_modality<1, WIDE>(a, md, agent, m, t0, nc, q, zv, sobs, llo, first);
        else if (R <= 2)
            zv_tile_modality<2, WIDE>(a, md, agent, m, t0, nc, q, zv, sobs, llo, first);
        else if (R <= 4)
            zv_tile_modality<4, WIDE>(a, md, agent, m, t0, nc, q, zv, sobs, llo, first);
        else if (R <= 8)
            zv_tile_modality<8, WIDE>(a, md, agent, m, t0, nc, q, zv, sobs, llo, first);
        else   // (blocks of 12 rows beyond: 16 would spill at three workgroups per CU)
            zv_tile_modality<12, WIDE>(a, md, agent, m, t0, nc, q, zv, sobs, llo, first);
        first += nc * tile_nch(md.C);
        llo += md.slice;
    }
}

// Phase 2: lam of contexts [t0, t0 + nc) into lam[t][ntot].  TILE: Z/V in the
// tile layout (Z as per-chunk partial sums; MIXED: only for the modalities in
// a.tilemask, the others Z [R] then V [C]).
// lam of state s of factor f in chunk context c (qt: the marginals of its step)
template <bool TILE, int BT, bool WIDE, bool MIXED>
__device__ inline double lam_one(const AgentArgs &a, int c, int f, int s, const double *qt, const double *zv)
{
    double acc = 0.0;
    for (int m = 0; m < a.M; ++m) {
        const ModDesc &md = a.mods[m];
        const double *Z = zv + c * a.zvpc + (TILE ? a.zt[m] : md.zv_off);
        const bool tiled = TILE && (!MIXED || ((a.tilemask >> m) & 1));
        const int nch = tiled ? tile_nch(md.C) : 1;
        const double *V = Z + (tiled ? (md.nrow > 0 ? nch * md.R : 0) : md.R);
        // Z[k]: the sum of its column chunks' partial sums
        auto zat = [&](int k) {
            double z = Z[k];
            for (int cb = 1; cb < nch; ++cb) z += Z[cb * md.R + k];
            return z;
        };
        if (WIDE && (md.nrow > 2 || md.ncol > 2)) {
            // a side of more than two factors: the lines whose digit of f
            // is s, weighted by the side's other marginals
            for (int side = 0; side < 2; ++side) {
                const int k = side ? md.ncol : md.nrow;
                const int32_t *sf = side ? md.cf : md.rf, *sn = side ? md.cn : md.rn;
                for (int p = 0; p < k; ++p) {
                    if (sf[p] != f) continue;
                    int low = 1;
                    for (int g = p + 1; g < k; ++g) low *= sn[g];
                    const int np = sn[p], len = (side ? md.C : md.R) / np;
                    auto line = [&](int jj) {
                        const int hi = jj / low;
                        return (hi * np + s) * low + (jj - hi * low);
                    };
                    acc += dot8<BT>(len, [&](int jj) { return side ? V[line(jj)] : zat(line(jj)); },
                                    [&](int jj) { return side_weight(a, qt, sf, sn, k, line(jj), p); });
                }
            }
        } else if (md.nrow >= 1 && md.rf[0] == f) {
            if (md.nrow == 1) {
                acc += zat(s);
            } else {
                const double *q1 = qt + a.facs[md.rf[1]].q_off;
                const int n1 = md.rn[1];
                acc += dot8<BT>(n1, [&](int r1) { return zat(s * n1 + r1); }, [&](int r1) { return q1[r1]; });
            }
        } else if (md.nrow == 2 && md.rf[1] == f) {
            const double *q0 = qt + a.facs[md.rf[0]].q_off;
            const int n0 = md.rn[0], n1 = md.rn[1];
            acc += dot8<BT>(n0, [&](int r0) { return zat(r0 * n1 + s); }, [&](int r0) { return q0[r0]; });
        } else if (md.cf[0] == f) {
            if (md.ncol == 1) {
                acc += V[s];
            } else {
                const double *q1 = qt + a.facs[md.cf[1]].q_off;
                const int n1 = md.cn[1];
                acc += dot8<BT>(n1, [&](int c1) { return V[s * n1 + c1]; }, [&](int c1) { return q1[c1]; });
            }
        } else if (md.ncol == 2 && md.cf[1] == f) {
            const double *q0 = qt + a.facs[md.cf[0]].q_off;
            const int n0 = md.cn[0], n1 = md.cn[1];
            acc += dot8<BT>(n0, [&](int c0) { return V[c0 * n1 + s]; }, [&](int c0) { return q0[c0]; });
        }
    }
    return acc;
}

template <bool TILE, int BT, bool WIDE, bool MIXED = false>
__device__ void phase_lam(const AgentArgs &a, int t0, int nc, const double *q, const double *zv, const int *sfac,
                          double *lam)
{
    for (int i = threadIdx.x; i < nc * a.ntot; i += kThreads) {
        const int c = i / a.ntot, j = i - c * a.ntot;
        const int f = sfac[j];
        lam[(t0 + c) * a.ntot + j] =
            lam_one<TILE, BT, WIDE, MIXED>(a, c, f, j - a.facs[f].q_off, q + (t0 + c) * a.ntot, zv);
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

// batch of the LDS dot products in the window kernel (see dot8)
template <int SRC> constexpr int kBatch = SRC == kSrcLdsShort ? 1 : 8;

// lam for every context of the window (phases 1 and 2 over context chunks;
// staged chunks are copied to LDS first unless the whole window is resident).
template <int SRC, bool WIDE>
__device__ void window_lam(const AgentArgs &a, int agent, const double *q, double *zv, double *stg, const int *sfac,
                           const int *sobs, double *lam)
{
    for (int t0 = 0; t0 < a.T; t0 += a.nc) {
        const int nc = min(a.nc, a.T - t0);
        if (a.stage == kStageChunk) {
            stage_slices(a, agent, t0, nc, stg);
            __syncthreads();
        }
        if (SRC == kSrcTile)
            phase_zv_tile<WIDE, false>(a, agent, t0, nc, q, zv, sobs);
        else
            phase_zv<SRC == kSrcGlobal, kBatch<SRC>, WIDE>(a, agent, t0, nc, q, zv, stg,
                                                           a.stage == kStageWindow ? t0 : 0);
        __syncthreads();
        phase_lam<SRC == kSrcTile, kBatch<SRC>, WIDE>(a, t0, nc, q, zv, sfac, lam);
        __syncthreads();
    }
}

// Copy the window's outcomes [T][M] into LDS (tile form).
__device__ void stage_obs(const AgentArgs &a, int agent, int *sobs)
{
    const int n = a.T * a.M;
    for (int i = threadIdx.x; i < n; i += kThreads) sobs[i] = a.obs[(int64_t)agent * n + i];
}

// Copy the agent's B (fp32) or log B (fp64, lb) of every factor into tab.
__device__ void stage_b(const AgentArgs &a, int agent, bool lb, double *tab)
{
    const int64_t am = a.shared ? 0 : agent;
    for (int f = 0; f < a.F; ++f) {
        const FacDesc &fd = a.facs[f];
        const int cnt = fd.U * fd.n * fd.bstates;
        if (lb) {
            const double *src = at<double>(a.base, fd.lb_off) + am * fd.b_agent;
            for (int i = threadIdx.x; i < cnt; i += kThreads) tab[a.bo[f] + i] = src[i];
        } else {
            const float *src = at<float>(a.base, fd.b_off) + am * fd.b_agent;
            float *dst = reinterpret_cast<float *>(tab) + a.bo[f];
            for (int i = threadIdx.x; i < cnt; i += kThreads) dst[i] = src[i];
        }
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

// Segmented softmax over the window: logits v[t][j] of every (step, state)
// are in LDS; each thread owns states i = threadIdx.x + k * kThreads and
// reads its (t, f) segment for the max and, after the exponentials are
// written to e, for the sum.  Every lane works whatever the factor sizes
// (a wave per (t, f) would leave 64 - n_f lanes idle).  Writes out (damped
// towards cur when tau != 1).  Three barriers.
template <int BT>
__device__ void window_softmax(const AgentArgs &a, const int *sfac, const double *v, double *e, const double *cur,
                               double *out)
{
    const int TN = a.T * a.ntot;
    for (int i = threadIdx.x; i < TN; i += kThreads) {
        const int t = i / a.ntot, j = i - t * a.ntot;
        const FacDesc &fd = a.facs[sfac[j]];
        const double mx = seg_max<BT>(v + t * a.ntot + fd.q_off, fd.n);
        e[i] = exp(v[i] - mx);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < TN; i += kThreads) {
        const int t = i / a.ntot, j = i - t * a.ntot;
        const FacDesc &fd = a.facs[sfac[j]];
        const double sum = seg_sum<BT>(e + t * a.ntot + fd.q_off, fd.n);
        const double qn = e[i] / sum;
        out[i] = a.tau != 1.0 ? (1.0 - a.tau) * cur[i] + a.tau * qn : qn;
    }
    __syncthreads();
}

// Transition messages and masked softmax of every (step, factor), trivial
// B-dependency lists: one segment of a.sw lanes (a power of two >= every n_f)
// per (t, f), a lane per state; the segment's maximum and sum come from lane
// exchanges, so the update is one pass with no LDS round trip or barrier
// between its phases (a thread per state took three passes, each reading the
// (t, f) segment back from LDS).  Writes the new marginals to nxt.
template <int ALGO, int BT>
__device__ void window_update_seg(const AgentArgs &a, int agent, int64_t am, const double *cur, const double *lam,
                                  const double *btab, double *nxt)
{
    const int SW = a.sw, sl = (int)threadIdx.x % SW;
    for (int sg = (int)threadIdx.x / SW; sg < a.T * a.F; sg += kThreads / SW) {
        const int t = sg / a.F, f = sg - t * a.F;
        const FacDesc &fd = a.facs[f];
        const int n = fd.n, s = min(sl, n - 1);
        const int j = fd.q_off + s, i = t * a.ntot + j;
        const double *LB = a.bst ? btab + a.bo[f] : at<double>(a.base, fd.lb_off) + am * fd.b_agent;
        const float *Bf = a.bst ? reinterpret_cast<const float *>(btab) + a.bo[f]
                                : at<float>(a.base, fd.b_off) + am * fd.b_agent;
        double fwd, bwd = 0.0;
        if (t == 0) {
            fwd = a.prior ? ln_clamped((double)a.prior[(int64_t)agent * a.ntot + j])
                          : at<double>(a.base, fd.ld_off)[am * fd.ld_agent + s];
        } else {
            const int up = a.act[((int64_t)agent * (a.T - 1) + t - 1) * a.F + f];
            const double *qprev = cur + (t - 1) * a.ntot + fd.q_off;
            if (ALGO == BI_ALGO_VMP) {
                const double *row = LB + (int64_t)up * n * n + s * n;   // [i][j]
                fwd = dot8<BT>(n, [&](int jj) { return row[jj]; }, [&](int jj) { return qprev[jj]; });
            } else {
                const float *row = Bf + (int64_t)up * n * n + s * n;
                fwd = ln_clamped(dot8<BT>(n, [&](int jj) { return (double)row[jj]; }, [&](int jj) { return qprev[jj]; }));
            }
        }
        if (t + 1 < a.T) {
            const int un = a.act[((int64_t)agent * (a.T - 1) + t) * a.F + f];
            const double *qnext = cur + (t + 1) * a.ntot + fd.q_off;
            if (ALGO == BI_ALGO_VMP) {
                const double *col = LB + (int64_t)un * n * n + s;
                bwd = dot8<BT>(n, [&](int ii) { return qnext[ii]; }, [&](int ii) { return col[ii * n]; });
            } else {
                const float *col = Bf + (int64_t)un * n * n + s;
                bwd = ln_clamped(
                    dot8<BT>(n, [&](int ii) { return qnext[ii]; }, [&](int ii) { return (double)col[ii * n]; }));
            }
        }
        const double lm = lam[i];
        const double v = ALGO == BI_ALGO_VMP ? lm + fwd + bwd : t + 1 < a.T ? lm + 0.5 * (fwd + bwd) : lm + fwd;
        const bool act = sl < n;
        const double mx = seg_allreduce<true>(act ? v : -INFINITY, SW);
        const double e = act ? exp(v - mx) : 0.0;
        const double sum = seg_allreduce<false>(e, SW);
        if (act) {
            const double qn = e / sum;
            nxt[i] = a.tau != 1.0 ? (1.0 - a.tau) * cur[i] + a.tau * qn : qn;
        }
    }
}

// ALGO: BI_ALGO_VMP or BI_ALGO_MMP; SRC: where phase 1 reads the slices; TB:
// every B-dependency list is {f} (the row / column transition products;
// otherwise the general contractions of transition.h)
template <int ALGO, int SRC, bool TB, bool WIDE>
__global__ __launch_bounds__(kThreads, SRC == kSrcTile ? 3 : 4) void agent_window_kernel(AgentArgs a)
{
    extern __shared__ double smem[];
    const int agent = blockIdx.x;
    const int TN = a.T * a.ntot;
    double *qa = smem, *qb = qa + TN, *lam = qb + TN, *zv = lam + TN, *stg = zv + a.nc * a.zvpc;
    const int nstg = a.stage == kStageWindow ? a.T : a.stage == kStageChunk ? a.nc : 0;
    double *btab = stg + (int64_t)nstg * a.sctx;
    int *sfac = reinterpret_cast<int *>(btab + a.bdoubles);
    int *sobs = sfac + a.ntot;
    init_tables(a, sfac);
    if (SRC == kSrcTile && !a.ll) stage_obs(a, agent, sobs);
    if (a.bst) stage_b(a, agent, ALGO == BI_ALGO_VMP, btab);
    if (a.stage == kStageWindow) stage_slices(a, agent, 0, a.T, stg);   // every iteration reads them from LDS
    __syncthreads();
    for (int i = threadIdx.x; i < TN; i += kThreads) qa[i] = 1.0 / a.facs[sfac[i % a.ntot]].n;
    __syncthreads();
    const int64_t am = a.shared ? 0 : agent;
    double *cur = qa, *nxt = qb;
    for (int k = 0; k < a.iters; ++k) {
        window_lam<SRC, WIDE>(a, agent, cur, zv, stg, sfac, sobs, lam);
        if (TB && a.sw) {
            window_update_seg<ALGO, kBatch<SRC>>(a, agent, am, cur, lam, btab, nxt);
            __syncthreads();
            double *tmp = cur;
            cur = nxt;
            nxt = tmp;
            continue;
        }
        // logits of every (t, state) into nxt, one thread per state
        for (int i = threadIdx.x; i < TN; i += kThreads) {
            const int t = i / a.ntot, j = i - t * a.ntot;
            const int f = sfac[j];
            const FacDesc &fd = a.facs[f];
            const int n = fd.n, s = j - fd.q_off;
            const double *qprev = t > 0 ? cur + (t - 1) * a.ntot + fd.q_off : nullptr;
            const double *qnext = t + 1 < a.T ? cur + (t + 1) * a.ntot + fd.q_off : nullptr;
            const int up = t > 0 ? a.act[((int64_t)agent * (a.T - 1) + t - 1) * a.F + f] : 0;
            const int un = t + 1 < a.T ? a.act[((int64_t)agent * (a.T - 1) + t) * a.F + f] : 0;
            // VMP uses log B, MMP the linear B (log taken after the product)
            const double *LB = a.bst ? btab + a.bo[f] : at<double>(a.base, fd.lb_off) + am * fd.b_agent;
            const float *Bf = a.bst ? reinterpret_cast<const float *>(btab) + a.bo[f]
                                    : at<float>(a.base, fd.b_off) + am * fd.b_agent;
            double fwd, bwd = 0.0;
            if (!TB) {
                // general B-dependencies: forward message from the factors f
                // depends on, one backward message per child j of f
                const BDep df = bdep_of(a.facs, fd);
                const int bs = df.bs;
                if (t == 0)
                    fwd = a.prior ? ln_clamped((double)a.prior[(int64_t)agent * a.ntot + j])
                                  : at<double>(a.base, fd.ld_off)[am * fd.ld_agent + s];
                else if (ALGO == BI_ALGO_VMP)
                    fwd = bdep_row(df, LB + ((int64_t)up * n + s) * bs, cur + (t - 1) * a.ntot, -1, 0);
                else
                    fwd = ln_clamped(bdep_row(df, Bf + ((int64_t)up * n + s) * bs, cur + (t - 1) * a.ntot, -1, 0));
                int children = 0;
                if (t + 1 < a.T) {
                    for (int c = 0; c < fd.nch; ++c) {
                        const int jf = fd.ch[c], pos = fd.chpos[c];
                        const FacDesc &fj = a.facs[jf];
                        const BDep dj = bdep_of(a.facs, fj);
                        const int nj = fj.n;
                        const int uj = a.act[((int64_t)agent * (a.T - 1) + t) * a.F + jf];
                        const int64_t tab = (int64_t)uj * nj * dj.bs;
                        const double *qn = cur + (t + 1) * a.ntot + fj.q_off;
                        double msg = 0.0;
                        if (ALGO == BI_ALGO_VMP) {
                            const double *LBj =
                                (a.bst ? btab + a.bo[jf] : at<double>(a.base, fj.lb_off) + am * fj.b_agent) + tab;
                            for (int sn = 0; sn < nj; ++sn)
                                msg = fma(qn[sn], bdep_row(dj, LBj + (int64_t)sn * dj.bs, cur + t * a.ntot, pos, s),
                                          msg);
                            bwd += msg;
                        } else {
                            const float *Bj = (a.bst ? reinterpret_cast<const float *>(btab) + a.bo[jf]
                                                     : at<float>(a.base, fj.b_off) + am * fj.b_agent) + tab;
                            for (int sn = 0; sn < nj; ++sn)
                                msg = fma(qn[sn], bdep_row(dj, Bj + (int64_t)sn * dj.bs, cur + t * a.ntot, pos, s),
                                          msg);
                            bwd += ln_clamped(msg);
                        }
                        ++children;
                    }
                }
                const double lm = lam[i];
                if (ALGO == BI_ALGO_VMP)
                    nxt[i] = lm + fwd + bwd;
                else
                    nxt[i] = children > 0 ? lm + (fwd + bwd) / (double)(1 + children) : lm + fwd;
                continue;
            }
            if (t == 0) {
                fwd = a.prior ? ln_clamped((double)a.prior[(int64_t)agent * a.ntot + j])
                              : at<double>(a.base, fd.ld_off)[am * fd.ld_agent + s];
            } else if (ALGO == BI_ALGO_VMP) {
                const double *row = LB + (int64_t)up * n * n + s * n;   // [i][j]
                fwd = dot8<kBatch<SRC>>(n, [&](int jj) { return row[jj]; }, [&](int jj) { return qprev[jj]; });
            } else {
                const float *row = Bf + (int64_t)up * n * n + s * n;
                fwd = ln_clamped(dot8<kBatch<SRC>>(n, [&](int jj) { return (double)row[jj]; }, [&](int jj) { return qprev[jj]; }));
            }
            if (qnext) {
                if (ALGO == BI_ALGO_VMP) {
                    const double *col = LB + (int64_t)un * n * n + s;
                    bwd = dot8<kBatch<SRC>>(n, [&](int ii) { return qnext[ii]; }, [&](int ii) { return col[ii * n]; });
                } else {
                    const float *col = Bf + (int64_t)un * n * n + s;
                    bwd = ln_clamped(
                        dot8<kBatch<SRC>>(n, [&](int ii) { return qnext[ii]; }, [&](int ii) { return (double)col[ii * n]; }));
                }
            }
            const double lm = lam[i];
            if (ALGO == BI_ALGO_VMP)
                nxt[i] = lm + fwd + bwd;
            else
                nxt[i] = qnext ? lm + 0.5 * (fwd + bwd) : lm + fwd;
        }
        __syncthreads();
        // lam is free again: it takes the exponentials
        window_softmax<kBatch<SRC>>(a, sfac, nxt, lam, cur, nxt);
        double *tmp = cur;
        cur = nxt;
        nxt = tmp;
    }
    float *out = a.q + (int64_t)agent * TN;
    for (int i = threadIdx.x; i < TN; i += kThreads) out[i] = (float)cur[i];
}

// GX: slices read from global memory (TILE: in the tile form); TB: trivial
// B-dependency lists; WIDE: some modality has a side of more than two factors
template <bool GX, bool TB, bool WIDE, bool TILE>
__global__ __launch_bounds__(kThreads, TILE ? 3 : 4) void agent_filter_kernel(AgentArgs a)
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
    double *btab = stg + (int64_t)nstg * a.sctx;
    int *sfac = reinterpret_cast<int *>(btab + a.bdoubles);
    int *sobs = sfac + a.ntot;
    init_tables(a, sfac);
    if (TILE && !a.ll) stage_obs(a, agent, sobs);
    if (a.bst) stage_b(a, agent, false, btab);
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
                const float *Bp = (a.bst ? reinterpret_cast<const float *>(btab) + a.bo[f]
                                         : at<float>(a.base, fd.b_off) + am * fd.b_agent) +
                                  (int64_t)u * n * fd.bstates;
                if (TB) {
                    const double *qp = qfin + (t - 1) * a.ntot + fd.q_off;
                    for (int s = lane; s < n; s += 64)
                        lp[s] = ln_clamped(
                            dot8<8>(n, [&](int j) { return (double)Bp[s * n + j]; }, [&](int j) { return qp[j]; }));
                } else {   // predictive marginal under the factorised q_{t-1}
                    const BDep df = bdep_of(a.facs, fd);
                    for (int s = lane; s < n; s += 64)
                        lp[s] = ln_clamped(bdep_row(df, Bp + (int64_t)s * df.bs, qfin + (t - 1) * a.ntot, -1, 0));
                }
            }
        }
        double *qt = cur + t * a.ntot;
        for (int j = threadIdx.x; j < a.ntot; j += kThreads) qt[j] = 1.0 / a.facs[sfac[j]].n;
        if (a.stage == kStageChunk) stage_slices(a, agent, t, 1, stg);   // step t's slices, for all its iterations
        __syncthreads();
        // with factor segments (a.sw) the iterate alternates between row t
        // of cur and of lam: each iteration reads one and writes the other
        double *qa = cur, *qb = lam;
        for (int k = 0; k < a.iters; ++k) {
            if (TILE)
                phase_zv_tile<WIDE, true>(a, agent, t, 1, qa, zv, sobs);
            else
                phase_zv<GX, 8, WIDE>(a, agent, t, 1, qa, zv, stg, a.stage == kStageWindow ? t : 0);
            __syncthreads();
            if (a.sw) {
                // one segment of a.sw lanes per factor, a lane per state: its
                // lam, the prior, and the softmax from lane exchanges, in one
                // pass (instead of a lam pass, a barrier and a wave per factor)
                const int SW = a.sw, sl = (int)threadIdx.x % SW, f = (int)threadIdx.x / SW;
                if (f < a.F) {
                    const FacDesc &fd = a.facs[f];
                    const int n = fd.n, s = min(sl, n - 1);
                    const double *qr = qa + t * a.ntot;
                    const double v = lam_one<TILE, 8, WIDE, true>(a, 0, f, s, qr, zv) + logp[fd.q_off + s];
                    const bool act = sl < n;
                    const double mx = seg_allreduce<true>(act ? v : -INFINITY, SW);
                    const double e = act ? exp(v - mx) : 0.0;
                    const double sum = seg_allreduce<false>(e, SW);
                    if (act) {
                        const double qn = e / sum;
                        qb[t * a.ntot + fd.q_off + s] = a.tau != 1.0 ? (1.0 - a.tau) * qr[fd.q_off + s] + a.tau * qn : qn;
                    }
                }
                __syncthreads();
                double *tmp = qa;
                qa = qb;
                qb = tmp;
                continue;
            }
            phase_lam<TILE, 8, WIDE, true>(a, t, 1, cur, zv, sfac, lam);
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
        for (int j = threadIdx.x; j < a.ntot; j += kThreads) qfin[t * a.ntot + j] = qa[t * a.ntot + j];
        __syncthreads();
    }
    float *out = a.q + (int64_t)agent * TN;
    for (int i = threadIdx.x; i < TN; i += kThreads) out[i] = (float)qfin[i];
}

constexpr size_t kLdsMax = 160 * 1024;
#ifndef BI_SEG_UPDATE
#define BI_SEG_UPDATE 1
#endif
constexpr bool kSegUpdate = BI_SEG_UPDATE;


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
    // lanes per (step, factor) segment of the window kernels' update: the
    // power of two covering the largest factor, up to a wave
    // (FPI: segments of every factor in one pass of the workgroup)
    a.sw = 0;
    if (algo == BI_ALGO_FPI || m->trivial_b) {
        int nmax = 1;
        for (const FacDesc &fd : m->facs) nmax = std::max(nmax, (int)fd.n);
        int sw = 1;
        while (sw < nmax) sw *= 2;
        const bool fits = sw <= 64 && (algo != BI_ALGO_FPI || (int64_t)m->F * sw <= kThreads);
        a.sw = kSegUpdate && fits ? sw : 0;
    }
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
    // transition tables: staged when they fit kBStageMax
    {
        int64_t elems = 0;
        for (int f = 0; f < m->F && f <= kStageMaxF; ++f) {
            if (f < kStageMaxF) a.bo[f] = (int)elems;
            elems += (int64_t)m->facs[f].U * m->facs[f].n * m->facs[f].bstates;
        }
        const size_t bytes = (size_t)elems * (algo == BI_ALGO_VMP ? 8 : 4);
        a.bst = m->F <= kStageMaxF && bytes <= kBStageMax;
        a.bdoubles = a.bst ? (int)((bytes + 7) / 8) : 0;
    }
    const size_t bt = 8 * (size_t)a.bdoubles;
    size_t fixed, per_ctx = (size_t)m->zvpc * 8, lds;
    a.stage = kStageNone;
    if (algo == BI_ALGO_FPI) {
        fixed = (3 * TN + m->ntot) * 8 + (size_t)m->ntot * 4 + per_ctx + bt;
        a.nc = 1;
        if (can_stage && fixed + T * sb <= budget2)
            a.stage = kStageWindow;
        else if (can_stage && fixed + sb <= kLdsMax)
            a.stage = kStageChunk;
        lds = fixed + (a.stage == kStageWindow ? T * sb : a.stage == kStageChunk ? sb : 0);
    } else {
        fixed = 3 * TN * 8 + (size_t)m->ntot * 4 + bt;
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
    // Slices from global memory: the tile form of phase 1 when its Z/V layout
    // fits (per context: the Z partial sums of every column chunk and V), with
    // the window's outcomes in LDS; FPI only for the modalities of at most
    // kTileMaxRows rows (the others one dot product per thread).
    a.tile = 0;
    a.tilemask = 0;
    for (int i = 0; i < m->M && i < kStageMaxM; ++i)
        if (algo != BI_ALGO_FPI || m->mods[i].R <= kTileMaxRows) a.tilemask |= 1u << i;
    if (a.stage == kStageNone && m->M <= kStageMaxM && a.tilemask != 0) {
        int zt = 0;
        for (int i = 0; i < m->M; ++i) {
            a.zt[i] = zt;
            zt += tile_block(m->mods[i], (a.tilemask >> i) & 1);
        }
        a.zt[m->M] = zt;
        const size_t pc = (size_t)zt * 8, so = (size_t)T * m->M * 4;
        // the whole window in one chunk when it fits 80 KB, else as many
        // contexts as 160 KB allow (chunks sized for three workgroups per CU
        // measured 5% slower on the model sweep: more barriers per sweep)
        const size_t fx = fixed + so - (algo == BI_ALGO_FPI ? per_ctx : 0);
        size_t nc = algo == BI_ALGO_FPI ? 1 : T;
        if (algo != BI_ALGO_FPI && fx + nc * pc > budget2) nc = fx < kLdsMax ? (kLdsMax - fx) / pc : 0;
        if (nc > (size_t)T) nc = T;
        const size_t lt = fx + nc * pc;
        if (nc >= 1 && lt <= kLdsMax) {
            a.tile = 1;
            a.nc = (int)nc;
            a.zvpc = zt;
            lds = lt;
        }
    }
    if (a.nc < 1 || lds > kLdsMax)
        return fail(BI_ERR_UNSUPPORTED, "agent working set (%zu bytes of LDS) exceeds the 160 KB budget", lds);
    int src = a.tile ? kSrcTile : a.stage == kStageNone ? kSrcGlobal : kSrcLds;
    if (src == kSrcLds) {
        int longest = 0;
        for (const FacDesc &fd : m->facs) longest = std::max(longest, (int)fd.n);
        for (const ModDesc &md : m->mods) longest = std::max(longest, (int)std::max(md.R, md.C));
        if (longest <= 8) src = kSrcLdsShort;
    }
    const bool tb = m->trivial_b;
    // instantiation tables [src][tb][wide]; wide: some modality has a side of
    // more than two factors (the general side code is compiled only there)
    bool wide = false;
    for (const ModDesc &md : m->mods) wide = wide || md.nrow > 2 || md.ncol > 2;
#define BI_FILTER(GX, TB) \
    { (const void *)agent_filter_kernel<GX, TB, false, false>, (const void *)agent_filter_kernel<GX, TB, true, false> }
#define BI_FILTER_TILE(TB) \
    { (const void *)agent_filter_kernel<true, TB, false, true>, (const void *)agent_filter_kernel<true, TB, true, true> }
#define BI_WINDOW(ALGO, SRC, TB) \
    { (const void *)agent_window_kernel<ALGO, SRC, TB, false>, (const void *)agent_window_kernel<ALGO, SRC, TB, true> }
    static const void *const kFilter[3][2][2] = {{BI_FILTER(false, false), BI_FILTER(false, true)},
                                                 {BI_FILTER(true, false), BI_FILTER(true, true)},
                                                 {BI_FILTER_TILE(false), BI_FILTER_TILE(true)}};
    static const void *const kVmp[4][2][2] = {
        {BI_WINDOW(BI_ALGO_VMP, kSrcLds, false), BI_WINDOW(BI_ALGO_VMP, kSrcLds, true)},
        {BI_WINDOW(BI_ALGO_VMP, kSrcGlobal, false), BI_WINDOW(BI_ALGO_VMP, kSrcGlobal, true)},
        {BI_WINDOW(BI_ALGO_VMP, kSrcTile, false), BI_WINDOW(BI_ALGO_VMP, kSrcTile, true)},
        {BI_WINDOW(BI_ALGO_VMP, kSrcLdsShort, false), BI_WINDOW(BI_ALGO_VMP, kSrcLdsShort, true)}};
    static const void *const kMmp[4][2][2] = {
        {BI_WINDOW(BI_ALGO_MMP, kSrcLds, false), BI_WINDOW(BI_ALGO_MMP, kSrcLds, true)},
        {BI_WINDOW(BI_ALGO_MMP, kSrcGlobal, false), BI_WINDOW(BI_ALGO_MMP, kSrcGlobal, true)},
        {BI_WINDOW(BI_ALGO_MMP, kSrcTile, false), BI_WINDOW(BI_ALGO_MMP, kSrcTile, true)},
        {BI_WINDOW(BI_ALGO_MMP, kSrcLdsShort, false), BI_WINDOW(BI_ALGO_MMP, kSrcLdsShort, true)}};
#undef BI_FILTER
#undef BI_FILTER_TILE
#undef BI_WINDOW
    const void *fn = algo == BI_ALGO_FPI ? kFilter[a.tile ? 2 : a.stage == kStageNone ? 1 : 0][tb][wide]
                     : algo == BI_ALGO_VMP ? kVmp[src][tb][wide]
                                           : kMmp[src][tb][wide];
    hipError_t e = func_max_lds(fn, (int)kLdsMax);
    if (e == hipSuccess) {
        ProfScope p(algo == BI_ALGO_FPI ? (a.tile ? "agent_filter_tile" : "agent_filter")
                                    : a.tile ? "agent_window_tile" : "agent_window",
                stream);
        void *args[] = {&a};
        e = hipLaunchKernel(fn, dim3(b), dim3(kThreads), args, lds, stream);
    }
    if (e != hipSuccess) return fail(BI_ERR_DEVICE, "kernel launch failed: %s", hipGetErrorString(e));
    return BI_OK;
}

}  // namespace bi
