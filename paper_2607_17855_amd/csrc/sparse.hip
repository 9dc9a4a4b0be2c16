// Sparse likelihood messages (BI_SPARSE_A, models shared by every agent):
// fp64 gathers over the nonzero entries of the observed slices.
//
// With the slice X = LN(A_m[o]) - ln(eps) (layout.h) the structural zeros of
// A are exact zeros of X and drop out of both contractions of the two-sided
// view (Sec. IV marginalisation; the dropped constant ln(eps) times the
// product of the other factors' marginals is the same for every state of the
// receiving factor, so it cancels in the softmax):
//   Z[c][r]   = sum_{(r,col) in X} X[r][col] q_c0[col_0] q_c1[col_1]   (CSR lines)
//   V[c][col] = sum_{(r,col) in X} X[r][col] q_r0[r_0]   q_r1[r_1]     (CSC lines)
// followed by the fold of the line values into the line factors' messages.
// Both contractions are one "line" kernel: role 0 runs over the rows with the
// column factors as the entry side, role 1 over the columns with the row
// factors as the entry side.
//
// A workgroup (16 waves) owns one tile of lines of one (modality, role,
// outcome).  Its lanes are the contexts that observed the outcome, 64 at a
// time; every wave walks its lines' entries in order (the entry stream is
// uniform across the wave, so entries come in through scalar loads) and each
// lane gathers its own context's entry-side marginals from LDS tables
// (laid out [state][lane], conflict-free).  Line values go to an LDS tile;
// after a barrier the tile is folded into the line factors' messages in a
// fixed order and written as partial messages: the first line factor's
// messages of the tile's line groups directly (tiles own disjoint groups),
// the second line factor's as one partial vector per tile (summed by the
// update kernel).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "internal.h"
#include "stream.h"

namespace bi {
namespace {

constexpr int kSpThreads = 768;  // 12 waves, two workgroups per CU: 24 waves hide the latency
constexpr int kSpWaves = kSpThreads / 64;
constexpr int kSpLanes = 48;     // contexts per pass (lanes 48..63 of a wave idle)
constexpr int kSpLines = 128;    // target lines per tile
constexpr int kZS = kSpLanes + 1;  // padded line-tile stride (doubles)
constexpr int kSpBatch = 16;     // entries per gather round (4 x 64-byte scalar loads)

// Entries and line pointers are read through the constant address space:
// the addresses are wave-uniform, so every load is a wide scalar load.
#define BI_CONST __attribute__((address_space(4)))
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// Geometry of one role of a modality.
struct Side {
    int lines, nline, ln0, ln1, lf0, lf1;   // line side
    int nent, en0, en1, ef0, ef1;           // entry side
    int64_t ptr_off, ent_off;
};

__host__ __device__ inline Side side_of(const ModDesc &md, int role)
{
    Side s;
    const bool rows = role == 0;
    s.nline = rows ? md.nrow : md.ncol;
    s.lines = rows ? md.R : md.C;
    s.lf0 = rows ? md.rf[0] : md.cf[0];
    s.lf1 = rows ? md.rf[1] : md.cf[1];
    s.ln0 = s.nline >= 1 ? (rows ? md.rn[0] : md.cn[0]) : 1;
    s.ln1 = s.nline == 2 ? (rows ? md.rn[1] : md.cn[1]) : 1;
    s.nent = rows ? md.ncol : md.nrow;
    s.ef0 = rows ? md.cf[0] : md.rf[0];
    s.ef1 = rows ? md.cf[1] : md.rf[1];
    s.en0 = s.nent >= 1 ? (rows ? md.cn[0] : md.rn[0]) : 1;
    s.en1 = s.nent == 2 ? (rows ? md.cn[1] : md.rn[1]) : 1;
    s.ptr_off = rows ? md.csr_ptr_off : md.csc_ptr_off;
    s.ent_off = rows ? md.csr_ent_off : md.csc_ent_off;
    return s;
}

// sum_{i < n} z[i * zs] w[i] in fp64, in order, with the loads issued 8 at a
// time (the fold's operands sit in LDS and L2: one wait per 8 terms)
__device__ inline double dot_batched(const double *z, int zs, const double *w, int n)
{
    double acc = 0.0;
    int i = 0;
    for (; i + 8 <= n; i += 8) {
        double zv[8], wv[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            zv[k] = z[(i + k) * zs];
            wv[k] = w[i + k];
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) acc = fma(zv[k], wv[k], acc);
    }
    for (; i < n; ++i) acc = fma(z[i * zs], w[i], acc);
    return acc;
}

// line groups per tile: whole first-factor states, about kSpLines lines
__host__ __device__ inline int groups_per_tile(const Side &s)
{
    return s.nline == 2 ? std::max(1, kSpLines / s.ln1) : kSpLines;
}

__global__ __launch_bounds__(kSpThreads, 6) void sparse_lik_kernel(StreamArgs a, const char *__restrict__ mbase,
                                                                   const double *__restrict__ q,
                                                                   double *__restrict__ part)
{
    extern __shared__ double sd[];
    __shared__ int ctxs[kSpLanes];

    const int wg = a.flip ? (int)gridDim.x - 1 - (int)blockIdx.x : (int)blockIdx.x;   // grid = a.nwg
    int ti = 0;
    while (ti + 1 < a.ntask && a.task[ti + 1].wg0 <= wg) ++ti;
    const SpTask tk = a.task[ti];
    const ModDesc &md = a.mods[tk.m];
    const Side sd_ = side_of(md, tk.role);
    const int local = wg - tk.wg0;
    const int o = local / tk.tiles, tile = local - o * tk.tiles;
    const int32_t *start = a.bstart + a.sm[tk.m].bofs;
    const int b0 = start[o], J = start[o + 1] - b0;
    if (J == 0) return;

    // the tile's lines: groups [g0, g0 + ng) of the first line factor
    const int G = tk.G;
    const int g0 = tile * G;
    const int ng = min(G, sd_.ln0 - g0);
    const int lb = g0 * sd_.ln1, le = (g0 + ng) * sd_.ln1;
    const int nl = le - lb;

    const int ntab = sd_.en0 + sd_.en1;
    double *tab = sd;                       // [en0 + en1][64]: entry-side marginals
    double *zt = sd + ntab * kSpLanes;      // [lines of the tile][kZS]
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: entry stream via scalar loads

    const BI_CONST int32_t *lptr = (const BI_CONST int32_t *)(mbase + sd_.ptr_off) + (int64_t)o * (sd_.lines + 1);
    const BI_CONST u32x4 *ent = (const BI_CONST u32x4 *)(mbase + sd_.ent_off);   // SpEntry as 4 dwords
    const SpEntry *ent_v = reinterpret_cast<const SpEntry *>(mbase + sd_.ent_off);
    const int off_e0 = sd_.nent >= 1 ? a.facs[sd_.ef0].q_off : -1;
    const int off_e1 = sd_.nent == 2 ? a.facs[sd_.ef1].q_off : -1;
    const int off_l0 = a.facs[sd_.lf0].q_off;
    const int off_l1 = sd_.nline == 2 ? a.facs[sd_.lf1].q_off : -1;
    const int en0 = sd_.en0;

    // Pull a line's entries into L2: one dword per 64-byte line of them, by
    // vector loads whose values are only consumed one line later, so that the
    // scalar entry stream of the line being processed never waits on them.
    auto touch = [&](int l) {
        int v = 0;
        if (l < le) {
            const int idx = lptr[l] + 4 * lane;
            if (idx < lptr[l + 1]) v = *reinterpret_cast<const int *>(ent_v + idx);
        }
        return v;
    };
    int pf = 0, sink = 0;

    for (int c0 = 0; c0 < J; c0 += kSpLanes) {
        const int jc = min(kSpLanes, J - c0);
        pf = touch(lb + wave);   // first line of this wave, overlapping the table build
        if (tid < kSpLanes) ctxs[tid] = tid < jc ? a.bctx[(int64_t)tk.m * a.nlist + b0 + c0 + tid] : -1;
        __syncthreads();
        // entry-side marginal tables (1.0 for an absent factor)
        for (int i = tid; i < ntab * kSpLanes; i += kSpThreads) {
            const int c = i % kSpLanes, s = i / kSpLanes;
            const int ctx = ctxs[c];
            double v = 0.0;
            if (ctx >= 0) {
                const double *qc = q + (int64_t)(ctx >> a.vshift) * a.ntot;
                if (s < en0)
                    v = off_e0 >= 0 ? qc[off_e0 + s] : 1.0;
                else
                    v = off_e1 >= 0 ? qc[off_e1 + s - en0] : 1.0;
            }
            tab[i] = v;
        }
        __syncthreads();

        // line values: wave w takes lines lb + w, lb + w + kSpWaves, ...
        const double *t0 = tab + lane;
        const double *t1 = tab + en0 * kSpLanes + lane;
        for (int l = lb + wave; l < le; l += kSpWaves) {
            const int e0 = lptr[l], e1 = lptr[l + 1];
            // the touches of this line have landed; start those of the next
            sink ^= pf;
            pf = touch(l + kSpWaves);
            double acc = 0.0;
            int e = e0;
            // batches of kSpBatch entries: one round of scalar loads, one of
            // LDS gathers, then the FMAs (in entry order)
            for (; e + kSpBatch <= e1; e += kSpBatch) {
                double v[kSpBatch], p[kSpBatch];
                uint32_t ia[kSpBatch], ib[kSpBatch];
                const BI_CONST u32x4 *eb = ent + e;   // one base, constant offsets
#pragma unroll
                for (int k = 0; k < kSpBatch; ++k) {
                    const u32x4 x = eb[k];
                    v[k] = __hiloint2double((int)x.y, (int)x.x);
                    ia[k] = x.z;
                    ib[k] = x.w;
                }
#pragma unroll
                for (int k = 0; k < kSpBatch; ++k) p[k] = t0[ia[k] * kSpLanes] * t1[ib[k] * kSpLanes];
#pragma unroll
                for (int k = 0; k < kSpBatch; ++k) acc = fma(v[k], p[k], acc);
            }
            for (; e < e1; ++e) {
                const u32x4 x = ent[e];
                acc = fma(__hiloint2double((int)x.y, (int)x.x), t0[x.z * kSpLanes] * t1[x.w * kSpLanes], acc);
            }
            if (lane < kSpLanes) zt[(l - lb) * kZS + lane] = acc;
        }
        sink ^= pf;
        __syncthreads();

        // fold and write
        const int64_t ps = a.pstride;
        if (sd_.nline == 1) {
            // messages of the single line factor are the line values
            for (int i = tid; i < jc * nl; i += kSpThreads) {
                const int c = i / nl, k = i - c * nl;
                part[(int64_t)ctxs[c] * ps + tk.so + lb + k] = zt[k * kZS + c];
            }
        } else {
            const int ln1 = sd_.ln1;
            // first line factor: one message per (context, group), summed over l1
            for (int i = tid; i < jc * ng; i += kSpThreads) {
                const int c = i / ng, g = i - c * ng;
                const double *qc = q + (int64_t)(ctxs[c] >> a.vshift) * a.ntot + off_l1;
                part[(int64_t)ctxs[c] * ps + tk.so + g0 + g] = dot_batched(zt + g * ln1 * kZS + c, kZS, qc, ln1);
            }
            // second line factor: the tile's partial, summed over its groups
            for (int i = tid; i < jc * ln1; i += kSpThreads) {
                const int c = i / ln1, l1 = i - c * ln1;
                const double *qc = q + (int64_t)(ctxs[c] >> a.vshift) * a.ntot + off_l0 + g0;
                part[(int64_t)ctxs[c] * ps + tk.so + sd_.ln0 + (int64_t)tile * ln1 + l1] =
                    dot_batched(zt + l1 * kZS + c, ln1 * kZS, qc, ng);
            }
        }
        __syncthreads();
    }
    if (sink == 0x5a5a5a5a && a.nlist < 0) part[0] = 0.0;   // never true (nlist >= 1): keeps the touches
}

inline size_t lds_for(const Side &s)
{
    const int G = groups_per_tile(s);
    const int lines = std::min(G, s.ln0) * s.ln1;
    return sizeof(double) * ((size_t)(s.en0 + s.en1) * kSpLanes + (size_t)lines * kZS);
}

}  // namespace

bool sparse_eligible(const bi_model *m, int algo)
{
    if (!(m->flags & BI_SPARSE_A) || m->mb != 1 || algo == BI_ALGO_FPI) return false;
    if (sq_eligible(m)) return true;   // the sparse fp16-pair tiles (split.hip)
    if (m->M > kStreamMaxM) return false;
    int64_t pstride = 0;
    for (const ModDesc &md : m->mods) {
        if (md.csr_ptr_off < 0 || md.K > kStreamMaxK) return false;
        for (int role = 0; role < 2; ++role) {
            const Side s = side_of(md, role);
            if (s.nline == 0) continue;
            if (lds_for(s) > 160 * 1024) return false;
            const int G = groups_per_tile(s);
            const int64_t tiles = s.nline == 2 ? (s.ln0 + G - 1) / G : (s.lines + G - 1) / G;
            pstride += s.nline == 2 ? s.ln0 + tiles * s.ln1 : s.lines;
        }
    }
    return pstride < (int64_t)1 << 30;
}

size_t sparse_lds_bytes(const bi_model *m)
{
    size_t most = 0;
    for (const ModDesc &md : m->mods)
        for (int role = 0; role < 2; ++role) {
            const Side s = side_of(md, role);
            if (s.nline > 0) most = std::max(most, lds_for(s));
        }
    return most;
}

int64_t sparse_plan(const bi_model *m, StreamArgs *a)
{
    int wg = 0;
    int64_t so = 0;
    a->ntask = 0;
    a->nmsg = 0;
    for (int i = 0; i < m->M; ++i) {
        const ModDesc &md = m->mods[i];
        for (int role = 0; role < 2; ++role) {
            const Side s = side_of(md, role);
            if (s.nline == 0) continue;   // no row factors
            SpTask &tk = a->task[a->ntask++];
            tk.m = (int8_t)i;
            tk.role = (int8_t)role;
            const int G = groups_per_tile(s);
            tk.G = (int16_t)G;
            tk.tiles = s.nline == 2 ? (s.ln0 + G - 1) / G : (s.lines + G - 1) / G;
            tk.wg0 = wg;
            wg += md.K * tk.tiles;
            tk.so = (int32_t)so;
            MsgSrc &m0 = a->msg[a->nmsg++];
            m0.f = s.lf0;
            m0.copies = 1;
            m0.stride = 0;
            m0.off = (int32_t)so;
            if (s.nline == 2) {
                MsgSrc &m1 = a->msg[a->nmsg++];
                m1.f = s.lf1;
                m1.copies = tk.tiles;
                m1.stride = s.ln1;
                m1.off = (int32_t)(so + s.ln0);
                so += s.ln0 + (int64_t)tk.tiles * s.ln1;
            } else {
                so += s.lines;
            }
        }
    }
    a->nwg = wg;
    return so;
}

int sparse_prepare(const bi_model *m)
{
    const size_t lds = sparse_lds_bytes(m);
    if (lds > 160 * 1024) return fail(BI_ERR_UNSUPPORTED, "sparse working set exceeds LDS");
    const hipError_t e = func_max_lds((const void *)sparse_lik_kernel, (int)lds);
    if (e != hipSuccess) return fail(BI_ERR_DEVICE, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    return BI_OK;
}

void sparse_lik_launch(const bi_model *m, const StreamArgs &a, const double *q, double *part, hipStream_t stream)
{
    const size_t lds = sparse_lds_bytes(m);
    hipLaunchKernelGGL(sparse_lik_kernel, dim3(a.nwg), dim3(kSpThreads), lds, stream, a, (const char *)m->dev, q,
                       part);
}

}  // namespace bi
