// Dense likelihood messages on fp32 matrix cores, one contraction per
// workgroup (BI_FAST_F32, models shared by every agent, every modality with
// two factors on each side, the second factors of 16 or 32 states and the
// first factors of an even number of states up to 32).
//
// The two leave-one-out contractions of a slice X (two-sided view of
// layout.h, Sec. IV marginalisation) are done by separate workgroups, each
// over "lines" of X and contracting the other side (the "entries"):
//   role 0 (lines = rows):    Z[c][r]   = sum_{e0,e1} q_e0[c][e0] q_e1[c][e1] X[r][(e0,e1)]
//   role 1 (lines = columns): V[c][col] = sum_{e0,e1} q_e0[c][e0] q_e1[c][e1] X[(e0,e1)][col]
// For each state e0 of the entry side's first factor, the contraction over
// e1 is a 16x16x4 fp32 MFMA chain whose A operand is q_e1 scaled by
// q_e0[c][e0] (one multiply per operand element), so the outer product of the
// marginals is never built and the result accumulates in registers over the
// whole slice.  The B operand is streamed from HBM straight into registers
// (one 16-byte load per lane feeds four MFMAs); a wave owns 64 lines, a
// workgroup 4 waves.  At the end the line values go through LDS and are
// folded into the line factors' messages (fixed order, no atomics): the
// first line factor's messages of the tile's line groups directly, the
// second line factor's as one partial vector per tile.  Both roles of a slice
// are dispatched next to each other, so the second read of the slice mostly
// hits the last-level cache.
//
// With fp16 pairs (BI_F16_PAIRS) the same tiles run on fp16 matrix cores:
// the slice is read from its pair copy (4 columns per 16 bytes: high parts,
// then residuals), the A operand is q_e1 scaled by 2^15 and split into an
// fp16 high part and residual once per pass, and each first-factor state e0
// is one 16x16x32 (16x16x16 for 16-state second factors) product chain of
// three fp16 MFMAs: (A high, X high), (A high, X residual), (A residual,
// X high).  The chain starts from zero and is added to the accumulators with
// the weight q_e0[c][e0] 2^-15 in fp32, so nothing but the operand split ever
// leaves fp32 and the scaling keeps the small marginals clear of the fp16
// subnormals.
//
// The sparse fp16-pair layout (BI_SPARSE_A with BI_F16_PAIRS) runs the same
// products from the nonzeros alone: for every first-factor state e0 a wave
// scatters the nonzeros of its 64 lines with that e0 (one contiguous run of
// 8-byte entries, layout.h) into a zeroed 64 x en1 block in LDS, reads the B
// operands of its four 16-line MFMA tiles from there, puts the zeros back at
// the scattered places and runs the fp16-pair product chains.  The matrix
// cores do the dense work of the slice; memory carries only the nonzeros.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>

#include "internal.h"
#include "profile.h"
#include "stream.h"

namespace bi {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kWaveLines = 64;                 // lines per wave
constexpr int kTileLines = kWaves * kWaveLines; // lines per workgroup (at most)
constexpr int kMaxKb = 3;                      // 16-context MFMA blocks per pass
constexpr int kCtx = 16 * kMaxKb;
constexpr int kMaxT = 8;                       // k-steps per first-factor state (second factor <= 32)
constexpr int kZS = kCtx + 1;                  // line-tile stride (floats)
constexpr int kXcds = 8;                       // accelerator dies; workgroup i runs on die i % 8
constexpr size_t kMaxLds = 80 * 1024;          // two workgroups per CU

typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));
typedef uint32_t u2 __attribute__((ext_vector_type(2)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h4 __attribute__((ext_vector_type(4)));
constexpr float kPairScale = 32768.0f;   // 2^15: q_e1 in [0, 1] scaled below the fp16 maximum

// Sparse pairs: a wave's B block in LDS is two planes (high parts, then
// residuals) of the shape layout.h fixes (16-byte pad, then per line KS
// values and a 16-byte pad, so the 16 lines of one operand load start on
// different banks); sized for KS = 32.  Entries in flight per lane for one
// state e0: kSqR.
constexpr int kSqWaveBytes = 2 * sq_plane_bytes(32);
constexpr int kSqR = 4;
constexpr int kSqDepth = 4;   // a ring of states: the entries of 3 fetched ahead of the one in use
constexpr uint32_t kBufWord3 = 0x00020000u;   // buffer resource config word of the gfx9 family: raw dwords

// kernel variants: dense fp32 slices, dense fp16 pairs, sparse fp16 pairs
enum { kDenseF32 = 0, kDensePairs = 1, kSparsePairs = 2 };

struct Geo {
    int lines, ln0, ln1, lf0, lf1;   // line side (two factors)
    int en0, en1, ef0, ef1;          // entry side (two factors)
};

__host__ __device__ inline Geo geo_of(const ModDesc &md, int role)
{
    Geo g;
    const bool rows = role == 0;
    g.lines = rows ? md.R : md.C;
    g.lf0 = rows ? md.rf[0] : md.cf[0];
    g.lf1 = rows ? md.rf[1] : md.cf[1];
    g.ln0 = rows ? md.rn[0] : md.cn[0];
    g.ln1 = rows ? md.rn[1] : md.cn[1];
    g.ef0 = rows ? md.cf[0] : md.rf[0];
    g.ef1 = rows ? md.cf[1] : md.rf[1];
    g.en0 = rows ? md.cn[0] : md.rn[0];
    g.en1 = rows ? md.cn[1] : md.rn[1];
    return g;
}

// sum_{i < n} z[i * zs] w[i] in fp32, in order, with the loads issued 8 at a
// time (the fold's operands sit in LDS and L2: one wait per 8 terms)
__device__ inline float dot_batched(const float *z, int zs, const float *w, int n)
{
    float acc = 0.0f;
    int i = 0;
    for (; i + 8 <= n; i += 8) {
        float zv[8], wv[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            zv[k] = z[(i + k) * zs];
            wv[k] = w[i + k];
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) acc = fmaf(zv[k], wv[k], acc);
    }
    for (; i < n; ++i) acc = fmaf(z[i * zs], w[i], acc);
    return acc;
}

// line groups per tile: whole first-factor states, at most kTileLines lines
__host__ __device__ inline int split_groups(const Geo &g) { return std::max(1, kTileLines / g.ln1); }

template <int NKB, int ROLE, int NT>
__device__ void split_tile(const StreamArgs &a, const Geo &g, const float *__restrict__ X, int64_t Cp, int lb,
                           int le, const float *qe0, const float *qe1, float *zt)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wl0 = lb + kWaveLines * wave;
    if (wl0 >= le) return;
    const int li = lane & 15, lg = lane >> 4;
    // NT = en1 / 4 k-steps per first-factor state.  A operand of k-step t,
    // before the scaling by q_e0: q_e1[ctx][e1(t)]
    float a1[NT][NKB];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int e1 = ROLE == 0 ? 16 * (t >> 2) + 4 * lg + (t & 3) : 4 * t + lg;
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) a1[t][kb] = qe1[(16 * kb + li) * kMaxT * 4 + e1];
    }
    f4 acc[4][NKB];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) acc[j][kb] = f4{0.f, 0.f, 0.f, 0.f};

    // B operand loads of one first-factor state, 16 bytes per lane each:
    //   role 0: slot H j + h = line wl0 + 16 j + li, entries e0*en1 + 16 h + 4 lg .. +3 (H = NT / 4)
    //   role 1: slot t = entry e0*en1 + 4 t + lg, lines wl0 + 4 li .. +3
    // (lines past the tile are clamped to a valid one; their results are dropped)
    // byte offsets inside the slice (a slice is below 2 GiB: 32-bit offsets
    // from the wave-uniform slice base)
    constexpr int H = NT / 4, NS = ROLE == 0 ? 4 * H : NT;
    uint32_t bo[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        if (ROLE == 0) {
            const int line = min(wl0 + 16 * (s / H) + li, le - 1);
            bo[s] = 4u * (uint32_t)(line * (int)Cp + 16 * (s % H) + 4 * lg);
        } else {
            const int line = min(wl0 + 4 * li, le - 4);
            bo[s] = 4u * (uint32_t)((4 * s + lg) * (int)Cp + line);
        }
    }
    const uint32_t step = 4u * (ROLE == 0 ? 4 * NT : 4 * NT * (uint32_t)Cp);   // to the next first-factor state
    const char *Xb = reinterpret_cast<const char *>(X);
    auto load = [&](f4 (&b)[NS], int e0) {
        const uint32_t eo = (uint32_t)e0 * step;
#pragma unroll
        for (int s = 0; s < NS; ++s) b[s] = *reinterpret_cast<const f4 *>(Xb + (bo[s] + eo));
    };
    auto use = [&](const f4 (&b)[NS], int e0) {
        float s0[NKB];
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) s0[kb] = qe0[(16 * kb + li) * 32 + e0];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            float at[NKB];
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) at[kb] = a1[t][kb] * s0[kb];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float bv = ROLE == 0 ? b[H * j + (t >> 2)][t & 3] : b[t][j];
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb)
                    acc[j][kb] = __builtin_amdgcn_mfma_f32_16x16x4f32(at[kb], bv, acc[j][kb], 0, 0, 0);
            }
        }
    };
    // ping-pong: the loads of state e0 + 1 are in flight while state e0 is used
    // (en0 is even; the last round re-reads the last state, unused)
    // (the scheduling barriers keep each batch of loads ahead of the MFMAs
    // that do not need it; left alone, the compiler sinks them to their use)
    f4 ba[NS], bb[NS];
    load(ba, 0);
    for (int e0 = 0; e0 < g.en0; e0 += 2) {
        load(bb, e0 + 1);
        __builtin_amdgcn_sched_barrier(0);
        use(ba, e0);
        __builtin_amdgcn_sched_barrier(0);
        load(ba, min(e0 + 2, g.en0 - 1));
        __builtin_amdgcn_sched_barrier(0);
        use(bb, e0 + 1);
        __builtin_amdgcn_sched_barrier(0);
    }
    // D[ctx][line]: lane holds contexts 16 kb + 4 lg + v of line n = li
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int line = ROLE == 0 ? wl0 + 16 * j + li : wl0 + 4 * li + j;
        if (line < le)
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
                for (int v = 0; v < 4; ++v) zt[(line - lb) * kZS + 16 * kb + 4 * lg + v] = acc[j][kb][v];
    }
}

__device__ inline uint32_t pack_halves(_Float16 lo, _Float16 hi)
{
    return (uint32_t)__builtin_bit_cast(uint16_t, lo) | ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
}

// The fp16-pair version of split_tile.  KS = en1 (16 or 32) is the MFMA's K:
// a lane holds KW = KS / 4 consecutive k values (entries e1 = KW lg + i) of
// its A row (context 16 kb + li) and of its B column (line).  qe0t holds
// q_e0 2^-15 as [e0][kCtx], so a lane reads the weights of its 4
// accumulator rows (contexts 16 kb + 4 lg + v) as one float4.
template <int NKB, int ROLE, int KS>
__device__ void split16_tile(const StreamArgs &a, const Geo &g, const char *__restrict__ P, int64_t Cp, int lb,
                             int le, const float *qe0t, const float *qe1, float *zt)
{
    constexpr int KW = KS / 4;   // k values per lane
    constexpr int DW = KW / 2;   // dwords per operand
    using HV = std::conditional_t<KS == 32, h8, h4>;
    using UV = std::conditional_t<KS == 32, u4, u2>;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wl0 = lb + kWaveLines * wave;
    if (wl0 >= le) return;
    const int li = lane & 15, lg = lane >> 4;
    // A operand: q_e1 2^15 = high + residual, both fp16
    HV ah[NKB], al[NKB];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
        UV hd, ld;
#pragma unroll
        for (int p = 0; p < DW; ++p) {
            const float *src = qe1 + (16 * kb + li) * kMaxT * 4 + KW * lg + 2 * p;
            const float v0 = src[0] * kPairScale, v1 = src[1] * kPairScale;
            const _Float16 h0 = (_Float16)v0, h1 = (_Float16)v1;
            hd[p] = pack_halves(h0, h1);
            ld[p] = pack_halves((_Float16)(v0 - (float)h0), (_Float16)(v1 - (float)h1));
        }
        ah[kb] = __builtin_bit_cast(HV, hd);
        al[kb] = __builtin_bit_cast(HV, ld);
    }
    f4 acc[4][NKB];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) acc[j][kb] = f4{0.f, 0.f, 0.f, 0.f};

    // 16-byte loads of one first-factor state (4 columns of a row: 4 high
    // parts, 4 residuals):
    //   role 0: slot (KW / 4) j + h = line wl0 + 16 j + li, entries e0*KS + KW lg + 4 h .. +3
    //   role 1: slot i = entry e0*KS + KW lg + i, lines wl0 + 4 li .. +3
    // (lines past the tile are clamped to a valid one; their results are dropped)
    constexpr int H = KW / 4, NS = ROLE == 0 ? 4 * H : KW;
    uint32_t bo[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        if (ROLE == 0) {
            const int line = min(wl0 + 16 * (s / H) + li, le - 1);
            bo[s] = 4u * (uint32_t)(line * (int)Cp + KW * lg + 4 * (s % H));
        } else {
            const int line = min(wl0 + 4 * li, le - 4);
            bo[s] = 4u * (uint32_t)((KW * lg + s) * (int)Cp + line);
        }
    }
    const uint32_t step = 4u * (ROLE == 0 ? KS : KS * (uint32_t)Cp);   // to the next first-factor state
    auto load = [&](u4 (&b)[NS], int e0) {
        const uint32_t eo = (uint32_t)e0 * step;
#pragma unroll
        for (int s = 0; s < NS; ++s) b[s] = *reinterpret_cast<const u4 *>(P + (bo[s] + eo));
    };
    auto use = [&](const u4 (&b)[NS], int e0) {
        f4 w[NKB];
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) w[kb] = *reinterpret_cast<const f4 *>(qe0t + e0 * kCtx + 16 * kb + 4 * lg);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            UV xh, xl;
            if (ROLE == 0) {
                // the lane's KW entries of line j: consecutive columns of one row
#pragma unroll
                for (int h = 0; h < H; ++h) {
                    xh[2 * h] = b[H * j + h][0];
                    xh[2 * h + 1] = b[H * j + h][1];
                    xl[2 * h] = b[H * j + h][2];
                    xl[2 * h + 1] = b[H * j + h][3];
                }
            } else {
                // column j of the KW rows: one half of every load, paired up
                const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
#pragma unroll
                for (int p = 0; p < DW; ++p) {
                    xh[p] = __builtin_amdgcn_perm(b[2 * p + 1][j >> 1], b[2 * p][j >> 1], sel);
                    xl[p] = __builtin_amdgcn_perm(b[2 * p + 1][2 + (j >> 1)], b[2 * p][2 + (j >> 1)], sel);
                }
            }
            const HV bh = __builtin_bit_cast(HV, xh), bl = __builtin_bit_cast(HV, xl);
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) {
                f4 d = f4{0.f, 0.f, 0.f, 0.f};
                if constexpr (KS == 32) {
                    d = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[kb], bh, d, 0, 0, 0);
                    d = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[kb], bl, d, 0, 0, 0);
                    d = __builtin_amdgcn_mfma_f32_16x16x32_f16(al[kb], bh, d, 0, 0, 0);
                } else {
                    d = __builtin_amdgcn_mfma_f32_16x16x16f16(ah[kb], bh, d, 0, 0, 0);
                    d = __builtin_amdgcn_mfma_f32_16x16x16f16(ah[kb], bl, d, 0, 0, 0);
                    d = __builtin_amdgcn_mfma_f32_16x16x16f16(al[kb], bh, d, 0, 0, 0);
                }
#pragma unroll
                for (int v = 0; v < 4; ++v) acc[j][kb][v] = fmaf(w[kb][v], d[v], acc[j][kb][v]);
            }
        }
    };
    u4 ba[NS], bb[NS];
    load(ba, 0);
    for (int e0 = 0; e0 < g.en0; e0 += 2) {
        load(bb, e0 + 1);
        __builtin_amdgcn_sched_barrier(0);
        use(ba, e0);
        __builtin_amdgcn_sched_barrier(0);
        load(ba, min(e0 + 2, g.en0 - 1));
        __builtin_amdgcn_sched_barrier(0);
        use(bb, e0 + 1);
        __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int line = ROLE == 0 ? wl0 + 16 * j + li : wl0 + 4 * li + j;
        if (line < le)
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
                for (int v = 0; v < 4; ++v) zt[(line - lb) * kZS + 16 * kb + 4 * lg + v] = acc[j][kb][v];
    }
}

// The sparse fp16-pair tile.  A wave owns the 64 lines of one block of the
// sparse layout; for each state e0 the block's run of nonzeros is scattered
// into the wave's zeroed B block, the B operands of the four 16-line tiles
// are read back, the run's places are zeroed again and the product chains
// run as in split16_tile.  Entries arrive by bounds-checked buffer loads
// (a slot past the run reads 0: pair 0 at offset 0, the block's leading
// pad), and each carries its byte offset in the block, so a slot costs one
// address add and two 16-bit stores.  Only this wave touches its block, and
// LDS operations of one wave take effect in program order, so the block
// needs no barrier; the scheduling barriers keep the compiler from moving
// LDS operations across the phases.  The entries of state e0 + 1 are loaded
// while state e0 is used.  Ends with a workgroup barrier (every wave reaches
// it) and the line values written to zt, which overlays the blocks.
template <int NKB, int KS>
__device__ void sq_tile(const Geo &g, const uint32_t *__restrict__ ptr, const SqEntry *__restrict__ ent, int lb,
                        int le, const float *qe0t, const float *qe1, char *blocks, float *zt)
{
    constexpr int KW = KS / 4;   // k values per lane
    constexpr int DW = KW / 2;   // dwords per operand
    constexpr int SH = sq_line_bytes(KS), PL = sq_plane_bytes(KS);
    using HV = std::conditional_t<KS == 32, h8, h4>;
    using UV = std::conditional_t<KS == 32, u4, u2>;
    typedef uint32_t w2 __attribute__((ext_vector_type(2)));
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wl0 = lb + kWaveLines * wave;
    const bool active = wl0 < le;
    const int li = lane & 15, lg = lane >> 4;
    f4 acc[4][NKB];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) acc[j][kb] = f4{0.f, 0.f, 0.f, 0.f};
    if (active) {
        // A operand: q_e1 2^15 = high + residual, both fp16
        HV ah[NKB], al[NKB];
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
            UV hd, ld;
#pragma unroll
            for (int p = 0; p < DW; ++p) {
                const float *src = qe1 + (16 * kb + li) * kMaxT * 4 + KW * lg + 2 * p;
                const float v0 = src[0] * kPairScale, v1 = src[1] * kPairScale;
                const _Float16 h0 = (_Float16)v0, h1 = (_Float16)v1;
                hd[p] = pack_halves(h0, h1);
                ld[p] = pack_halves((_Float16)(v0 - (float)h0), (_Float16)(v1 - (float)h1));
            }
            ah[kb] = __builtin_bit_cast(HV, hd);
            al[kb] = __builtin_bit_cast(HV, ld);
        }
        const int en0 = g.en0;
        // lane i <= en0 holds the start of run i of the wave's block (run en0:
        // the block's end)
        const uint32_t *bp = ptr + (int64_t)(wl0 / kSqBlock) * en0;
        const int pv = (int)bp[min(lane, en0)];
        char *bk = blocks + wave * kSqWaveBytes;
        // buffer resource over the run of state e0 (its length bounds the loads)
        auto run_rsrc = [&](int e0, int &n) {
            const int rs = __builtin_amdgcn_readlane(pv, e0);
            n = __builtin_amdgcn_readlane(pv, e0 + 1) - rs;
            return __builtin_amdgcn_make_buffer_rsrc((void *)(ent + rs), (short)0, 8 * n, (int)kBufWord3);
        };
        auto fetch = [&](w2 (&E)[kSqR], int e0) {
            int n;
            const auto r = run_rsrc(e0, n);
#pragma unroll
            for (int i = 0; i < kSqR; ++i) E[i] = __builtin_amdgcn_raw_buffer_load_b64(r, 8 * (lane + 64 * i), 0, 0);
        };
        auto put = [&](w2 x, bool clear) {
            char *d = bk + x[1];
            *reinterpret_cast<uint16_t *>(d) = clear ? (uint16_t)0 : (uint16_t)(x[0] & 0xffffu);
            *reinterpret_cast<uint16_t *>(d + PL) = clear ? (uint16_t)0 : (uint16_t)(x[0] >> 16);
        };
        // scatter (or zero again) the run of state e0: the entries in flight,
        // then any beyond 64 kSqR straight from memory
        auto scatter = [&](const w2 (&E)[kSqR], int e0, bool clear) {
#pragma unroll
            for (int i = 0; i < kSqR; ++i) put(E[i], clear);
            int n;
            const auto r = run_rsrc(e0, n);
            for (int b0 = 64 * kSqR; b0 < n; b0 += 64) put(__builtin_amdgcn_raw_buffer_load_b64(r, 8 * (b0 + lane), 0, 0), clear);
        };
        auto step = [&](const w2 (&E)[kSqR], int e0) {
            scatter(E, e0, false);
            __builtin_amdgcn_sched_barrier(0);
            UV xh[4], xl[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const char *r = bk + kSqPad + (16 * j + li) * SH + 2 * KW * lg;
                xh[j] = *reinterpret_cast<const UV *>(r);
                xl[j] = *reinterpret_cast<const UV *>(r + PL);
            }
            __builtin_amdgcn_sched_barrier(0);
            scatter(E, e0, true);
            __builtin_amdgcn_sched_barrier(0);
            f4 w[NKB];
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb)
                w[kb] = *reinterpret_cast<const f4 *>(qe0t + e0 * kCtx + 16 * kb + 4 * lg);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const HV bh = __builtin_bit_cast(HV, xh[j]), bl = __builtin_bit_cast(HV, xl[j]);
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb) {
                    f4 d = f4{0.f, 0.f, 0.f, 0.f};
                    if constexpr (KS == 32) {
                        d = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[kb], bh, d, 0, 0, 0);
                        d = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah[kb], bl, d, 0, 0, 0);
                        d = __builtin_amdgcn_mfma_f32_16x16x32_f16(al[kb], bh, d, 0, 0, 0);
                    } else {
                        d = __builtin_amdgcn_mfma_f32_16x16x16f16(ah[kb], bh, d, 0, 0, 0);
                        d = __builtin_amdgcn_mfma_f32_16x16x16f16(ah[kb], bl, d, 0, 0, 0);
                        d = __builtin_amdgcn_mfma_f32_16x16x16f16(al[kb], bh, d, 0, 0, 0);
                    }
#pragma unroll
                    for (int v = 0; v < 4; ++v) acc[j][kb][v] = fmaf(w[kb][v], d[v], acc[j][kb][v]);
                }
            }
        };
        // a ring of kSqDepth states: the entries of the next kSqDepth - 1
        // states are in flight while one is used
        w2 E[kSqDepth][kSqR];
#pragma unroll
        for (int k = 0; k < kSqDepth - 1; ++k)
            if (k < en0) fetch(E[k], k);
        for (int e0 = 0; e0 < en0; e0 += kSqDepth) {
#pragma unroll
            for (int k = 0; k < kSqDepth; ++k) {
                const int e = e0 + k;
                if (e < en0) {
                    if (e + kSqDepth - 1 < en0) fetch(E[(k + kSqDepth - 1) % kSqDepth], e + kSqDepth - 1);
                    step(E[k], e);
                }
            }
        }
    }
    __syncthreads();   // every wave is done with its block: zt overlays them
    if (active) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int line = wl0 + 16 * j + li;
            if (line < le)
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
                    for (int v = 0; v < 4; ++v) zt[(line - lb) * kZS + 16 * kb + 4 * lg + v] = acc[j][kb][v];
        }
    }
}

template <int MODE>
__device__ void split_body(const StreamArgs &a, const float *__restrict__ q, float *__restrict__ part)
{
    constexpr bool PAIRS = MODE != kDenseF32;
    extern __shared__ float sh[];
    __shared__ int ctxs[kCtx];
    // decode (modality, outcome, role, tile): the two roles of a modality share
    // its workgroup range, outcome-major, so both roles of a slice run together.
    // Workgroups are dealt to the dies round-robin, so each die gets a
    // contiguous range of that order: both roles of a slice run on one die
    // (the second read of the slice can hit that die's L2), and every die
    // streams its own slices (consecutive workgroups on different dies would
    // put all first reads of the slices on half of them).
    // (odd iterations: the reverse order, a.flip)
    const int per_die = (a.nwg + kXcds - 1) / kXcds;
    const int bid = a.flip ? (int)gridDim.x - 1 - (int)blockIdx.x : (int)blockIdx.x;
    const int wg = (bid % kXcds) * per_die + bid / kXcds;
    if (wg >= a.nwg) return;
    int m = 0;
    while (m + 1 < a.M && a.task[2 * (m + 1)].wg0 <= wg) ++m;
    const SpTask t0 = a.task[2 * m], t1 = a.task[2 * m + 1];
    const int per_o = t0.tiles + t1.tiles;
    const int local = wg - t0.wg0;
    const int o = local / per_o, r = local - o * per_o;
    const int role = r < t0.tiles ? 0 : 1;
    const int tile = role ? r - t0.tiles : r;
    const SpTask tk = role ? t1 : t0;
    const ModDesc &md = a.mods[m];
    const Geo g = geo_of(md, role);
    const int32_t *start = a.bstart + a.sm[m].bofs;
    const int b0 = start[o], J = start[o + 1] - b0;
    if (J == 0) return;
    const int G = tk.G;
    const int gs = tile * G, ng = min(G, g.ln0 - gs);
    const int lb = gs * g.ln1, le = (gs + ng) * g.ln1;
    const float *X = MODE == kDenseF32 ? reinterpret_cast<const float *>(a.base + md.la32_off) + (int64_t)o * md.slice
                                       : nullptr;
    const char *P = MODE == kDensePairs ? a.base + md.lp16_off + 4 * (int64_t)o * md.slice : nullptr;
    // sparse pairs: this outcome's run pointers and the side's entries
    const uint32_t *sqp = nullptr;
    const SqEntry *sqe = nullptr;
    if (MODE == kSparsePairs) {
        const int64_t runs = (int64_t)((g.lines + kSqBlock - 1) / kSqBlock) * g.en0;
        sqp = reinterpret_cast<const uint32_t *>(a.base + md.sq_ptr_off[role]) + (int64_t)o * (runs + 1);
        sqe = reinterpret_cast<const SqEntry *>(a.base + md.sq_ent_off[role]);
    }
    float *qe0 = sh;                      // [kCtx][32]: marginals of the entry side's first factor
                                          // (pairs: [32][kCtx], times 2^-15)
    float *qe1 = qe0 + kCtx * 32;         // [kCtx][32]: second factor
    float *ql0 = qe1 + kCtx * 32;         // [kCtx][32]: the line side's first and second factors (fold)
    float *ql1 = ql0 + kCtx * 32;
    float *zt = ql1 + kCtx * 32;          // [tile lines][kZS] (sparse pairs: over the B blocks)
    char *blocks = reinterpret_cast<char *>(zt);
    const int tid = threadIdx.x;
    const int off_e0 = a.facs[g.ef0].q_off, off_e1 = a.facs[g.ef1].q_off;
    const int off_l0 = a.facs[g.lf0].q_off, off_l1 = a.facs[g.lf1].q_off;

    for (int c0 = 0; c0 < J; c0 += kCtx) {
        const int jc = min(kCtx, J - c0);
        if (tid < kCtx) ctxs[tid] = tid < jc ? a.bctx[(int64_t)m * a.nlist + b0 + c0 + tid] : -1;
        if (MODE == kSparsePairs)   // zero B blocks (the line tile of the last pass overlays them)
            for (int i = tid; i < kWaves * kSqWaveBytes / 16; i += kThreads)
                reinterpret_cast<u4 *>(blocks)[i] = u4{0u, 0u, 0u, 0u};
        __syncthreads();
        // marginal tables of the pass (zero for padded contexts and states):
        // the four loads of a (context, state) in flight together, two rounds
        // at a time, from addresses clamped to valid entries (a padded context
        // reads context 0, a padded state the factor's last state)
        static_assert(kCtx * 32 % (2 * kThreads) == 0, "table set-up assumes whole double rounds");
        for (int i0 = tid; i0 < kCtx * 32; i0 += 2 * kThreads) {
            float v[2][4];
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                const int i = i0 + k * kThreads, c = i >> 5, s = i & 31;
                const float *qc = q + (int64_t)(max(ctxs[c], 0) >> a.vshift) * a.ntot;
                v[k][0] = qc[off_e0 + min(s, g.en0 - 1)];
                v[k][1] = qc[off_e1 + min(s, g.en1 - 1)];
                v[k][2] = qc[off_l0 + min(s, g.ln0 - 1)];
                v[k][3] = qc[off_l1 + min(s, g.ln1 - 1)];
            }
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                const int i = i0 + k * kThreads, c = i >> 5, s = i & 31;
                const bool ok = ctxs[c] >= 0;
                const float e0 = ok && s < g.en0 ? v[k][0] : 0.0f;
                if (PAIRS)
                    qe0[s * kCtx + c] = e0 * (1.0f / kPairScale);
                else
                    qe0[c * 32 + s] = e0;
                qe1[c * 32 + s] = ok && s < g.en1 ? v[k][1] : 0.0f;
                ql0[c * 32 + s] = ok && s < g.ln0 ? v[k][2] : 0.0f;
                ql1[c * 32 + s] = ok && s < g.ln1 ? v[k][3] : 0.0f;
            }
        }
        __syncthreads();
        const int nkb = (jc + 15) >> 4;
        const int nt = g.en1 >> 2;
        // dispatch on (role, context blocks, k-steps per state); eligibility
        // admits second factors of 16 or 32 states
#define BI_SPLIT_TILE(R, K, T)                                                                     \
    do {                                                                                           \
        if constexpr (MODE == kSparsePairs) sq_tile<K, 4 * T>(g, sqp, sqe, lb, le, qe0, qe1, blocks, zt); \
        else if constexpr (MODE == kDensePairs) split16_tile<K, R, 4 * T>(a, g, P, md.Cp, lb, le, qe0, qe1, zt); \
        else split_tile<K, R, T>(a, g, X, md.Cp, lb, le, qe0, qe1, zt);                            \
    } while (0)
#define BI_SPLIT_NT(R, K) \
    if (nt == 8) BI_SPLIT_TILE(R, K, 8); \
    else BI_SPLIT_TILE(R, K, 4)
#define BI_SPLIT_KB(R) \
    if (nkb == 1) { BI_SPLIT_NT(R, 1); } \
    else if (nkb == 2) { BI_SPLIT_NT(R, 2); } \
    else { BI_SPLIT_NT(R, 3); }
        if (MODE == kSparsePairs || role == 0) {   // the sparse tile reads both sides the same way
            BI_SPLIT_KB(0)
        } else {
            BI_SPLIT_KB(1)
        }
#undef BI_SPLIT_KB
#undef BI_SPLIT_NT
#undef BI_SPLIT_TILE
        __syncthreads();
        // fold: first line factor per (context, group) over l1; second line
        // factor per (context, l1) over the tile's groups
        const int64_t ps = a.pstride;
        const int ln1 = g.ln1;
        for (int i = tid; i < jc * ng; i += kThreads) {
            const int c = i / ng, gg = i - c * ng;
            part[(int64_t)ctxs[c] * ps + tk.so + gs + gg] = dot_batched(zt + gg * ln1 * kZS + c, kZS, ql1 + c * 32, ln1);
        }
        for (int i = tid; i < jc * ln1; i += kThreads) {
            const int c = i / ln1, l1 = i - c * ln1;
            part[(int64_t)ctxs[c] * ps + tk.so + g.ln0 + (int64_t)tile * ln1 + l1] =
                dot_batched(zt + l1 * kZS + c, ln1 * kZS, ql0 + c * 32 + gs, ng);
        }
        __syncthreads();
    }
}

template <bool PAIRS>
__global__ __launch_bounds__(kThreads, 2) void split_lik_kernel(StreamArgs a, const float *__restrict__ q,
                                                             float *__restrict__ part)
{
    split_body<PAIRS ? kDensePairs : kDenseF32>(a, q, part);
}

__global__ __launch_bounds__(kThreads, 2) void sparse16_lik_kernel(StreamArgs a, const float *__restrict__ q,
                                                                float *__restrict__ part)
{
    split_body<kSparsePairs>(a, q, part);
}

size_t lds_bytes(const bi_model *m, bool sparse)
{
    size_t most = 0;
    for (const ModDesc &md : m->mods)
        for (int role = 0; role < 2; ++role) {
            const Geo g = geo_of(md, role);
            const size_t lines = (size_t)std::min(split_groups(g), g.ln0) * g.ln1;
            size_t tail = sizeof(float) * lines * kZS;
            if (sparse) tail = std::max(tail, (size_t)kWaves * kSqWaveBytes);
            most = std::max(most, sizeof(float) * (size_t)kCtx * 128 + tail);
        }
    return most;
}

}  // namespace

bool split_eligible(const bi_model *m)
{
    if (m->M > kStreamMaxM) return false;
    int64_t pstride = 0;
    for (const ModDesc &md : m->mods) {
        if (md.la32_off < 0 || md.nrow != 2 || md.ncol != 2 || md.Cp != md.C) return false;
        if (4 * (int64_t)md.R * md.Cp >= INT32_MAX) return false;   // 32-bit byte offsets inside a slice
        for (int role = 0; role < 2; ++role) {
            const Geo g = geo_of(md, role);
            // 4 or 8 k-steps per first-factor state (16 or 32 states)
            if ((g.en1 != 16 && g.en1 != 32) || g.en0 > 32 || g.en0 % 2 != 0 || g.ln1 > kTileLines || g.ln1 % 4 != 0)
                return false;
            const int G = split_groups(g);
            pstride += g.ln0 + (int64_t)((g.ln0 + G - 1) / G) * g.ln1;
        }
        if (md.K > kStreamMaxK) return false;
    }
    return lds_bytes(m, false) <= kMaxLds && pstride < (int64_t)1 << 30;
}

bool sq_eligible(const bi_model *m)
{
    if (m->M > kStreamMaxM || m->mods.empty()) return false;
    int64_t pstride = 0;
    for (const ModDesc &md : m->mods) {
        // the layout exists only for the shapes it serves (sq_shape)
        if (md.sq_ptr_off[0] < 0 || md.sq_ptr_off[1] < 0 || md.K > kStreamMaxK) return false;
        for (int role = 0; role < 2; ++role) {
            const Geo g = geo_of(md, role);
            const int G = split_groups(g);
            // tiles of whole 64-line blocks of the layout
            if (G * g.ln1 % kSqBlock != 0 && G < g.ln0) return false;
            pstride += g.ln0 + (int64_t)((g.ln0 + G - 1) / G) * g.ln1;
        }
    }
    return lds_bytes(m, true) <= kMaxLds && pstride < (int64_t)1 << 30;
}

int64_t split_plan(const bi_model *m, StreamArgs *a)
{
    int wg = 0;
    int64_t so = 0;
    a->ntask = 0;
    a->nmsg = 0;
    for (int i = 0; i < m->M; ++i) {
        const ModDesc &md = m->mods[i];
        const int wg0 = wg;
        for (int role = 0; role < 2; ++role) {
            const Geo g = geo_of(md, role);
            SpTask &tk = a->task[a->ntask++];
            tk.m = (int8_t)i;
            tk.role = (int8_t)role;
            const int G = split_groups(g);
            tk.G = (int16_t)G;
            tk.tiles = (g.ln0 + G - 1) / G;
            tk.wg0 = wg0;
            wg += md.K * tk.tiles;
            tk.so = (int32_t)so;
            MsgSrc &m0 = a->msg[a->nmsg++];
            m0.f = g.lf0;
            m0.copies = 1;
            m0.stride = 0;
            m0.off = (int32_t)so;
            MsgSrc &m1 = a->msg[a->nmsg++];
            m1.f = g.lf1;
            m1.copies = tk.tiles;
            m1.stride = g.ln1;
            m1.off = (int32_t)(so + g.ln0);
            so += g.ln0 + (int64_t)tk.tiles * g.ln1;
        }
    }
    a->nwg = wg;
    return so;
}

size_t split_lds_bytes(const bi_model *m, bool sparse) { return lds_bytes(m, sparse); }

int split_prepare(const bi_model *m, bool sparse)
{
    const void *fn = sparse ? (const void *)sparse16_lik_kernel
                     : split_pairs(m) ? (const void *)split_lik_kernel<true>
                                      : (const void *)split_lik_kernel<false>;
    const hipError_t e = func_max_lds(fn, (int)kMaxLds);
    if (e != hipSuccess) return fail(BI_ERR_DEVICE, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    return BI_OK;
}

bool split_pairs(const bi_model *m)
{
    for (const ModDesc &md : m->mods)
        if (md.lp16_off < 0 || md.lp16_order != 0) return false;   // row-ordered pairs only
    return !m->mods.empty();
}

void split_lik_launch(const bi_model *m, const StreamArgs &a, const float *q, float *part, hipStream_t stream,
                      bool sparse)
{
    const unsigned grid = (unsigned)((a.nwg + kXcds - 1) / kXcds * kXcds);
    const size_t lds = lds_bytes(m, sparse);
    if (sparse)
        hipLaunchKernelGGL(sparse16_lik_kernel, dim3(grid), dim3(kThreads), lds, stream, a, q, part);
    else if (split_pairs(m))
        hipLaunchKernelGGL(split_lik_kernel<true>, dim3(grid), dim3(kThreads), lds, stream, a, q, part);
    else
        hipLaunchKernelGGL(split_lik_kernel<false>, dim3(grid), dim3(kThreads), lds, stream, a, q, part);
}

}  // namespace bi
