// Dense likelihood messages from a single read of every slice, on fp16
// matrix cores (BI_F16_PAIRS; models shared by every agent whose modalities
// all have two factors on each side, both second factors of 32 states, the
// first column factor of an even number of states up to 32 and the first row
// factor of at most 32).
//
// A slice X of the two-sided view (layout.h; the marginalisation of Sec. IV)
// has rows (r0, r1) and columns (c0, c1).  For the contexts c that observed
// it, the messages of its four factors are
//   Y[c][r]        = sum_{c0,c1} q_c0[c0] q_c1[c1] X[r][(c0,c1)]
//   m_r0[c][r0]    = sum_{r1} q_r1[r1] Y[c][(r0,r1)]
//   m_r1[c][r1]    = sum_{r0} q_r0[r0] Y[c][(r0,r1)]
//   m_c0[c][c0]    = sum_{r} q_r0 q_r1[r] sum_{c1} q_c1[c1] X[r][(c0,c1)]
//   m_c1[c][c1]    = sum_{c0} q_c0[c0] sum_{r} q_r0 q_r1[r] X[r][(c0,c1)]
// A workgroup owns 8 states of r0 (256 rows), one per wave.  For each state
// c0 (32 columns) a wave loads its 32 x 32 block of fp16 pairs once (one
// contiguous 4 KB block of the blocked pair copy, layout.h), stages it in
// LDS and runs two product chains over it, the slice block as the matrix
// cores' A operand and the marginals as B, so that every lane ends up with
// one context's values:
//   rows    (K = c1): d_row[r1][c] = sum_{c1} X[(r0,r1)][(c0,c1)] (q_c1 2^15)[c][c1]
//   columns (K = r1): d_col[c1][c] = sum_{r1} X[(r0,r1)][(c0,c1)] (q_r0[r0] q_r1 2^15)[c][r1]
// each as three fp16 products per fp32 product (high/high, high/residual,
// residual/high) started from zero.  Then, in fp32:
//   Y   += q_c0[c0] 2^-15 d_row          (accumulated over c0 in registers)
//   U   += q_c0[c0] 2^-15 d_col          (this wave's share of m_c1)
//   m_c0[c][c0] (this wave's share) = sum_{r1} q_r0 q_r1 2^-15 d_row: the lane's
//                4 rows per block in registers, then across the 4 lane rows
// so the slice leaves HBM once and nothing larger than a message vector is
// kept.  At the end the waves' shares are summed in LDS in wave order (no
// atomics) and written as partial message vectors, one per row tile, that
// the update kernel adds up.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "internal.h"
#include "stream.h"

namespace bi {
namespace {

constexpr int kWaves = 8;                 // states of r0 per workgroup, one per wave
constexpr int kThreads = 64 * kWaves;
constexpr int kN1 = 32;                   // states of each side's second factor
constexpr int kMaxKb = 3;                 // 16-context matrix-core blocks per pass
constexpr int kCtx = 16 * kMaxKb;
constexpr float kPairScale = 32768.0f;    // 2^15: marginals in [0, 1] scaled below the fp16 maximum
constexpr float kPairInv = 1.0f / 32768.0f;

// A wave's staged block of one state c0: 32 rows r1 of 8 sixteen-byte units
// (unit 2 g: the high parts of columns 8 g .. 8 g + 7; unit 2 g + 1: their
// residuals), 128 bytes per row, unit u of row rho at position u ^ (rho & 7)
// so that the 8 lanes serving consecutive rows of one unit, or one row's
// units, hit distinct banks.  Blocks arrive by direct global-to-LDS loads
// (1 KB per instruction, lane L to bytes 16 L of it) in a ring of three per
// wave: the loads of the next two states are in flight while one is used.
constexpr int kBlockBytes = kN1 * 128;
constexpr int kRing = 3;

// LDS (bytes)
constexpr int kTab = kCtx * 32 * 4;                   // one [kCtx][32] (or [32][kCtx]) fp32 table
constexpr int kOffQc0 = 0;                            // [32][kCtx]  q_c0 2^-15, by state
constexpr int kOffQr1 = kTab;                         // [kCtx][32]  q_r1
constexpr int kOffQr0w = 2 * kTab;                    // [kWaves][kCtx]  q_r0 of each wave's state
// Shares of a message summed over the waves: [kWaves][kCtx][kSh] with the
// 32 states of a context contiguous and an odd pitch, so that the sums (32
// consecutive states of one context per 32 lanes) and the writes from the
// accumulators (16 consecutive contexts per 16 lanes) fall on distinct banks
// (a pitch of kCtx states had put 32 lanes on 4 banks)
constexpr int kSh = 33;
constexpr int kShares = kWaves * kCtx * kSh * 4;
constexpr int kOffM3 = kOffQr0w + kWaves * kCtx * 4;  // shares of m_c0
constexpr int kOffRing = kOffM3 + kShares;            // [kRing][kWaves] blocks; before the loop the
constexpr int kRingBytes = kRing * kWaves * kBlockBytes;   // third ring slot holds q_c1 and q_r0 [kCtx][32];
constexpr int kLds = kOffRing + kRingBytes;           // after it, the shares of m_c1 / m_r1
static_assert(2 * kTab <= kWaves * kBlockBytes, "set-up tables exceed a ring slot");
static_assert(kShares <= kRingBytes, "shares exceed the ring");
static_assert(kOffRing % 16 == 0, "ring slots must be 16-byte aligned");
static_assert(kLds + 4 * kCtx <= 160 * 1024, "LDS of the workgroup exceeds 160 KB");

typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));

__device__ inline uint32_t pack_halves(_Float16 lo, _Float16 hi)
{
    return (uint32_t)__builtin_bit_cast(uint16_t, lo) | ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
}

// fp16 high parts and residuals of v[0..7] * s
__device__ inline void split8(const float *v, float s, h8 &hi, h8 &lo)
{
    u4 hd, ld;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const float v0 = v[2 * p] * s, v1 = v[2 * p + 1] * s;
        const _Float16 h0 = (_Float16)v0, h1 = (_Float16)v1;
        hd[p] = pack_halves(h0, h1);
        ld[p] = pack_halves((_Float16)(v0 - (float)h0), (_Float16)(v1 - (float)h1));
    }
    hi = __builtin_bit_cast(h8, hd);
    lo = __builtin_bit_cast(h8, ld);
}

// (fp16 high, residual) x (fp16 high, residual) product chain from zero
__device__ inline f4 chain3(const h8 &ah, const h8 &al, const h8 &bh, const h8 &bl)
{
    f4 d = f4{0.f, 0.f, 0.f, 0.f};
    d = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, bh, d, 0, 0, 0);
    d = __builtin_amdgcn_mfma_f32_16x16x32_f16(ah, bl, d, 0, 0, 0);
    d = __builtin_amdgcn_mfma_f32_16x16x32_f16(al, bh, d, 0, 0, 0);
    return d;
}

struct Pass {
    const char *P;      // the slice's fp16 pairs
    int Cp;             // row pitch (values)
    int rn0, cn0;       // states of r0 and c0
    int tile, jc;       // row tile; contexts of this pass
    int64_t ps;         // partial values per context
    int64_t o_r0, o_r1, o_c0, o_c1;   // offsets of the four message vectors (o_r1, o_c*: this tile's copy)
    int off_r0, off_r1, off_c0, off_c1;   // the factors' offsets in a marginal vector
};

// sum over the 4 lane rows (lanes l, l + 16, l + 32, l + 48); the four
// lanes end with the same value (fp32 addition is commutative)
__device__ inline float rows_sum4(float x)
{
    x += __shfl_xor(x, 16);
    x += __shfl_xor(x, 32);
    return x;
}

// One pass over the workgroup's row tile for up to kCtx contexts (NKB blocks
// of 16).  Every wave reaches every barrier.
template <int NKB>
__device__ void rc_pass(const StreamArgs &a, const Pass &p, const float *__restrict__ q, float *__restrict__ part,
                        const int *ctxs, char *lds)
{
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int li = lane & 15, lg = lane >> 4;
    const int r0 = 8 * p.tile + wave;
    const bool active = r0 < p.rn0;
    float *qc0t = reinterpret_cast<float *>(lds + kOffQc0);
    float *qr1t = reinterpret_cast<float *>(lds + kOffQr1);
    float *qr0w = reinterpret_cast<float *>(lds + kOffQr0w);
    float *m3 = reinterpret_cast<float *>(lds + kOffM3);
    float *shares = reinterpret_cast<float *>(lds + kOffRing);
    char *ring = lds + kOffRing + wave * kBlockBytes;   // slot k of this wave at + k * kWaves * kBlockBytes

    // Direct loads of state c0 into ring slot c0 % 3: the block of (r0, c0)
    // is contiguous; instruction i (0..3) brings its bytes 1024 i ..
    // 1024 i + 1023, lane L the unit at position L & 7 of row 8 i + (L >> 3),
    // i.e. unit (L & 7) ^ (L >> 3).  Byte offsets inside the slice fit 32
    // bits (checked at eligibility).
    const uint32_t gofs = 4096u * (uint32_t)(r0 * p.cn0) + 128u * (uint32_t)(lane >> 3) +
                          16u * (uint32_t)((lane & 7) ^ (lane >> 3));
    auto dma = [&](int c0) {
        char *dst = ring + (c0 % kRing) * (kWaves * kBlockBytes);
        const uint32_t o = gofs + 4096u * (uint32_t)c0;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            __builtin_amdgcn_global_load_lds((const void *)(p.P + (o + 1024u * i)),
                                             (__attribute__((address_space(3))) void *)(dst + 1024 * i), 16, 0, 0);
    };
    if (active) {   // the first two states' loads overlap the table set-up (slots 0 and 1)
        dma(0);
        dma(1);
    }

    // tables of this pass's marginals (zero for padded contexts and states);
    // q_c1 and q_r0 [kCtx][32] sit in ring slot 2 until the loop starts
    float *qc1t = reinterpret_cast<float *>(lds + kOffRing + 2 * kWaves * kBlockBytes);
    float *qr0t = qc1t + kCtx * 32;
    // the four loads of a round in flight at once: addresses clamped to valid
    // entries (a padded context reads context 0, a padded state the last
    // state), the values selected after the loads (few registers: the main
    // loop below is at the register limit)
#pragma unroll 1
    for (int i = tid; i < kCtx * 32; i += kThreads) {
        const int c = i >> 5, s = i & 31, ctx = ctxs[c];
        const float *qc = q + (int64_t)(max(ctx, 0) >> a.vshift) * a.ntot;
        const float v0 = qc[p.off_c0 + min(s, p.cn0 - 1)], v1 = qc[p.off_c1 + s];
        const float v2 = qc[p.off_r0 + min(s, p.rn0 - 1)], v3 = qc[p.off_r1 + s];
        const bool ok = ctx >= 0;
        qc0t[s * kCtx + c] = ok && s < p.cn0 ? v0 * kPairInv : 0.0f;
        qc1t[c * 32 + s] = ok ? v1 : 0.0f;
        qr0t[c * 32 + s] = ok && s < p.rn0 ? v2 : 0.0f;
        qr1t[c * 32 + s] = ok ? v3 : 0.0f;
    }
    __syncthreads();
    if (tid < kWaves * kCtx) {
        const int w = tid / kCtx, c = tid - w * kCtx;
        qr0w[w * kCtx + c] = 8 * p.tile + w < p.rn0 ? qr0t[c * 32 + 8 * p.tile + w] : 0.0f;
    }

    // B operands (context 16 kb + li, k = 8 lg .. 8 lg + 7):
    //   rows:    q_c1 2^15;  columns: q_r0[r0] q_r1 2^15
    // and the m_c0 weights q_r0[r0] q_r1[16 j + 4 lg + v] 2^-15 of the lane's
    // context 16 kb + li and accumulator rows
    h8 rbh[NKB], rbl[NKB], cbh[NKB], cbl[NKB];
    float wq[2][NKB][4];
    if (active) {
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
            const int c = 16 * kb + li;
            split8(qc1t + c * 32 + 8 * lg, kPairScale, rbh[kb], rbl[kb]);
            split8(qr1t + c * 32 + 8 * lg, qr0t[c * 32 + r0] * kPairScale, cbh[kb], cbl[kb]);
            const float w0 = qr0t[c * 32 + r0] * kPairInv;
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int v = 0; v < 4; ++v) wq[j][kb][v] = w0 * qr1t[c * 32 + 16 * j + 4 * lg + v];
        }
    }
    __syncthreads();   // slot 2 is read by every wave before any loads a block into it

    // Y[j][kb][v]: row 16 j + 4 lg + v, context 16 kb + li
    // U[jj][kb][v]: column 8 lg + 2 v + jj, context 16 kb + li
    f4 Y[2][NKB], U[2][NKB];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
            Y[j][kb] = f4{0.f, 0.f, 0.f, 0.f};
            U[j][kb] = f4{0.f, 0.f, 0.f, 0.f};
        }

    if (active) {
        // row operands: row 16 j + li, units 2 lg (high parts of columns
        // 8 lg .. 8 lg + 7) and 2 lg + 1 (residuals)
        const int roh = 128 * li + 16 * ((2 * lg) ^ (li & 7));
        const int rol = 128 * li + 16 * ((2 * lg + 1) ^ (li & 7));
        // column operands: rows 8 lg + i, the dword of columns 2 li and
        // 2 li + 1 in units 2 (li >> 2) (high parts) and 2 (li >> 2) + 1; for
        // i = 2 i' + b the two units sit at 32 ((li >> 2) ^ i') + 16 b' (b' = 0 / 1)
        int cob[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) cob[e] = 1024 * lg + 256 * e + 32 * ((li >> 2) ^ e) + 4 * (li & 3);
        for (int c0 = 0; c0 < p.cn0; ++c0) {
            // ring slot (c0 + 2) % 3 was last read at state c0 - 1, whose
            // operands are consumed: load state c0 + 2 into it, then wait for
            // the loads of state c0 (those of c0 + 1 and c0 + 2 may stay out)
            __builtin_amdgcn_sched_barrier(0);
            if (c0 + 2 < p.cn0) {
                dma(c0 + 2);
                asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
            } else if (c0 + 1 < p.cn0) {
                asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
            } else {
                asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            }
            __builtin_amdgcn_sched_barrier(0);
            const char *blk = ring + (c0 % kRing) * (kWaves * kBlockBytes);
            float w[NKB];
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) w[kb] = qc0t[c0 * kCtx + 16 * kb + li];
            uint32_t ch[8], cl[8];
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int b = 0; b < 2; ++b) {
                    // row 8 lg + 2 e + b: high-part unit at position ((2 (li >> 2)) ^ (2 e + b)),
                    // residual unit at the other position of the same pair
                    const char *g = blk + cob[e] + 128 * b;
                    ch[2 * e + b] = *reinterpret_cast<const uint32_t *>(g + 16 * b);
                    cl[2 * e + b] = *reinterpret_cast<const uint32_t *>(g + 16 * (1 - b));
                }
            // rows: Y and this state's m_c0 share
            float s3[NKB];
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) s3[kb] = 0.0f;
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const h8 ah = *reinterpret_cast<const h8 *>(blk + roh + 2048 * j);
                const h8 al = *reinterpret_cast<const h8 *>(blk + rol + 2048 * j);
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb) {
                    const f4 d = chain3(ah, al, rbh[kb], rbl[kb]);
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        Y[j][kb][v] = fmaf(w[kb], d[v], Y[j][kb][v]);
                        s3[kb] = fmaf(wq[j][kb][v], d[v], s3[kb]);
                    }
                }
            }
            // columns: column 2 li + jj of the state
#pragma unroll
            for (int jj = 0; jj < 2; ++jj) {
                const uint32_t sel = jj ? 0x07060302u : 0x05040100u;
                u4 xh, xl;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    xh[e] = __builtin_amdgcn_perm(ch[2 * e + 1], ch[2 * e], sel);
                    xl[e] = __builtin_amdgcn_perm(cl[2 * e + 1], cl[2 * e], sel);
                }
                const h8 ah = __builtin_bit_cast(h8, xh), al = __builtin_bit_cast(h8, xl);
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb) {
                    const f4 d = chain3(ah, al, cbh[kb], cbl[kb]);
#pragma unroll
                    for (int v = 0; v < 4; ++v) U[jj][kb][v] = fmaf(w[kb], d[v], U[jj][kb][v]);
                }
            }
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) s3[kb] = rows_sum4(s3[kb]);
            if (lg == 0)
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb) m3[(wave * kCtx + 16 * kb + li) * kSh + c0] = s3[kb];
        }
        __builtin_amdgcn_sched_barrier(0);
        // m_r0[r0] = sum_{r1} q_r1 Y, over the lane's rows, then the lane rows
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
            const int c = 16 * kb + li;
            float x = 0.0f;
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
                for (int v = 0; v < 4; ++v) x = fmaf(Y[j][kb][v], qr1t[c * 32 + 16 * j + 4 * lg + v], x);
            x = rows_sum4(x);
            if (lg == 0 && c < p.jc) part[(int64_t)ctxs[c] * p.ps + p.o_r0 + r0] = x;
        }
    }
    __syncthreads();   // every wave is done with its ring: it holds the shares next

    const int nw = min(kWaves, p.rn0 - 8 * p.tile);
    // m_c1 shares
    if (active)
#pragma unroll
        for (int jj = 0; jj < 2; ++jj)
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    shares[(wave * kCtx + 16 * kb + li) * kSh + 8 * lg + 2 * v + jj] = U[jj][kb][v];
    __syncthreads();
    for (int i = tid; i < p.jc * 32; i += kThreads) {
        const int c = i >> 5, s = i & 31;
        float acc = 0.0f;
        for (int w = 0; w < nw; ++w) acc += shares[(w * kCtx + c) * kSh + s];
        part[(int64_t)ctxs[c] * p.ps + p.o_c1 + s] = acc;
    }
    for (int i = tid; i < p.jc * p.cn0; i += kThreads) {
        const int c = i / p.cn0, s = i - c * p.cn0;
        float acc = 0.0f;
        for (int w = 0; w < nw; ++w) acc += m3[(w * kCtx + c) * kSh + s];
        part[(int64_t)ctxs[c] * p.ps + p.o_c0 + s] = acc;
    }
    __syncthreads();
    // m_r1 shares: q_r0[r0] Y
    if (active)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) {
                const float wr = qr0w[wave * kCtx + 16 * kb + li];
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    shares[(wave * kCtx + 16 * kb + li) * kSh + 16 * j + 4 * lg + v] = wr * Y[j][kb][v];
            }
    __syncthreads();
    for (int i = tid; i < p.jc * 32; i += kThreads) {
        const int c = i >> 5, s = i & 31;
        float acc = 0.0f;
        for (int w = 0; w < nw; ++w) acc += shares[(w * kCtx + c) * kSh + s];
        part[(int64_t)ctxs[c] * p.ps + p.o_r1 + s] = acc;
    }
    __syncthreads();   // the tables and the ring are refilled by the next pass
}

__global__ __launch_bounds__(kThreads, 1) void rowcol16_lik_kernel(StreamArgs a, const float *__restrict__ q,
                                                                   float *__restrict__ part)
{
    extern __shared__ __attribute__((aligned(16))) char lds[];
    __shared__ int ctxs[kCtx];
    const int wg = a.flip ? (int)gridDim.x - 1 - (int)blockIdx.x : (int)blockIdx.x;
    if (wg >= a.nwg) return;
    int m = 0;
    while (m + 1 < a.M && a.task[m + 1].wg0 <= wg) ++m;
    const SpTask tk = a.task[m];
    const int local = wg - tk.wg0;
    const int o = local / tk.tiles, tile = local - o * tk.tiles;
    const ModDesc &md = a.mods[m];
    const int32_t *start = a.bstart + a.sm[m].bofs;
    const int b0 = start[o], J = start[o + 1] - b0;
    if (J == 0) return;
    Pass p;
    p.P = a.base + md.lp16_off + 4 * (int64_t)o * md.slice;
    p.Cp = md.Cp;
    p.rn0 = md.rn[0];
    p.cn0 = md.cn[0];
    p.tile = tile;
    p.ps = a.pstride;
    p.o_r0 = tk.so;
    p.o_r1 = tk.so + p.rn0 + (int64_t)tile * kN1;
    p.o_c0 = tk.so + p.rn0 + (int64_t)tk.tiles * kN1 + (int64_t)tile * p.cn0;
    p.o_c1 = tk.so + p.rn0 + (int64_t)tk.tiles * (kN1 + p.cn0) + (int64_t)tile * kN1;
    p.off_r0 = a.facs[md.rf[0]].q_off;
    p.off_r1 = a.facs[md.rf[1]].q_off;
    p.off_c0 = a.facs[md.cf[0]].q_off;
    p.off_c1 = a.facs[md.cf[1]].q_off;
    for (int c0 = 0; c0 < J; c0 += kCtx) {
        p.jc = min(kCtx, J - c0);
        if (threadIdx.x < kCtx)
            ctxs[threadIdx.x] = (int)threadIdx.x < p.jc ? a.bctx[(int64_t)m * a.nlist + b0 + c0 + threadIdx.x] : -1;
        __syncthreads();
        const int nkb = (p.jc + 15) >> 4;
        if (nkb == 1) rc_pass<1>(a, p, q, part, ctxs, lds);
        else if (nkb == 2) rc_pass<2>(a, p, q, part, ctxs, lds);
        else rc_pass<3>(a, p, q, part, ctxs, lds);
    }
}

}  // namespace

bool rc_eligible(const bi_model *m)
{
    if (m->M > kStreamMaxM || m->mods.empty()) return false;
    int64_t ps = 0;
    for (const ModDesc &md : m->mods) {
        // the blocked pair copy exists only for the shapes this kernel serves (rc_shape)
        if (md.lp16_off < 0 || md.lp16_order != 1 || !rc_shape(md) || md.K > kStreamMaxK) return false;
        if (4 * (int64_t)md.R * md.Cp >= INT32_MAX) return false;   // 32-bit byte offsets inside a slice
        const int tiles = (md.rn[0] + kWaves - 1) / kWaves;
        ps += md.rn[0] + (int64_t)tiles * (2 * kN1 + md.cn[0]);
    }
    return ps < (int64_t)1 << 30;
}

int64_t rc_plan(const bi_model *m, StreamArgs *a)
{
    int wg = 0;
    int64_t so = 0;
    a->ntask = 0;
    a->nmsg = 0;
    for (int i = 0; i < m->M; ++i) {
        const ModDesc &md = m->mods[i];
        const int rn0 = md.rn[0], cn0 = md.cn[0];
        const int tiles = (rn0 + kWaves - 1) / kWaves;
        SpTask &tk = a->task[a->ntask++];
        tk.m = (int8_t)i;
        tk.role = 0;
        tk.G = (int16_t)kWaves;
        tk.tiles = tiles;
        tk.wg0 = wg;
        tk.so = (int32_t)so;
        wg += md.K * tiles;
        const int32_t f[4] = {md.rf[0], md.rf[1], md.cf[0], md.cf[1]};
        const int32_t copies[4] = {1, tiles, tiles, tiles};
        const int32_t stride[4] = {0, kN1, cn0, kN1};
        const int64_t off[4] = {so, so + rn0, so + rn0 + (int64_t)tiles * kN1,
                                so + rn0 + (int64_t)tiles * (kN1 + cn0)};
        for (int k = 0; k < 4; ++k) {
            MsgSrc &s = a->msg[a->nmsg++];
            s.f = f[k];
            s.copies = copies[k];
            s.stride = stride[k];
            s.off = (int32_t)off[k];
        }
        so += rn0 + (int64_t)tiles * (2 * kN1 + cn0);
    }
    a->nwg = wg;
    return so;
}

size_t rc_lds_bytes() { return kLds; }

int rc_prepare()
{
    const hipError_t e = func_max_lds((const void *)rowcol16_lik_kernel, kLds);
    if (e != hipSuccess) return fail(BI_ERR_DEVICE, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    return BI_OK;
}

void rc_lik_launch(const StreamArgs &a, const float *q, float *part, hipStream_t stream)
{
    hipLaunchKernelGGL(rowcol16_lik_kernel, dim3(a.nwg), dim3(kThreads), kLds, stream, a, q, part);
}

}  // namespace bi
