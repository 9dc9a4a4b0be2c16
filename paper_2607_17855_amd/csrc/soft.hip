// Soft observations: the log-likelihood tensors of every context.
//
// With an observation vector w_{t,m} over the K_m outcomes of modality m (a
// distribution; one-hot for an integer outcome), the observed slice of the
// integer case becomes the expected log-likelihood
//   LL_{t,m}[r][c] = sum_o w_{t,m}[o] X_m[o][r][c],
// the log(A) . o contraction of Sec. III-C, here taken over the stored
// two-sided slices (layout.h).  All modalities of a context are written one
// after another, modality m at the sum of the slice sizes before it (the
// block-diagonal merge of the Appendix without its zero blocks), so the
// agent-resident kernels read LL_{t,m} exactly where they would read an
// observed slice.  The per-slice shifts of the stored logs become
// sum_o w[o] c_{m,o}, again a constant per (context, modality) that the
// softmax removes.
//
// For one agent and modality this is a dense product: LL_m = W_m X_m with
// W_m the [T][K_m] observation vectors and X_m the [K_m][slice] stored logs,
// done on the fp64 matrix cores (v_mfma_f64_16x16x4f64: 16 steps x 16
// elements per tile, 4 outcomes per product).  A wave owns 64 consecutive
// elements of one modality (4 tiles) and 32 steps (2 row tiles) at a time,
// so every value of X_m leaves memory once per 32 steps; the weights come in
// as fp32 and are widened.  Operand layouts (lane l): A[l % 16][l / 16],
// B[l / 16][l % 16], result element i at row 4 i + l / 16, column l % 16, so
// a store writes 4 steps x 16 consecutive elements.  Out-of-range steps,
// outcomes and elements are read from clamped addresses and enter as zeros.
// The sums over o are exact for one-hot vectors (zeros added to the one
// product), so they reproduce the integer observations' slices bit for bit.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "internal.h"
#include "profile.h"

namespace bi {

namespace {

constexpr int kSoftWaves = 4;
constexpr int kSoftThreads = 64 * kSoftWaves;
constexpr int kSoftNB = 4;                     // 16-element tiles per wave
constexpr int kSoftRT = 2;                     // 16-step tiles per pass
constexpr int kSoftCols = 16 * kSoftNB;        // elements per wave
constexpr int kSoftBlock = kSoftCols * kSoftWaves;

typedef double d4 __attribute__((ext_vector_type(4)));

struct SoftArgs {
    const char *base;
    const ModDesc *mods;
    int M, T, ksum, shared, b;
    int64_t llpc;            // values per context
    const float *w;          // [agent][T][ksum]
    double *ll;              // [agent][T][llpc]
};

__global__ __launch_bounds__(kSoftThreads) void soft_ll_kernel(SoftArgs a)
{
    // block -> (modality, first element): the blocks of each modality in turn
    int blk = blockIdx.x, m = 0, k0m = 0;
    int64_t po = 0;
    for (; m < a.M; ++m) {
        const int nb = (a.mods[m].slice + kSoftBlock - 1) / kSoftBlock;
        if (blk < nb) break;
        blk -= nb;
        po += a.mods[m].slice;
        k0m += a.mods[m].K;
    }
    if (m >= a.M) return;
    const ModDesc &md = a.mods[m];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int e0 = blk * kSoftBlock + wave * kSoftCols;
    if (e0 >= md.slice) return;
    const int li = lane & 15, lg = lane >> 4;
    const int K = md.K, S = md.slice;
    for (int agent = blockIdx.y; agent < a.b; agent += gridDim.y) {
        const double *X = reinterpret_cast<const double *>(a.base + md.la_off) +
                          (a.shared ? 0 : (int64_t)agent * md.la_agent);
        const float *wa = a.w + (int64_t)agent * a.T * a.ksum + k0m;
        double *out = a.ll + (int64_t)agent * a.T * a.llpc + po;
        for (int t0 = 0; t0 < a.T; t0 += 16 * kSoftRT) {
            d4 acc[kSoftRT][kSoftNB];
#pragma unroll
            for (int r = 0; r < kSoftRT; ++r)
#pragma unroll
                for (int nb = 0; nb < kSoftNB; ++nb) acc[r][nb] = d4{0.0, 0.0, 0.0, 0.0};
            for (int k0 = 0; k0 < K; k0 += 4) {
                const int o = k0 + lg;
                const bool ok = o < K;
                const int oc = min(o, K - 1);
                double av[kSoftRT], bv[kSoftNB];
#pragma unroll
                for (int r = 0; r < kSoftRT; ++r) {
                    const int t = t0 + 16 * r + li;
                    const float wv = wa[(int64_t)min(t, a.T - 1) * a.ksum + oc];
                    av[r] = ok && t < a.T ? (double)wv : 0.0;
                }
#pragma unroll
                for (int nb = 0; nb < kSoftNB; ++nb) {
                    const int e = e0 + 16 * nb + li;
                    const double xv = X[(int64_t)oc * S + min(e, S - 1)];
                    bv[nb] = ok && e < S ? xv : 0.0;
                }
#pragma unroll
                for (int r = 0; r < kSoftRT; ++r)
#pragma unroll
                    for (int nb = 0; nb < kSoftNB; ++nb)
                        acc[r][nb] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[r], bv[nb], acc[r][nb], 0, 0, 0);
            }
#pragma unroll
            for (int r = 0; r < kSoftRT; ++r)
#pragma unroll
                for (int nb = 0; nb < kSoftNB; ++nb) {
                    const int e = e0 + 16 * nb + li;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int t = t0 + 16 * r + 4 * i + lg;
                        if (t < a.T && e < S) out[(int64_t)t * a.llpc + e] = acc[r][nb][i];
                    }
                }
        }
    }
}

}  // namespace

int64_t soft_values_per_context(const bi_model *m)
{
    int64_t v = 0;
    for (const ModDesc &md : m->mods) v += md.slice;
    return v;
}

int launch_soft_ll(const bi_model *m, int b, int T, const float *w, double *ll, hipStream_t stream)
{
    SoftArgs a;
    a.base = m->dev;
    a.mods = reinterpret_cast<const ModDesc *>(m->dev);
    a.M = m->M;
    a.T = T;
    a.ksum = 0;
    for (int k : m->K) a.ksum += k;
    a.shared = m->mb == 1;
    a.b = b;
    a.llpc = soft_values_per_context(m);
    a.w = w;
    a.ll = ll;
    int64_t blocks = 0;
    for (const ModDesc &md : m->mods) blocks += (md.slice + kSoftBlock - 1) / kSoftBlock;
    if (blocks > INT32_MAX)
        return fail(BI_ERR_UNSUPPORTED, "soft log-likelihood grid of %lld blocks too large", (long long)blocks);
    {
        ProfScope p("soft_ll", stream);
        hipLaunchKernelGGL(soft_ll_kernel, dim3((unsigned)blocks, (unsigned)std::min(b, 65535)), dim3(kSoftThreads),
                           0, stream, a);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(BI_ERR_DEVICE, "kernel launch failed: %s", hipGetErrorString(e));
    return BI_OK;
}

}  // namespace bi
