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
// One thread per slice element and agent: it reads X_m[o][e] once per group
// of 8 steps and keeps 8 fp64 sums, the weights being wave-uniform loads.
// Per agent the kernel reads K_m values and writes T values per element:
// HBM bound (the model of a shared batch comes from L2).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "internal.h"
#include "profile.h"

namespace bi {

namespace {

constexpr int kSoftThreads = 256;
constexpr int kSoftT = 8;   // steps per pass over the outcomes

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
    // block -> (modality, first element): blocks of each modality in turn
    int blk = blockIdx.x, m = 0, k0 = 0;
    int64_t po = 0;
    for (; m < a.M; ++m) {
        const int nb = (a.mods[m].slice + kSoftThreads - 1) / kSoftThreads;
        if (blk < nb) break;
        blk -= nb;
        po += a.mods[m].slice;
        k0 += a.mods[m].K;
    }
    if (m >= a.M) return;
    const ModDesc &md = a.mods[m];
    const int e = blk * kSoftThreads + (int)threadIdx.x;
    if (e >= md.slice) return;
    for (int agent = blockIdx.y; agent < a.b; agent += gridDim.y) {
        const double *X = reinterpret_cast<const double *>(a.base + md.la_off) +
                          (a.shared ? 0 : (int64_t)agent * md.la_agent) + e;
        const float *wa = a.w + (int64_t)agent * a.T * a.ksum + k0;
        double *out = a.ll + (int64_t)agent * a.T * a.llpc + po + e;
        for (int t0 = 0; t0 < a.T; t0 += kSoftT) {
            double acc[kSoftT];
#pragma unroll
            for (int j = 0; j < kSoftT; ++j) acc[j] = 0.0;
            const int nt = min(kSoftT, a.T - t0);
            for (int o = 0; o < md.K; ++o) {
                const double x = X[(int64_t)o * md.slice];
#pragma unroll
                for (int j = 0; j < kSoftT; ++j)
                    if (j < nt) acc[j] = fma((double)wa[(int64_t)(t0 + j) * a.ksum + o], x, acc[j]);
            }
#pragma unroll
            for (int j = 0; j < kSoftT; ++j)
                if (j < nt) out[(int64_t)(t0 + j) * a.llpc] = acc[j];
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
    for (const ModDesc &md : m->mods) blocks += (md.slice + kSoftThreads - 1) / kSoftThreads;
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
