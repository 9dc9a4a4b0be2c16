// Predictive prior of the next step (Sec. III-B transition model): for every
// agent and factor, out_f(i) = sum_j B_f[i][j][u_f] q_f(j), the same product
// the filtering kernels form between steps.  It is what a caller carries into
// the next window when inference rolls forward one step at a time.
//
// One workgroup per agent, one wave per factor (waves stride the factors),
// one lane per next state i: the lane walks row i of B_f[u] (contiguous in
// the packed [u][i][j] layout) while every lane of the wave reads the same
// q_f(j), a broadcast.  Sums are fp64.  The op moves b * sum_f n_f floats in
// and out plus B, which stays in L2 for shared models: it is launch bound at
// any batch the filtering kernels serve, so it is kept simple.
#include <hip/hip_runtime.h>

#include "internal.h"
#include "transition.h"

namespace bi {

namespace {

struct PredictArgs {
    const char *base;
    const FacDesc *facs;
    int F, ntot, trivb;
    const float *q;
    int64_t q_stride;
    const int32_t *act;
    int64_t act_stride;
    float *out;
};

__global__ __launch_bounds__(256) void predict_kernel(PredictArgs a)
{
    const int agent = blockIdx.x;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const float *qa = a.q + (int64_t)agent * a.q_stride;
    const int32_t *ua = a.act + (int64_t)agent * a.act_stride;
    float *oa = a.out + (int64_t)agent * a.ntot;
    for (int f = wave; f < a.F; f += 4) {
        const FacDesc &fd = a.facs[f];
        const int n = fd.n;
        const int u = ua[f];
        const float *B = reinterpret_cast<const float *>(a.base + fd.b_off) + (int64_t)agent * fd.b_agent +
                         (int64_t)u * n * fd.bstates;
        if (!a.trivb) {   // B-dependency lists: the predictive marginal under the factorised q
            const BDep d = bdep_of(a.facs, fd);
            for (int i = lane; i < n; i += 64) oa[fd.q_off + i] = (float)bdep_row(d, B + (int64_t)i * d.bs, qa, -1, 0);
            continue;
        }
        const float *qf = qa + fd.q_off;
        for (int i = lane; i < n; i += 64) {
            const float *row = B + (int64_t)i * n;
            double acc = 0.0;
            for (int j = 0; j < n; ++j) acc = fma((double)row[j], (double)qf[j], acc);
            oa[fd.q_off + i] = (float)acc;
        }
    }
}

}  // namespace

int launch_predict(const bi_model *m, int b, const float *q, int64_t q_stride, const int32_t *act,
                   int64_t act_stride, float *out, hipStream_t stream)
{
    PredictArgs a;
    a.base = m->dev;
    a.facs = reinterpret_cast<const FacDesc *>(m->dev + align_up((int64_t)sizeof(ModDesc) * m->M, kAlign));
    a.F = m->F;
    a.ntot = m->ntot;
    a.trivb = m->trivial_b;
    a.q = q;
    a.q_stride = q_stride;
    a.act = act;
    a.act_stride = act_stride;
    a.out = out;
    hipLaunchKernelGGL(predict_kernel, dim3(b), dim3(256), 0, stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(BI_ERR_DEVICE, "kernel launch failed: %s", hipGetErrorString(e));
    return BI_OK;
}

}  // namespace bi
