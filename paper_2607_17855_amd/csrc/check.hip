// Input validation for models packed with BI_CHECK: one workgroup scans the
// observation and action arrays of a call, counts the values outside
// [0, K_m) / [0, U_f) and records the first offending index, then the host
// reads the two words back (the call synchronises its stream).  A single
// workgroup keeps it free of atomics and of any clearing of the status
// words: it is a few microseconds at every batch served here.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace bi {

namespace {

constexpr int kChkThreads = 1024;

struct CheckArgs {
    const ModDesc *mods;
    const FacDesc *facs;
    int M, F, T, b;
    const int32_t *obs;   // [b][T][M] or NULL
    const int32_t *act;   // [b][T-1][F] or NULL
    int32_t *status;      // [0] bad values, [1] first bad flat index (obs first, then act), [2] which (0 obs, 1 act)
};

__global__ __launch_bounds__(kChkThreads) void check_kernel(CheckArgs a)
{
    __shared__ int cnt[kChkThreads];
    __shared__ int64_t first[kChkThreads];
    const int tid = threadIdx.x;
    const int64_t nobs = a.obs ? (int64_t)a.b * a.T * a.M : 0;
    const int64_t nact = a.act && a.T > 1 ? (int64_t)a.b * (a.T - 1) * a.F : 0;
    int c = 0;
    int64_t f = INT64_MAX;
    for (int64_t i = tid; i < nobs + nact; i += kChkThreads) {
        bool bad;
        if (i < nobs) {
            const int v = a.obs[i];
            bad = v < 0 || v >= a.mods[i % a.M].K;
        } else {
            const int64_t j = i - nobs;
            const int v = a.act[j];
            bad = v < 0 || v >= a.facs[j % a.F].U;
        }
        if (bad) {
            ++c;
            if (i < f) f = i;
        }
    }
    cnt[tid] = c;
    first[tid] = f;
    __syncthreads();
    for (int s = kChkThreads / 2; s > 0; s >>= 1) {
        if (tid < s) {
            cnt[tid] += cnt[tid + s];
            first[tid] = min(first[tid], first[tid + s]);
        }
        __syncthreads();
    }
    if (tid == 0) {
        const int64_t i = first[0];
        a.status[0] = cnt[0];
        a.status[1] = cnt[0] == 0 ? -1 : (int32_t)min(i < nobs ? i : i - nobs, (int64_t)INT32_MAX);
        a.status[2] = cnt[0] == 0 ? -1 : (i < nobs ? 0 : 1);
    }
}

}  // namespace

int check_inputs(const bi_model *m, int b, int T, const int32_t *obs, const int32_t *act, int32_t *status,
                 hipStream_t stream)
{
    CheckArgs a;
    a.mods = reinterpret_cast<const ModDesc *>(m->dev);
    a.facs = reinterpret_cast<const FacDesc *>(m->dev + align_up((int64_t)sizeof(ModDesc) * m->M, kAlign));
    a.M = m->M;
    a.F = m->F;
    a.T = T;
    a.b = b;
    a.obs = obs;
    a.act = act;
    a.status = status;
    hipLaunchKernelGGL(check_kernel, dim3(1), dim3(kChkThreads), 0, stream, a);
    hipError_t e = hipGetLastError();
    int32_t host[3] = {0, -1, -1};
    if (e == hipSuccess) e = hipMemcpyAsync(host, status, sizeof(host), hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return fail(BI_ERR_DEVICE, "input check failed: %s", hipGetErrorString(e));
    if (host[0] != 0) {
        if (host[2] == 0)
            return fail(BI_ERR_INVALID_ARG, "%d out-of-range inputs; first: obs[%d] (agent %d, step %d, modality %d)",
                        host[0], host[1], host[1] / (T * m->M), host[1] / m->M % T, host[1] % m->M);
        return fail(BI_ERR_INVALID_ARG, "%d out-of-range inputs; first: act[%d] (agent %d, step %d, factor %d)",
                    host[0], host[1], host[1] / ((T - 1) * m->F), host[1] / m->F % (T - 1), host[1] % m->F);
    }
    return BI_OK;
}

}  // namespace bi
