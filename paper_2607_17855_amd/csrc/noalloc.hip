// bi_infer_static: inference for callers that cannot allocate device memory
// (code under HIP graph capture, tight serving loops, harnesses that forbid
// hipMalloc).  The streaming kernel families need scratch memory (outcome
// buckets, partial messages, double-buffered marginals); instead of a
// caller's workspace they get it from a file-scope device array of fixed
// size, one copy per GPU, which lives until the process ends.
//
// Host code never passes the array's name to a kernel: on the host that name
// is a stand-in, not a device address.  The first call on a device, with
// that device current, asks the runtime for the array's address there
// (hipGetSymbolAddress) and keeps it per device; every call then hands that
// address to the same launches as bi_infer, as their workspace.  Nothing in
// the array needs to start at zero: every kernel that reads a workspace word
// has written it earlier in the same call.  Calls that overlap on one GPU
// share the array and race; callers serialise them (one stream, or events).
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.h"

namespace {

constexpr int kMaxDevices = 64;

static __device__ __align__(256) char scratch[BI_STATIC_SCRATCH_BYTES];

std::mutex g_lock;
void *g_ptr[kMaxDevices];   // the array's device address, per device (null until the first call there)

// The array's address on `device` (current), looked up once per device.
int scratch_on(int device, void **out)
{
    if (device < 0 || device >= kMaxDevices)
        return bi::fail(BI_ERR_UNSUPPORTED, "device %d beyond the %d devices the static scratch serves", device,
                        kMaxDevices);
    std::lock_guard<std::mutex> hold(g_lock);
    if (!g_ptr[device]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return bi::fail(BI_ERR_DEVICE, "hipGetSymbolAddress of the static scratch failed: %s",
                            hipGetErrorString(e));
        g_ptr[device] = p;
    }
    *out = g_ptr[device];
    return BI_OK;
}

}  // namespace

extern "C" int bi_infer_static(const bi_model *model, int32_t algo, int32_t b, int32_t T, const int32_t *obs_dev,
                               const int32_t *act_dev, int32_t iters, const bi_infer_opts *opts, float *q_dev,
                               void *hip_stream)
{
    try {
        if (!model) return bi::fail(BI_ERR_INVALID_ARG, "model is NULL");
        if (!model->dev) return bi::fail(BI_ERR_INVALID_ARG, "model has no device buffer (bi_attach_device_buffer)");
        if (model->flags & BI_CHECK)
            return bi::fail(BI_ERR_UNSUPPORTED, "bi_infer_static does not take models packed with BI_CHECK "
                                                "(the check copies its status to the host and synchronises)");
        if (algo < BI_ALGO_FPI || algo > BI_ALGO_MMP) return bi::fail(BI_ERR_INVALID_ARG, "unknown algorithm %d", algo);
        if (b < 1 || T < 1) return bi::fail(BI_ERR_INVALID_ARG, "b and T must be >= 1");
        size_t need = 0;
        int rc = bi_workspace_size(model, b, T, algo, &need);
        if (rc != BI_OK) return rc;
        if (need > BI_STATIC_SCRATCH_BYTES)
            return bi::fail(BI_ERR_UNSUPPORTED, "b=%d T=%d needs %zu bytes of scratch, above the static %zu bytes",
                            b, T, need, (size_t)BI_STATIC_SCRATCH_BYTES);
        int device = -1;
        if (hipGetDevice(&device) != hipSuccess) return bi::fail(BI_ERR_DEVICE, "hipGetDevice failed");
        if (device != model->device)
            return bi::fail(BI_ERR_INVALID_ARG, "device %d is current but the model lives on device %d", device,
                            model->device);
        void *ws = nullptr;
        if (need > 0) {
            rc = scratch_on(device, &ws);
            if (rc != BI_OK) return rc;
        }
        const float *prior = opts ? opts->prior_dev : nullptr;
        const double tau = opts ? opts->damping : 1.0;
        return bi::infer_impl(algo, model, b, T, obs_dev, act_dev, prior, tau, iters, q_dev, ws,
                              need > 0 ? (size_t)BI_STATIC_SCRATCH_BYTES : 0, hip_stream);
    } catch (...) {
        return bi::fail(BI_ERR_INVALID_ARG, "unexpected host exception");
    }
}
