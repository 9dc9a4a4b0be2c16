// extern "C" entry points of libbi (declared in include/bi.h).
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <set>
#include <tuple>

#include "internal.h"
#include "stream.h"

namespace bi {
const char *last_error();
int fill(const bi_model *m, const float *const *A, const float *const *B, const float *const *D, char *host,
         int64_t *nnz_out);
}  // namespace bi

using bi::fail;

namespace {

enum class Path { Agent = BI_PATH_AGENT, Stream = BI_PATH_STREAM, Sparse = BI_PATH_SPARSE };

// BI_CHECK: status words of the input check, after the call's own workspace
constexpr size_t kStatusBytes = 256;

// Dispatch among the kernel families the packed model is eligible for: the
// agent-resident fp64 kernels (always), the dense streaming kernels (shared
// model, BI_FAST_F32: the caller opted into fp32 contractions) and the
// sparse streaming kernels (shared model, BI_SPARSE_A).  With more than one
// eligible, the measured selector decides (selector.cpp).
// BI_FORCE_PATH=agent|stream|sparse overrides the choice (tests, timing
// sweeps), never the eligibility.
Path choose_path(const bi_model *m, int algo, int b, int T)
{
    const bool stream = bi::stream_eligible(m, algo), sparse = bi::sparse_eligible(m, algo);
    const char *env = std::getenv("BI_FORCE_PATH");
    if (env) {
        if (std::strcmp(env, "agent") == 0) return Path::Agent;
        if (std::strcmp(env, "stream") == 0 && stream) return Path::Stream;
        if (std::strcmp(env, "sparse") == 0 && sparse) return Path::Sparse;
    }
    if (!stream && !sparse) return Path::Agent;
    return static_cast<Path>(bi::select_path(m, algo, b, T, stream, sparse));
}

// Why a model is not eligible for a streaming family (NULL: eligible).
const char *stream_refusal(const bi_model *m, int algo, bool sparse)
{
    if (sparse ? !(m->flags & BI_SPARSE_A) : !(m->flags & BI_FAST_F32))
        return sparse ? "not packed with BI_SPARSE_A" : "not packed with BI_FAST_F32";
    if (m->mb != 1) return "per-agent model (the streaming kernels share one model among all agents)";
    if (algo == BI_ALGO_FPI) return "FPI runs agent-resident (sequential over the window)";
    for (const bi::ModDesc &md : m->mods)
        if (md.nrow > bi::kStreamSide || md.ncol > bi::kStreamSide)
            return "a modality depends on more than 4 factors (the streaming layouts serve up to 2 per side)";
    if (sparse ? bi::sparse_eligible(m, algo) : bi::stream_eligible(m, algo)) return nullptr;
    return "a modality's shape exceeds the streaming kernels' limits (outcomes, modalities or LDS tiles)";
}

// The family a call with soft observation vectors runs.  On the streaming
// kernels a vector weighting k outcomes costs about k likelihood launches'
// work, on the agent-resident ones the log-likelihood tensors cost little
// more than the integer call, so soft vectors stream only where the agent
// path is far behind: models beyond the selector's timed range (on the
// shared F=4x32 model, 33 ms against 722 ms per call; on the sweep models
// the selector streams, the agent path was 3-12x faster with soft vectors),
// or when BI_FORCE_PATH names the family; and only when the slots fit the
// streaming limits (stream_soft_ok).
Path soft_path(const bi_model *m, int algo, int b, int T)
{
    const Path p = choose_path(m, algo, b, T);
    if (p == Path::Agent || !bi::stream_soft_ok(m, b, T, p == Path::Sparse)) return Path::Agent;
    const char *env = std::getenv("BI_FORCE_PATH");
    const bool forced = env && std::strcmp(env, p == Path::Sparse ? "sparse" : "stream") == 0;
    return forced || bi::beyond_timed_range(m) ? p : Path::Agent;
}

}  // namespace

namespace bi {
hipError_t func_max_lds(const void *fn, int bytes)
{
    static std::mutex mu;
    static std::set<std::tuple<int, const void *, int>> done;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) dev = -1;
    const auto key = std::make_tuple(dev, fn, bytes);
    {
        std::lock_guard<std::mutex> g(mu);
        if (done.count(key)) return hipSuccess;
    }
    const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e == hipSuccess) {
        std::lock_guard<std::mutex> g(mu);
        done.insert(key);
    }
    return e;
}

int infer_impl(int algo, const bi_model *model, int32_t b, int32_t T, const int32_t *obs, const int32_t *act,
                   const float *prior, double tau, int32_t iters, float *q, void *ws, size_t ws_bytes, void *stream)
{
    try {
        if (!model) return fail(BI_ERR_INVALID_ARG, "model is NULL");
        if (!model->dev) return fail(BI_ERR_INVALID_ARG, "model has no device buffer (bi_attach_device_buffer)");
        if (b < 1 || T < 1 || iters < 1) return fail(BI_ERR_INVALID_ARG, "b, T and iters must be >= 1");
        if (model->mb != 1 && model->mb != b)
            return fail(BI_ERR_SHAPE, "b=%d but the model holds %d agents", b, model->mb);
        if (!obs || !q) return fail(BI_ERR_INVALID_ARG, "obs and q must be non-NULL");
        if (T > 1 && !act) return fail(BI_ERR_INVALID_ARG, "act must be non-NULL when T > 1");
        if (!(tau > 0.0 && tau <= 1.0)) return fail(BI_ERR_INVALID_ARG, "damping %g is not in (0, 1]", tau);
        size_t need = 0;
        int rc = bi_workspace_size(model, b, T, algo, &need);
        if (rc != BI_OK) return rc;
        if (ws_bytes < need) return fail(BI_ERR_BUFFER_TOO_SMALL, "ws_bytes %zu < %zu required", ws_bytes, need);
        if (need > 0 && !ws) return fail(BI_ERR_INVALID_ARG, "ws is NULL");
        if (need > 0 && reinterpret_cast<uintptr_t>(ws) % bi::kAlign)
            return fail(BI_ERR_INVALID_ARG, "ws must be %d-byte aligned", bi::kAlign);
        hipStream_t s = reinterpret_cast<hipStream_t>(stream);
        if (model->flags & BI_CHECK) {
            rc = bi::check_inputs(model, b, T, obs, act,
                                  reinterpret_cast<int32_t *>(static_cast<char *>(ws) + need - kStatusBytes), s);
            if (rc != BI_OK) return rc;
        }
        const Path p = choose_path(model, algo, b, T);
        if (p != Path::Agent)
            return bi::launch_stream(model, algo, b, T, obs, act, prior, tau, iters, q, ws, s, p == Path::Sparse);
        return bi::launch_agent(model, algo, b, T, obs, nullptr, act, prior, tau, iters, q, s);
    } catch (...) {
        return fail(BI_ERR_INVALID_ARG, "unexpected host exception");
    }
}
}  // namespace bi

extern "C" {

const char *bi_last_error(void) { return bi::last_error(); }

int bi_plan_model(const bi_model_desc *desc, size_t *device_bytes)
{
    try {
        if (!device_bytes) return fail(BI_ERR_INVALID_ARG, "device_bytes is NULL");
        bi_model m;
        const int rc = bi::plan(desc, &m);
        if (rc != BI_OK) return rc;
        *device_bytes = (size_t)m.bytes;
        return BI_OK;
    } catch (const std::bad_alloc &) {
        return fail(BI_ERR_INVALID_ARG, "host allocation failed");
    } catch (...) {
        return fail(BI_ERR_INVALID_ARG, "unexpected host exception");
    }
}

// Plan + fill into host memory; on success *out owns the metadata.
static int pack_host(const bi_model_desc *desc, const float *const *A, const float *const *B, const float *const *D,
                     char *host, size_t host_bytes, bi_model **out)
{
    *out = nullptr;
    if (!A || !B || !D) return fail(BI_ERR_INVALID_ARG, "A, B and D must be non-NULL");
    if (desc && desc->M > 0)
        for (int i = 0; i < desc->M; ++i)
            if (!A[i]) return fail(BI_ERR_INVALID_ARG, "A[%d] is NULL", i);
    bi_model *m = new bi_model;
    int rc = bi::plan(desc, m, A);
    if (rc != BI_OK) {
        delete m;
        return rc;
    }
    for (int i = 0; i < m->F; ++i)
        if (!B[i] || !D[i]) {
            delete m;
            return fail(BI_ERR_INVALID_ARG, "B[%d] or D[%d] is NULL", i, i);
        }
    if (host == nullptr) {  // caller only wanted the plan checked
        *out = m;
        return BI_OK;
    }
    if ((int64_t)host_bytes < m->bytes) {
        const long long need = (long long)m->bytes;
        delete m;
        return fail(BI_ERR_BUFFER_TOO_SMALL, "buffer of %zu bytes < %lld required", host_bytes, need);
    }
    std::memset(host, 0, (size_t)m->bytes);
    int64_t nnz = 0;
    bi::fill(m, A, B, D, host, &nnz);
    m->stats.a_nnz = nnz;
    *out = m;
    return BI_OK;
}

int bi_plan_model_exact(const bi_model_desc *desc, const float *const *A, size_t *device_bytes)
{
    try {
        if (!device_bytes) return fail(BI_ERR_INVALID_ARG, "device_bytes is NULL");
        if (!A) return fail(BI_ERR_INVALID_ARG, "A is NULL");
        if (desc && desc->M > 0)
            for (int i = 0; i < desc->M; ++i)
                if (!A[i]) return fail(BI_ERR_INVALID_ARG, "A[%d] is NULL", i);
        bi_model m;
        const int rc = bi::plan(desc, &m, A);
        if (rc != BI_OK) return rc;
        *device_bytes = (size_t)m.bytes;
        return BI_OK;
    } catch (const std::bad_alloc &) {
        return fail(BI_ERR_INVALID_ARG, "host allocation failed");
    } catch (...) {
        return fail(BI_ERR_INVALID_ARG, "unexpected host exception");
    }
}

int bi_pack_model_host(const bi_model_desc *desc, const float *const *A, const float *const *B,
                       const float *const *D, void *host_buf, size_t host_bytes, bi_model **out)
{
    try {
        if (!out) return fail(BI_ERR_INVALID_ARG, "out is NULL");
        *out = nullptr;
        if (!host_buf) return fail(BI_ERR_INVALID_ARG, "host_buf is NULL");
        if (reinterpret_cast<uintptr_t>(host_buf) % bi::kAlign)
            return fail(BI_ERR_INVALID_ARG, "host_buf must be %d-byte aligned", bi::kAlign);
        return pack_host(desc, A, B, D, reinterpret_cast<char *>(host_buf), host_bytes, out);
    } catch (const std::bad_alloc &) {
        return fail(BI_ERR_INVALID_ARG, "host allocation failed");
    } catch (...) {
        return fail(BI_ERR_INVALID_ARG, "unexpected host exception");
    }
}

int bi_attach_device_buffer(bi_model *model, void *dev_buf, size_t dev_bytes)
{
    if (!model || !dev_buf) return fail(BI_ERR_INVALID_ARG, "model and dev_buf must be non-NULL");
    if (reinterpret_cast<uintptr_t>(dev_buf) % bi::kAlign)
        return fail(BI_ERR_INVALID_ARG, "dev_buf must be %d-byte aligned", bi::kAlign);
    if ((int64_t)dev_bytes < model->bytes)
        return fail(BI_ERR_BUFFER_TOO_SMALL, "dev_bytes %zu < %lld required", dev_bytes, (long long)model->bytes);
    model->dev = reinterpret_cast<char *>(dev_buf);
    if (hipGetDevice(&model->device) != hipSuccess) model->device = 0;
    return BI_OK;
}

int bi_pack_model(const bi_model_desc *desc, const float *const *A, const float *const *B, const float *const *D,
                  void *dev_buf, size_t dev_bytes, void *hip_stream, bi_model **out)
{
    try {
        if (!out) return fail(BI_ERR_INVALID_ARG, "out is NULL");
        *out = nullptr;
        if (!dev_buf) return fail(BI_ERR_INVALID_ARG, "dev_buf is NULL");
        if (reinterpret_cast<uintptr_t>(dev_buf) % bi::kAlign)
            return fail(BI_ERR_INVALID_ARG, "dev_buf must be %d-byte aligned", bi::kAlign);
        bi_model *m = nullptr;
        int rc = pack_host(desc, A, B, D, nullptr, 0, &m);  // validate before allocating
        if (rc != BI_OK) return rc;
        if ((int64_t)dev_bytes < m->bytes) {
            const long long need = (long long)m->bytes;
            delete m;
            return fail(BI_ERR_BUFFER_TOO_SMALL, "dev_bytes %zu < %lld required", dev_bytes, need);
        }
        const size_t bytes = (size_t)m->bytes;
        delete m;
        char *host = nullptr;
        const hipError_t he = hipHostMalloc((void **)&host, bytes, hipHostMallocDefault);
        if (he != hipSuccess)
            return fail(BI_ERR_DEVICE, "hipHostMalloc of %zu bytes failed: %s", bytes, hipGetErrorString(he));
        rc = pack_host(desc, A, B, D, host, bytes, &m);
        if (rc != BI_OK) {
            hipHostFree(host);
            return rc;
        }
        hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
        hipError_t e = hipMemcpyAsync(dev_buf, host, bytes, hipMemcpyHostToDevice, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        hipHostFree(host);
        if (e != hipSuccess) {
            delete m;
            return fail(BI_ERR_DEVICE, "copy to device failed: %s", hipGetErrorString(e));
        }
        m->dev = reinterpret_cast<char *>(dev_buf);
        if (hipGetDevice(&m->device) != hipSuccess) m->device = 0;
        *out = m;
        return BI_OK;
    } catch (const std::bad_alloc &) {
        return fail(BI_ERR_INVALID_ARG, "host allocation failed");
    } catch (...) {
        return fail(BI_ERR_INVALID_ARG, "unexpected host exception");
    }
}

int bi_get_model_stats(const bi_model *model, bi_model_stats *out)
{
    if (!model || !out) return fail(BI_ERR_INVALID_ARG, "model and out must be non-NULL");
    *out = model->stats;
    return BI_OK;
}

int bi_workspace_size(const bi_model *model, int32_t b, int32_t T, int32_t algo, size_t *bytes)
{
    if (!model || !bytes) return fail(BI_ERR_INVALID_ARG, "model and bytes must be non-NULL");
    if (b < 1 || T < 1) return fail(BI_ERR_INVALID_ARG, "b and T must be >= 1");
    if (algo < BI_ALGO_FPI || algo > BI_ALGO_MMP) return fail(BI_ERR_INVALID_ARG, "unknown algorithm %d", algo);
    const Path p = choose_path(model, algo, b, T);
    *bytes = p == Path::Agent ? 0 : bi::stream_workspace(model, b, T, p == Path::Sparse);
    if (model->flags & BI_CHECK) *bytes = (size_t)bi::align_up((int64_t)*bytes, bi::kAlign) + kStatusBytes;
    return BI_OK;
}

int bi_vfilter(const bi_model *model, int32_t b, int32_t T, const int32_t *obs_dev, const int32_t *act_dev,
               int32_t iters, float *q_dev, void *ws_dev, size_t ws_bytes, void *hip_stream)
{
    return bi::infer_impl(BI_ALGO_FPI, model, b, T, obs_dev, act_dev, nullptr, 1.0, iters, q_dev, ws_dev, ws_bytes, hip_stream);
}

int bi_vmp(const bi_model *model, int32_t b, int32_t T, const int32_t *obs_dev, const int32_t *act_dev,
           int32_t iters, float *q_dev, void *ws_dev, size_t ws_bytes, void *hip_stream)
{
    return bi::infer_impl(BI_ALGO_VMP, model, b, T, obs_dev, act_dev, nullptr, 1.0, iters, q_dev, ws_dev, ws_bytes, hip_stream);
}

int bi_mmp(const bi_model *model, int32_t b, int32_t T, const int32_t *obs_dev, const int32_t *act_dev,
           int32_t iters, float *q_dev, void *ws_dev, size_t ws_bytes, void *hip_stream)
{
    return bi::infer_impl(BI_ALGO_MMP, model, b, T, obs_dev, act_dev, nullptr, 1.0, iters, q_dev, ws_dev, ws_bytes, hip_stream);
}

int bi_vfilter_prior(const bi_model *model, int32_t b, int32_t T, const int32_t *obs_dev, const int32_t *act_dev,
                     const float *prior_dev, int32_t iters, float *q_dev, void *ws_dev, size_t ws_bytes,
                     void *hip_stream)
{
    if (!prior_dev) return fail(BI_ERR_INVALID_ARG, "prior is NULL");
    return bi::infer_impl(BI_ALGO_FPI, model, b, T, obs_dev, act_dev, prior_dev, 1.0, iters, q_dev, ws_dev, ws_bytes, hip_stream);
}

int bi_vmp_prior(const bi_model *model, int32_t b, int32_t T, const int32_t *obs_dev, const int32_t *act_dev,
                 const float *prior_dev, int32_t iters, float *q_dev, void *ws_dev, size_t ws_bytes,
                 void *hip_stream)
{
    if (!prior_dev) return fail(BI_ERR_INVALID_ARG, "prior is NULL");
    return bi::infer_impl(BI_ALGO_VMP, model, b, T, obs_dev, act_dev, prior_dev, 1.0, iters, q_dev, ws_dev, ws_bytes, hip_stream);
}

int bi_mmp_prior(const bi_model *model, int32_t b, int32_t T, const int32_t *obs_dev, const int32_t *act_dev,
                 const float *prior_dev, int32_t iters, float *q_dev, void *ws_dev, size_t ws_bytes,
                 void *hip_stream)
{
    if (!prior_dev) return fail(BI_ERR_INVALID_ARG, "prior is NULL");
    return bi::infer_impl(BI_ALGO_MMP, model, b, T, obs_dev, act_dev, prior_dev, 1.0, iters, q_dev, ws_dev, ws_bytes, hip_stream);
}

int bi_infer(const bi_model *model, int32_t algo, int32_t b, int32_t T, const int32_t *obs_dev,
             const int32_t *act_dev, int32_t iters, const bi_infer_opts *opts, float *q_dev, void *ws_dev,
             size_t ws_bytes, void *hip_stream)
{
    if (algo < BI_ALGO_FPI || algo > BI_ALGO_MMP) return fail(BI_ERR_INVALID_ARG, "unknown algorithm %d", algo);
    const float *prior = opts ? opts->prior_dev : nullptr;
    const double tau = opts ? opts->damping : 1.0;
    return bi::infer_impl(algo, model, b, T, obs_dev, act_dev, prior, tau, iters, q_dev, ws_dev, ws_bytes, hip_stream);
}

int bi_query_path(const bi_model *model, int32_t b, int32_t T, int32_t algo, int32_t *path)
{
    if (!model || !path) return fail(BI_ERR_INVALID_ARG, "model and path must be non-NULL");
    if (b < 1 || T < 1) return fail(BI_ERR_INVALID_ARG, "b and T must be >= 1");
    if (algo < BI_ALGO_FPI || algo > BI_ALGO_MMP) return fail(BI_ERR_INVALID_ARG, "unknown algorithm %d", algo);
    *path = static_cast<int32_t>(choose_path(model, algo, b, T));
    return BI_OK;
}

int bi_explain_path(const bi_model *model, int32_t b, int32_t T, int32_t algo, char *buf, size_t cap)
{
    if (!model || !buf || cap == 0) return fail(BI_ERR_INVALID_ARG, "model and buf must be non-NULL, cap > 0");
    if (b < 1 || T < 1) return fail(BI_ERR_INVALID_ARG, "b and T must be >= 1");
    if (algo < BI_ALGO_FPI || algo > BI_ALGO_MMP) return fail(BI_ERR_INVALID_ARG, "unknown algorithm %d", algo);
    static const char *names[] = {"agent", "stream", "sparse"};
    const Path p = choose_path(model, algo, b, T);
    const char *rs = stream_refusal(model, algo, false), *rp = stream_refusal(model, algo, true);
    const char *env = std::getenv("BI_FORCE_PATH");
    const char *how = (rs && rp) ? "the only eligible family"
                      : (env && std::strcmp(env, names[static_cast<int>(p)]) == 0) ? "forced by BI_FORCE_PATH"
                                                                                      : "chosen by the selector";
    std::snprintf(buf, cap, "%s (%s); stream: %s; sparse: %s", names[static_cast<int>(p)], how,
                  rs ? rs : "eligible", rp ? rp : "eligible");
    return BI_OK;
}

int bi_workspace_size_soft(const bi_model *model, int32_t b, int32_t T, int32_t algo, size_t *bytes)
{
    if (!model || !bytes) return fail(BI_ERR_INVALID_ARG, "model and bytes must be non-NULL");
    if (b < 1 || T < 1) return fail(BI_ERR_INVALID_ARG, "b and T must be >= 1");
    if (algo < BI_ALGO_FPI || algo > BI_ALGO_MMP) return fail(BI_ERR_INVALID_ARG, "unknown algorithm %d", algo);
    const Path p = soft_path(model, algo, b, T);
    if (p != Path::Agent) {
        *bytes = bi::stream_workspace(model, b, T, p == Path::Sparse, true);
    } else {
        const int64_t vals = bi::soft_values_per_context(model);
        if (vals > (INT64_MAX / 8) / ((int64_t)b * T))
            return fail(BI_ERR_UNSUPPORTED, "soft log-likelihood tensors of b=%d T=%d overflow", b, T);
        *bytes = (size_t)bi::align_up((int64_t)b * T * vals * 8, bi::kAlign);
    }
    if (model->flags & BI_CHECK) *bytes += kStatusBytes;
    return BI_OK;
}

int bi_infer_soft(const bi_model *model, int32_t algo, int32_t b, int32_t T, const float *obs_dev,
                  const int32_t *act_dev, int32_t iters, const bi_infer_opts *opts, float *q_dev, void *ws_dev,
                  size_t ws_bytes, void *hip_stream)
{
    try {
        if (!model) return fail(BI_ERR_INVALID_ARG, "model is NULL");
        if (!model->dev) return fail(BI_ERR_INVALID_ARG, "model has no device buffer (bi_attach_device_buffer)");
        if (algo < BI_ALGO_FPI || algo > BI_ALGO_MMP) return fail(BI_ERR_INVALID_ARG, "unknown algorithm %d", algo);
        if (b < 1 || T < 1 || iters < 1) return fail(BI_ERR_INVALID_ARG, "b, T and iters must be >= 1");
        if (model->mb != 1 && model->mb != b)
            return fail(BI_ERR_SHAPE, "b=%d but the model holds %d agents", b, model->mb);
        if (!obs_dev || !q_dev) return fail(BI_ERR_INVALID_ARG, "obs and q must be non-NULL");
        if (T > 1 && !act_dev) return fail(BI_ERR_INVALID_ARG, "act must be non-NULL when T > 1");
        const float *prior = opts ? opts->prior_dev : nullptr;
        const double tau = opts ? opts->damping : 1.0;
        if (!(tau > 0.0 && tau <= 1.0)) return fail(BI_ERR_INVALID_ARG, "damping %g is not in (0, 1]", tau);
        size_t need = 0;
        int rc = bi_workspace_size_soft(model, b, T, algo, &need);
        if (rc != BI_OK) return rc;
        if (ws_bytes < need) return fail(BI_ERR_BUFFER_TOO_SMALL, "ws_bytes %zu < %zu required", ws_bytes, need);
        if (!ws_dev) return fail(BI_ERR_INVALID_ARG, "ws is NULL");
        if (reinterpret_cast<uintptr_t>(ws_dev) % bi::kAlign)
            return fail(BI_ERR_INVALID_ARG, "ws must be %d-byte aligned", bi::kAlign);
        hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
        if (model->flags & BI_CHECK) {
            rc = bi::check_inputs(model, b, T, nullptr, act_dev,
                                  reinterpret_cast<int32_t *>(static_cast<char *>(ws_dev) + need - kStatusBytes), s);
            if (rc != BI_OK) return rc;
        }
        const Path p = soft_path(model, algo, b, T);
        if (p != Path::Agent)
            return bi::launch_stream(model, algo, b, T, nullptr, act_dev, prior, tau, iters, q_dev, ws_dev, s,
                                     p == Path::Sparse, obs_dev);
        double *ll = reinterpret_cast<double *>(ws_dev);
        rc = bi::launch_soft_ll(model, b, T, obs_dev, ll, s);
        if (rc != BI_OK) return rc;
        return bi::launch_agent(model, algo, b, T, nullptr, ll, act_dev, prior, tau, iters, q_dev, s);
    } catch (...) {
        return fail(BI_ERR_INVALID_ARG, "unexpected host exception");
    }
}

int bi_predict(const bi_model *model, int32_t b, const float *q_dev, int64_t q_stride, const int32_t *act_dev,
               int64_t act_stride, float *out_dev, void *hip_stream)
{
    try {
        if (!model) return fail(BI_ERR_INVALID_ARG, "model is NULL");
        if (!model->dev) return fail(BI_ERR_INVALID_ARG, "model has no device buffer (bi_attach_device_buffer)");
        if (b < 1) return fail(BI_ERR_INVALID_ARG, "b must be >= 1");
        if (model->mb != 1 && model->mb != b)
            return fail(BI_ERR_SHAPE, "b=%d but the model holds %d agents", b, model->mb);
        if (!q_dev || !act_dev || !out_dev) return fail(BI_ERR_INVALID_ARG, "q, act and out must be non-NULL");
        if (q_stride < model->ntot)
            return fail(BI_ERR_INVALID_ARG, "q_stride %lld < %d states", (long long)q_stride, model->ntot);
        if (act_stride < model->F)
            return fail(BI_ERR_INVALID_ARG, "act_stride %lld < %d factors", (long long)act_stride, model->F);
        return bi::launch_predict(model, b, q_dev, q_stride, act_dev, act_stride, out_dev,
                                  reinterpret_cast<hipStream_t>(hip_stream));
    } catch (...) {
        return fail(BI_ERR_INVALID_ARG, "unexpected host exception");
    }
}

void bi_free_model(bi_model *model) { delete model; }

}  // extern "C"
