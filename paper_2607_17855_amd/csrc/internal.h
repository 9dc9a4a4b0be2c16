// Host-side state of libbi (internal).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "../../include/bi.h"
#include "layout.h"

struct bi_model {
    int32_t F = 0, M = 0, mb = 1;
    uint32_t flags = BI_DENSE_A;
    std::vector<int32_t> n, U, K, dep_off, dep;
    std::vector<int32_t> bdep_off, bdep;   // B-dependency lists ({f} each when trivial)
    bool trivial_b = true;   // every B-dependency list is {f}
    std::vector<bi::ModDesc> mods;
    std::vector<bi::FacDesc> facs;
    int32_t ntot = 0;      // sum of n
    int32_t zvpc = 0;      // floats of Z/V scratch per context: sum_m (R_m + C_m)
    int32_t max_rank = 0;
    int64_t bytes = 0;     // bytes of the packed device buffer in use
    char *dev = nullptr;   // caller's device buffer
    int device = 0;        // HIP device the buffer lives on
    bi_model_stats stats{};
};

namespace bi {

// Record a failure for bi_last_error() and return `code`.
int fail(int code, const char *fmt, ...);

// Layout planning shared by bi_plan_model and bi_pack_model; fills the
// descriptors and offsets of `m` (no data).  Returns BI_OK or an error code.
// A (host) is optional: with it the sparse layout is sized exactly, without
// it for fully dense A (an upper bound).
int plan(const bi_model_desc *desc, bi_model *m, const float *const *A = nullptr);

// Agent-resident launches (one workgroup per agent, every iteration in-kernel).
// Returns BI_OK or an error code.
// `prior` (nullable, device fp32 [b][ntot]) replaces D at the first step;
// `tau` in (0, 1] damps every update: q <- (1 - tau) q + tau q_new.  With
// soft observations obs is NULL and ll holds every context's log-likelihood
// tensors (launch_soft_ll).
// hipFuncSetAttribute(fn, MaxDynamicSharedMemorySize, bytes), issued once per
// (device, kernel, size): every launch asks for it, and the runtime call costs
// host time on launch-bound calls (one-step online filtering).
hipError_t func_max_lds(const void *fn, int bytes);

int launch_agent(const bi_model *m, int algo, int b, int T, const int32_t *obs, const double *ll,
                 const int32_t *act, const float *prior, double tau, int iters, float *q, hipStream_t stream);

// Soft observations (soft.hip): values per context of the log-likelihood
// tensors, and the launch that forms them from w [b][T][sum K].
int64_t soft_values_per_context(const bi_model *m);
int launch_soft_ll(const bi_model *m, int b, int T, const float *w, double *ll, hipStream_t stream);

// BI_CHECK (check.hip): scan obs (may be NULL) and act for out-of-range
// values, using 3 int32 status words of device memory; synchronises `stream`.
// Returns BI_OK or BI_ERR_INVALID_ARG naming the first offending entry.
int check_inputs(const bi_model *m, int b, int T, const int32_t *obs, const int32_t *act, int32_t *status,
                 hipStream_t stream);

// Kernel-family selector (selector.cpp): one of BI_PATH_* among the eligible
// ones (agent always; stream / sparse as flagged), for algo over b agents and
// a window of T steps.
int select_path(const bi_model *m, int algo, int b, int T, bool stream, bool sparse);
// Whether the model holds more A entries than any model the selector was
// fitted on (the selector then decides by a rule).
bool beyond_timed_range(const bi_model *m);

// The inference call behind bi_infer and the named entry points (capi.cpp):
// host validation, optional input check, then the chosen kernel family with
// ws (ws_bytes) as its workspace.  Returns BI_OK or an error code.
int infer_impl(int algo, const bi_model *m, int32_t b, int32_t T, const int32_t *obs, const int32_t *act,
               const float *prior, double tau, int32_t iters, float *q, void *ws, size_t ws_bytes, void *stream);

// Predictive prior B_f[:, :, u] q for every agent and factor (predict.hip).
int launch_predict(const bi_model *m, int b, const float *q, int64_t q_stride, const int32_t *act,
                   int64_t act_stride, float *out, hipStream_t stream);

}  // namespace bi
