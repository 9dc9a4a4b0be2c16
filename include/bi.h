/*
 * bi.h — C-ABI of libbi, MI355X (gfx950) belief updates for discrete
 * HMM / POMDP generative models: variational filtering (FPI), variational
 * message passing (VMP) and marginal message passing (MMP).
 *
 * The generative model is the factorised POMDP of Sec. III-B of "A
 * Hardware-oriented Approach for Efficient Bayesian Inference Computation and
 * Deployment" (joint over o_{1:T}, s_{1:T} given u_{1:T-1}; emission tensors
 * A_m with A-dependency lists of up to 10 factors, transition tensors B_f
 * with B-dependency lists of up to 4 factors, prior D; lists of more than 4
 * likelihood factors run on the agent-resident kernels only).  The three
 * updates are built from the likelihood
 * and transition messages of Sec. IV, each an instance of the coordinate
 * update of Sec. III-A; the exact readings are stated per entry point.
 *
 * Conventions shared by every entry point:
 *  - Every function returns 0 (BI_OK) or a negative BI_ERR_* code and never
 *    throws; bi_last_error() then describes the failure (thread-local).
 *  - "host" pointers are ordinary CPU memory; "device" pointers are HIP device
 *    memory of the current device (e.g. torch tensors).  The caller owns all
 *    memory; the library borrows device pointers until the work it enqueued
 *    on the given stream has completed.
 *  - hip_stream is a hipStream_t passed as void* (NULL = the null stream).
 *    Inference calls only enqueue kernels on it: no host synchronisation, no
 *    device allocation, no host<->device copies.  Arguments are validated on
 *    the host before anything is enqueued.  So a call on a stream under HIP
 *    graph capture is recorded as its kernels and can be replayed (the output
 *    and workspace must then stay allocated; not with BI_CHECK, whose check
 *    synchronises, nor inside bi_profile_begin / _end).
 *  - Layouts are C row-major.  sum_n = n_0 + ... + n_{F-1}.
 */
#ifndef BI_H
#define BI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
#define BI_OK 0
#define BI_ERR_INVALID_ARG (-1)      /* null pointer, non-positive size, bad enum, ... */
#define BI_ERR_SHAPE (-2)            /* inconsistent shapes or dependency lists       */
#define BI_ERR_BUFFER_TOO_SMALL (-3) /* dev_bytes / ws_bytes below what is required   */
#define BI_ERR_UNSUPPORTED (-4)      /* valid, but beyond what this library handles   */
#define BI_ERR_DEVICE (-5)           /* a HIP runtime call failed                     */

/* bi_model_desc.flags: layout of the emission tensors on the device, ORed
 * with an optional precision policy. */
#define BI_DENSE_A 1u  /* dense log-domain slices (default)                         */
#define BI_SPARSE_A 2u /* also store the nonzero entries of every slice (by rows and by
                          columns); models shared by every agent run VMP and MMP on
                          sparse kernels (fp64 arithmetic; fp16-pair matrix cores with
                          BI_F16_PAIRS).  FPI keeps the dense path. */
/* Precision policy.  Without it every update is computed in fp64, which
 * reproduces the fp64 definition to output rounding even where the Jacobi
 * iterations amplify rounding errors by 10^3-10^4 (near-bifurcation models).
 * With BI_FAST_F32 a model shared by all agents (model_batch == 1) runs VMP and
 * MMP through the streaming kernels, whose slice contractions use fp32 matrix
 * cores (messages, sums and the softmax stay fp64; the marginals between
 * iterations and the transition tables are fp32: B for MMP, log B rounded
 * to fp32 for VMP).  Use it for models whose marginals are insensitive to
 * fp32 rounding of the log-likelihoods; it stores an extra fp32 copy of the
 * slices and of log B.
 * Limit (tested at 16 sweeps): the result stays within 1e-5 of the fp64
 * definition exactly when the definition itself moves by less than that under
 * a relative perturbation of log A at the class's rounding scale (2^-24 here,
 * 2^-21 with BI_F16_PAIRS).  Dense Dirichlet models (the seeded sweeps, the
 * large shared model) are far inside it (<= 2e-6); small models with many
 * exact zeros in A can be chaotic under the iteration (the definition moves by
 * up to 1 after 16 sweeps), and then only the fp64 classes reproduce it. */
#define BI_FAST_F32 4u
/* (Both streaming families, BI_FAST_F32 and BI_SPARSE_A, take models shared
 * by every agent, VMP and MMP; with B-dependency lists their update forms the
 * general transition messages.  bi_explain_path tells which family runs.) */
/* With BI_FAST_F32 and the dense layout, a shared model also stores every
 * slice as pairs of fp16 values (high part, rounded residual: 22 significant
 * bits, 4 bytes per entry like the fp32 copy), and the slice contractions of
 * the shapes the matrix-core kernel takes (two factors on each side of the
 * two-sided view, second factors of 16 or 32 states) run on fp16 matrix cores:
 * three fp16 products per fp32 product (high x high, high x residual,
 * residual x high), accumulated in fp32.  The contraction then moves the same
 * bytes at a fraction of the fp32 matrix-core time.
 * With BI_FAST_F32 and BI_SPARSE_A, the nonzero entries of such shapes are
 * stored as fp16 pairs too (8 bytes per nonzero and side, in blocks of 64
 * lines), and the sparse path runs the same fp16 matrix-core products from
 * them: each wave scatters the nonzeros of one first-factor state into a
 * zeroed block in LDS and contracts it.  No dense pair copy is stored then.
 * The stored nonzeros are log(A) - log(1e-16), up to 36.8 in size, so the
 * rounding error relative to the messages grows with the share of nonzeros;
 * the selector takes this path for at most half the entries nonzero. */
#define BI_F16_PAIRS 16u
/* Input checking.  Out-of-range observations or actions are undefined
 * behaviour by default.  With BI_CHECK every inference call first scans obs
 * and act on the device, synchronises its stream and returns
 * BI_ERR_INVALID_ARG (naming the first bad entry, bi_last_error) before any
 * inference kernel runs; the workspace sizes grow by 256 bytes for the check's
 * status words, and such calls cannot be captured in a HIP graph.
 * bi_predict is not checked. */
#define BI_CHECK 8u

/* Kernel families (bi_query_path). */
#define BI_PATH_AGENT 0  /* agent-resident fp64 kernels: one workgroup per agent, all iterations in-kernel */
#define BI_PATH_STREAM 1 /* dense streaming kernels: fp32 (or, with BI_F16_PAIRS, fp16-pair) matrix-core
                            contractions (shared model, BI_FAST_F32) */
#define BI_PATH_SPARSE 2 /* sparse streaming kernels: fp64 gathers over the nonzeros, or with BI_F16_PAIRS
                            fp16-pair matrix-core tiles fed from them (shared model, BI_SPARSE_A) */

/* Algorithm ids (bi_workspace_size). */
#define BI_ALGO_FPI 0
#define BI_ALGO_VMP 1
#define BI_ALGO_MMP 2

/*
 * Shape of a generative model (Sec. III-B).
 *   F factors with n[f] states and U[f] actions each; M modalities with K[m]
 *   outcomes each; modality m depends on the factors
 *   dep[dep_off[m] .. dep_off[m+1]-1], a non-empty, strictly ascending list
 *   (the A-dependency list).  model_batch is 1 when every agent shares the
 *   model, otherwise the number of agents, each with its own parameters (the
 *   batch axis b of Sec. III-B).  flags: BI_DENSE_A or BI_SPARSE_A (0 = dense),
 *   optionally ORed with BI_FAST_F32 (and then BI_F16_PAIRS) and BI_CHECK.
 */
typedef struct bi_model_desc {
    int32_t F;
    const int32_t *n;       /* [F] host */
    const int32_t *U;       /* [F] host */
    int32_t M;
    const int32_t *K;       /* [M] host */
    const int32_t *dep_off; /* [M+1] host, dep_off[0] = 0 */
    const int32_t *dep;     /* [dep_off[M]] host */
    int32_t model_batch;
    uint32_t flags;
    /* B-dependency lists (Sec. III-B, transition model): factor f's next state
     * depends on the current states of bdep[bdep_off[f] .. bdep_off[f+1]),
     * ascending, 1 to 4 factors, each factor in at most 8 lists; B[f] is then
     * [model_batch][n_f][n_{g_1}]..[n_{g_k}][U_f].  NULL (both): every list is
     * {f}, B[f] = [model_batch][n_f][n_f][U_f].  Every kernel family takes
     * such lists (the streaming families' update then forms the general
     * transition messages, one lane per state). */
    const int32_t *bdep_off;
    const int32_t *bdep;
} bi_model_desc;

/* Opaque handle: host-side metadata of a packed model (the packed tensors
 * live in the caller's device buffer). */
typedef struct bi_model bi_model;

/* Parameter counts of a packed model (the paper's memory proxy, Sec. V). */
typedef struct bi_model_stats {
    int64_t a_raw;        /* entries of the A tensors as given                 */
    int64_t a_stored;     /* A entries stored on the device (dense incl. pad)  */
    int64_t a_nnz;        /* nonzero A entries                                 */
    int64_t device_bytes; /* bytes of the packed device buffer in use          */
} bi_model_stats;

/* Boundary plumbing (no passage of the paper): thread-local description of
 * the last error (never NULL). */
const char *bi_last_error(void);

/*
 * Boundary plumbing (sizing; the layout it sizes is that of bi_pack_model).
 * Size of the device buffer that bi_pack_model needs for this model shape.
 * Host only.  For BI_SPARSE_A the size depends on the values of A, so this
 * returns an upper bound (every entry nonzero); bi_plan_model_exact gives the
 * exact size.
 */
int bi_plan_model(const bi_model_desc *desc, size_t *device_bytes);

/* Exact size of the packed buffer for these A tensors (layout as
 * bi_pack_model).  Host only; A as in bi_pack_model. */
int bi_plan_model_exact(const bi_model_desc *desc, const float *const *A, size_t *device_bytes);

/*
 * Pack a model into the caller's device buffer (the one-time layout step of
 * Sec. III-C: "performed only once during initialization").
 *   A[m]: host float [model_batch][K_m][n_{d1}]..[n_{dk}], P(o^m | s^{dep(m)})
 *   B[f]: host float [model_batch][n_f][n_f][U_f], B[i][j][u] = P(s'=i | s=j, u)
 *   D[f]: host float [model_batch][n_f], p(s_1^f)
 *   dev_buf: device memory of at least bi_plan_model bytes, 256-byte aligned.
 * The host arrays are read before the call returns (they may be freed
 * afterwards).  The call copies to the device on hip_stream and synchronises
 * that stream before returning.  *out receives a handle to free with
 * bi_free_model; the caller keeps dev_buf alive while the handle is used.
 * Probabilities are not required to be normalised; zeros are allowed (their
 * logarithm is clamped to log(1e-16)).
 */
int bi_pack_model(const bi_model_desc *desc, const float *const *A, const float *const *B,
                  const float *const *D, void *dev_buf, size_t dev_bytes, void *hip_stream, bi_model **out);

/*
 * Host-only variant of bi_pack_model: writes the same packed image into host
 * memory (host_buf, at least bi_plan_model bytes, 256-byte aligned) and
 * returns a handle that has no device buffer yet.  Copy the image to a device
 * buffer yourself (or save it and reload it later) and declare it with
 * bi_attach_device_buffer before inference.  Needs no GPU.
 */
int bi_pack_model_host(const bi_model_desc *desc, const float *const *A, const float *const *B,
                       const float *const *D, void *host_buf, size_t host_bytes, bi_model **out);

/*
 * Declare that dev_buf (device memory, 256-byte aligned, dev_bytes >= the
 * packed size) holds a byte-identical copy of the image that
 * bi_pack_model_host wrote for this handle.  The library does not check the
 * contents.  Replaces any buffer attached before.
 */
int bi_attach_device_buffer(bi_model *model, void *dev_buf, size_t dev_bytes);

/* Parameter counts of a packed model. */
int bi_get_model_stats(const bi_model *model, bi_model_stats *out);

/*
 * Boundary plumbing (sizing).  Device workspace (bytes, 256-byte aligned start
 * required) that an inference call with b agents, window T and algorithm algo
 * needs; may be 0, in which case ws_dev may be NULL.  The workspace holds the
 * streaming paths' outcome buckets, partial messages and double-buffered
 * marginals; its contents need not be initialised and are scratch after the
 * call.
 */
int bi_workspace_size(const bi_model *model, int32_t b, int32_t T, int32_t algo, size_t *bytes);

/*
 * Variational filtering ("FPI", Sec. I and IV): for t = 0..T-1 in order, the
 * prior of step t is D (t = 0) or B_f[:,:,u_{t-1,f}] q_{t-1,f} (the final
 * marginal of the previous step); q_t starts uniform and takes `iters`
 * Jacobi sweeps of q_{t,f} = softmax(lam_{t,f} + log prior_{t,f}), where the
 * likelihood message is
 *   lam_{t,f}(s) = sum_{m: f in dep(m)} sum_{s_dep: s_f = s}
 *                  log A_m[o_{t,m}, s_dep] prod_{g in dep(m), g != f} q_{t,g}(s_g)
 * (the marginalisation step of Sec. IV).
 *   obs_dev: device int32 [b][T][M], 0 <= obs < K_m
 *   act_dev: device int32 [b][T-1][F], 0 <= act < U_f (may be NULL if T == 1)
 *   q_dev:   device float [b][T][sum_n], output posterior marginals
 *   ws_dev:  device workspace of ws_bytes >= bi_workspace_size(..., BI_ALGO_FPI)
 * b must equal model_batch unless model_batch == 1.  Out-of-range obs/act
 * values are undefined behaviour.
 */
int bi_vfilter(const bi_model *model, int32_t b, int32_t T, const int32_t *obs_dev, const int32_t *act_dev,
               int32_t iters, float *q_dev, void *ws_dev, size_t ws_bytes, void *hip_stream);

/*
 * Variational message passing over the window (Sec. III-A update applied to
 * the joint of Sec. III-B with q = prod_{t,f} q_{t,f}): q starts uniform and
 * takes `iters` Jacobi sweeps over every (t, f) of
 *   q_{t,f} = softmax(lam_{t,f} + fwd_{t,f} + bwd_{t,f}),
 *   fwd = log D_f (t = 0), else sum_{s'} log B_f[s, s', u_{t-1}] q_{t-1,f}(s'),
 *   bwd = 0 (t = T-1),    else sum_{s''} q_{t+1,f}(s'') log B_f[s'', s, u_t].
 * Arguments as bi_vfilter.
 */
int bi_vmp(const bi_model *model, int32_t b, int32_t T, const int32_t *obs_dev, const int32_t *act_dev,
           int32_t iters, float *q_dev, void *ws_dev, size_t ws_bytes, void *hip_stream);

/*
 * Marginal message passing over the window (Sec. I and IV): as bi_vmp but with
 * the marginal (log-of-expectation) transition messages
 *   fwd = log D_f (t = 0), else log(B_f[:,:,u_{t-1}] q_{t-1,f}),
 *   bwd = log(B_f[:,:,u_t]^T q_{t+1,f}) (t < T-1),
 * averaged over the messages present:
 *   q_{t,f} = softmax(lam + (fwd + bwd) / 2) for t < T-1, softmax(lam + fwd) at t = T-1.
 * Arguments as bi_vfilter.
 */
int bi_mmp(const bi_model *model, int32_t b, int32_t T, const int32_t *obs_dev, const int32_t *act_dev,
           int32_t iters, float *q_dev, void *ws_dev, size_t ws_bytes, void *hip_stream);

/*
 * Rolling (online) inference.  The window of Sec. III-B is the current step
 * and the h steps before it; when it slides, the belief about its first step
 * comes from what was inferred before rather than from D.  These three calls
 * are bi_vfilter / bi_vmp / bi_mmp with p(s_1) = D replaced by the caller's
 * prior over the window's first step:
 *   prior_dev: device fp32 [b][sum_f n_f], factor f's block at sum_{g<f} n_g,
 *              each block a distribution over the factor's states (zeros
 *              allowed: their logarithm is clamped to log(1e-16)); read only,
 *              must stay valid until the stream work completes; NULL is
 *              BI_ERR_INVALID_ARG.
 * Every other argument, the workspace and the errors are those of the call
 * without a prior.  Typical use: prior = bi_predict of an earlier marginal.
 */
int bi_vfilter_prior(const bi_model *model, int32_t b, int32_t T, const int32_t *obs_dev, const int32_t *act_dev,
                     const float *prior_dev, int32_t iters, float *q_dev, void *ws_dev, size_t ws_bytes,
                     void *hip_stream);
int bi_vmp_prior(const bi_model *model, int32_t b, int32_t T, const int32_t *obs_dev, const int32_t *act_dev,
                 const float *prior_dev, int32_t iters, float *q_dev, void *ws_dev, size_t ws_bytes,
                 void *hip_stream);
int bi_mmp_prior(const bi_model *model, int32_t b, int32_t T, const int32_t *obs_dev, const int32_t *act_dev,
                 const float *prior_dev, int32_t iters, float *q_dev, void *ws_dev, size_t ws_bytes,
                 void *hip_stream);

/*
 * Options of bi_infer (all calls above are bi_infer with some of them fixed).
 *   prior_dev: NULL (the first step's prior is D) or as for bi_vfilter_prior.
 *   damping:   step tau in (0, 1] of a damped update: every sweep (every
 *              iteration of FPI at a step; every Jacobi sweep of VMP / MMP)
 *              mixes the new marginal with the current one,
 *                q <- (1 - tau) q + tau q_new,
 *              q_new being the update stated above for that algorithm.
 *              1 is the plain update; a fixed point of the plain update is
 *              one of the damped update, which oscillates less.
 */
typedef struct bi_infer_opts {
    const float *prior_dev;
    double damping;
} bi_infer_opts;

/*
 * Inference with options: algo is BI_ALGO_FPI / _VMP / _MMP; opts NULL means
 * { NULL, 1.0 }.  Other arguments, the workspace (bi_workspace_size for the
 * same algo) and the errors are those of bi_vfilter; a damping outside
 * (0, 1] (or NaN) is BI_ERR_INVALID_ARG, as is an unknown algo.
 */
int bi_infer(const bi_model *model, int32_t algo, int32_t b, int32_t T, const int32_t *obs_dev,
             const int32_t *act_dev, int32_t iters, const bi_infer_opts *opts, float *q_dev, void *ws_dev,
             size_t ws_bytes, void *hip_stream);

/*
 * No-allocation inference, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): bi_infer without a workspace.  The scratch the streaming kernel
 * families need lives in a static device array of BI_STATIC_SCRATCH_BYTES
 * that the library holds on every GPU it runs on until the process ends; the
 * caller still passes inputs and outputs (and the packed model), and the call
 * allocates nothing (no hipMalloc / hipFree, no allocating library routine).
 *   - Arguments, results and errors are those of bi_infer, on the device
 *     that is current, which must be the model's (else BI_ERR_INVALID_ARG).
 *   - A call whose bi_workspace_size exceeds BI_STATIC_SCRATCH_BYTES returns
 *     BI_ERR_UNSUPPORTED before enqueueing anything; models packed with
 *     BI_CHECK are refused the same way (the check synchronises and copies).
 *   - Every call on a GPU shares that GPU's array and leaves its contents
 *     behind (nothing needs to start at zero).  Calls that overlap in time on
 *     one GPU (several streams or threads) race on it: serialise them.
 *   - The first call on a device looks up the array's address there (once);
 *     after that a call only enqueues kernels, so it can be captured.
 */
#define BI_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
int bi_infer_static(const bi_model *model, int32_t algo, int32_t b, int32_t T, const int32_t *obs_dev,
                    const int32_t *act_dev, int32_t iters, const bi_infer_opts *opts, float *q_dev,
                    void *hip_stream);

/*
 * The kernel family a call with these sizes will run (BI_PATH_*).  FPI always
 * runs agent-resident.  VMP and MMP on a model shared by every agent may
 * also run the dense streaming kernels (packed with BI_FAST_F32) or the
 * sparse ones (packed with BI_SPARSE_A); among the families the packing
 * allows, a selector fitted to timings of seeded sweep models on MI355X
 * picks the one expected to be fastest for (model, algo, b, T).  Host only.
 *
 * Test and timing hook: the environment variable BI_FORCE_PATH = "agent",
 * "stream" or "sparse", read at every call, overrides the selector's choice
 * among the eligible families (never the eligibility itself); any other
 * value is ignored.  It exists so tests and timing sweeps can run each
 * family; production callers leave it unset.
 */
int bi_query_path(const bi_model *model, int32_t b, int32_t T, int32_t algo, int32_t *path);

/*
 * Boundary plumbing (no passage of the paper): a one-line, NUL-terminated
 * account of the family bi_query_path returns for these arguments and of why
 * each streaming family is or is not eligible (e.g. "agent (the only
 * eligible family); stream: B-dependency lists are not trivial ...; sparse:
 * not packed with BI_SPARSE_A"), truncated to cap bytes.  Host only.
 */
int bi_explain_path(const bi_model *model, int32_t b, int32_t T, int32_t algo, char *buf, size_t cap);

/*
 * Soft observations (Sec. III-C: the log-likelihood of a modality is the
 * contraction log(A_m) . o_m of its A-array with an observation vector).
 * Instead of integer outcomes, every context carries one vector per modality:
 *   obs_dev: device fp32 [b][T][sum_m K_m], modality m's vector over its K_m
 *            outcomes at offset sum_{m' < m} K_m' (a distribution, e.g. a
 *            noisy sensor's output; one-hot reproduces the integer call).
 * Every log A_m[o_{t,m}, s_dep] in the updates above becomes the expected
 * log-likelihood sum_o o_{t,m}[o] log A_m[o, s_dep].  Which kernels run:
 *   - when bi_query_path picks a streaming family for these arguments (a
 *     shared model packed for it; VMP or MMP), the model holds more A
 *     entries than the models the selector was timed on (about 4.3 million;
 *     there the agent-resident kernels are far slower) or BI_FORCE_PATH names that
 *     family, and every modality has at most 256 outcomes: that family, over
 *     slots (t, o) of each context, slot o
 *     observing outcome o in every modality whose vector gives o a nonzero
 *     weight; the update sums a context's slot messages weighted by its
 *     vectors (fp64).  The likelihood work grows with the nonzero weights per
 *     vector (one-hot vectors cost the integer call and give its bits);
 *   - otherwise (FPI, per-agent models, the agent-resident choice): the
 *     expected log-likelihood tensors, formed once per call before the
 *     iterations (b * T * sum_m prod_{f in dep(m)} n_f doubles, the slices
 *     padded as in the packed model), and the agent-resident kernels on the
 *     dense fp64 planes.
 *   ws_bytes >= bi_workspace_size_soft(model, b, T, algo), 256-byte aligned
 *   (the streaming workspace with its slots, or the tensors).
 * algo, opts and the other arguments are those of bi_infer; the same errors.
 */
int bi_workspace_size_soft(const bi_model *model, int32_t b, int32_t T, int32_t algo, size_t *bytes);
int bi_infer_soft(const bi_model *model, int32_t algo, int32_t b, int32_t T, const float *obs_dev,
                  const int32_t *act_dev, int32_t iters, const bi_infer_opts *opts, float *q_dev, void *ws_dev,
                  size_t ws_bytes, void *hip_stream);

/*
 * Predictive prior of the next step (the product FPI uses between steps,
 * Sec. III-B transition model): for every agent a and factor f
 *   out[a][f](i) = sum_j B_f[i][j][u_{a,f}] q[a][f](j)      (fp64 sums)
 *   q_dev:    device fp32 marginals of agent a at q_dev + a * q_stride
 *             (q_stride >= sum_f n_f floats; e.g. one step of a bi_vfilter
 *             output with q_stride = T * sum_f n_f);
 *   act_dev:  device int32 actions of agent a at act_dev + a * act_stride
 *             (act_stride >= F), u_{a,f} in [0, U_f);
 *   out_dev:  device fp32 [b][sum_f n_f], written.
 * b must equal the model's agent count when the model is per-agent.  Errors:
 * BI_ERR_INVALID_ARG (NULL pointers, b < 1, strides too small),
 * BI_ERR_SHAPE (b versus model_batch).  Asynchronous on hip_stream; allocates
 * nothing.
 */
int bi_predict(const bi_model *model, int32_t b, const float *q_dev, int64_t q_stride, const int32_t *act_dev,
               int64_t act_stride, float *out_dev, void *hip_stream);

/* Boundary plumbing: free the host metadata of a packed model (not the
 * caller's device buffer).  NULL is ignored. */
void bi_free_model(bi_model *model);

/*
 * Kernel timing (profiling aid).  Between bi_profile_begin and bi_profile_end
 * every kernel the library enqueues is bracketed by a pair of HIP events on
 * the call's stream (the recording adds two small packets per launch).
 * bi_profile_end waits for those events and reports, per kernel class
 * ("lik", "update", "bucket", "init", "agent_window", "agent_filter"), the
 * number of launches and their summed duration in milliseconds, in at most
 * `cap` entries of `out`; *n_out receives the number of classes seen.
 * Process-wide; not for concurrent use from several threads.
 */
typedef struct bi_profile_entry {
    char name[32];
    int64_t launches;
    double total_ms;
} bi_profile_entry;

int bi_profile_begin(void);
int bi_profile_end(bi_profile_entry *out, int32_t cap, int32_t *n_out);

#ifdef __cplusplus
}
#endif

#endif /* BI_H */
