// Streaming paths (models shared by every agent): internal API.
//
// Both streaming paths run VMP / MMP over the b*T contexts of a call as one
// likelihood launch + one update launch per iteration, with the marginals
// double-buffered in the workspace:
//   dense  (BI_FAST_F32): fp32 matrix-core contractions over the dense slices
//          (stream.hip), fp32 marginals between iterations;
//   sparse (BI_SPARSE_A): fp64 gathers over the nonzero entries of the slices
//          (sparse.hip), fp64 marginals between iterations.
// Contexts are bucketed by observed outcome per modality first; the
// likelihood kernels write partial message vectors per context, which the
// update kernel sums in a fixed order (no atomics: bitwise reproducible).
#pragma once

#include "internal.h"

namespace bi {

constexpr int kStreamMaxM = 16;
constexpr int kStreamMaxK = 8000;           // outcomes per modality (bucket histogram in LDS)
constexpr int kStreamMaxMsg = 4 * kStreamMaxM;
constexpr int kStreamMaxTask = 2 * kStreamMaxM;

struct StreamMod {
    int K;        // outcomes
    int ntiles;   // row tiles of a slice (dense path)
    int wg0;      // first workgroup of this modality in the dense likelihood grid
    int bofs;     // offset of this modality's K+1 bucket starts
    int fofs;     // offset of its outcomes in a soft observation vector (sum of the earlier K)
    int pbeg;     // first value of its partial messages inside a context's partial block
    int64_t poff; // offset of its partial messages inside a context's partial block (dense path)
};

// One source of likelihood messages for factor f: `copies` vectors of n_f
// values at off + k*stride (k < copies) inside a context's partial block.
struct MsgSrc {
    int32_t f;
    int32_t copies;
    int32_t stride;
    int32_t off;
};

// Sparse likelihood task: one side of one modality.  role 0 = row lines (the
// row factors' messages, from the CSR entries), role 1 = column lines (the
// column factors' messages, from the CSC entries).
struct SpTask {
    int8_t m, role;
    int16_t G;      // line groups (first-factor states) per tile
    int32_t wg0;    // first workgroup of the task
    int32_t tiles;  // tiles per outcome
    int32_t so;     // offset of the task's messages inside a context's partial block
};

// Per-factor fields the update kernel reads (kernel arguments, so scalar
// loads): the first kStreamFacs factors; later ones are read from FacDesc.
constexpr int kStreamFacs = 16;
struct StreamFac {
    int64_t lb_off, b_off, ld_off;   // byte offsets of log B, B and log D in the packed buffer
    int32_t n, q_off;
    int64_t lb32_off;                // log B in fp32 (fp32 marginals), or -1
};

struct StreamArgs {
    const char *base;
    const ModDesc *mods;
    const FacDesc *facs;
    int F, M, T, nctx, ntot, nwg;
    int64_t pstride;            // values of partial messages per context
    const int32_t *obs;
    const int32_t *act;
    const float *prior;         // optional [agent][ntot] prior of the first step (replaces D)
    double tau;                 // damping step: q <- (1 - tau) q + tau q_new (1: plain update)
    int32_t *bstart, *bctx;
    int nmsg, ntask;
    int stage;                  // update: partial messages and neighbour marginals staged in LDS
    // Soft observations: every context c stands for 2^vshift slots c 2^vshift + o,
    // slot o observing outcome o of every modality whose vector gives it a
    // nonzero weight.  The likelihood kernels treat slots as contexts (bucket
    // lists and partial blocks per slot, marginals of slot >> vshift); the
    // update sums a context's slots weighted by its vectors.  vshift = 0 and
    // soft = NULL for integer observations.
    int vshift;
    int nlist;                  // bucket-list length per modality: nctx << vshift
    int ksum;                   // values per soft observation vector (sum of K)
    const float *soft;          // [nctx][ksum] soft observation vectors, or NULL
    int flip;                   // likelihood launches: walk the work items in reverse order (odd iterations)
    int trivb;                  // every B-dependency list is {f} (else the update's general transition messages)
    StreamMod sm[kStreamMaxM];
    MsgSrc msg[kStreamMaxMsg];
    SpTask task[kStreamMaxTask];
    StreamFac fac[kStreamFacs];
};

// Whether `m` can run `algo` on the dense streaming kernels.
bool stream_eligible(const bi_model *m, int algo);
// Whether `m` can run `algo` on the sparse streaming kernels.
bool sparse_eligible(const bi_model *m, int algo);
// Workspace bytes of a streaming call with b agents and window T (soft:
// observation vectors instead of outcomes).
size_t stream_workspace(const bi_model *m, int b, int T, bool sparse, bool soft = false);
// Whether a streaming call with soft observation vectors fits its limits (the
// slots' partial blocks staged in the update's LDS, 32-bit slot indices).
bool stream_soft_ok(const bi_model *m, int b, int T, bool sparse);
// Enqueue a streaming VMP / MMP call (dense or sparse likelihood kernels);
// with soft != NULL the [b][T][sum K] observation vectors replace obs.
int launch_stream(const bi_model *m, int algo, int b, int T, const int32_t *obs, const int32_t *act,
                  const float *prior, double tau, int iters, float *q, void *ws, hipStream_t stream, bool sparse,
                  const float *soft = nullptr);

// Dense likelihood kernel with one contraction per workgroup (split.hip), for
// models whose modalities all have two factors per side (second factors of
// 16 or 32 states, first factors of at most 32): eligibility, planning (tasks and message sources; returns the
// values of partial messages per context) and one launch.
bool split_eligible(const bi_model *m);
int64_t split_plan(const bi_model *m, StreamArgs *a);
size_t split_lds_bytes(const bi_model *m, bool sparse);
int split_prepare(const bi_model *m, bool sparse);   // once per call, before the launches
// every modality has its fp16-pair copy (BI_F16_PAIRS): the fp16 matrix-core tiles run
bool split_pairs(const bi_model *m);
// every modality has the sparse fp16-pair layout (BI_SPARSE_A with
// BI_F16_PAIRS): the sparse path runs the same tiles from the nonzeros
// (same plan and partial layout as the dense kernel)
bool sq_eligible(const bi_model *m);
// sparse: the sparse fp16-pair kernel, else the dense one of the model's copy
void split_lik_launch(const bi_model *m, const StreamArgs &a, const float *q, float *part, hipStream_t stream,
                      bool sparse);

// Dense likelihood kernel reading every slice once (rowcol.hip), for models
// with the fp16-pair copy (BI_F16_PAIRS) whose modalities all have two
// factors per side, both second factors of 32 states, the first column
// factor of an even number of states up to 32 and the first row factor of at
// most 32: eligibility, planning (tasks and message sources; returns the
// values of partial messages per context), the dynamic LDS size, the
// once-per-call kernel attribute and one launch.
bool rc_eligible(const bi_model *m);
int64_t rc_plan(const bi_model *m, StreamArgs *a);
size_t rc_lds_bytes();
int rc_prepare();
void rc_lik_launch(const StreamArgs &a, const float *q, float *part, hipStream_t stream);

// Sparse likelihood kernel (sparse.hip): task planning and one launch.
// sparse_plan fills a->task / a->ntask / a->nwg and the message sources,
// and returns the values of partial messages per context.
int64_t sparse_plan(const bi_model *m, StreamArgs *a);
size_t sparse_lds_bytes(const bi_model *m);
int sparse_prepare(const bi_model *m);   // once per call, before the launches
void sparse_lik_launch(const bi_model *m, const StreamArgs &a, const double *q, double *part, hipStream_t stream);

}  // namespace bi
