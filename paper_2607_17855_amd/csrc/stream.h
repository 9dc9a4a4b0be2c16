// Streaming path (models shared by every agent, BI_FAST_F32): internal API.
#pragma once

#include "internal.h"

namespace bi {

constexpr int kStreamMaxM = 16;
constexpr int kStreamMaxK = 8000;   // outcomes per modality (bucket histogram in LDS)

struct StreamMod {
    int K;        // outcomes
    int ntiles;   // row tiles of a slice
    int wg0;      // first workgroup of this modality in the likelihood grid
    int bofs;     // offset of this modality's K+1 bucket starts
    int fofs;     // (reserved)
    int pad;
    int64_t poff; // offset of its partial messages inside a context's partial block
};

struct StreamArgs {
    const char *base;
    const ModDesc *mods;
    const FacDesc *facs;
    int F, M, T, nctx, ntot, nwg;
    int64_t pstride;            // floats of partial messages per context
    const int32_t *obs;
    const int32_t *act;
    int32_t *bstart, *bctx;
    StreamMod sm[kStreamMaxM];
};

// Whether `m` can run `algo` on the streaming kernels.
bool stream_eligible(const bi_model *m, int algo);
// Workspace bytes of a streaming call with b agents and window T.
size_t stream_workspace(const bi_model *m, int b, int T);
// Enqueue a streaming VMP / MMP call.
int launch_stream(const bi_model *m, int algo, int b, int T, const int32_t *obs, const int32_t *act, int iters,
                  float *q, void *ws, hipStream_t stream);

}  // namespace bi
