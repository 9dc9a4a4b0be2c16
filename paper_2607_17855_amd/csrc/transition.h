// Transition messages with B-dependency lists (device code shared by the
// agent-resident kernels and the predict kernel).  B_f conditions the next
// state of factor f on the current states of the factors of its list
// (Sec. III-B, transition model); the messages contract B_f (or log B_f)
// with the marginals of the list.
#pragma once

#include <hip/hip_runtime.h>

#include "layout.h"

namespace bi {

// sum over the B-dependency states of factor fd of Bu[i][flat] times the
// marginals (of one step, q[sum n]) of the dependencies other than list
// position skip, whose state is held at fixv (skip -1: none).  Bu is B_f or
// log B_f at one action, [n][bstates].  With the list {f} and skip -1 this is
// the matrix-vector product B_f[u] q_f; the loops are unrolled over the
// at most kMaxBDep positions so the indices stay in registers.
template <typename BT, typename QT>
__device__ inline double bdep_sum(const FacDesc *facs, const FacDesc &fd, const BT *Bu, int i, const QT *q,
                                  int skip, int fixv)
{
    const int k = fd.nbd;
    int m[kMaxBDep], off[kMaxBDep], nn[kMaxBDep];
#pragma unroll
    for (int p = 0; p < kMaxBDep; ++p) {
        m[p] = p == skip ? fixv : 0;
        off[p] = p < k ? facs[fd.bd[p]].q_off : 0;
        nn[p] = fd.bdn[p];
    }
    const BT *row = Bu + (int64_t)i * fd.bstates;
    double acc = 0.0;
    bool more = true;
    while (more) {
        int flat = 0;
        double w = 1.0;
#pragma unroll
        for (int p = 0; p < kMaxBDep; ++p)
            if (p < k) {
                flat = flat * nn[p] + m[p];
                if (p != skip) w *= (double)q[off[p] + m[p]];
            }
        acc = fma((double)row[flat], w, acc);
        more = false;   // odometer over the free positions, last fastest
#pragma unroll
        for (int p = kMaxBDep - 1; p >= 0; --p)
            if (!more && p < k && p != skip) {
                if (++m[p] < nn[p])
                    more = true;
                else
                    m[p] = 0;
            }
    }
    return acc;
}

}  // namespace bi
