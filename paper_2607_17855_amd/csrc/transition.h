// Transition messages with B-dependency lists (device code shared by the
// agent-resident kernels and the predict kernel).  B_f conditions the next
// state of factor f on the current states of the factors of its list
// (Sec. III-B, transition model); the messages contract B_f (or log B_f)
// with the marginals of the list.
#pragma once

#include <hip/hip_runtime.h>

#include "layout.h"

namespace bi {

// The B-dependency list of one factor, read once from its descriptor: list
// length, dependency-state count, and per position the offset of the
// listed factor's marginals in a step's marginal vector and its state count.
struct BDep {
    int k, bs;
    int off[kMaxBDep], nn[kMaxBDep];
};

__device__ inline BDep bdep_of(const FacDesc *facs, const FacDesc &fd)
{
    BDep d;
    d.k = fd.nbd;
    d.bs = fd.bstates;
#pragma unroll
    for (int p = 0; p < kMaxBDep; ++p) {
        d.off[p] = p < d.k ? facs[fd.bd[p]].q_off : 0;
        d.nn[p] = fd.bdn[p];
    }
    return d;
}

// sum over the dependency states of row[flat] times the marginals (of one
// step, q[sum n]) of the listed factors other than list position skip, whose
// state is held at fixv (skip -1: none).  row is row i of B_f or log B_f at
// one action ([bstates]).  With the list {f} and skip -1 this is the row
// times q_f; the loops are unrolled over the at most kMaxBDep positions so
// the indices stay in registers.
template <typename BT, typename QT>
__device__ inline double bdep_row(const BDep &d, const BT *row, const QT *q, int skip, int fixv)
{
    // lists of one or two factors: plain and nested dot products
    if (d.k == 1) {
        if (skip == 0) return (double)row[fixv];
        const QT *q0 = q + d.off[0];
        double acc = 0.0;
        for (int j = 0; j < d.nn[0]; ++j) acc = fma((double)row[j], (double)q0[j], acc);
        return acc;
    }
    if (d.k == 2) {
        const QT *q0 = q + d.off[0], *q1 = q + d.off[1];
        const int n1 = d.nn[1];
        if (skip == 0) {
            const BT *r = row + fixv * n1;
            double acc = 0.0;
            for (int j = 0; j < n1; ++j) acc = fma((double)r[j], (double)q1[j], acc);
            return acc;
        }
        if (skip == 1) {
            double acc = 0.0;
            for (int j = 0; j < d.nn[0]; ++j) acc = fma((double)row[j * n1 + fixv], (double)q0[j], acc);
            return acc;
        }
        double acc = 0.0;
        for (int j0 = 0; j0 < d.nn[0]; ++j0) {
            const BT *r = row + j0 * n1;
            double in = 0.0;
            for (int j1 = 0; j1 < n1; ++j1) in = fma((double)r[j1], (double)q1[j1], in);
            acc = fma((double)q0[j0], in, acc);
        }
        return acc;
    }
    // three or four factors: odometer
    int m[kMaxBDep];
#pragma unroll
    for (int p = 0; p < kMaxBDep; ++p) m[p] = p == skip ? fixv : 0;
    double acc = 0.0;
    bool more = true;
    while (more) {
        int flat = 0;
        double w = 1.0;
#pragma unroll
        for (int p = 0; p < kMaxBDep; ++p)
            if (p < d.k) {
                flat = flat * d.nn[p] + m[p];
                if (p != skip) w *= (double)q[d.off[p] + m[p]];
            }
        acc = fma((double)row[flat], w, acc);
        more = false;   // odometer over the free positions, last fastest
#pragma unroll
        for (int p = kMaxBDep - 1; p >= 0; --p)
            if (!more && p < d.k && p != skip) {
                if (++m[p] < d.nn[p])
                    more = true;
                else
                    m[p] = 0;
            }
    }
    return acc;
}

}  // namespace bi
