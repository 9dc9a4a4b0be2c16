// Kernel-family selector: which of the eligible families (agent-resident,
// dense streaming, sparse streaming) a VMP / MMP call should run.
//
// The families trade differently with the model and the batch: the
// agent-resident kernels keep one agent per workgroup and pay per agent,
// the streaming kernels read every observed slice once per iteration for
// all the contexts that share it and pay per slice.  The choice is a small
// decision tree per (candidate set, algorithm) over features of the packed
// model and the call, fitted to timings of every family on the seeded
// sweep models (uniform and skewed dimension regimes) on MI355X; the tree
// tables are generated (selector_table.h, written by selector/fit.py) and
// hold no code.  Without a table for a candidate set, or for a model with
// more A entries than any timed one, the rule below applies: sparse when
// packed sparse, otherwise the dense streaming kernels once the largest
// slice reaches 16384 entries.
//
// Models packed with fp16 pairs (BI_F16_PAIRS) have trees of their own (the
// candidate sets + 4), fitted to timings of the pair kernels: with the dense
// layout the dense streaming family reads the pair copy; with the sparse
// layout the sparse family runs the pair tiles from 8 bytes per nonzero and
// the dense streaming family the fp32 kernels (no dense pair copy is stored).
// The timed models have no zeros in A, so where the tree (or the rule)
// picks a streaming family for a model with the sparse pair layout, the
// sparse pairs are taken while at most half the entries are nonzero, the
// dense fp32 kernels otherwise.
#include <algorithm>
#include <cmath>

#include "internal.h"
#include "selector_table.h"
#include "stream.h"

namespace bi {

namespace {

double lg2(double x) { return std::log2(std::max(1.0, x)); }

// The features the trees split on (the order of selector_table.h).
void features(const bi_model *m, int b, int T, double *x)
{
    double slices = 0.0, biggest = 0.0, afloats = 0.0;
    int rank = 0, ksum = 0;
    for (const ModDesc &md : m->mods) {
        const double p = (double)md.R * md.C;
        slices += p;
        biggest = std::max(biggest, p);
        afloats += p * md.K;
        rank = std::max(rank, (int)md.rank);
        ksum += md.K;
    }
    x[kFeatContexts] = lg2((double)b * T);
    x[kFeatSlices] = lg2(slices);
    x[kFeatBiggest] = lg2(biggest);
    x[kFeatAFloats] = lg2(afloats);
    x[kFeatT] = T;
    x[kFeatF] = m->F;
    x[kFeatM] = m->M;
    x[kFeatRank] = rank;
    x[kFeatStates] = m->ntot;
    x[kFeatOutcomes] = ksum;
}

int fallback(const bi_model *m, bool stream, bool sparse)
{
    if (sparse) return BI_PATH_SPARSE;
    int64_t biggest = 0;
    for (const ModDesc &md : m->mods) biggest = std::max<int64_t>(biggest, (int64_t)md.R * md.C);
    return stream && biggest >= 16384 ? BI_PATH_STREAM : BI_PATH_AGENT;
}

// Between the two streaming families of a model with the sparse fp16-pair
// layout (rule above).
int streaming_pairs(const bi_model *m, bool stream)
{
    double nnz = 0.0, entries = 0.0;
    for (const ModDesc &md : m->mods) {
        nnz += (double)md.nnz;
        entries += (double)md.K * md.R * md.C;
    }
    return (!stream || nnz <= 0.5 * entries) ? BI_PATH_SPARSE : BI_PATH_STREAM;
}

}  // namespace

bool beyond_timed_range(const bi_model *m)
{
    double x[kNumFeatures];
    features(m, 1, 1, x);
    return x[kFeatAFloats] > kSelMaxAFloats;
}

int select_path(const bi_model *m, int algo, int b, int T, bool stream, bool sparse)
{
    // 1: {agent, stream}, 2: {agent, sparse}, 3: all three; + 4 when the
    // model carries fp16 pairs (the streaming families then run the pair
    // kernels: dense pairs with the dense layout, sparse pairs with the sparse one)
    const int set = (stream ? 1 : 0) | (sparse ? 2 : 0) | (m->flags & BI_F16_PAIRS ? 4 : 0);
    const SelTree *tree = nullptr;
    for (const SelTree &t : kSelTrees)
        if (t.set == set && t.algo == algo) tree = &t;
    double x[kNumFeatures];
    features(m, b, T, x);
    // no timings for this candidate set, or a model larger than every timed
    // one (the trees would extrapolate): the rule
    if (!tree || tree->nodes == 0 || x[kFeatAFloats] > kSelMaxAFloats) {
        const int path = fallback(m, stream, sparse);
        return path != BI_PATH_AGENT && sparse && sq_eligible(m) ? streaming_pairs(m, stream) : path;
    }
    int i = 0;
    while (kSelNodes[tree->first + i].feature >= 0) {
        const SelNode &nd = kSelNodes[tree->first + i];
        i = x[nd.feature] <= nd.threshold ? nd.left : nd.right;
    }
    int path = kSelNodes[tree->first + i].leaf;
    if ((path == BI_PATH_STREAM && !stream) || (path == BI_PATH_SPARSE && !sparse)) path = fallback(m, stream, sparse);
    // the timed models have no zeros in A, so between the two streaming
    // families of the sparse fp16-pair layout the share of nonzeros decides
    if (path != BI_PATH_AGENT && sparse && sq_eligible(m)) path = streaming_pairs(m, stream);
    return path;
}

}  // namespace bi
