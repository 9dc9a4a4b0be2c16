// Host packer: validates a model description, plans the device layout of
// layout.h and converts the user's A / B / D tensors into it.  This is the
// one-time padding/merging step of Sec. III-C (done once at initialisation,
// no cost at inference time); the layout itself is the two-sided slice view
// described in layout.h rather than the paper's axis-aligned or
// block-diagonal merge.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <thread>

#include "internal.h"

namespace bi {

static thread_local std::string g_err = "no error";

int fail(int code, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

const char *last_error() { return g_err.c_str(); }

static int64_t prod(const int32_t *n, const int32_t *f, int k)
{
    int64_t p = 1;
    for (int i = 0; i < k; ++i) p *= n[f[i]];
    return p;
}

int plan(const bi_model_desc *d, bi_model *m, const float *const *A)
{
    if (!d) return fail(BI_ERR_INVALID_ARG, "desc is NULL");
    if (d->F < 1 || d->M < 1) return fail(BI_ERR_INVALID_ARG, "F and M must be >= 1 (F=%d, M=%d)", d->F, d->M);
    if (!d->n || !d->U || !d->K || !d->dep_off || !d->dep)
        return fail(BI_ERR_INVALID_ARG, "desc has a NULL array");
    if (d->model_batch < 1) return fail(BI_ERR_INVALID_ARG, "model_batch must be >= 1");
    uint32_t flags = d->flags ? d->flags : BI_DENSE_A;
    if ((flags & ~(BI_DENSE_A | BI_SPARSE_A | BI_FAST_F32 | BI_F16_PAIRS | BI_CHECK)) != 0)
        return fail(BI_ERR_INVALID_ARG, "unknown bits in flags");
    if ((flags & BI_F16_PAIRS) && !(flags & BI_FAST_F32))
        return fail(BI_ERR_INVALID_ARG, "BI_F16_PAIRS needs BI_FAST_F32");
    if ((flags & (BI_DENSE_A | BI_SPARSE_A)) == 0) flags |= BI_DENSE_A;
    if ((flags & BI_DENSE_A) && (flags & BI_SPARSE_A))
        return fail(BI_ERR_INVALID_ARG, "flags must hold one of BI_DENSE_A and BI_SPARSE_A");
    if ((flags & BI_SPARSE_A) && d->model_batch != 1)
        return fail(BI_ERR_UNSUPPORTED, "the sparse A layout is for models shared by every agent");
    m->F = d->F;
    m->M = d->M;
    m->mb = d->model_batch;
    m->flags = flags;
    m->n.assign(d->n, d->n + d->F);
    m->U.assign(d->U, d->U + d->F);
    m->K.assign(d->K, d->K + d->M);
    m->dep_off.assign(d->dep_off, d->dep_off + d->M + 1);
    for (int f = 0; f < d->F; ++f) {
        if (d->n[f] < 1 || d->U[f] < 1) return fail(BI_ERR_SHAPE, "factor %d: n and U must be >= 1", f);
        if (d->n[f] > 65535) return fail(BI_ERR_UNSUPPORTED, "factor %d: more than 65535 states", f);
    }
    if (d->dep_off[0] != 0) return fail(BI_ERR_SHAPE, "dep_off[0] must be 0");
    for (int mm = 0; mm < d->M; ++mm) {
        const int k = d->dep_off[mm + 1] - d->dep_off[mm];
        if (k < 1) return fail(BI_ERR_SHAPE, "modality %d: empty dependency list", mm);
        if (d->K[mm] < 1) return fail(BI_ERR_SHAPE, "modality %d: K must be >= 1", mm);
        for (int i = d->dep_off[mm]; i < d->dep_off[mm + 1]; ++i) {
            if (d->dep[i] < 0 || d->dep[i] >= d->F)
                return fail(BI_ERR_SHAPE, "modality %d: dependency %d out of range", mm, d->dep[i]);
            if (i > d->dep_off[mm] && d->dep[i] <= d->dep[i - 1])
                return fail(BI_ERR_SHAPE, "modality %d: dependency list not strictly ascending", mm);
        }
        if (k > 2 * kMaxSide)
            return fail(BI_ERR_UNSUPPORTED, "modality %d depends on %d factors; this library handles up to %d", mm, k,
                        2 * kMaxSide);
    }
    m->dep.assign(d->dep, d->dep + d->dep_off[d->M]);
    // B-dependency lists (NULL: trivial)
    if ((d->bdep_off == nullptr) != (d->bdep == nullptr))
        return fail(BI_ERR_INVALID_ARG, "bdep_off and bdep must both be set or both be NULL");
    m->bdep_off.clear();
    m->bdep.clear();
    for (int f = 0; f <= d->F; ++f) m->bdep_off.push_back(f);
    for (int f = 0; f < d->F; ++f) m->bdep.push_back(f);
    if (d->bdep_off) {
        if (d->bdep_off[0] != 0) return fail(BI_ERR_SHAPE, "bdep_off[0] must be 0");
        for (int f = 0; f < d->F; ++f) {
            const int k = d->bdep_off[f + 1] - d->bdep_off[f];
            if (k < 1) return fail(BI_ERR_SHAPE, "factor %d: empty B-dependency list", f);
            if (k > kMaxBDep)
                return fail(BI_ERR_UNSUPPORTED, "factor %d: %d B-dependencies; this library handles up to %d", f, k,
                            kMaxBDep);
            for (int i = d->bdep_off[f]; i < d->bdep_off[f + 1]; ++i) {
                if (d->bdep[i] < 0 || d->bdep[i] >= d->F)
                    return fail(BI_ERR_SHAPE, "factor %d: B-dependency %d out of range", f, d->bdep[i]);
                if (i > d->bdep_off[f] && d->bdep[i] <= d->bdep[i - 1])
                    return fail(BI_ERR_SHAPE, "factor %d: B-dependency list not strictly ascending", f);
            }
        }
        m->bdep_off.assign(d->bdep_off, d->bdep_off + d->F + 1);
        m->bdep.assign(d->bdep, d->bdep + d->bdep_off[d->F]);
    }
    m->trivial_b = true;
    for (int f = 0; f < d->F; ++f)
        if (m->bdep_off[f + 1] - m->bdep_off[f] != 1 || m->bdep[m->bdep_off[f]] != f) m->trivial_b = false;

    // descriptor tables first
    int64_t off = 0;
    off += (int64_t)sizeof(ModDesc) * m->M;
    off = align_up(off, kAlign);
    off += (int64_t)sizeof(FacDesc) * m->F;
    off = align_up(off, kAlign);

    m->mods.assign(m->M, ModDesc{});
    m->facs.assign(m->F, FacDesc{});
    int32_t qoff = 0;
    for (int f = 0; f < m->F; ++f) {
        FacDesc &fd = m->facs[f];
        fd.n = m->n[f];
        fd.U = m->U[f];
        fd.q_off = qoff;
        qoff += m->n[f];
        fd.nbd = m->bdep_off[f + 1] - m->bdep_off[f];
        int64_t bs = 1;
        for (int i = 0; i < kMaxBDep; ++i) {
            fd.bd[i] = i < fd.nbd ? m->bdep[m->bdep_off[f] + i] : -1;
            fd.bdn[i] = i < fd.nbd ? m->n[fd.bd[i]] : 1;
            bs *= fd.bdn[i];
        }
        if (bs * fd.n * fd.U > INT32_MAX / 2) return fail(BI_ERR_UNSUPPORTED, "factor %d: B too large", f);
        fd.bstates = (int32_t)bs;
        fd.nch = 0;
        for (int i = 0; i < kMaxCh; ++i) fd.ch[i] = fd.chpos[i] = -1;
    }
    m->ntot = qoff;
    for (int j = 0; j < m->F; ++j)   // children: j is a child of every factor on its list
        for (int p = 0; p < m->facs[j].nbd; ++p) {
            FacDesc &fd = m->facs[m->facs[j].bd[p]];
            if (fd.nch == kMaxCh)
                return fail(BI_ERR_UNSUPPORTED, "factor %d is on more than %d B-dependency lists", m->facs[j].bd[p],
                            kMaxCh);
            fd.ch[fd.nch] = j;
            fd.chpos[fd.nch] = p;
            ++fd.nch;
        }

    int64_t a_raw = 0, a_stored = 0;
    int32_t zv = 0;
    m->max_rank = 0;
    for (int mm = 0; mm < m->M; ++mm) {
        ModDesc &md = m->mods[mm];
        const int32_t *dl = m->dep.data() + m->dep_off[mm];
        const int k = m->dep_off[mm + 1] - m->dep_off[mm];
        m->max_rank = std::max(m->max_rank, k);
        // rows = first p factors, columns = the rest, at most L per side (L =
        // kStreamSide for lists of up to 4 factors, which keeps them in the
        // streaming layouts' shape, else kMaxSide), 1 <= k-p, chosen to
        // balance the two sides
        const int L = k <= 2 * kStreamSide ? kStreamSide : kMaxSide;
        int best_p = -1;
        int64_t best = INT64_MAX;
        for (int p = std::max(0, k - L); p <= std::min(L, k - 1); ++p) {
            const int64_t R = prod(m->n.data(), dl, p), C = prod(m->n.data(), dl + p, k - p);
            const int64_t cost = R > C ? R - C : C - R;
            if (cost < best) {
                best = cost;
                best_p = p;
            }
        }
        const int p = best_p;
        const int64_t R = prod(m->n.data(), dl, p), C = prod(m->n.data(), dl + p, k - p);
        const int64_t Cp = align_up(C, 4);
        if (R * Cp > INT32_MAX / 2) return fail(BI_ERR_UNSUPPORTED, "modality %d: slice too large", mm);
        md.K = m->K[mm];
        md.rank = k;
        md.R = (int32_t)R;
        md.C = (int32_t)C;
        md.Cp = (int32_t)Cp;
        md.slice = (int32_t)(R * Cp);
        md.nrow = p;
        md.ncol = k - p;
        for (int i = 0; i < kMaxSide; ++i) {
            md.rf[i] = i < p ? dl[i] : -1;
            md.rn[i] = i < p ? m->n[dl[i]] : 1;
            md.cf[i] = i < k - p ? dl[p + i] : -1;
            md.cn[i] = i < k - p ? m->n[dl[p + i]] : 1;
        }
        md.zv_off = zv;
        zv += (int32_t)(R + C);
        md.dsum = 0;
        for (int i = 0; i < k; ++i) md.dsum += m->n[dl[i]];
        md.la_off = off;
        md.la_agent = m->mb == 1 ? 0 : (int64_t)md.K * md.slice;
        off = align_up(off + 8 * (int64_t)m->mb * md.K * md.slice, kAlign);
        // the streaming layouts (fp32 copy, fp16 pairs, sparse planes) serve
        // modalities with at most kStreamSide factors per side; a wider one
        // leaves its model to the agent-resident kernels
        const bool narrow = p <= kStreamSide && k - p <= kStreamSide;
        md.la32_off = -1;
        if ((flags & BI_FAST_F32) && narrow) {
            md.la32_off = off;
            off = align_up(off + 4 * (int64_t)m->mb * md.K * md.slice, kAlign);
        }
        md.lp16_off = -1;
        // dense pairs (the matrix-core kernels serve shared models; with the
        // sparse layout the pairs are stored with the nonzeros instead)
        if ((flags & BI_F16_PAIRS) && (flags & BI_DENSE_A) && m->mb == 1 && narrow) {
            md.lp16_off = off;
            off = align_up(off + 4 * (int64_t)md.K * md.slice, kAlign);
        }
        md.csr_ptr_off = md.csr_ent_off = md.csc_ptr_off = md.csc_ent_off = -1;
        md.nnz = 0;
        if ((flags & BI_SPARSE_A) && narrow) {
            // exact entry count when A is given, else an upper bound (dense)
            int64_t nnz = (int64_t)md.K * R * C;
            if (A) {
                nnz = 0;
                const float *a = A[mm];
                const int64_t tot = (int64_t)md.K * R * C;
                for (int64_t e = 0; e < tot; ++e) nnz += (double)a[e] > kEps;
            }
            if (nnz > INT32_MAX) return fail(BI_ERR_UNSUPPORTED, "modality %d: too many nonzero entries", mm);
            md.nnz = nnz;
            md.csr_ptr_off = off;
            off = align_up(off + 4 * (int64_t)md.K * (R + 1), kAlign);
            md.csr_ent_off = off;
            off = align_up(off + (int64_t)sizeof(SpEntry) * nnz, kAlign);
            md.csc_ptr_off = off;
            off = align_up(off + 4 * (int64_t)md.K * (C + 1), kAlign);
            md.csc_ent_off = off;
            off = align_up(off + (int64_t)sizeof(SpEntry) * nnz, kAlign);
        }
        for (int side = 0; side < 2; ++side) md.sq_ptr_off[side] = md.sq_ent_off[side] = -1;
        if ((flags & BI_SPARSE_A) && (flags & BI_F16_PAIRS) && sq_shape(md)) {
            for (int side = 0; side < 2; ++side) {
                const int64_t lines = side ? C : R;
                const int64_t runs = (lines + kSqBlock - 1) / kSqBlock * (side ? md.rn[0] : md.cn[0]);
                md.sq_ptr_off[side] = off;
                off = align_up(off + 4 * (int64_t)md.K * (runs + 1), kAlign);
                md.sq_ent_off[side] = off;
                off = align_up(off + (int64_t)sizeof(SqEntry) * md.nnz, kAlign);
            }
        }
        a_raw += (int64_t)m->mb * md.K * R * C;
        a_stored += (int64_t)m->mb * md.K * md.slice;
    }
    m->zvpc = zv;
    // the pair copies are blocked when every modality has the single-read
    // kernel's shape (layout.h)
    {
        bool all = true;
        for (const ModDesc &md : m->mods) all = all && md.lp16_off >= 0 && rc_shape(md);
        for (ModDesc &md : m->mods) {
            md.lp16_order = all ? 1 : 0;
            md.pad0 = 0;
        }
    }
    for (int f = 0; f < m->F; ++f) {
        FacDesc &fd = m->facs[f];
        const int64_t per = (int64_t)fd.U * fd.n * fd.bstates;
        fd.b_agent = m->mb == 1 ? 0 : per;
        fd.b_off = off;
        off = align_up(off + 4 * per * m->mb, kAlign);
        fd.lb_off = off;
        off = align_up(off + 8 * per * m->mb, kAlign);
        fd.lb32_off = -1;
        if (flags & BI_FAST_F32) {
            fd.lb32_off = off;
            off = align_up(off + 4 * per * m->mb, kAlign);
        }
        fd.ld_agent = m->mb == 1 ? 0 : fd.n;
        fd.ld_off = off;
        off = align_up(off + 8 * (int64_t)fd.n * m->mb, kAlign);
    }
    m->bytes = off;
    m->stats.a_raw = a_raw;
    m->stats.a_stored = a_stored;
    m->stats.a_nnz = 0;
    m->stats.device_bytes = off;
    return BI_OK;
}

// Run fn(i) for i in [0, count) on up to 16 host threads.
template <class Fn>
static void parallel_for(int64_t count, Fn fn)
{
    const int64_t nt = std::max<int64_t>(1, std::min<int64_t>({16, (int64_t)std::thread::hardware_concurrency(), count}));
    if (nt <= 1) {
        for (int64_t i = 0; i < count; ++i) fn(i);
        return;
    }
    std::atomic<int64_t> next{0};
    std::vector<std::thread> th;
    for (int64_t t = 0; t < nt; ++t)
        th.emplace_back([&] {
            for (int64_t i; (i = next.fetch_add(1)) < count;) fn(i);
        });
    for (auto &x : th) x.join();
}

static inline double ln_clamped(double x) { return std::log(x > kEps ? x : kEps); }

// IEEE binary16 bits of v rounded to nearest, ties to even (|v| below 65504;
// subnormals kept), and the value they hold in *rounded.  Directly from the
// double, so there is no second rounding through fp32.
static uint16_t half_rne(double v, double *rounded)
{
    const uint16_t sign = std::signbit(v) ? 0x8000 : 0;
    const double a = std::fabs(v);
    uint16_t bits = 0;
    double r = 0.0;
    if (a > 0.0) {
        int e;
        std::frexp(a, &e);                 // a = f 2^e, f in [0.5, 1)
        int E = std::max(e - 1, -14);      // binade (the subnormals share the lowest)
        double k = std::nearbyint(std::ldexp(a, 10 - E));   // 11-bit significand, ties to even
        if (k >= 2048.0) {                 // rounded up into the next binade
            k = 1024.0;
            ++E;
        }
        r = std::ldexp(k, E - 10);
        bits = k < 1024.0 ? (uint16_t)k : (uint16_t)(((E + 15) << 10) | ((int)k - 1024));
    }
    if (rounded) *rounded = sign ? -r : r;
    return sign | bits;
}

int fill(const bi_model *m, const float *const *A, const float *const *B, const float *const *D, char *host,
         int64_t *nnz_out)
{
    std::memcpy(host, m->mods.data(), sizeof(ModDesc) * m->M);
    std::memcpy(host + align_up((int64_t)sizeof(ModDesc) * m->M, kAlign), m->facs.data(), sizeof(FacDesc) * m->F);
    std::atomic<int64_t> nnz{0};
    for (int mm = 0; mm < m->M; ++mm) {
        const ModDesc &md = m->mods[mm];
        const int64_t RC = (int64_t)md.R * md.C;
        const float *src = A[mm];
        parallel_for((int64_t)m->mb * md.K, [&](int64_t s) {
            const float *a = src + s * RC;
            double *dst = reinterpret_cast<double *>(host + md.la_off) + s * md.slice;
            std::vector<double> lv(RC);
            int64_t cnt = 0;
            for (int64_t e = 0; e < RC; ++e) {
                lv[e] = ln_clamped((double)a[e]);
                cnt += a[e] != 0.0f;
            }
            // shift: the slice median (exact in the updates, see layout.h)
            std::vector<double> tmp(lv);
            std::nth_element(tmp.begin(), tmp.begin() + RC / 2, tmp.end());
            const double c = tmp[RC / 2];
            for (int64_t r = 0; r < md.R; ++r) {
                for (int64_t col = 0; col < md.C; ++col) dst[r * md.Cp + col] = lv[r * md.C + col] - c;
                for (int64_t col = md.C; col < md.Cp; ++col) dst[r * md.Cp + col] = 0.0;
            }
            if (md.la32_off >= 0) {
                float *d32 = reinterpret_cast<float *>(host + md.la32_off) + s * md.slice;
                for (int64_t e = 0; e < md.slice; ++e) d32[e] = (float)dst[e];
            }
            if (md.lp16_off >= 0 && md.lp16_order == 1) {   // shared model: s is the outcome
                uint16_t *p = reinterpret_cast<uint16_t *>(host + md.lp16_off) + 2 * s * md.slice;
                for (int64_t r = 0; r < md.R; ++r)
                    for (int64_t col = 0; col < md.C; ++col) {
                        const int64_t i = rc_pair_index(md, r, col);
                        double hi;
                        p[i] = half_rne(dst[r * md.Cp + col], &hi);
                        p[i + 8] = half_rne(dst[r * md.Cp + col] - hi, nullptr);
                    }
            } else if (md.lp16_off >= 0) {
                uint16_t *p = reinterpret_cast<uint16_t *>(host + md.lp16_off) + 2 * s * md.slice;
                for (int64_t e = 0; e < md.slice; e += 4)
                    for (int i = 0; i < 4; ++i) {
                        double hi;
                        p[2 * e + i] = half_rne(dst[e + i], &hi);
                        p[2 * e + 4 + i] = half_rne(dst[e + i] - hi, nullptr);
                    }
            }
            nnz += cnt;
        });
    }
    for (int mm = 0; mm < m->M; ++mm) {
        const ModDesc &md = m->mods[mm];
        if (md.csr_ptr_off < 0) continue;
        const int64_t R = md.R, C = md.C, RC = R * C;
        const float *src = A[mm];
        int32_t *rptr = reinterpret_cast<int32_t *>(host + md.csr_ptr_off);
        int32_t *cptr = reinterpret_cast<int32_t *>(host + md.csc_ptr_off);
        SpEntry *rent = reinterpret_cast<SpEntry *>(host + md.csr_ent_off);
        SpEntry *cent = reinterpret_cast<SpEntry *>(host + md.csc_ent_off);
        const double lne = std::log(kEps);
        // split of a row / column index over its side's factors
        const int rn1 = md.nrow == 2 ? md.rn[1] : 1;
        const int cn1 = md.ncol == 2 ? md.cn[1] : 1;
        auto rentry = [&](double v, int64_t r) { return SpEntry{v, (uint32_t)(r / rn1), (uint32_t)(r % rn1)}; };
        auto centry = [&](double v, int64_t c) { return SpEntry{v, (uint32_t)(c / cn1), (uint32_t)(c % cn1)}; };
        int64_t e = 0;
        for (int o = 0; o < md.K; ++o) {
            const float *a = src + (int64_t)o * RC;
            for (int64_t r = 0; r < R; ++r) {
                rptr[(int64_t)o * (R + 1) + r] = (int32_t)e;
                for (int64_t c = 0; c < C; ++c) {
                    const double x = a[r * C + c];
                    if (x > kEps) rent[e++] = centry(std::log(x) - lne, c);
                }
            }
            rptr[(int64_t)o * (R + 1) + R] = (int32_t)e;
        }
        e = 0;
        for (int o = 0; o < md.K; ++o) {
            const float *a = src + (int64_t)o * RC;
            for (int64_t c = 0; c < C; ++c) {
                cptr[(int64_t)o * (C + 1) + c] = (int32_t)e;
                for (int64_t r = 0; r < R; ++r) {
                    const double x = a[r * C + c];
                    if (x > kEps) cent[e++] = rentry(std::log(x) - lne, r);
                }
            }
            cptr[(int64_t)o * (C + 1) + C] = (int32_t)e;
        }
    }
    for (int mm = 0; mm < m->M; ++mm) {
        const ModDesc &md = m->mods[mm];
        if (md.sq_ptr_off[0] < 0) continue;
        const int64_t R = md.R, C = md.C, RC = R * C;
        const float *src = A[mm];
        const double lne = std::log(kEps);
        // entries per outcome (the same on both sides), then each (side,
        // outcome) fills its own range
        std::vector<int64_t> first(md.K + 1, 0);
        parallel_for(md.K, [&](int64_t o) {
            const float *a = src + o * RC;
            int64_t cnt = 0;
            for (int64_t e = 0; e < RC; ++e) cnt += (double)a[e] > kEps;
            first[o + 1] = cnt;
        });
        for (int o = 0; o < md.K; ++o) first[o + 1] += first[o];
        parallel_for(2 * (int64_t)md.K, [&](int64_t i) {
            const int side = (int)(i / md.K), o = (int)(i % md.K);
            const float *a = src + (int64_t)o * RC;
            const int64_t lines = side ? C : R;
            const int e0n = side ? md.rn[0] : md.cn[0], e1n = side ? md.rn[1] : md.cn[1];
            const int64_t nblk = (lines + kSqBlock - 1) / kSqBlock, runs = nblk * e0n;
            uint32_t *ptr = reinterpret_cast<uint32_t *>(host + md.sq_ptr_off[side]) + (int64_t)o * (runs + 1);
            SqEntry *ent = reinterpret_cast<SqEntry *>(host + md.sq_ent_off[side]);
            int64_t e = first[o];
            for (int64_t blk = 0; blk < nblk; ++blk)
                for (int e0 = 0; e0 < e0n; ++e0) {
                    ptr[blk * e0n + e0] = (uint32_t)e;
                    const int64_t l1 = std::min(lines, (blk + 1) * kSqBlock);
                    for (int64_t l = blk * kSqBlock; l < l1; ++l)
                        for (int e1 = 0; e1 < e1n; ++e1) {
                            const int64_t other = (int64_t)e0 * e1n + e1;
                            const double x = side ? a[other * C + l] : a[l * C + other];
                            if (!(x > kEps)) continue;
                            const double v = std::log(x) - lne;
                            double hi;
                            const uint16_t h = half_rne(v, &hi), r = half_rne(v - hi, nullptr);
                            ent[e++] = SqEntry{(uint32_t)h | (uint32_t)r << 16,
                                               sq_pos((int)(l - blk * kSqBlock), e1, e1n)};
                        }
                }
            ptr[runs] = (uint32_t)e;
        });
    }
    for (int f = 0; f < m->F; ++f) {
        const FacDesc &fd = m->facs[f];
        const int n = fd.n, U = fd.U, bs = fd.bstates;
        for (int a = 0; a < m->mb; ++a) {
            const float *src = B[f] + (int64_t)a * n * bs * U;          // [i][j][u], j over the dependency states
            float *b = reinterpret_cast<float *>(host + fd.b_off) + (int64_t)a * U * n * bs;   // [u][i][j]
            double *lb = reinterpret_cast<double *>(host + fd.lb_off) + (int64_t)a * U * n * bs;
            float *lb32 = fd.lb32_off >= 0 ? reinterpret_cast<float *>(host + fd.lb32_off) + (int64_t)a * U * n * bs
                                           : nullptr;
            for (int u = 0; u < U; ++u)
                for (int i = 0; i < n; ++i)
                    for (int j = 0; j < bs; ++j) {
                        const float v = src[((int64_t)i * bs + j) * U + u];
                        const int64_t e = ((int64_t)u * n + i) * bs + j;
                        b[e] = v;
                        lb[e] = ln_clamped((double)v);
                        if (lb32) lb32[e] = (float)lb[e];
                    }
            const float *dsrc = D[f] + (int64_t)a * n;
            double *ld = reinterpret_cast<double *>(host + fd.ld_off) + (int64_t)a * n;
            for (int s = 0; s < n; ++s) ld[s] = ln_clamped((double)dsrc[s]);
        }
    }
    *nnz_out = nnz.load();
    return BI_OK;
}

}  // namespace bi
