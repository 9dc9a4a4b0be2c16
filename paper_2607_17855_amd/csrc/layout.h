// Device layout of a packed model (internal to libbi; not part of the ABI).
//
// The packed buffer starts with the descriptor tables, followed by the
// parameter arrays, each 256-byte aligned (all offsets below are in bytes):
//
//   ModDesc[M] | FacDesc[F] | LA (dense, fp64) | LA32 (fp32, BI_FAST_F32 only) |
//   fp16 pairs (BI_F16_PAIRS) | sparse A (BI_SPARSE_A only) | B (fp32) | LB (fp64) | LD (fp64)
//
// Sparse A (models shared by every agent).  Every slice X of LA - shifted by
// log(1e-16) instead of its median, so that the structural zeros of A are
// exactly 0 and drop out - is stored twice, by rows (CSR) and by columns
// (CSC).  An entry is {double value; uint32 a; uint32 b} where (a, b) is the
// split of the other side's index over that side's one or two factors (row
// entries carry the column's (c0, c1), column entries the row's (r0, r1)), so
// the kernels never divide.  Inside a line the entries are ordered by (a, b).
//
// Sparse fp16 pairs (BI_SPARSE_A with BI_F16_PAIRS, modalities with two
// factors on each side whose second factors have 16 or 32 states and whose
// first factors an even number up to 32).  The same nonzeros, once per side
// (side 0: lines = rows, entries = columns; side 1 the transpose), as
// SqEntry {uint32 pair; uint32 pos}: pair = the binary16 high part of the
// value (low half) and the binary16 rounding of its residual (high half),
// pos = the byte offset of the entry's high part in the matrix-core kernel's
// LDS block of its 64 lines, sq_pos(line - first line of its block, e1, en1)
// below (a 16-byte pad, then per line en1 high parts and a 16-byte pad; the
// residuals sit in a second plane of the same shape).  The lines of an outcome
// are cut into blocks of 64; inside an outcome the entries run block by
// block, and inside a block by the state e0 of the entry side's first
// factor, then by line, then by e1 (the entry side's second factor).  The
// pointer array [K][nblk * en0 + 1] (uint32, indices into the side's entry
// array) gives the start of every (block, e0) run and, last, the end of the
// outcome.
//
// Precision.  The mean-field fixed-point iterations are ill-conditioned for
// some models: a relative perturbation of 1e-7 in A (fp32 rounding) moves
// some marginals by more than 1e-4 after 16 Jacobi sweeps.  Everything in the
// log domain is therefore stored and combined in double precision; B keeps
// the caller's fp32 values exactly.
//
// Emission slices ("two-sided" view).  For modality m with A-dependency list
// (d_1 < ... < d_k) the slice LA_m[o] of every outcome o is stored as a
// matrix X[r][c] with the first p dependency axes flattened into rows and the
// remaining k-p into columns (row-major, last axis fastest, exactly the order
// of the user's A).  Columns are padded with zeros to a multiple of 4 so that
// every row starts 32-byte aligned.  The stored value is the shifted log
//   X = log(max(A, 1e-16)) - c_{m,o}
// where c_{m,o} is the median of the slice (dense) or log(1e-16) (sparse).
// The shift is exact in the updates: it adds c * prod_{g != f} sum_s q_g(s) to
// every entry of lam_f, a constant over the states of f that the softmax
// removes.
//
// With this view the likelihood messages of one context need two passes over
// the slice, Z = X t and V = s X, where t is the outer product of the column
// factors' marginals and s that of the row factors'; every lam_f of the
// modality is then a small contraction of Z (row factors) or V (column
// factors).
#pragma once

#include <stdint.h>

namespace bi {

constexpr double kEps = 1e-16;
constexpr int kMaxSide = 5;      // factors per side of the two-sided view (dependency lists of up to 10)
constexpr int kStreamSide = 2;   // factors per side the streaming layouts serve (rank <= 4)
constexpr int kAlign = 256;   // byte alignment of every array in the packed buffer

struct ModDesc {
    int64_t la_off;    // byte offset of the dense fp64 slices [agent][K][R][Cp]
    int64_t la_agent;  // elements per agent (0 when the model is shared)
    int32_t K;         // outcomes
    int32_t slice;     // elements per outcome slice = R * Cp
    int32_t rank;      // |dep(m)|
    int32_t R, C, Cp;  // rows, columns, padded columns
    int32_t nrow;      // factors on the row side (0..2)
    int32_t ncol;      // factors on the column side (1..2)
    int32_t rf[kMaxSide], rn[kMaxSide];  // row factors, ascending, and their sizes
    int32_t cf[kMaxSide], cn[kMaxSide];  // column factors, ascending, and sizes
    int32_t zv_off;    // offset of this modality's Z (R values) then V (C values) in a context's block
    int32_t dsum;      // sum of n over dep(m): length of one partial message vector
    int64_t la32_off;  // byte offset of the fp32 copy of the slices (same shape), or -1
    // sparse layout (BI_SPARSE_A): line pointers int32 [K][R+1] / [K][C+1]
    // (entry indices from the modality's first entry) and SpEntry arrays
    int64_t csr_ptr_off, csr_ent_off;   // byte offsets, or -1
    int64_t csc_ptr_off, csc_ent_off;
    int64_t nnz;                        // entries of the modality (each stored twice)
    // fp16 pairs (BI_F16_PAIRS): the slices [K][R][Cp] in groups of 4 columns,
    // 16 bytes each: the 4 high parts, then the 4 residuals; or -1
    int64_t lp16_off;
    // sparse fp16 pairs (BI_SPARSE_A with BI_F16_PAIRS), per side: pointer
    // array and SqEntry array, or -1
    int64_t sq_ptr_off[2], sq_ent_off[2];
    // order of the fp16 pairs: 0 = by rows in groups of 4 columns (above);
    // 1 = in 32 x 32 blocks (rc_shape below)
    int32_t lp16_order;
    int32_t pad0;
};

constexpr int kSqBlock = 64;   // lines per block of the sparse fp16-pair layout
constexpr int kSqPad = 16;     // bytes of padding before a block and after every line

// Bytes per line of one plane of a block (en1 binary16 values and the pad),
// and the byte offset of (line, e1) in the plane.  Offset 0 (the leading pad)
// stands for an empty slot: the kernel's writes for it land in pads that no
// operand read covers.
constexpr int sq_line_bytes(int en1) { return 2 * en1 + kSqPad; }
constexpr int sq_plane_bytes(int en1) { return kSqPad + kSqBlock * sq_line_bytes(en1); }
constexpr uint32_t sq_pos(int line, int e1, int en1) { return (uint32_t)(kSqPad + line * sq_line_bytes(en1) + 2 * e1); }

// Whether a modality has the shape of the sparse fp16-pair layout (and of the
// matrix-core kernels): two factors on each side, second factors of 16 or 32
// states, first factors of an even number of states up to 32.
inline bool sq_shape(const ModDesc &md)
{
    if (md.nrow != 2 || md.ncol != 2 || md.Cp != md.C) return false;
    for (int side = 0; side < 2; ++side) {
        const int n0 = side ? md.cn[0] : md.rn[0], n1 = side ? md.cn[1] : md.rn[1];
        if ((n1 != 16 && n1 != 32) || n0 > 32 || n0 % 2 != 0) return false;
    }
    return true;
}

// Blocked fp16 pairs (lp16_order = 1).  When every modality of a shared
// model has two factors on each side, both second factors of 32 states, the
// first column factor an even number of states up to 32 and the first row
// factor at most 32, the pair copy of slice o is stored as 4096-byte blocks,
// one per (r0, c0) in that order (r0 the first row factor's state, c0 the
// first column factor's).  A block holds the 32 rows r1 of the second row
// factor, 128 bytes each: for u = 0..3 the binary16 high parts of columns
// c1 = 8u .. 8u + 7, then their residuals.  One block is what one wave of
// the single-read kernel contracts per step, so it streams contiguous memory.
inline bool rc_shape(const ModDesc &md)
{
    return md.nrow == 2 && md.ncol == 2 && md.Cp == md.C && md.rn[1] == 32 && md.cn[1] == 32 && md.rn[0] <= 32 &&
           md.cn[0] <= 32 && md.cn[0] % 2 == 0;
}
// uint16 index of the high part of (r, col) in a blocked slice (residual: + 8)
inline int64_t rc_pair_index(const ModDesc &md, int64_t r, int64_t col)
{
    const int64_t r0 = r >> 5, r1 = r & 31, c0 = col >> 5, c1 = col & 31;
    return ((r0 * md.cn[0] + c0) * 32 + r1) * 64 + 16 * (c1 >> 3) + (c1 & 7);
}

constexpr int kMaxBDep = 4;   // B-dependencies per factor
constexpr int kMaxCh = 8;     // factors whose B-dependencies hold a given factor

struct FacDesc {
    int64_t b_off;    // byte offset of fp32 B as [agent][u][i][j] = P(s'=i | s_dep=j, u), j the
                      // dependency states flattened (row-major over bd); trivial: j = s^f
    int64_t lb_off;   // byte offset of fp64 log B, same layout
    int64_t ld_off;   // byte offset of fp64 log D as [agent][n]
    int64_t b_agent;  // elements per agent of B / LB (0 when shared)
    int32_t ld_agent; // elements per agent of LD (0 when shared)
    int32_t n, U;
    int32_t q_off;    // offset of this factor in a context's marginal vector
    int32_t nbd;                  // B-dependencies (factors whose states at t condition s_{t+1}^f)
    int32_t bd[kMaxBDep];         // ascending; trivial: {f}
    int32_t bdn[kMaxBDep];        // their state counts
    int32_t bstates;              // prod of bdn (B_f is [u][n][bstates])
    int32_t nch;                  // children: factors j with f in bd(j)
    int32_t ch[kMaxCh], chpos[kMaxCh];   // the children and the position of f in their lists
    int64_t lb32_off;             // byte offset of log B rounded to fp32 (BI_FAST_F32: the streaming
                                  // families' VMP update with fp32 marginals), or -1
};

struct SpEntry {
    double v;       // log(max(A, 1e-16)) - log(1e-16) > 0
    uint32_t a, b;  // split of the other side's index over that side's factors
};

struct SqEntry {
    uint32_t pair;  // binary16 high part | binary16 residual << 16 of log(max(A, 1e-16)) - log(1e-16)
    uint32_t pos;   // sq_pos(line - block start, e1, en1)
};

inline int64_t align_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

}  // namespace bi
