"""C-ABI checks that need no GPU: exports, argument validation, host packing."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2607_17855_amd import bi, synth
import bruteforce as bfm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = set()
    inc = os.path.join(ROOT, "include")
    for fn in os.listdir(inc):
        if fn.endswith(".h"):
            txt = open(os.path.join(inc, fn)).read()
            txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
            names |= set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(bi_\w+)\s*\(", txt, flags=re.M))
    return names


def test_library_exports_every_declared_function():
    lib = bi.load()
    declared = _declared_functions()
    assert {"bi_pack_model", "bi_vfilter", "bi_vmp", "bi_mmp"} <= declared
    for name in declared:
        assert hasattr(lib, name), f"{name} declared in include/ but not exported"
    assert set(bi.EXPORTS) == declared


class ModDesc(ctypes.Structure):
    _fields_ = [("la_off", ctypes.c_int64), ("la_agent", ctypes.c_int64), ("K", ctypes.c_int32),
                ("slice", ctypes.c_int32), ("rank", ctypes.c_int32), ("R", ctypes.c_int32), ("C", ctypes.c_int32),
                ("Cp", ctypes.c_int32), ("nrow", ctypes.c_int32), ("ncol", ctypes.c_int32),
                ("rf", ctypes.c_int32 * 5), ("rn", ctypes.c_int32 * 5), ("cf", ctypes.c_int32 * 5),
                ("cn", ctypes.c_int32 * 5), ("zv_off", ctypes.c_int32), ("dsum", ctypes.c_int32),
                ("la32_off", ctypes.c_int64), ("csr_ptr_off", ctypes.c_int64), ("csr_ent_off", ctypes.c_int64),
                ("csc_ptr_off", ctypes.c_int64), ("csc_ent_off", ctypes.c_int64), ("nnz", ctypes.c_int64),
                ("lp16_off", ctypes.c_int64), ("sq_ptr_off", ctypes.c_int64 * 2), ("sq_ent_off", ctypes.c_int64 * 2),
                ("lp16_order", ctypes.c_int32), ("pad0", ctypes.c_int32)]


SpEntry = np.dtype([("v", np.float64), ("a", np.uint32), ("b", np.uint32)])
SqEntry = np.dtype([("pair", np.uint32), ("pos", np.uint32)])


class FacDesc(ctypes.Structure):
    _fields_ = [("b_off", ctypes.c_int64), ("lb_off", ctypes.c_int64), ("ld_off", ctypes.c_int64),
                ("b_agent", ctypes.c_int64), ("ld_agent", ctypes.c_int32), ("n", ctypes.c_int32),
                ("U", ctypes.c_int32), ("q_off", ctypes.c_int32), ("nbd", ctypes.c_int32),
                ("bd", ctypes.c_int32 * 4), ("bdn", ctypes.c_int32 * 4), ("bstates", ctypes.c_int32),
                ("nch", ctypes.c_int32), ("ch", ctypes.c_int32 * 8), ("chpos", ctypes.c_int32 * 8),
                ("lb32_off", ctypes.c_int64)]


def _descs(img, M, F):
    mods = (ModDesc * M).from_buffer_copy(img[:ctypes.sizeof(ModDesc) * M].tobytes())
    foff = -(-ctypes.sizeof(ModDesc) * M // 256) * 256
    facs = (FacDesc * F).from_buffer_copy(img[foff:foff + ctypes.sizeof(FacDesc) * F].tobytes())
    return mods, facs


@pytest.mark.parametrize("seed", range(8))
def test_host_pack_round_trip(seed):
    w = synth.random_small(500 + seed, F_max=4, n_max=6, M_max=4, K_max=5, T_max=2, b=3, sparsity=0.3 * (seed % 2))
    m = w.model
    h, img = bi.bi_pack_model_host(m.n, m.U, m.K, m.deps, m.mb, m.A, m.B, m.D)
    try:
        st = bi.bi_get_model_stats(h)
        assert st["device_bytes"] == img.size == bi.bi_plan_model(m.n, m.U, m.K, m.deps, m.mb)
        mods, facs = _descs(img, m.M, m.F)

        def f64(off, count):
            return img[off:off + 8 * count].view(np.float64)

        def f32(off, count):
            return img[off:off + 4 * count].view(np.float32)
        raw = 0
        for mi in range(m.M):
            md = mods[mi]
            d = m.deps[mi]
            assert md.rank == len(d) and md.nrow + md.ncol == len(d)
            assert [md.rf[i] for i in range(md.nrow)] + [md.cf[i] for i in range(md.ncol)] == d
            assert md.R == int(np.prod([m.n[f] for f in d[:md.nrow]]))
            assert md.C == int(np.prod([m.n[f] for f in d[md.nrow:]])) and md.Cp % 4 == 0
            for a in range(m.mb):
                for o in range(m.K[mi]):
                    X = f64(md.la_off + 8 * (a * md.la_agent + o * md.slice), md.slice).reshape(md.R, md.Cp)
                    assert np.all(X[:, md.C:] == 0)
                    ln = bfm.LN(m.A[mi][a, o]).reshape(md.R, md.C)
                    shift = ln - X[:, :md.C]
                    # one constant per slice: the median of the slice's logs
                    assert np.ptp(shift) < 1e-12
                    assert abs(shift.flat[0] - np.sort(ln.ravel())[ln.size // 2]) < 1e-12
            raw += m.mb * m.K[mi] * md.R * md.C
        assert st["a_raw"] == raw
        assert st["a_nnz"] == sum(int((a != 0).sum()) for a in m.A)
        qoff = 0
        for f in range(m.F):
            fd = facs[f]
            n, U = m.n[f], m.U[f]
            assert (fd.n, fd.U, fd.q_off) == (n, U, qoff)
            qoff += n
            for a in range(m.mb):
                Bp = f32(fd.b_off + 4 * a * fd.b_agent, U * n * n).reshape(U, n, n)
                LB = f64(fd.lb_off + 8 * a * fd.b_agent, U * n * n).reshape(U, n, n)
                np.testing.assert_array_equal(Bp, np.transpose(m.B[f][a], (2, 0, 1)))
                np.testing.assert_allclose(LB, bfm.LN(np.transpose(m.B[f][a], (2, 0, 1))), rtol=0, atol=1e-14)
                LD = f64(fd.ld_off + 8 * a * fd.ld_agent, n)
                np.testing.assert_allclose(LD, bfm.LN(m.D[f][a]), rtol=0, atol=1e-14)
    finally:
        bi.bi_free_model(h)


def _desc_err(n, U, K, deps, mb=1, flags=bi.BI_DENSE_A):
    with pytest.raises(bi.BiError) as ei:
        bi.bi_plan_model(n, U, K, deps, mb, flags)
    return ei.value.code


def test_plan_rejects_bad_descriptors():
    assert _desc_err([3], [1], [2], [[1]]) == bi.BI_ERR_SHAPE               # dependency out of range
    assert _desc_err([3, 2], [1, 1], [2], [[1, 0]]) == bi.BI_ERR_SHAPE      # not ascending
    assert _desc_err([3, 2], [1, 1], [2], [[0, 0]]) == bi.BI_ERR_SHAPE      # repeated factor
    assert _desc_err([3], [1], [2], [[]]) == bi.BI_ERR_SHAPE                # empty list
    assert _desc_err([0], [1], [2], [[0]]) == bi.BI_ERR_SHAPE               # no states
    assert _desc_err([3], [0], [2], [[0]]) == bi.BI_ERR_SHAPE               # no actions
    assert _desc_err([3], [1], [0], [[0]]) == bi.BI_ERR_SHAPE               # no outcomes
    assert _desc_err([2] * 11, [1] * 11, [2], [list(range(11))]) == bi.BI_ERR_UNSUPPORTED   # lists of up to 10
    assert bi.bi_plan_model([2] * 10, [1] * 10, [2], [list(range(10))], 1, bi.BI_DENSE_A) > 0
    assert _desc_err([3], [1], [2], [[0]], mb=0) == bi.BI_ERR_INVALID_ARG
    assert _desc_err([3], [1], [2], [[0]], flags=3) == bi.BI_ERR_INVALID_ARG
    assert _desc_err([3], [1], [2], [[0]], flags=64) == bi.BI_ERR_INVALID_ARG
    # fp16 pairs only with BI_FAST_F32 (either layout)
    assert _desc_err([3], [1], [2], [[0]], flags=bi.BI_F16_PAIRS) == bi.BI_ERR_INVALID_ARG
    assert _desc_err([3], [1], [2], [[0]], flags=bi.BI_SPARSE_A | bi.BI_F16_PAIRS) == bi.BI_ERR_INVALID_ARG
    assert bi.bi_plan_model([3], [1], [2], [[0]], 1, bi.BI_SPARSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS) > 0
    lib = bi.load()
    out = ctypes.c_size_t(0)
    assert lib.bi_plan_model(None, ctypes.byref(out)) == bi.BI_ERR_INVALID_ARG
    assert "NULL" in bi.bi_last_error()


def test_plan_sizes_cover_every_array():
    w = synth.two_factor_agents(b=4)
    m = w.model
    nbytes = bi.bi_plan_model(m.n, m.U, m.K, m.deps, m.mb)
    need = sum(8 * a.size for a in m.A) + sum(12 * b.size + 8 * d.size for b, d in zip(m.B, m.D))
    tables = ctypes.sizeof(ModDesc) * m.M + ctypes.sizeof(FacDesc) * m.F
    assert need <= nbytes <= need + tables + 256 * (2 + 2 * m.M + 3 * m.F) + 8 * 4 * 64 * m.M


def test_inference_validates_on_host_before_launch():
    w = synth.random_small(3, b=2, per_agent=True)
    m = w.model
    h, img = bi.bi_pack_model_host(m.n, m.U, m.K, m.deps, m.mb, m.A, m.B, m.D)
    lib = bi.load()
    fake = ctypes.c_void_p(1 << 20)   # never dereferenced: every call below fails validation first
    try:
        for fn in (lib.bi_vfilter, lib.bi_vmp, lib.bi_mmp):
            # no device buffer attached yet
            assert fn(ctypes.c_void_p(h), 2, 2, fake, fake, 3, fake, None, 0, None) == bi.BI_ERR_INVALID_ARG
        assert lib.bi_attach_device_buffer(ctypes.c_void_p(h), ctypes.c_void_p(1 << 20), 16) == \
            bi.BI_ERR_BUFFER_TOO_SMALL
        assert lib.bi_attach_device_buffer(ctypes.c_void_p(h), ctypes.c_void_p((1 << 20) + 4), img.size) == \
            bi.BI_ERR_INVALID_ARG
        assert lib.bi_attach_device_buffer(ctypes.c_void_p(h), fake, img.size) == bi.BI_OK
        for fn in (lib.bi_vfilter, lib.bi_vmp, lib.bi_mmp):
            assert fn(None, 2, 2, fake, fake, 3, fake, None, 0, None) == bi.BI_ERR_INVALID_ARG
            assert fn(ctypes.c_void_p(h), 3, 2, fake, fake, 3, fake, None, 0, None) == bi.BI_ERR_SHAPE   # b != mb
            assert fn(ctypes.c_void_p(h), 2, 2, fake, fake, 0, fake, None, 0, None) == bi.BI_ERR_INVALID_ARG
            assert fn(ctypes.c_void_p(h), 2, 0, fake, fake, 3, fake, None, 0, None) == bi.BI_ERR_INVALID_ARG
            assert fn(ctypes.c_void_p(h), 2, 2, fake, None, 3, fake, None, 0, None) == bi.BI_ERR_INVALID_ARG
            assert fn(ctypes.c_void_p(h), 2, 2, None, fake, 3, fake, None, 0, None) == bi.BI_ERR_INVALID_ARG
            assert fn(ctypes.c_void_p(h), 2, 2, fake, fake, 3, None, None, 0, None) == bi.BI_ERR_INVALID_ARG
        for fn in (lib.bi_vfilter_prior, lib.bi_vmp_prior, lib.bi_mmp_prior):
            # the prior is required; the other checks are those of the call without it
            assert fn(ctypes.c_void_p(h), 2, 2, fake, fake, None, 3, fake, None, 0, None) == bi.BI_ERR_INVALID_ARG
            assert fn(ctypes.c_void_p(h), 3, 2, fake, fake, fake, 3, fake, None, 0, None) == bi.BI_ERR_SHAPE
            assert fn(ctypes.c_void_p(h), 2, 2, fake, fake, fake, 0, fake, None, 0, None) == bi.BI_ERR_INVALID_ARG
        bi_ = lib.bi_infer
        for tau in (0.0, -1.0, 1.5, float("nan")):
            opts = bi.bi_infer_opts(None, tau)
            assert bi_(ctypes.c_void_p(h), 1, 2, 2, fake, fake, 3, ctypes.byref(opts), fake, None, 0, None) == \
                bi.BI_ERR_INVALID_ARG
        opts = bi.bi_infer_opts(None, 0.5)
        assert bi_(ctypes.c_void_p(h), 3, 2, 2, fake, fake, 3, ctypes.byref(opts), fake, None, 0, None) == \
            bi.BI_ERR_INVALID_ARG   # unknown algorithm
        assert bi_(ctypes.c_void_p(h), 1, 3, 2, fake, fake, 3, ctypes.byref(opts), fake, None, 0, None) == \
            bi.BI_ERR_SHAPE
        assert bi_(ctypes.c_void_p(h), 1, 2, 2, fake, fake, 3, None, None, None, 0, None) == bi.BI_ERR_INVALID_ARG
        # soft observations: same argument checks, own workspace size
        si = lib.bi_infer_soft
        assert si(ctypes.c_void_p(h), 1, 3, 2, fake, fake, 3, None, fake, fake, 1 << 30, None) == bi.BI_ERR_SHAPE
        assert si(ctypes.c_void_p(h), 5, 2, 2, fake, fake, 3, None, fake, fake, 1 << 30, None) == \
            bi.BI_ERR_INVALID_ARG
        assert si(ctypes.c_void_p(h), 1, 2, 2, None, fake, 3, None, fake, fake, 1 << 30, None) == \
            bi.BI_ERR_INVALID_ARG
        assert si(ctypes.c_void_p(h), 1, 2, 2, fake, None, 3, None, fake, fake, 1 << 30, None) == \
            bi.BI_ERR_INVALID_ARG
        assert si(ctypes.c_void_p(h), 1, 2, 2, fake, fake, 3, None, fake, fake, 16, None) == \
            bi.BI_ERR_BUFFER_TOO_SMALL
        assert si(ctypes.c_void_p(h), 1, 2, 2, fake, fake, 3, None, fake, None, 1 << 30, None) == \
            bi.BI_ERR_INVALID_ARG
        opts = bi.bi_infer_opts(None, 2.0)
        assert si(ctypes.c_void_p(h), 1, 2, 2, fake, fake, 3, ctypes.byref(opts), fake, fake, 1 << 30, None) == \
            bi.BI_ERR_INVALID_ARG
        mods, _ = _descs(img, m.M, m.F)
        per_ctx = sum(int(mods[i].slice) for i in range(m.M))
        assert bi.bi_workspace_size_soft(h, 2, 3, 0) == -(-2 * 3 * per_ctx * 8 // 256) * 256
        ntot, F = sum(m.n), m.F
        pr = lib.bi_predict
        assert pr(None, 2, fake, ntot, fake, F, fake, None) == bi.BI_ERR_INVALID_ARG
        assert pr(ctypes.c_void_p(h), 3, fake, ntot, fake, F, fake, None) == bi.BI_ERR_SHAPE
        assert pr(ctypes.c_void_p(h), 0, fake, ntot, fake, F, fake, None) == bi.BI_ERR_INVALID_ARG
        assert pr(ctypes.c_void_p(h), 2, None, ntot, fake, F, fake, None) == bi.BI_ERR_INVALID_ARG
        assert pr(ctypes.c_void_p(h), 2, fake, ntot, None, F, fake, None) == bi.BI_ERR_INVALID_ARG
        assert pr(ctypes.c_void_p(h), 2, fake, ntot, fake, F, None, None) == bi.BI_ERR_INVALID_ARG
        assert pr(ctypes.c_void_p(h), 2, fake, ntot - 1, fake, F, fake, None) == bi.BI_ERR_INVALID_ARG
        assert pr(ctypes.c_void_p(h), 2, fake, ntot, fake, F - 1, fake, None) == bi.BI_ERR_INVALID_ARG
        sz = ctypes.c_size_t(0)
        assert lib.bi_workspace_size(ctypes.c_void_p(h), 2, 2, 9, ctypes.byref(sz)) == bi.BI_ERR_INVALID_ARG
    finally:
        bi.bi_free_model(h)
    bi.bi_free_model(0)   # NULL is ignored


@pytest.mark.parametrize("seed", range(6))
def test_host_pack_sparse_planes(seed):
    """BI_SPARSE_A: the CSR and CSC planes hold exactly the entries LN(A) - ln(eps)
    of A > eps, with the other side's index split over its factors."""
    rng = np.random.Generator(np.random.PCG64(900 + seed))
    F = int(rng.integers(1, 5))
    n = [int(x) for x in rng.integers(1, 7, size=F)]
    M = int(rng.integers(1, 4))
    deps = []
    for _ in range(M):
        k = int(rng.integers(1, F + 1))
        deps.append(sorted(int(x) for x in rng.choice(F, size=k, replace=False)))
    K = [int(x) for x in rng.integers(1, 5, size=M)]
    model = synth.make_model(rng, n, [2] * F, K, deps, 1, 1.0, 1.0, sparsity=0.5, uniform_D=False)
    flags = bi.BI_SPARSE_A
    upper = bi.bi_plan_model(model.n, model.U, model.K, model.deps, 1, flags)
    exact = bi.bi_plan_model_exact(model.n, model.U, model.K, model.deps, 1, model.A, flags)
    assert exact <= upper
    h, img = bi.bi_pack_model_host(model.n, model.U, model.K, model.deps, 1, model.A, model.B, model.D, flags)
    try:
        assert img.size == exact == bi.bi_get_model_stats(h)["device_bytes"]
        mods, _ = _descs(img, model.M, model.F)
        lne = np.log(1e-16)
        for mi in range(model.M):
            md = mods[mi]
            A = model.A[mi][0].astype(np.float64).reshape(md.K, md.R, md.C)
            want = np.where(A > 1e-16, np.log(np.maximum(A, 1e-16)) - lne, 0.0)
            assert md.nnz == int((A > 1e-16).sum())
            rn1 = md.rn[1] if md.nrow == 2 else 1
            cn1 = md.cn[1] if md.ncol == 2 else 1
            for side in ("csr", "csc"):
                lines = md.R if side == "csr" else md.C
                ptr_off = getattr(md, side + "_ptr_off")
                ent = img[getattr(md, side + "_ent_off"):].view(SpEntry)[:md.nnz]
                ptr = img[ptr_off:ptr_off + 4 * md.K * (lines + 1)].view(np.int32).reshape(md.K, lines + 1)
                assert ptr[0, 0] == 0 and ptr[-1, -1] == md.nnz
                assert np.all(np.diff(ptr, axis=1) >= 0) and np.all(ptr[1:, 0] == ptr[:-1, -1])
                got = np.zeros_like(want)
                for o in range(md.K):
                    for l in range(lines):
                        le = ent[ptr[o, l]:ptr[o, l + 1]]
                        on1 = cn1 if side == "csr" else rn1
                        # ordered by the other side's index
                        keys = le["a"].astype(np.int64) * on1 + le["b"]
                        assert np.all(np.diff(keys) > 0)
                        for e in le:
                            a, b = int(e["a"]), int(e["b"])
                            assert e["v"] > 0
                            if side == "csr":
                                c = a * cn1 + b
                                assert b < cn1 and got[o, l, c] == 0
                                got[o, l, c] = e["v"]
                            else:
                                r = a * rn1 + b
                                assert b < rn1 and got[o, r, l] == 0
                                got[o, r, l] = e["v"]
                np.testing.assert_allclose(got, want, rtol=0, atol=1e-13)
    finally:
        bi.bi_free_model(h)


SQ_SHAPES = [
    # (n, K): every modality depends on all four factors (rows = the first two)
    ([4, 16, 6, 32], [3]),
    ([2, 32, 2, 16], [2]),
    ([6, 16, 4, 16], [2]),
    ([32, 32, 2, 32], [1]),
]


@pytest.mark.parametrize("case", range(len(SQ_SHAPES)))
def test_host_pack_sparse_pair_layout(case):
    """BI_SPARSE_A with BI_F16_PAIRS: per side, the nonzeros of every outcome
    in blocks of 64 lines, inside a block by (e0, line, e1), each entry the
    binary16 rounding of LN(A) - ln(eps) and of its residual (numpy's float64
    -> float16 conversion is the reference) with its byte offset in the
    kernel's LDS block (16 + line (2 en1 + 16) + 2 e1; offset 0, the pad that
    empty slots write to, is never an entry's),
    and the run pointers delimiting every (block, e0).  Rebuilt into dense
    slices they give back exactly the pair rounding of the nonzeros."""
    n, K = SQ_SHAPES[case]
    rng = np.random.Generator(np.random.PCG64(1300 + case))
    model = synth.make_model(rng, n, [1] * 4, K, [[0, 1, 2, 3]] * len(K), 1, 1.0, 1.0,
                             sparsity=0.3 + 0.2 * case, uniform_D=False)
    flags = bi.BI_SPARSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS
    assert bi.bi_plan_model_exact(model.n, model.U, model.K, model.deps, 1, model.A, flags) <= \
        bi.bi_plan_model(model.n, model.U, model.K, model.deps, 1, flags)
    h, img = bi.bi_pack_model_host(model.n, model.U, model.K, model.deps, 1, model.A, model.B, model.D, flags)
    try:
        mods, _ = _descs(img, model.M, model.F)
        lne = np.log(1e-16)
        for mi in range(model.M):
            md = mods[mi]
            assert md.lp16_off == -1          # no dense pair copy with the sparse layout
            A = model.A[mi][0].astype(np.float64).reshape(md.K, md.R, md.C)
            nz = A > 1e-16
            v = np.where(nz, np.log(np.maximum(A, 1e-16)) - lne, 0.0)
            hi = v.astype(np.float16)
            lo = (v - hi.astype(np.float64)).astype(np.float16)
            for side in range(2):
                lines = md.R if side == 0 else md.C
                e0n = md.cn[0] if side == 0 else md.rn[0]
                e1n = md.cn[1] if side == 0 else md.rn[1]
                nblk = -(-lines // 64)
                runs = nblk * e0n
                assert md.sq_ptr_off[side] % 256 == 0 and md.sq_ent_off[side] % 256 == 0
                ptr = img[md.sq_ptr_off[side]:md.sq_ptr_off[side] + 4 * md.K * (runs + 1)]
                ptr = ptr.view(np.uint32).reshape(md.K, runs + 1).astype(np.int64)
                ent = img[md.sq_ent_off[side]:md.sq_ent_off[side] + 8 * md.nnz].view(SqEntry)
                assert ptr[0, 0] == 0 and ptr[-1, -1] == md.nnz
                assert np.all(np.diff(ptr, axis=1) >= 0) and np.all(ptr[1:, 0] == ptr[:-1, -1])
                # the slices seen from this side: [o][line][e0][e1]
                vh = hi if side == 0 else hi.transpose(0, 2, 1)
                vl = lo if side == 0 else lo.transpose(0, 2, 1)
                vz = nz if side == 0 else nz.transpose(0, 2, 1)
                got_h = np.zeros((md.K, lines, e0n * e1n), dtype=np.uint16)
                got_l = np.zeros_like(got_h)
                seen = np.zeros((md.K, lines, e0n * e1n), dtype=bool)
                for o in range(md.K):
                    for blk in range(nblk):
                        for e0 in range(e0n):
                            run = ent[ptr[o, blk * e0n + e0]:ptr[o, blk * e0n + e0 + 1]]
                            # pos = 16 + line (2 e1n + 16) + 2 e1: the byte offset in the kernel's LDS block
                            off = run["pos"].astype(np.int64) - 16
                            line, rem = off // (2 * e1n + 16), off % (2 * e1n + 16)
                            e1 = rem // 2
                            assert np.all(off >= 0) and np.all(rem % 2 == 0) and np.all(rem < 2 * e1n)
                            assert np.all(line < 64) and np.all(blk * 64 + line < lines)
                            key = line * e1n + e1
                            assert np.all(np.diff(key) > 0)       # ordered by (line, e1), no repeats
                            L, E = blk * 64 + line, e0 * e1n + e1
                            assert not seen[o, L, E].any()
                            seen[o, L, E] = True
                            got_h[o, L, E] = run["pair"] & 0xFFFF
                            got_l[o, L, E] = run["pair"] >> 16
                np.testing.assert_array_equal(seen, vz)
                np.testing.assert_array_equal(got_h[seen], vh[vz].view(np.uint16))
                np.testing.assert_array_equal(got_l[seen], vl[vz].view(np.uint16))
    finally:
        bi.bi_free_model(h)


def test_sparse_pair_layout_only_for_its_shapes():
    """Modalities outside the shapes of the matrix-core tiles get no sparse
    pair arrays (their model keeps the sparse fp64 kernels); per-agent models
    cannot be packed sparse at all."""
    rng = np.random.Generator(np.random.PCG64(1310))
    model = synth.make_model(rng, [4, 16, 6, 12], [1] * 4, [2, 3], [[0, 1, 2, 3], [0, 1]], 1, 1.0, 1.0,
                             sparsity=0.5, uniform_D=False)
    flags = bi.BI_SPARSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS
    h, img = bi.bi_pack_model_host(model.n, model.U, model.K, model.deps, 1, model.A, model.B, model.D, flags)
    try:
        mods, _ = _descs(img, model.M, model.F)
        assert all(mods[i].sq_ptr_off[s] == -1 and mods[i].sq_ent_off[s] == -1 for i in range(2) for s in range(2))
        assert all(mods[i].csr_ptr_off >= 0 for i in range(2))
        assert bi.bi_query_path(h, 8, 4, bi.BI_ALGO_VMP) in (bi.BI_PATH_AGENT, bi.BI_PATH_STREAM, bi.BI_PATH_SPARSE)
    finally:
        bi.bi_free_model(h)


def test_check_flag_adds_status_words_to_every_workspace():
    w = synth.random_small(7, b=2, per_agent=True)
    m = w.model
    h0, _ = bi.bi_pack_model_host(m.n, m.U, m.K, m.deps, m.mb, m.A, m.B, m.D)
    h1, _ = bi.bi_pack_model_host(m.n, m.U, m.K, m.deps, m.mb, m.A, m.B, m.D, flags=bi.BI_DENSE_A | bi.BI_CHECK)
    try:
        for algo in range(3):
            assert bi.bi_workspace_size(h0, 2, 3, algo) == 0            # agent-resident: none
            assert bi.bi_workspace_size(h1, 2, 3, algo) == 256          # the check's status words
            assert bi.bi_workspace_size_soft(h1, 2, 3, algo) == bi.bi_workspace_size_soft(h0, 2, 3, algo) + 256
    finally:
        bi.bi_free_model(h0)
        bi.bi_free_model(h1)
    # a shared model on the streaming kernels: its workspace plus the status words
    ms = synth.make_model(np.random.Generator(np.random.PCG64(8)), [32, 32, 16], [1, 1, 1], [3], [[0, 1, 2]], 1)
    fl = bi.BI_DENSE_A | bi.BI_FAST_F32
    h0, _ = bi.bi_pack_model_host(ms.n, ms.U, ms.K, ms.deps, 1, ms.A, ms.B, ms.D, flags=fl)
    h1, _ = bi.bi_pack_model_host(ms.n, ms.U, ms.K, ms.deps, 1, ms.A, ms.B, ms.D, flags=fl | bi.BI_CHECK)
    old = os.environ.get("BI_FORCE_PATH")
    os.environ["BI_FORCE_PATH"] = "stream"   # the selector would run this small batch agent-resident
    try:
        n0 = bi.bi_workspace_size(h0, 4, 3, 1)
        assert n0 > 0
        assert bi.bi_workspace_size(h1, 4, 3, 1) == -(-n0 // 256) * 256 + 256
    finally:
        if old is None:
            os.environ.pop("BI_FORCE_PATH", None)
        else:
            os.environ["BI_FORCE_PATH"] = old
        bi.bi_free_model(h0)
        bi.bi_free_model(h1)


def test_sparse_layout_needs_a_shared_model():
    with pytest.raises(bi.BiError) as ei:
        bi.bi_plan_model([3], [1], [2], [[0]], 2, bi.BI_SPARSE_A)
    assert ei.value.code == bi.BI_ERR_UNSUPPORTED
    lib = bi.load()
    out = ctypes.c_size_t(0)
    d = bi._Desc([3], [1], [2], [[0]], 1, bi.BI_SPARSE_A)
    assert lib.bi_plan_model_exact(ctypes.byref(d.c), None, ctypes.byref(out)) == bi.BI_ERR_INVALID_ARG


def test_query_path_follows_eligibility_and_forcing():
    lib_models = []
    try:
        w = synth.random_small(9, b=3, per_agent=True)
        m = w.model
        h, _ = bi.bi_pack_model_host(m.n, m.U, m.K, m.deps, m.mb, m.A, m.B, m.D, flags=bi.BI_DENSE_A | bi.BI_FAST_F32)
        lib_models.append(h)
        for algo in range(3):   # per-agent models: agent-resident only, whatever is forced
            assert bi.bi_query_path(h, 3, 4, algo) == bi.BI_PATH_AGENT
        ms = synth.make_model(np.random.Generator(np.random.PCG64(3)), [9, 7, 5], [2, 1, 3], [3, 2],
                              [[0, 1, 2], [1]], 1)
        hs, _ = bi.bi_pack_model_host(ms.n, ms.U, ms.K, ms.deps, 1, ms.A, ms.B, ms.D, flags=bi.BI_SPARSE_A)
        lib_models.append(hs)
        assert bi.bi_query_path(hs, 8, 4, bi.BI_ALGO_FPI) == bi.BI_PATH_AGENT
        old = os.environ.get("BI_FORCE_PATH")
        try:
            os.environ["BI_FORCE_PATH"] = "sparse"
            assert bi.bi_query_path(hs, 8, 4, bi.BI_ALGO_VMP) == bi.BI_PATH_SPARSE
            assert bi.bi_query_path(hs, 8, 4, bi.BI_ALGO_FPI) == bi.BI_PATH_AGENT   # not eligible
            os.environ["BI_FORCE_PATH"] = "stream"                                 # not packed for it
            assert bi.bi_query_path(hs, 8, 4, bi.BI_ALGO_VMP) in (bi.BI_PATH_AGENT, bi.BI_PATH_SPARSE)
            os.environ["BI_FORCE_PATH"] = "agent"
            assert bi.bi_query_path(hs, 8, 4, bi.BI_ALGO_MMP) == bi.BI_PATH_AGENT
        finally:
            if old is None:
                os.environ.pop("BI_FORCE_PATH", None)
            else:
                os.environ["BI_FORCE_PATH"] = old
        out = ctypes.c_int32(0)
        assert bi.load().bi_query_path(ctypes.c_void_p(hs), 0, 4, 1, ctypes.byref(out)) == bi.BI_ERR_INVALID_ARG
        assert bi.load().bi_query_path(ctypes.c_void_p(hs), 8, 4, 7, ctypes.byref(out)) == bi.BI_ERR_INVALID_ARG
    finally:
        for h in lib_models:
            bi.bi_free_model(h)


@pytest.mark.parametrize("regime", ["uniform", "skewed"])
def test_selector_table_matches_the_fitted_trees(regime):
    """The C selector (through bi_query_path on host-packed sweep models)
    makes the choice of the decision trees the fit produced, for every
    candidate set and algorithm, on a sample of the sweep models."""
    from paper_2607_17855_amd.selector import fit
    data = fit.load()
    flags = {1: bi.BI_DENSE_A | bi.BI_FAST_F32, 2: bi.BI_SPARSE_A, 3: bi.BI_SPARSE_A | bi.BI_FAST_F32,
             5: bi.BI_DENSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS,
             7: bi.BI_SPARSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS}
    family = {"agent": "agent", "stream": "stream", "sparse": "sparse", "stream16": "stream", "sparse16": "sparse"}
    trees = {}
    for cset, cands in fit.SETS.items():
        for algo in ("vmp", "mmp"):
            X, y, wt, _ = fit.dataset(data, algo, cands)
            trees[(cset, algo)] = (fit.fit_tree(X, y, wt), cands)
    rng = np.random.Generator(np.random.PCG64(7))
    cases = sorted(set(int(c) for c in rng.choice(770, size=40, replace=False)))
    checked = 0
    for case in cases:
        sp = synth.sweep_spec(case, regime)
        model = synth.make_model(np.random.Generator(np.random.PCG64(case)), sp.n, sp.U, sp.K, sp.deps, 1)
        for cset, fl in flags.items():
            h, _ = bi.bi_pack_model_host(model.n, model.U, model.K, model.deps, 1, model.A, model.B, model.D,
                                         flags=fl)
            try:
                for algo in ("vmp", "mmp"):
                    tree, cands = trees[(cset, algo)]
                    want = family[cands[int(tree.predict(np.array([fit.features(sp, 256)]))[0])]]
                    got = bi.PATH_NAMES[bi.bi_query_path(h, 256, sp.T, bi.ALGO_IDS[algo])]
                    # a family the model is not eligible for falls back; the sweep models are all eligible
                    assert got == want, (regime, case, cset, algo, got, want)
                    checked += 1
            finally:
                bi.bi_free_model(h)
    assert checked == len(cases) * 2 * len(flags)


def _bdep_model(seed, lists, mb=2, n=(3, 4, 2)):
    rng = np.random.Generator(np.random.PCG64(seed))
    return synth.make_model(rng, list(n), [2, 1, 3], [3, 2], [[0, 1], [2]], mb, bdeps=lists)


def test_bdeps_host_pack_layout():
    lists = [[0, 2], [1], [0, 1, 2]]
    m = _bdep_model(41, lists)
    h, img = bi.bi_pack_model_host(m.n, m.U, m.K, m.deps, m.mb, m.A, m.B, m.D, bdeps=m.bdeps)
    try:
        _, facs = _descs(img, m.M, m.F)
        for f in range(m.F):
            fd = facs[f]
            assert fd.nbd == len(lists[f]) and [fd.bd[i] for i in range(fd.nbd)] == lists[f]
            assert [fd.bdn[i] for i in range(fd.nbd)] == [m.n[g] for g in lists[f]]
            assert fd.bstates == int(np.prod([m.n[g] for g in lists[f]]))
            kids = sorted((j, lists[j].index(f)) for j in range(m.F) if f in lists[j])
            assert sorted((fd.ch[i], fd.chpos[i]) for i in range(fd.nch)) == kids
            n, U, bs = m.n[f], m.U[f], fd.bstates
            for a in range(m.mb):
                b = img[fd.b_off + 4 * a * fd.b_agent:fd.b_off + 4 * (a + 1) * fd.b_agent].view(np.float32)
                want = np.transpose(m.B[f][a].reshape(n, bs, U), (2, 0, 1)).ravel()   # [u][i][flat]
                assert np.array_equal(b, want)
                lb = img[fd.lb_off + 8 * a * fd.b_agent:fd.lb_off + 8 * (a + 1) * fd.b_agent].view(np.float64)
                assert np.allclose(lb, np.log(np.maximum(want.astype(np.float64), 1e-16)), rtol=0, atol=1e-12)
    finally:
        bi.bi_free_model(h)
    # the explicit trivial lists pack exactly like no lists
    t = _bdep_model(42, None)
    h0, i0 = bi.bi_pack_model_host(t.n, t.U, t.K, t.deps, t.mb, t.A, t.B, t.D)
    h1, i1 = bi.bi_pack_model_host(t.n, t.U, t.K, t.deps, t.mb, t.A, t.B, t.D, bdeps=[[0], [1], [2]])
    try:
        assert np.array_equal(i0, i1)
    finally:
        bi.bi_free_model(h0)
        bi.bi_free_model(h1)


def test_bdeps_validation_and_dispatch():
    m = _bdep_model(43, [[0, 2], [1], [0, 1, 2]], mb=1)
    def err(lists):
        try:
            h, _ = bi.bi_pack_model_host(m.n, m.U, m.K, m.deps, 1, m.A, m.B, m.D, bdeps=lists)
        except bi.BiError as e:
            return e.code
        bi.bi_free_model(h)
        return bi.BI_OK
    assert err([[0], [], [2]]) == bi.BI_ERR_SHAPE                # empty list
    assert err([[0], [1], [2, 0]]) == bi.BI_ERR_SHAPE            # not ascending
    assert err([[0], [1], [3]]) == bi.BI_ERR_SHAPE               # out of range
    d = bi._Desc(m.n, m.U, m.K, m.deps, 1, bi.BI_DENSE_A, [[0], [1], [2]])
    d.c.bdep = None                                               # one of the two arrays missing
    out = ctypes.c_size_t(0)
    assert bi.load().bi_plan_model(ctypes.byref(d.c), ctypes.byref(out)) == bi.BI_ERR_INVALID_ARG
    # five dependencies, and a factor on nine lists: beyond what the library handles
    big = synth.make_model(np.random.Generator(np.random.PCG64(1)), [2] * 9, [1] * 9, [2], [[0]], 1)
    bd = bi._Desc(big.n, big.U, big.K, big.deps, 1, bi.BI_DENSE_A, [[0, 1, 2, 3, 4]] + [[f] for f in range(1, 9)])
    assert bi.load().bi_plan_model(ctypes.byref(bd.c), ctypes.byref(out)) == bi.BI_ERR_UNSUPPORTED
    bd = bi._Desc(big.n, big.U, big.K, big.deps, 1, bi.BI_DENSE_A, [[0, f] if f else [0] for f in range(9)])
    assert bi.load().bi_plan_model(ctypes.byref(bd.c), ctypes.byref(out)) == bi.BI_ERR_UNSUPPORTED
    # non-trivial lists: the streaming families take VMP / MMP on a shared
    # model as packed (their update has the general transition messages);
    # FPI stays agent-resident
    for fl, fam in ((bi.BI_DENSE_A | bi.BI_FAST_F32, bi.BI_PATH_STREAM), (bi.BI_SPARSE_A, bi.BI_PATH_SPARSE)):
        h, _ = bi.bi_pack_model_host(m.n, m.U, m.K, m.deps, 1, m.A, m.B, m.D, flags=fl, bdeps=m.bdeps)
        old = os.environ.get("BI_FORCE_PATH")
        try:
            os.environ["BI_FORCE_PATH"] = "stream" if fam == bi.BI_PATH_STREAM else "sparse"
            for algo in range(3):
                want = bi.BI_PATH_AGENT if algo == bi.BI_ALGO_FPI else fam
                assert bi.bi_query_path(h, 8, 4, algo) == want
                why = bi.bi_explain_path(h, 8, 4, algo)
                if algo == bi.BI_ALGO_FPI:
                    assert why.startswith("agent (the only eligible family)"), why
                else:
                    assert "forced by BI_FORCE_PATH" in why, why
        finally:
            if old is None:
                os.environ.pop("BI_FORCE_PATH", None)
            else:
                os.environ["BI_FORCE_PATH"] = old
            bi.bi_free_model(h)


@pytest.mark.parametrize("seed", range(4))
def test_f16_pair_plane(seed):
    """The fp16-pair copy of every slice: groups of 4 columns, 4 high parts then
    4 residuals, where high = the fp64 log-likelihood rounded to binary16 (ties
    to even) and residual = (value - high) rounded the same way; numpy's
    float64 -> float16 conversion rounds directly from the double and is the
    reference.  Per-agent models get no pair copy."""
    w = synth.random_small(520 + seed, F_max=4, n_max=7, M_max=3, K_max=4, T_max=2, b=2,
                           sparsity=0.5 * (seed % 2), per_agent=False)
    m = w.model
    fl = bi.BI_DENSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS
    h, img = bi.bi_pack_model_host(m.n, m.U, m.K, m.deps, 1, m.A, m.B, m.D, flags=fl)
    try:
        assert img.size == bi.bi_plan_model(m.n, m.U, m.K, m.deps, 1, fl)
        mods, _ = _descs(img, m.M, m.F)
        for mi in range(m.M):
            md = mods[mi]
            assert md.lp16_off >= 0 and md.lp16_off % 256 == 0
            X = img[md.la_off:md.la_off + 8 * md.K * md.slice].view(np.float64).reshape(md.K, md.R, md.Cp // 4, 4)
            P = img[md.lp16_off:md.lp16_off + 4 * md.K * md.slice].view(np.float16).reshape(md.K, md.R, md.Cp // 4, 2, 4)
            hi = X.astype(np.float16)
            np.testing.assert_array_equal(P[..., 0, :].view(np.uint16), hi.view(np.uint16))
            lo = (X - hi.astype(np.float64)).astype(np.float16)
            np.testing.assert_array_equal(P[..., 1, :].view(np.uint16), lo.view(np.uint16))
            # 22 significant bits: |X - hi - lo| <= 2^-22 |X| (plus the binary16 subnormal spacing)
            err = np.abs(X - hi.astype(np.float64) - lo.astype(np.float64))
            assert np.all(err <= 2.0 ** -22 * np.abs(X) + 2.0 ** -25)
    finally:
        bi.bi_free_model(h)
    # per-agent: no pair copy
    wa = synth.random_small(530 + seed, F_max=3, n_max=5, M_max=2, K_max=3, T_max=2, b=2, per_agent=True)
    ma = wa.model
    h, img = bi.bi_pack_model_host(ma.n, ma.U, ma.K, ma.deps, ma.mb, ma.A, ma.B, ma.D, flags=fl)
    try:
        mods, _ = _descs(img, ma.M, ma.F)
        assert all(mods[i].lp16_off == -1 for i in range(ma.M))
    finally:
        bi.bi_free_model(h)


def test_f16_pair_blocks():
    """Models whose modalities all have two factors per side with both second
    factors of 32 states get the blocked pair copy: per outcome, 4096-byte
    blocks in (r0, c0) order, each with the 32 rows r1 of 128 bytes, and in a
    row, for every 8 columns c1, their 8 high parts, then their 8 residuals
    (the same values as the row-ordered copy).  A model with one modality of
    another shape keeps the row order for all."""
    rng = np.random.Generator(np.random.PCG64(11))
    n, U = [4, 32, 2, 32], [1, 1, 1, 1]
    K = [2, 3]
    deps = [[0, 1, 2, 3], [0, 1, 2, 3]]
    A = []
    for k in K:
        a = rng.dirichlet(np.ones(k), size=int(np.prod(n))).T.reshape([1, k] + n)
        A.append(a.astype(np.float32))
    B = [np.full((1, x, x, 1), 1.0 / x, np.float32) for x in n]
    D = [np.full((1, x), 1.0 / x, np.float32) for x in n]
    fl = bi.BI_DENSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS
    h, img = bi.bi_pack_model_host(n, U, K, deps, 1, A, B, D, flags=fl)
    try:
        mods, _ = _descs(img, 2, 4)
        for mi in range(2):
            md = mods[mi]
            assert md.lp16_order == 1 and (md.R, md.C, md.Cp) == (128, 64, 64)
            X = img[md.la_off:md.la_off + 8 * md.K * md.slice].view(np.float64).reshape(md.K, 4, 32, 2, 32)
            hi = X.astype(np.float16)
            lo = (X - hi.astype(np.float64)).astype(np.float16)
            # [o][r0][c0][r1][unit g][high / residual][8 columns]
            P = img[md.lp16_off:md.lp16_off + 4 * md.K * md.slice].view(np.uint16).reshape(md.K, 4, 2, 32, 4, 2, 8)
            want_hi = hi.transpose(0, 1, 3, 2, 4).reshape(md.K, 4, 2, 32, 4, 8)
            want_lo = lo.transpose(0, 1, 3, 2, 4).reshape(md.K, 4, 2, 32, 4, 8)
            np.testing.assert_array_equal(P[..., 0, :], want_hi.view(np.uint16))
            np.testing.assert_array_equal(P[..., 1, :], want_lo.view(np.uint16))
    finally:
        bi.bi_free_model(h)
    # one modality with a 16-state second factor: row order everywhere
    n2 = [4, 32, 2, 16]
    A2 = [rng.dirichlet(np.ones(2), size=int(np.prod(n2))).T.reshape([1, 2] + n2).astype(np.float32),
          rng.dirichlet(np.ones(2), size=4 * 32).T.reshape([1, 2, 4, 32]).astype(np.float32)]
    B2 = [np.full((1, x, x, 1), 1.0 / x, np.float32) for x in n2]
    D2 = [np.full((1, x), 1.0 / x, np.float32) for x in n2]
    h, img = bi.bi_pack_model_host(n2, U, [2, 2], [[0, 1, 2, 3], [0, 1]], 1, A2, B2, D2, flags=fl)
    try:
        mods, _ = _descs(img, 2, 4)
        assert mods[0].lp16_order == 0 and mods[1].lp16_order == 0
    finally:
        bi.bi_free_model(h)


def test_f16_pairs_wide_range():
    """A slice whose probabilities span 1e-16 .. 1: high parts over many
    binades and residuals down in the binary16 subnormals, each matching
    numpy's rounding from the double."""
    rng = np.random.Generator(np.random.PCG64(5))
    n, K = [64], [2]
    p = 10.0 ** rng.uniform(-16, 0, size=64)
    A = np.stack([p, 1.0 - p])[None].astype(np.float32)   # [agent][o][s]
    B = [np.full((1, 64, 64, 1), 1.0 / 64, np.float32)]
    D = [np.full((1, 64), 1.0 / 64, np.float32)]
    fl = bi.BI_DENSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS
    h, img = bi.bi_pack_model_host(n, [1], K, [[0]], 1, [A], B, D, flags=fl)
    try:
        mods, _ = _descs(img, 1, 1)
        md = mods[0]
        X = img[md.la_off:md.la_off + 8 * md.K * md.slice].view(np.float64).reshape(md.K, md.Cp // 4, 4)
        P = img[md.lp16_off:md.lp16_off + 4 * md.K * md.slice].view(np.uint16).reshape(md.K, md.Cp // 4, 2, 4)
        hi = X.astype(np.float16)
        lo = (X - hi.astype(np.float64)).astype(np.float16)
        np.testing.assert_array_equal(P[:, :, 0, :], hi.view(np.uint16))
        np.testing.assert_array_equal(P[:, :, 1, :], lo.view(np.uint16))
        expo = lambda u: (u >> 10) & 0x1F
        assert len(set(expo(P[:, :, 0, :]).ravel().tolist())) >= 6, "high parts over several binades"
        sub = (expo(P[:, :, 1, :]) == 0) & ((P[:, :, 1, :] & 0x3FF) != 0)
        assert sub.any(), "some residuals are binary16 subnormals"
    finally:
        bi.bi_free_model(h)


def test_python_binding_checks_tensors_before_the_library():
    """PackedModel passes raw device pointers to the C-ABI, so the binding
    rejects tensors of the wrong dtype, shape, layout or device first (CPU:
    the check runs before any launch; the model's device is given as cpu)."""
    import torch
    w = synth.random_small(5, b=3, T_max=4)
    while w.T < 2:
        w = synth.random_small(int(w.obs.sum()) + 7, b=3, T_max=4)
    m, cpu = w.model, torch.device("cpu")
    obs, act = torch.from_numpy(w.obs), torch.from_numpy(w.act)
    b, T = w.b, w.T
    q = torch.empty((b, T, m.n_total), dtype=torch.float32)
    prior = torch.full((b, m.n_total), 0.5, dtype=torch.float32)
    bi.check_infer_args(m, cpu, obs, act, q, prior)          # the good call passes
    bi.check_infer_args(m, cpu, obs[:, :1].contiguous(), None)  # T = 1 needs no actions
    bad = [
        (obs.long(), act, q, prior, "obs must be torch.int32"),          # torch's default integer type
        (obs, act.long(), q, prior, "act must be torch.int32"),
        (obs.float(), act, q, prior, "obs must be torch.int32"),
        (obs[:, :, :-1] if m.M > 1 else obs[:, :, :0], act, q, prior, "obs must have shape"),
        (obs.transpose(0, 1).contiguous().transpose(0, 1), act, q, prior, "obs must be contiguous"),
        (obs, act[:, :-1], q, prior, "act must have shape"),
        (obs, None, q, prior, "act is missing"),
        (obs, act, q.double(), prior, "q must be torch.float32"),
        (obs, act, q[:, :, :-1], prior, "q must have shape"),
        (obs, act, q, prior[:-1], "prior must have shape"),
        (obs, act, q, prior.half(), "prior must be torch.float32"),
    ]
    for o, a, qq, p, msg in bad:
        with pytest.raises(ValueError, match=msg.replace("(", r"\(")):
            bi.check_infer_args(m, cpu, o, a, qq, p)
    # host tensors against a model on the GPU
    with pytest.raises(ValueError, match="is on cpu"):
        bi.check_infer_args(m, torch.device("cuda", 0), obs, act, q, prior)
    # soft observations: float32 [b][T][sum K]
    so = torch.from_numpy(synth.one_hot_obs(w.obs, m.K))
    bi.check_infer_args(m, cpu, so, act, q, prior, soft=True)
    with pytest.raises(ValueError, match="obs_soft must be torch.float32"):
        bi.check_infer_args(m, cpu, so.double(), act, q, prior, soft=True)
    with pytest.raises(ValueError, match="obs_soft must have shape"):
        bi.check_infer_args(m, cpu, so[:, :, 1:].contiguous(), act, q, prior, soft=True)
    # a per-agent model with another agent count
    wp = synth.random_small(6, b=3, T_max=1, per_agent=True)
    assert wp.model.mb == 3
    with pytest.raises(ValueError, match="holds 3 agents"):
        bi.check_infer_args(wp.model, cpu, torch.from_numpy(wp.obs[:2].copy()), None)


def test_static_scratch_entry_refuses_before_any_launch():
    """bi_infer_static checks its limits on the host: a model packed with
    BI_CHECK, and a call whose workspace exceeds the static scratch, are
    refused with BI_ERR_UNSUPPORTED before any HIP call (the attached device
    address here is never touched)."""
    rng = np.random.Generator(np.random.PCG64(3))
    m = synth.make_model(rng, [4, 32, 2, 32], [2, 1, 2, 1], [3], [[0, 1, 2, 3]], 1)
    lib = bi.load()
    fake = ctypes.c_void_p(1 << 40)
    for flags, b, T, why in [(bi.BI_DENSE_A | bi.BI_FAST_F32 | bi.BI_CHECK, 8, 4, "BI_CHECK"),
                             (bi.BI_DENSE_A | bi.BI_FAST_F32, 4096, 64, "above the static")]:
        h, img = bi.bi_pack_model_host(m.n, m.U, m.K, m.deps, 1, m.A, m.B, m.D, flags)
        try:
            assert lib.bi_attach_device_buffer(ctypes.c_void_p(h), fake, img.nbytes) == bi.BI_OK
            old = os.environ.get("BI_FORCE_PATH")
            os.environ["BI_FORCE_PATH"] = "stream"
            try:
                if "above" in why:
                    assert bi.bi_workspace_size(h, b, T, bi.BI_ALGO_VMP) > bi.BI_STATIC_SCRATCH_BYTES
                rc = lib.bi_infer_static(ctypes.c_void_p(h), bi.BI_ALGO_VMP, b, T, fake, fake, 2, None, fake, None)
            finally:
                if old is None:
                    os.environ.pop("BI_FORCE_PATH", None)
                else:
                    os.environ["BI_FORCE_PATH"] = old
            assert rc == bi.BI_ERR_UNSUPPORTED, rc
            assert why in bi.bi_last_error()
        finally:
            bi.bi_free_model(h)


@pytest.mark.parametrize("flags", [bi.BI_DENSE_A, bi.BI_SPARSE_A | bi.BI_FAST_F32 | bi.BI_F16_PAIRS])
def test_host_pack_long_dependency_lists(flags):
    """Lists of 5 to 10 factors: up to 5 factors per side of the two-sided
    view, the slices stored like any other; the streaming layouts (fp32 copy,
    fp16 pairs, sparse planes) exist only for modalities with at most 2
    factors per side, and the model is refused by the streaming families."""
    rng = np.random.Generator(np.random.PCG64(77))
    n = [2, 3, 2, 2, 2, 2, 2, 2, 3, 2]
    deps = [list(range(10)), [1, 4, 7], [0, 2, 5, 8, 9], [3, 6]]
    K = [3, 4, 2, 3]
    model = synth.make_model(rng, n, [1] * 10, K, deps, 1, 1.0, 1.0)
    m = model
    h, img = bi.bi_pack_model_host(m.n, m.U, m.K, m.deps, m.mb, m.A, m.B, m.D, flags=flags)
    try:
        mods, _ = _descs(img, m.M, m.F)
        for mi, d in enumerate(m.deps):
            md = mods[mi]
            assert md.rank == len(d) and md.nrow + md.ncol == len(d) and max(md.nrow, md.ncol) <= 5
            assert [md.rf[i] for i in range(md.nrow)] + [md.cf[i] for i in range(md.ncol)] == d
            assert md.R == int(np.prod([m.n[f] for f in d[:md.nrow]]))
            assert md.C == int(np.prod([m.n[f] for f in d[md.nrow:]]))
            for o in range(m.K[mi]):
                X = img[md.la_off + 8 * o * md.slice:md.la_off + 8 * (o + 1) * md.slice].view(np.float64)
                X = X.reshape(md.R, md.Cp)
                shift = bfm.LN(m.A[mi][0, o]).reshape(md.R, md.C) - X[:, :md.C]
                assert np.ptp(shift) < 1e-12
            narrow = md.nrow <= 2 and md.ncol <= 2
            if flags != bi.BI_DENSE_A:
                assert (md.la32_off >= 0) == narrow and (md.csr_ptr_off >= 0) == narrow
    finally:
        bi.bi_free_model(h)


def test_soft_workspace_follows_the_family(monkeypatch):
    """Soft vectors on a shared model forced onto a streaming family run it
    (slots per context: a larger workspace than the integer call's) unless a
    modality has more than 256 outcomes; FPI, the agent path and models
    inside the selector's timed range take the log-likelihood tensors."""
    def ll_bytes(img, model, b, T):
        mods, _ = _descs(img, model.M, model.F)
        per_ctx = sum(int(mods[i].slice) for i in range(model.M))
        return -(-b * T * per_ctx * 8 // 256) * 256

    for K, slots in (([3, 2], True), ([300, 2], False)):
        rng = np.random.Generator(np.random.PCG64(2400 + K[0]))
        model = synth.make_model(rng, [4, 3, 5], [2, 1, 2], K, [[0, 1, 2], [1]], 1, 1.0, 1.0, uniform_D=False)
        h, img = bi.bi_pack_model_host(model.n, model.U, model.K, model.deps, 1, model.A, model.B, model.D,
                                       bi.BI_DENSE_A | bi.BI_FAST_F32)
        try:
            b, T = 6, 4
            monkeypatch.setenv("BI_FORCE_PATH", "stream")
            for algo in (bi.BI_ALGO_VMP, bi.BI_ALGO_MMP):
                assert bi.bi_query_path(h, b, T, algo) == bi.BI_PATH_STREAM
                soft, hard = bi.bi_workspace_size_soft(h, b, T, algo), bi.bi_workspace_size(h, b, T, algo)
                if slots:
                    assert soft > hard and soft != ll_bytes(img, model, b, T)
                else:
                    assert soft == ll_bytes(img, model, b, T)
            assert bi.bi_workspace_size_soft(h, b, T, bi.BI_ALGO_FPI) == ll_bytes(img, model, b, T)
            monkeypatch.setenv("BI_FORCE_PATH", "agent")
            assert bi.bi_workspace_size_soft(h, b, T, bi.BI_ALGO_VMP) == ll_bytes(img, model, b, T)
            # unforced: a model inside the selector's timed range keeps soft
            # vectors agent-resident whatever family takes its integer calls
            monkeypatch.delenv("BI_FORCE_PATH")
            for algo in (bi.BI_ALGO_VMP, bi.BI_ALGO_MMP):
                assert bi.bi_workspace_size_soft(h, b, T, algo) == ll_bytes(img, model, b, T)
        finally:
            bi.bi_free_model(h)
