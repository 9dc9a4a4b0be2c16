"""Thin ctypes binding of libbi's C-ABI (include/bi.h).

Functions keep the C names.  Device buffers are torch tensors on the current
HIP device; streams are torch streams.  This module only marshals arguments:
every step of the belief updates runs in the HIP kernels of libbi.so, and the
module raises if the library is missing or cannot be loaded.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libbi.so")

BI_OK = 0
BI_ERR_INVALID_ARG = -1
BI_ERR_SHAPE = -2
BI_ERR_BUFFER_TOO_SMALL = -3
BI_ERR_UNSUPPORTED = -4
BI_ERR_DEVICE = -5
BI_DENSE_A = 1
BI_SPARSE_A = 2
BI_FAST_F32 = 4
BI_F16_PAIRS = 16
BI_CHECK = 8
BI_ALGO_FPI, BI_ALGO_VMP, BI_ALGO_MMP = 0, 1, 2
ALGO_IDS = {"fpi": BI_ALGO_FPI, "vmp": BI_ALGO_VMP, "mmp": BI_ALGO_MMP}

EXPORTS = ("bi_last_error", "bi_plan_model", "bi_plan_model_exact", "bi_pack_model", "bi_pack_model_host", "bi_attach_device_buffer",
           "bi_get_model_stats", "bi_workspace_size", "bi_vfilter", "bi_vmp", "bi_mmp", "bi_vfilter_prior",
           "bi_vmp_prior", "bi_mmp_prior", "bi_infer", "bi_infer_static", "bi_query_path", "bi_explain_path", "bi_workspace_size_soft", "bi_infer_soft", "bi_predict", "bi_free_model",
           "bi_profile_begin", "bi_profile_end")


class BiError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{msg} (code {code})")
        self.code = code


class bi_model_desc(ctypes.Structure):
    _fields_ = [("F", ctypes.c_int32), ("n", ctypes.POINTER(ctypes.c_int32)), ("U", ctypes.POINTER(ctypes.c_int32)),
                ("M", ctypes.c_int32), ("K", ctypes.POINTER(ctypes.c_int32)),
                ("dep_off", ctypes.POINTER(ctypes.c_int32)), ("dep", ctypes.POINTER(ctypes.c_int32)),
                ("model_batch", ctypes.c_int32), ("flags", ctypes.c_uint32),
                ("bdep_off", ctypes.POINTER(ctypes.c_int32)), ("bdep", ctypes.POINTER(ctypes.c_int32))]


class bi_profile_entry(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("launches", ctypes.c_int64), ("total_ms", ctypes.c_double)]


class bi_model_stats(ctypes.Structure):
    _fields_ = [("a_raw", ctypes.c_int64), ("a_stored", ctypes.c_int64), ("a_nnz", ctypes.c_int64),
                ("device_bytes", ctypes.c_int64)]


class bi_infer_opts(ctypes.Structure):
    _fields_ = [("prior_dev", ctypes.c_void_p), ("damping", ctypes.c_double)]


_lib = None


def load(path: str = LIB_PATH):
    """Load libbi.so (built in-tree by paper_2607_17855_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"libbi.so not found at {path}: build it with `python -m paper_2607_17855_amd.build`")
    # One HIP runtime per process: torch ships its own, and libbi must bind to
    # that one.  Loading libbi first pulls in the system runtime beside it,
    # and the second runtime to start then finds no device.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(path)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    P = ctypes.POINTER
    lib.bi_last_error.restype = ctypes.c_char_p
    lib.bi_last_error.argtypes = []
    lib.bi_plan_model.argtypes = [P(bi_model_desc), P(sz)]
    lib.bi_plan_model_exact.argtypes = [P(bi_model_desc), P(vp), P(sz)]
    lib.bi_pack_model.argtypes = [P(bi_model_desc), P(vp), P(vp), P(vp), vp, sz, vp, P(vp)]
    lib.bi_pack_model_host.argtypes = [P(bi_model_desc), P(vp), P(vp), P(vp), vp, sz, P(vp)]
    lib.bi_attach_device_buffer.argtypes = [vp, vp, sz]
    lib.bi_get_model_stats.argtypes = [vp, P(bi_model_stats)]
    lib.bi_workspace_size.argtypes = [vp, i32, i32, i32, P(sz)]
    for name in ("bi_vfilter", "bi_vmp", "bi_mmp"):
        getattr(lib, name).argtypes = [vp, i32, i32, vp, vp, i32, vp, vp, sz, vp]
    for name in ("bi_vfilter_prior", "bi_vmp_prior", "bi_mmp_prior"):
        getattr(lib, name).argtypes = [vp, i32, i32, vp, vp, vp, i32, vp, vp, sz, vp]
    lib.bi_infer.argtypes = [vp, i32, i32, i32, vp, vp, i32, P(bi_infer_opts), vp, vp, sz, vp]
    lib.bi_infer_static.argtypes = [vp, i32, i32, i32, vp, vp, i32, P(bi_infer_opts), vp, vp]
    lib.bi_workspace_size_soft.argtypes = [vp, i32, i32, i32, P(sz)]
    lib.bi_query_path.argtypes = [vp, i32, i32, i32, P(i32)]
    lib.bi_explain_path.argtypes = [vp, i32, i32, i32, ctypes.c_char_p, sz]
    lib.bi_infer_soft.argtypes = [vp, i32, i32, i32, vp, vp, i32, P(bi_infer_opts), vp, vp, sz, vp]
    lib.bi_predict.argtypes = [vp, i32, vp, ctypes.c_int64, vp, ctypes.c_int64, vp, vp]
    lib.bi_free_model.argtypes = [vp]
    lib.bi_free_model.restype = None
    lib.bi_profile_begin.argtypes = []
    lib.bi_profile_end.argtypes = [P(bi_profile_entry), i32, P(i32)]
    for name in EXPORTS[1:]:
        if name != "bi_free_model":
            getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def bi_last_error() -> str:
    return load().bi_last_error().decode()


def _check(rc: int):
    if rc != BI_OK:
        raise BiError(rc, bi_last_error())


class _Desc:
    """Keeps the int32 arrays of a bi_model_desc alive."""

    def __init__(self, n, U, K, deps, model_batch: int, flags: int, bdeps=None):
        self.n = np.ascontiguousarray(n, dtype=np.int32)
        self.U = np.ascontiguousarray(U, dtype=np.int32)
        self.K = np.ascontiguousarray(K, dtype=np.int32)
        self.dep_off = np.ascontiguousarray(np.cumsum([0] + [len(d) for d in deps]), dtype=np.int32)
        self.dep = np.ascontiguousarray([f for d in deps for f in d], dtype=np.int32)
        if self.dep.size == 0:
            self.dep = np.zeros(1, dtype=np.int32)
        ip = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))  # noqa: E731
        if bdeps is None:
            bo = bd = None
        else:
            self.bdep_off = np.ascontiguousarray(np.cumsum([0] + [len(d) for d in bdeps]), dtype=np.int32)
            self.bdep = np.ascontiguousarray([g for d in bdeps for g in d] or [0], dtype=np.int32)
            bo, bd = ip(self.bdep_off), ip(self.bdep)
        self.c = bi_model_desc(len(self.n), ip(self.n), ip(self.U), len(self.K), ip(self.K), ip(self.dep_off),
                               ip(self.dep), int(model_batch), int(flags), bo, bd)


def bi_plan_model(n, U, K, deps, model_batch: int, flags: int = BI_DENSE_A, bdeps=None) -> int:
    d = _Desc(n, U, K, deps, model_batch, flags, bdeps)
    out = ctypes.c_size_t(0)
    _check(load().bi_plan_model(ctypes.byref(d.c), ctypes.byref(out)))
    return int(out.value)


def _f32_list(arrs):
    return [np.ascontiguousarray(a, dtype=np.float32) for a in arrs]


def _ptrs(arrs):
    return (ctypes.c_void_p * len(arrs))(*[a.ctypes.data for a in arrs])


def bi_plan_model_exact(n, U, K, deps, model_batch: int, A, flags: int = BI_DENSE_A, bdeps=None) -> int:
    """Exact packed size for these A tensors (differs from bi_plan_model for BI_SPARSE_A)."""
    d = _Desc(n, U, K, deps, model_batch, flags, bdeps)
    A = _f32_list(A)
    out = ctypes.c_size_t(0)
    _check(load().bi_plan_model_exact(ctypes.byref(d.c), _ptrs(A), ctypes.byref(out)))
    return int(out.value)


def _stream_ptr(stream) -> Optional[int]:
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream)


def bi_pack_model(n, U, K, deps, model_batch: int, A: Sequence[np.ndarray], B: Sequence[np.ndarray],
                  D: Sequence[np.ndarray], dev_buf, flags: int = BI_DENSE_A, stream=None, bdeps=None) -> int:
    """Pack host float32 A/B/D into the device tensor ``dev_buf``; returns the handle."""
    d = _Desc(n, U, K, deps, model_batch, flags, bdeps)
    A = [np.ascontiguousarray(a, dtype=np.float32) for a in A]
    B = [np.ascontiguousarray(b, dtype=np.float32) for b in B]
    D = [np.ascontiguousarray(x, dtype=np.float32) for x in D]
    ptrs = lambda arrs: (ctypes.c_void_p * len(arrs))(*[a.ctypes.data for a in arrs])  # noqa: E731
    out = ctypes.c_void_p(0)
    nbytes = dev_buf.numel() * dev_buf.element_size()
    _check(load().bi_pack_model(ctypes.byref(d.c), ptrs(A), ptrs(B), ptrs(D), ctypes.c_void_p(dev_buf.data_ptr()),
                                nbytes, ctypes.c_void_p(_stream_ptr(stream)), ctypes.byref(out)))
    return int(out.value)


def bi_pack_model_host(n, U, K, deps, model_batch: int, A, B, D, flags: int = BI_DENSE_A, bdeps=None):
    """Pack into host memory; returns (handle, uint8 numpy image)."""
    d = _Desc(n, U, K, deps, model_batch, flags, bdeps)
    nbytes = bi_plan_model_exact(n, U, K, deps, model_batch, A, flags, bdeps)
    raw = np.zeros(nbytes + 512, dtype=np.uint8)
    start = (-raw.ctypes.data) % 256
    img = raw[start:start + nbytes]
    A = [np.ascontiguousarray(a, dtype=np.float32) for a in A]
    B = [np.ascontiguousarray(b, dtype=np.float32) for b in B]
    D = [np.ascontiguousarray(x, dtype=np.float32) for x in D]
    ptrs = lambda arrs: (ctypes.c_void_p * len(arrs))(*[a.ctypes.data for a in arrs])  # noqa: E731
    out = ctypes.c_void_p(0)
    _check(load().bi_pack_model_host(ctypes.byref(d.c), ptrs(A), ptrs(B), ptrs(D), ctypes.c_void_p(img.ctypes.data),
                                     nbytes, ctypes.byref(out)))
    return int(out.value), img


def bi_attach_device_buffer(handle: int, dev_buf):
    nbytes = dev_buf.numel() * dev_buf.element_size()
    _check(load().bi_attach_device_buffer(ctypes.c_void_p(handle), ctypes.c_void_p(dev_buf.data_ptr()), nbytes))


def bi_get_model_stats(handle: int) -> dict:
    st = bi_model_stats()
    _check(load().bi_get_model_stats(ctypes.c_void_p(handle), ctypes.byref(st)))
    return {k: int(getattr(st, k)) for k, _ in bi_model_stats._fields_}


def bi_workspace_size(handle: int, b: int, T: int, algo: int) -> int:
    out = ctypes.c_size_t(0)
    _check(load().bi_workspace_size(ctypes.c_void_p(handle), int(b), int(T), int(algo), ctypes.byref(out)))
    return int(out.value)


def _infer(fn_name, handle, b, T, obs, act, iters, q, ws, stream, prior=None):
    ws_ptr = ws.data_ptr() if ws is not None else 0
    ws_bytes = ws.numel() * ws.element_size() if ws is not None else 0
    act_ptr = act.data_ptr() if act is not None and act.numel() > 0 else 0
    head = (ctypes.c_void_p(handle), int(b), int(T), ctypes.c_void_p(obs.data_ptr()), ctypes.c_void_p(act_ptr))
    if fn_name.endswith("_prior"):
        head += (ctypes.c_void_p(prior.data_ptr() if prior is not None else 0),)
    _check(getattr(load(), fn_name)(*head, int(iters), ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(ws_ptr),
                                    ws_bytes, ctypes.c_void_p(_stream_ptr(stream))))


def bi_vfilter(handle, b, T, obs, act, iters, q, ws=None, stream=None):
    _infer("bi_vfilter", handle, b, T, obs, act, iters, q, ws, stream)


def bi_vmp(handle, b, T, obs, act, iters, q, ws=None, stream=None):
    _infer("bi_vmp", handle, b, T, obs, act, iters, q, ws, stream)


def bi_mmp(handle, b, T, obs, act, iters, q, ws=None, stream=None):
    _infer("bi_mmp", handle, b, T, obs, act, iters, q, ws, stream)


def bi_vfilter_prior(handle, b, T, obs, act, prior, iters, q, ws=None, stream=None):
    _infer("bi_vfilter_prior", handle, b, T, obs, act, iters, q, ws, stream, prior)


def bi_vmp_prior(handle, b, T, obs, act, prior, iters, q, ws=None, stream=None):
    _infer("bi_vmp_prior", handle, b, T, obs, act, iters, q, ws, stream, prior)


def bi_mmp_prior(handle, b, T, obs, act, prior, iters, q, ws=None, stream=None):
    _infer("bi_mmp_prior", handle, b, T, obs, act, iters, q, ws, stream, prior)


def bi_infer(handle, algo: int, b, T, obs, act, iters, q, ws=None, stream=None, prior=None, damping: float = 1.0):
    """The general entry point: any algorithm, optional first-step prior and damping."""
    ws_ptr = ws.data_ptr() if ws is not None else 0
    ws_bytes = ws.numel() * ws.element_size() if ws is not None else 0
    act_ptr = act.data_ptr() if act is not None and act.numel() > 0 else 0
    opts = bi_infer_opts(ctypes.c_void_p(prior.data_ptr() if prior is not None else 0), float(damping))
    _check(load().bi_infer(ctypes.c_void_p(handle), int(algo), int(b), int(T), ctypes.c_void_p(obs.data_ptr()),
                           ctypes.c_void_p(act_ptr), int(iters), ctypes.byref(opts), ctypes.c_void_p(q.data_ptr()),
                           ctypes.c_void_p(ws_ptr), ws_bytes, ctypes.c_void_p(_stream_ptr(stream))))


BI_STATIC_SCRATCH_BYTES = 64 << 20


def bi_infer_static(handle, algo: int, b, T, obs, act, iters, q, stream=None, prior=None, damping: float = 1.0):
    """bi_infer without a workspace: the library's static device scratch (no allocation)."""
    act_ptr = act.data_ptr() if act is not None and act.numel() > 0 else 0
    opts = bi_infer_opts(ctypes.c_void_p(prior.data_ptr() if prior is not None else 0), float(damping))
    _check(load().bi_infer_static(ctypes.c_void_p(handle), int(algo), int(b), int(T),
                                  ctypes.c_void_p(obs.data_ptr()), ctypes.c_void_p(act_ptr), int(iters),
                                  ctypes.byref(opts), ctypes.c_void_p(q.data_ptr()),
                                  ctypes.c_void_p(_stream_ptr(stream))))


BI_PATH_AGENT, BI_PATH_STREAM, BI_PATH_SPARSE = 0, 1, 2
PATH_NAMES = {BI_PATH_AGENT: "agent", BI_PATH_STREAM: "stream", BI_PATH_SPARSE: "sparse"}


def bi_query_path(handle: int, b: int, T: int, algo: int) -> int:
    out = ctypes.c_int32(-1)
    _check(load().bi_query_path(ctypes.c_void_p(handle), int(b), int(T), int(algo), ctypes.byref(out)))
    return int(out.value)


def bi_explain_path(handle: int, b: int, T: int, algo: int) -> str:
    buf = ctypes.create_string_buffer(512)
    _check(load().bi_explain_path(ctypes.c_void_p(handle), int(b), int(T), int(algo), buf, 512))
    return buf.value.decode()


def bi_workspace_size_soft(handle: int, b: int, T: int, algo: int) -> int:
    out = ctypes.c_size_t(0)
    _check(load().bi_workspace_size_soft(ctypes.c_void_p(handle), int(b), int(T), int(algo), ctypes.byref(out)))
    return int(out.value)


def bi_infer_soft(handle, algo: int, b, T, obs_soft, act, iters, q, ws, stream=None, prior=None,
                  damping: float = 1.0):
    """Soft observations obs_soft [b][T][sum K] float32 (device)."""
    ws_bytes = ws.numel() * ws.element_size() if ws is not None else 0
    act_ptr = act.data_ptr() if act is not None and act.numel() > 0 else 0
    opts = bi_infer_opts(ctypes.c_void_p(prior.data_ptr() if prior is not None else 0), float(damping))
    _check(load().bi_infer_soft(ctypes.c_void_p(handle), int(algo), int(b), int(T),
                                ctypes.c_void_p(obs_soft.data_ptr()), ctypes.c_void_p(act_ptr), int(iters),
                                ctypes.byref(opts), ctypes.c_void_p(q.data_ptr()),
                                ctypes.c_void_p(ws.data_ptr() if ws is not None else 0), ws_bytes,
                                ctypes.c_void_p(_stream_ptr(stream))))


def bi_predict(handle, b, q, q_stride, act, act_stride, out, stream=None):
    """out[a] = B[:, :, act[a]] q[a] per factor; q / act rows at a * q_stride / a * act_stride elements."""
    _check(load().bi_predict(ctypes.c_void_p(handle), int(b), ctypes.c_void_p(q.data_ptr()), int(q_stride),
                             ctypes.c_void_p(act.data_ptr()), int(act_stride), ctypes.c_void_p(out.data_ptr()),
                             ctypes.c_void_p(_stream_ptr(stream))))


def bi_free_model(handle: int):
    load().bi_free_model(ctypes.c_void_p(handle))


def bi_profile_begin():
    _check(load().bi_profile_begin())


def bi_profile_end() -> dict:
    """{kernel class: (launches, total_ms)} of the launches since bi_profile_begin."""
    cap = 32
    arr = (bi_profile_entry * cap)()
    n = ctypes.c_int32(0)
    _check(load().bi_profile_end(arr, cap, ctypes.byref(n)))
    return {arr[i].name.decode(): (int(arr[i].launches), float(arr[i].total_ms)) for i in range(min(n.value, cap))}


def _check_tensor(name, t, dtype, shape, device):
    """Raise ValueError unless t is a contiguous tensor of this dtype, shape and device."""
    if t is None:
        raise ValueError(f"{name} is missing")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(int(x) for x in t.shape) != tuple(int(x) for x in shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, the model on {device}")


def check_infer_args(model, device, obs, act, q=None, prior=None, soft: bool = False):
    """Host-side check of an inference call's tensors against the model shape,
    before anything reaches the library (which reads them as raw device
    pointers): obs int32 [b][T][M] (soft: float32 [b][T][sum K]), act int32
    [b][T-1][F] (may be None or empty when T == 1), q float32 [b][T][sum n],
    prior float32 [b][sum n], all contiguous and on `device`."""
    import torch
    device = torch.device(device)
    if obs is None or obs.dim() != 3:
        raise ValueError("obs must be a 3-d tensor [b][T][M]")
    b, T = int(obs.shape[0]), int(obs.shape[1])
    if b < 1 or T < 1:
        raise ValueError("obs must hold at least one agent and one step")
    F, ntot = len(model.n), int(sum(model.n))
    if soft:
        _check_tensor("obs_soft", obs, torch.float32, (b, T, int(sum(model.K))), device)
    else:
        _check_tensor("obs", obs, torch.int32, (b, T, len(model.K)), device)
    if T > 1 or (act is not None and act.numel() > 0):
        _check_tensor("act", act, torch.int32, (b, T - 1, F), device)
    if q is not None:
        _check_tensor("q", q, torch.float32, (b, T, ntot), device)
    if prior is not None:
        _check_tensor("prior", prior, torch.float32, (b, ntot), device)
    if model.mb != 1 and model.mb != b:
        raise ValueError(f"b={b} but the model holds {model.mb} agents")


_ENTRY = {"fpi": bi_vfilter, "vmp": bi_vmp, "mmp": bi_mmp}
_ENTRY_PRIOR = {"fpi": bi_vfilter_prior, "vmp": bi_vmp_prior, "mmp": bi_mmp_prior}


class PackedModel:
    """A model packed into a torch device buffer, with its C handle."""

    def __init__(self, model, flags: int = BI_DENSE_A, device=None, stream=None):
        import torch
        self.model = model
        bdeps = getattr(model, "bdeps", None)
        nbytes = bi_plan_model_exact(model.n, model.U, model.K, model.deps, model.mb, model.A, flags, bdeps)
        self.buf = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device or "cuda")
        self.handle = bi_pack_model(model.n, model.U, model.K, model.deps, model.mb, model.A, model.B, model.D,
                                    self.buf, flags, stream, bdeps)
        self.flags = flags

    def stats(self) -> dict:
        return bi_get_model_stats(self.handle)

    def path(self, b: int, T: int, algo: str) -> str:
        """The kernel family ("agent", "stream" or "sparse") a call with these sizes runs."""
        return PATH_NAMES[bi_query_path(self.handle, b, T, ALGO_IDS[algo])]

    def explain_path(self, b: int, T: int, algo: str) -> str:
        """Which family a call runs and why the others are or are not eligible."""
        return bi_explain_path(self.handle, b, T, ALGO_IDS[algo])

    def workspace(self, b: int, T: int, algo: str):
        import torch
        nb = bi_workspace_size(self.handle, b, T, ALGO_IDS[algo])
        return torch.empty(nb, dtype=torch.uint8, device=self.buf.device) if nb else None

    def infer(self, algo: str, obs, act, iters: int, q=None, ws=None, stream=None, prior=None,
              damping: float = 1.0):
        """obs [b][T][M] / act [b][T-1][F] int32 device tensors -> q [b][T][sum n] float32.

        prior: optional float32 device tensor [b][sum n], the first step's prior in place of D.
        damping: step tau in (0, 1] of q <- (1 - tau) q + tau q_new (1 = plain update)."""
        import torch
        check_infer_args(self.model, self.buf.device, obs, act, q, prior)
        b, T = int(obs.shape[0]), int(obs.shape[1])
        if q is None:
            q = torch.empty((b, T, sum(self.model.n)), dtype=torch.float32, device=self.buf.device)
        if ws is None:
            ws = self.workspace(b, T, algo)
        if damping != 1.0:
            bi_infer(self.handle, ALGO_IDS[algo], b, T, obs, act, iters, q, ws, stream, prior, damping)
        elif prior is None:
            _ENTRY[algo](self.handle, b, T, obs, act, iters, q, ws, stream)
        else:
            _ENTRY_PRIOR[algo](self.handle, b, T, obs, act, prior, iters, q, ws, stream)
        return q

    def workspace_soft(self, b: int, T: int, algo: str):
        import torch
        nb = bi_workspace_size_soft(self.handle, b, T, ALGO_IDS[algo])
        return torch.empty(nb, dtype=torch.uint8, device=self.buf.device)

    def infer_soft(self, algo: str, obs_soft, act, iters: int, q=None, ws=None, stream=None, prior=None,
                   damping: float = 1.0):
        """obs_soft [b][T][sum K] float32 / act [b][T-1][F] int32 device tensors -> q [b][T][sum n]."""
        import torch
        check_infer_args(self.model, self.buf.device, obs_soft, act, q, prior, soft=True)
        b, T = int(obs_soft.shape[0]), int(obs_soft.shape[1])
        if q is None:
            q = torch.empty((b, T, sum(self.model.n)), dtype=torch.float32, device=self.buf.device)
        if ws is None:
            ws = self.workspace_soft(b, T, algo)
        bi_infer_soft(self.handle, ALGO_IDS[algo], b, T, obs_soft, act, iters, q, ws, stream, prior, damping)
        return q

    def predict(self, q, act, out=None, stream=None):
        """Predictive prior of the next step: q [b][..][sum n] marginals of the step to carry (the
        last dimension holds one step; other rows are skipped by the stride) and act [b][F] int32
        -> out [b][sum n] float32."""
        import torch
        b, ntot = int(q.shape[0]), sum(self.model.n)
        if q.stride(-1) != 1 or act.stride(-1) != 1:
            raise ValueError("q and act must be contiguous in their last dimension")
        if q.dtype != torch.float32 or act.dtype != torch.int32:
            raise ValueError("q must be float32 and act int32")
        if int(q.shape[-1]) < ntot or int(act.shape[0]) != b or int(act.shape[-1]) < len(self.model.n):
            raise ValueError("q must hold sum n marginals and act F actions per agent")
        if q.device != self.buf.device or act.device != self.buf.device:
            raise ValueError("q and act must be on the model's device")
        if out is not None:
            _check_tensor("out", out, torch.float32, (b, ntot), self.buf.device)
        if out is None:
            out = torch.empty((b, ntot), dtype=torch.float32, device=self.buf.device)
        bi_predict(self.handle, b, q, q.stride(0), act, act.stride(0), out, stream)
        return out

    def close(self):
        if getattr(self, "handle", 0):
            bi_free_model(self.handle)
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
