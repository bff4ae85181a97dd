"""Python binding of liboptcc (ctypes): argument marshalling only.

Every function here converts torch tensors to the pointers, sizes and the
stream the C ABI expects and calls the function of the same name in
liboptcc.so; all computation happens in the library's HIP kernels.  There is
no fallback: if the library is missing or fails to load, every call raises.

Tensors are row-major 2-D CUDA (HIP) tensors with unit column stride; the
leading dimension is taken from stride(0).  M is torch.float32 or
torch.bfloat16; err, P, Q and M_hat are torch.float32; P is rows x rank and Q
is cols x rank, contiguous.  Work is enqueued on torch's current stream.
"""

from __future__ import annotations

import ctypes
import os
import re

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "liboptcc.so")
HEADER = os.path.join(os.path.dirname(PKG), "include", "optcc.h")

OCC_OK = 0
OCC_F32, OCC_BF16 = 0, 1
OCC_F_NONFINITE, OCC_F_RANK_DEFICIENT, OCC_F_BAD_ROWS = 1, 2, 4
OCC_NO_MHAT = 1
OCC_DEC_SPLIT_BF16, OCC_DEC_OUT_BF16 = 1, 2
OCC_MAX_RANK = 128
OCC_NOALLOC_MAX_BYTES = 64 << 20
OCC_MAX_ITERS = 64

STATUS_NAMES = {
    0: "OCC_OK", 1: "OCC_E_NULL", 2: "OCC_E_SHAPE", 3: "OCC_E_RANK", 4: "OCC_E_ITERS",
    5: "OCC_E_DTYPE", 6: "OCC_E_ALIGN", 7: "OCC_E_ALIAS", 8: "OCC_E_WORKSPACE",
    9: "OCC_E_HIP", 10: "OCC_E_FLAGS",
}


class OccError(RuntimeError):
    """A liboptcc call returned a non-zero occ_status_t."""

    def __init__(self, fn: str, status: int):
        self.status = status
        self.code = STATUS_NAMES.get(status, str(status))
        super().__init__(f"{fn}: {self.code} ({occ_status_str(status)})")


class occ_mat_t(ctypes.Structure):
    _fields_ = [
        ("M", ctypes.c_void_p),
        ("m_dtype", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
        ("rows", ctypes.c_int64),
        ("cols", ctypes.c_int64),
        ("ldm", ctypes.c_int64),
        ("err", ctypes.c_void_p),
        ("lde", ctypes.c_int64),
        ("P", ctypes.c_void_p),
        ("Q", ctypes.c_void_p),
        ("M_hat", ctypes.c_void_p),
        ("ldh", ctypes.c_int64),
    ]


class occ_stage_t(ctypes.Structure):
    _fields_ = [
        ("bwd_done", ctypes.c_double),
        ("comm", ctypes.c_double),
        ("comm_compressed", ctypes.c_double),
        ("compress", ctypes.c_double),
    ]


class occ_kernel_time_t(ctypes.Structure):
    _fields_ = [
        ("name", ctypes.c_char * 48),
        ("launches", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
        ("total_ms", ctypes.c_double),
    ]


_lib = None

_SIGS = {
    "occ_abi_version": (ctypes.c_int, []),
    "occ_status_str": (ctypes.c_char_p, [ctypes.c_int]),
    "occ_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(occ_mat_t), ctypes.c_int,
                                              ctypes.c_int, ctypes.c_int]),
    "occ_compress_workspace_bytes": (ctypes.c_size_t, [ctypes.c_int64, ctypes.c_int64,
                                                       ctypes.c_int, ctypes.c_int, ctypes.c_int]),
    "occ_workspace_init": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "occ_compress": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_int64,
                                    ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                                    ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                    ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "occ_decompress": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                      ctypes.c_int64, ctypes.c_int, ctypes.c_void_p,
                                      ctypes.c_int64, ctypes.c_void_p]),
    "occ_decompress_ex": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                         ctypes.c_int64, ctypes.c_int, ctypes.c_uint,
                                         ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]),
    "occ_err_update": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int, ctypes.c_int64,
                                      ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p,
                                      ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
                                      ctypes.c_void_p, ctypes.c_void_p]),
    "occ_step": (ctypes.c_int, [ctypes.POINTER(occ_mat_t), ctypes.c_int, ctypes.c_int,
                                ctypes.c_uint, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "occ_step_batched": (ctypes.c_int, [ctypes.POINTER(occ_mat_t), ctypes.c_int, ctypes.c_int,
                                        ctypes.c_int, ctypes.c_uint, ctypes.c_void_p,
                                        ctypes.c_size_t, ctypes.c_void_p]),
    "occ_step_rows": (ctypes.c_int, [ctypes.POINTER(occ_mat_t), ctypes.c_void_p, ctypes.c_int64,
                                     ctypes.c_int, ctypes.c_int, ctypes.c_uint, ctypes.c_void_p,
                                     ctypes.c_size_t, ctypes.c_void_p]),
    "occ_step_rows_workspace_bytes": (ctypes.c_size_t, [ctypes.c_int64, ctypes.c_int64,
                                                        ctypes.c_int, ctypes.c_int, ctypes.c_int]),
    "occ_step_batched_noalloc": (ctypes.c_int, [ctypes.POINTER(occ_mat_t), ctypes.c_int,
                                                ctypes.c_int, ctypes.c_int, ctypes.c_uint,
                                                ctypes.c_void_p, ctypes.c_void_p]),
    "occ_get_flags": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_uint32),
                                     ctypes.c_int, ctypes.c_void_p]),
    "occ_pipeline_1f1b": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                         ctypes.c_double, ctypes.c_double,
                                         ctypes.POINTER(ctypes.c_double),
                                         ctypes.POINTER(ctypes.c_double)]),
    "occ_sc_select": (ctypes.c_int, [ctypes.POINTER(occ_stage_t), ctypes.c_int, ctypes.c_int,
                                     ctypes.POINTER(ctypes.c_uint8), ctypes.POINTER(ctypes.c_int),
                                     ctypes.POINTER(ctypes.c_double)]),
    "occ_profile_begin": (ctypes.c_int, []),
    "occ_profile_end": (ctypes.c_int, [ctypes.POINTER(occ_kernel_time_t), ctypes.c_int,
                                       ctypes.POINTER(ctypes.c_int)]),
}


def lib() -> ctypes.CDLL:
    """The loaded in-tree liboptcc.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        path = LIB_PATH
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with "
                               "`python -m paper_2301_09830_amd.build`")
        handle = ctypes.CDLL(path)
        for name, (res, args) in _SIGS.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def header_symbols() -> list:
    """Names of the functions declared in include/optcc.h."""
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(occ_[a-z_]+)\s*\(", text)))


def _check(fn: str, status: int) -> None:
    if status != OCC_OK:
        raise OccError(fn, status)


def occ_abi_version() -> int:
    return lib().occ_abi_version()


def occ_status_str(status: int) -> str:
    return lib().occ_status_str(status).decode()


# ----------------------------------------------------------------------------
# tensor marshalling
# ----------------------------------------------------------------------------
def _torch():
    import torch
    return torch


def _stream(stream=None) -> int:
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def _ptr(t) -> int | None:
    return None if t is None else int(t.data_ptr())


def _ld(t, name: str) -> int:
    if t.dim() != 2:
        raise ValueError(f"{name} must be 2-D")
    if t.shape[1] > 1 and t.stride(1) != 1:
        raise ValueError(f"{name} must have unit column stride (row-major)")
    return int(t.stride(0)) if t.shape[0] > 1 else int(t.shape[1])


def _mdtype(M) -> int:
    torch = _torch()
    if M.dtype == torch.float32:
        return OCC_F32
    if M.dtype == torch.bfloat16:
        return OCC_BF16
    raise TypeError("M must be float32 or bfloat16")


def _f32(t, name: str):
    torch = _torch()
    if t is not None and t.dtype != torch.float32:
        raise TypeError(f"{name} must be float32")
    return t


def make_mat(M, err, P, Q, M_hat=None) -> occ_mat_t:
    """occ_mat_t describing one matrix and its compressor state."""
    _f32(err, "err"), _f32(P, "P"), _f32(Q, "Q"), _f32(M_hat, "M_hat")
    if P.dim() != 2 or Q.dim() != 2 or P.shape[0] != M.shape[0] or Q.shape[0] != M.shape[1] \
            or P.shape[1] != Q.shape[1]:
        raise ValueError("P must be rows x rank and Q cols x rank")
    if not (P.is_contiguous() and Q.is_contiguous()):
        raise ValueError("P and Q must be contiguous")
    a = occ_mat_t()
    a.M = _ptr(M)
    a.m_dtype = _mdtype(M)
    a.rows, a.cols = int(M.shape[0]), int(M.shape[1])
    a.ldm = _ld(M, "M")
    a.err = _ptr(err)
    a.lde = _ld(err, "err")
    a.P = _ptr(P)
    a.Q = _ptr(Q)
    a.M_hat = _ptr(M_hat)
    a.ldh = _ld(M_hat, "M_hat") if M_hat is not None else 0
    return a


def occ_workspace_bytes(shapes, rank: int, iters: int, m_dtype: int = OCC_F32) -> int:
    """Workspace bytes for matrices of the given (rows, cols) shapes whose M
    has dtype m_dtype (OCC_F32 or OCC_BF16)."""
    arr = (occ_mat_t * len(shapes))()
    for a, (m, n) in zip(arr, shapes):
        a.rows, a.cols, a.ldm, a.m_dtype = m, n, n, m_dtype
    return int(lib().occ_workspace_bytes(arr, len(shapes), rank, iters))


def occ_compress_workspace_bytes(m: int, n: int, rank: int, iters: int,
                                 m_dtype: int = OCC_F32) -> int:
    return int(lib().occ_compress_workspace_bytes(m, n, m_dtype, rank, iters))


def alloc_workspace(nbytes: int, device="cuda", stream=None):
    """A zero-headed workspace tensor of at least nbytes (256-byte aligned)."""
    torch = _torch()
    ws = torch.empty(max(int(nbytes), 256) + 256, dtype=torch.uint8, device=device)
    off = (-ws.data_ptr()) % 256
    ws = ws[off:off + max(int(nbytes), 256)]
    occ_workspace_init(ws, stream)
    return ws


def occ_workspace_init(ws, stream=None) -> None:
    _check("occ_workspace_init", lib().occ_workspace_init(_ptr(ws), ws.numel(), _stream(stream)))


def occ_step(M, err, Q, rank: int, iters: int, P=None, M_hat=None, write_mhat: bool = True,
             ws=None, stream=None):
    """Fused compress + decompress + error update; err and Q updated in place.

    Returns (P, M_hat) (M_hat is None when write_mhat is False).
    """
    torch = _torch()
    m, n = M.shape
    if P is None:
        P = torch.empty((m, rank), dtype=torch.float32, device=M.device)
    if write_mhat and M_hat is None:
        M_hat = torch.empty((m, n), dtype=torch.float32, device=M.device)
    if P.shape[1] != rank:
        raise ValueError("P and Q must have `rank` columns")
    mat = make_mat(M, err, P, Q, M_hat if write_mhat else None)
    if ws is None:
        ws = alloc_workspace(lib().occ_workspace_bytes(ctypes.byref(mat), 1, rank, iters),
                             M.device, stream)
    flags = 0 if write_mhat else OCC_NO_MHAT
    _check("occ_step", lib().occ_step(ctypes.byref(mat), rank, iters, flags, _ptr(ws),
                                      ws.numel(), _stream(stream)))
    return P, (M_hat if write_mhat else None)


def occ_step_batched(items, rank: int, iters: int, write_mhat: bool = True, ws=None,
                     stream=None):
    """occ_step on independent matrices in one launch per pass.

    items: sequence of (M, err, Q, P, M_hat) tuples (P and M_hat preallocated;
    M_hat may be None when write_mhat is False).
    """
    arr = (occ_mat_t * len(items))()
    for a, (M, err, Q, P, M_hat) in zip(arr, items):
        ctypes.memmove(ctypes.byref(a), ctypes.byref(make_mat(M, err, P, Q,
                                                              M_hat if write_mhat else None)),
                       ctypes.sizeof(occ_mat_t))
    if ws is None:
        ws = alloc_workspace(lib().occ_workspace_bytes(arr, len(items), rank, iters),
                             items[0][0].device, stream)
    flags = 0 if write_mhat else OCC_NO_MHAT
    _check("occ_step_batched", lib().occ_step_batched(arr, len(items), rank, iters, flags,
                                                      _ptr(ws), ws.numel(), _stream(stream)))
    return ws


def occ_step_batched_noalloc(items, rank: int, iters: int, write_mhat: bool = True,
                             flags_out=None, stream=None) -> None:
    """occ_step_batched on the library's static per-GPU workspace (no device
    allocation by the library or by this binding).  items as for
    occ_step_batched; flags_out: optional int32 CUDA tensor of one element
    that receives the numeric flags (OR-ed in)."""
    arr = (occ_mat_t * len(items))()
    for a, (M, err, Q, P, M_hat) in zip(arr, items):
        ctypes.memmove(ctypes.byref(a), ctypes.byref(make_mat(M, err, P, Q,
                                                              M_hat if write_mhat else None)),
                       ctypes.sizeof(occ_mat_t))
    flags = 0 if write_mhat else OCC_NO_MHAT
    _check("occ_step_batched_noalloc",
           lib().occ_step_batched_noalloc(arr, len(items), rank, iters, flags, _ptr(flags_out),
                                          _stream(stream)))


def occ_step_rows_workspace_bytes(n_rows: int, cols: int, rank: int, iters: int,
                                  m_dtype: int = OCC_F32) -> int:
    return int(lib().occ_step_rows_workspace_bytes(n_rows, cols, m_dtype, rank, iters))


def occ_step_rows(M, err, Q, rows, rank: int, iters: int, P=None, M_hat=None,
                  write_mhat: bool = True, ws=None, stream=None):
    """Row-sparse step: compress the listed rows of M + err (rows: int32 CUDA
    tensor, strictly increasing); err and Q updated in place, only the listed
    rows of err and M_hat are written.  Returns (P, M_hat) with P compact
    (len(rows) x rank).  A newly allocated M_hat is zero-filled, so that its
    unlisted rows hold the dense step's zeros."""
    torch = _torch()
    m, n = M.shape
    if rows.dtype != torch.int32 or rows.dim() != 1 or not rows.is_contiguous():
        raise TypeError("rows must be a contiguous 1-D int32 tensor")
    n_rows = int(rows.numel())
    if P is None:
        P = torch.empty((n_rows, rank), dtype=torch.float32, device=M.device)
    if write_mhat and M_hat is None:
        M_hat = torch.zeros((m, n), dtype=torch.float32, device=M.device)
    _f32(err, "err"), _f32(P, "P"), _f32(Q, "Q"), _f32(M_hat, "M_hat")
    if P.shape != (n_rows, rank) or Q.shape != (n, rank) or not (P.is_contiguous() and
                                                                 Q.is_contiguous()):
        raise ValueError("P must be len(rows) x rank and Q cols x rank, both contiguous")
    a = occ_mat_t()
    a.M = _ptr(M)
    a.m_dtype = _mdtype(M)
    a.rows, a.cols = m, n
    a.ldm = _ld(M, "M")
    a.err = _ptr(err)
    a.lde = _ld(err, "err")
    a.P = _ptr(P) if n_rows else None
    a.Q = _ptr(Q)
    a.M_hat = _ptr(M_hat) if write_mhat else None
    a.ldh = _ld(M_hat, "M_hat") if write_mhat else 0
    if ws is None:
        ws = alloc_workspace(occ_step_rows_workspace_bytes(n_rows, n, rank, iters, a.m_dtype),
                             M.device, stream)
    flags = 0 if write_mhat else OCC_NO_MHAT
    _check("occ_step_rows", lib().occ_step_rows(ctypes.byref(a), _ptr(rows) if n_rows else None,
                                                n_rows, rank, iters, flags, _ptr(ws), ws.numel(),
                                                _stream(stream)))
    return P, (M_hat if write_mhat else None)


def occ_compress(M, err_prev, Q, rank: int, iters: int, P=None, ws=None, stream=None):
    """A = M + err_prev (err_prev may be None); Q updated in place; returns P_hat."""
    torch = _torch()
    m, n = M.shape
    _f32(err_prev, "err_prev"), _f32(Q, "Q")
    if P is None:
        P = torch.empty((m, rank), dtype=torch.float32, device=M.device)
    if ws is None:
        ws = alloc_workspace(occ_compress_workspace_bytes(m, n, rank, iters, _mdtype(M)),
                             M.device, stream)
    lde = _ld(err_prev, "err_prev") if err_prev is not None else 0
    _check("occ_compress", lib().occ_compress(_ptr(M), _mdtype(M), m, n, _ld(M, "M"),
                                              _ptr(err_prev), lde, _ptr(P), _ptr(Q), rank, iters,
                                              _ptr(ws), ws.numel(), _stream(stream)))
    return P


def occ_decompress(P, Q, M_hat=None, stream=None):
    """M_hat = P Q^T (fp32 products, fp32 M_hat)."""
    torch = _torch()
    _f32(P, "P"), _f32(Q, "Q"), _f32(M_hat, "M_hat")
    m, rank = P.shape
    n = Q.shape[0]
    if M_hat is None:
        M_hat = torch.empty((m, n), dtype=torch.float32, device=P.device)
    _check("occ_decompress", lib().occ_decompress(_ptr(P), _ptr(Q), m, n, rank, _ptr(M_hat),
                                                  _ld(M_hat, "M_hat"), _stream(stream)))
    return M_hat


def occ_decompress_ex(P, Q, flags: int = 0, M_hat=None, stream=None):
    """M_hat = P Q^T with OCC_DEC_* flags: OCC_DEC_SPLIT_BF16 runs the products
    occ_step uses for a bf16 M; OCC_DEC_OUT_BF16 stores M_hat as bfloat16."""
    torch = _torch()
    _f32(P, "P"), _f32(Q, "Q")
    m, rank = P.shape
    n = Q.shape[0]
    out_dtype = torch.bfloat16 if flags & OCC_DEC_OUT_BF16 else torch.float32
    if M_hat is None:
        M_hat = torch.empty((m, n), dtype=out_dtype, device=P.device)
    if M_hat.dtype != out_dtype:
        raise TypeError(f"M_hat must be {out_dtype} for these flags")
    _check("occ_decompress_ex", lib().occ_decompress_ex(_ptr(P), _ptr(Q), m, n, rank, flags,
                                                        _ptr(M_hat), _ld(M_hat, "M_hat"),
                                                        _stream(stream)))
    return M_hat


def occ_err_update(M, err_prev, M_hat, err_new=None, stream=None):
    """err_new = (M + err_prev) - M_hat; err_new may be err_prev (in place).
    err_prev and err_new share one leading dimension."""
    torch = _torch()
    m, n = M.shape
    if err_new is None:
        ld = _ld(err_prev, "err_prev") if err_prev is not None else n
        err_new = torch.empty((m, ld), dtype=torch.float32, device=M.device)[:, :n]
    lde = _ld(err_new, "err_new")
    if err_prev is not None and _ld(err_prev, "err_prev") != lde:
        raise ValueError("err_prev and err_new must share one leading dimension")
    _check("occ_err_update", lib().occ_err_update(_ptr(M), _mdtype(M), m, n, _ld(M, "M"),
                                                  _ptr(err_prev), lde, _ptr(M_hat),
                                                  _ld(M_hat, "M_hat"), _ptr(err_new),
                                                  _stream(stream)))
    return err_new


def occ_pipeline_1f1b(n_stages: int, n_micro: int, t_fwd: float, t_bwd: float,
                      t_p2p: float = 0.0):
    """(bwd_done per stage, end of the schedule) under one-forward-one-backward."""
    out = (ctypes.c_double * n_stages)()
    end = ctypes.c_double(0.0)
    _check("occ_pipeline_1f1b", lib().occ_pipeline_1f1b(n_stages, n_micro, t_fwd, t_bwd, t_p2p,
                                                        out, ctypes.byref(end)))
    return list(out), end.value


def occ_sc_select(stages, max_compressed: int):
    """stages: sequence of (bwd_done, comm, comm_compressed, compress).
    Returns (selected flags per stage, end of the last exchange)."""
    arr = (occ_stage_t * len(stages))(*[occ_stage_t(*map(float, t)) for t in stages])
    sel = (ctypes.c_uint8 * len(stages))()
    n = ctypes.c_int(0)
    end = ctypes.c_double(0.0)
    _check("occ_sc_select", lib().occ_sc_select(arr, len(stages), max_compressed, sel,
                                                ctypes.byref(n), ctypes.byref(end)))
    return [int(x) for x in sel], end.value


def occ_get_flags(ws, clear: bool = False, stream=None) -> int:
    out = ctypes.c_uint32(0)
    _check("occ_get_flags", lib().occ_get_flags(_ptr(ws), ctypes.byref(out), int(clear),
                                                _stream(stream)))
    return int(out.value)


def occ_profile_begin() -> None:
    _check("occ_profile_begin", lib().occ_profile_begin())


def occ_profile_end(max_kernels: int = 64) -> dict:
    """{kernel name: (launches, total_ms)} recorded since occ_profile_begin."""
    buf = (occ_kernel_time_t * max_kernels)()
    n = ctypes.c_int(0)
    _check("occ_profile_end", lib().occ_profile_end(buf, max_kernels, ctypes.byref(n)))
    return {buf[i].name.decode(): (int(buf[i].launches), float(buf[i].total_ms))
            for i in range(min(n.value, max_kernels))}
