"""Python binding for libfasq, the MI355X product-quantized matmul library.

The binding marshals arguments only: every computation runs in the HIP
kernels of ``libfasq.so``.  Torch is used for device buffers and streams.
If the library is not built, every call raises :class:`LibraryNotBuilt`;
there is no fallback.

Operation (FASQ, Sec. 3.1.2, Eq. lut-accumulate): ``y = x . W_hat^T`` where
``W_hat[n, s*d + i] = codebook[u(n, s), i]`` and ``u(n, s)`` are packed ids
(8, 12 or 16 bits, one least-significant-bit-first stream per output row).
The encoder (Sec. 3.1.1, Alg. 1) produces the codebook and the ids from dense
weights by k-means.
"""

from __future__ import annotations

import ctypes
import os
import threading
from typing import Optional

__all__ = [
    "FasqError",
    "LibraryNotBuilt",
    "LIB_PATH",
    "lib",
    "library_loaded",
    "abi_version",
    "idx_row_bytes",
    "plan",
    "status_string",
    "last_error",
    "pq_gemv",
    "pq_gemm",
    "pq_reconstruct",
    "pq_gemv_batched",
    "pq_encode",
    "pq_gemv_ex",
    "pq_gemm_lut",
    "gemm_lut_raw",
    "gemv_ex_raw",
    "gemv_ex_workspace_bytes",
    "pq_gemm_ex",
    "gemm_ex_raw",
    "gemm_ex_workspace_bytes",
    "encode_raw",
    "encode_workspace_bytes",
    "gemv_raw",
    "gemv_batched_raw",
    "gemm_raw",
    "reconstruct_raw",
    "FASQ_OK",
    "FASQ_ERR_INVALID_ARG",
    "FASQ_ERR_UNSUPPORTED",
    "FASQ_ERR_HIP",
    "FASQ_ERR_HOST_MEMORY",
    "LaunchList",
    "EXPORTED_SYMBOLS",
    "ABI_VERSION",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfasq.so")

ABI_VERSION = 6  # FASQ_ABI_VERSION of include/fasq.h

FASQ_OK = 0
FASQ_ERR_INVALID_ARG = 1
FASQ_ERR_UNSUPPORTED = 2
FASQ_ERR_HIP = 3
FASQ_ERR_HOST_MEMORY = 4

EXPORTED_SYMBOLS = (
    "fasq_pq_gemv",
    "fasq_pq_gemm",
    "fasq_pq_gemv_batched",
    "fasq_pq_reconstruct",
    "fasq_idx_row_bytes",
    "fasq_status_string",
    "fasq_last_error",
    "fasq_abi_version",
    "fasq_pq_plan",
    "fasq_pq_encode",
    "fasq_pq_encode_workspace_bytes",
    "fasq_pq_gemv_ex",
    "fasq_pq_gemv_ex_workspace_bytes",
    "fasq_pq_gemm_lut",
    "fasq_pq_gemm_ex",
    "fasq_pq_gemm_ex_workspace_bytes",
    "fasq_pq_gemv_ex_noalloc",
    "fasq_noalloc_scratch_bytes",
    "fasq_launch_list_create",
    "fasq_launch_list_begin",
    "fasq_launch_list_end",
    "fasq_launch_list_run",
    "fasq_launch_list_size",
    "fasq_launch_list_destroy",
)


class LibraryNotBuilt(ImportError):
    pass


class FasqError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{message} (status {status})")
        self.status = status


_lock = threading.Lock()
_lib: Optional[ctypes.CDLL] = None

_c_i64 = ctypes.c_int64
_c_int = ctypes.c_int
_c_vp = ctypes.c_void_p


def lib() -> ctypes.CDLL:
    """Load ``libfasq.so`` (once) and declare its signatures."""
    global _lib
    if _lib is not None:
        return _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(LIB_PATH):
            raise LibraryNotBuilt(f"{LIB_PATH} is missing; build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        mm = [_c_vp, _c_i64, _c_i64, _c_i64, _c_vp, _c_int, _c_int, _c_vp, _c_i64, _c_vp, _c_vp]
        for name in ("fasq_pq_gemv", "fasq_pq_gemm", "fasq_pq_gemm_lut"):
            f = getattr(L, name)
            f.argtypes = mm
            f.restype = _c_int
        _pp = ctypes.POINTER(_c_vp)
        _pi64 = ctypes.POINTER(_c_i64)
        L.fasq_pq_gemv_batched.argtypes = [_c_vp, _c_i64, _c_i64, _c_int, _pp, _pi64, _pp, _pi64, _pp, _c_int,
                                           _c_int, _c_vp]
        L.fasq_pq_gemv_batched.restype = _c_int
        L.fasq_pq_reconstruct.argtypes = [_c_vp, _c_i64, _c_i64, _c_int, _c_int, _c_vp, _c_i64, _c_vp, _c_vp]
        L.fasq_pq_reconstruct.restype = _c_int
        L.fasq_idx_row_bytes.argtypes = [_c_i64, _c_int, _c_int]
        L.fasq_idx_row_bytes.restype = _c_i64
        L.fasq_status_string.argtypes = [_c_int]
        L.fasq_status_string.restype = ctypes.c_char_p
        L.fasq_last_error.argtypes = []
        L.fasq_last_error.restype = ctypes.c_char_p
        L.fasq_abi_version.argtypes = []
        L.fasq_abi_version.restype = _c_int
        L.fasq_pq_plan.argtypes = [_c_int, _c_i64, _c_i64, _c_i64, _c_int, _c_int, _c_i64]
        L.fasq_pq_plan.restype = ctypes.c_char_p
        L.fasq_pq_encode.argtypes = [_c_vp, _c_i64, _c_i64, _c_int, _c_i64, _c_int, _c_vp, _c_int, _c_vp, _c_vp,
                                     _c_vp, _c_i64, _c_vp]
        L.fasq_pq_encode.restype = _c_int
        L.fasq_pq_encode_workspace_bytes.argtypes = [_c_i64, _c_i64, _c_int, _c_i64]
        L.fasq_pq_encode_workspace_bytes.restype = _c_i64
        L.fasq_pq_gemv_ex.argtypes = [_c_vp, _c_i64, _c_i64, _c_i64, _c_vp, _c_int, _c_int, _c_vp, _c_i64, _c_i64,
                                      _c_vp, _c_vp, _c_i64, _c_vp]
        L.fasq_pq_gemv_ex.restype = _c_int
        L.fasq_pq_gemv_ex_workspace_bytes.argtypes = [_c_i64, _c_i64, _c_i64, _c_int, _c_int, _c_i64, _c_i64]
        L.fasq_pq_gemv_ex_workspace_bytes.restype = _c_i64
        L.fasq_pq_gemm_ex.argtypes = [_c_vp, _c_i64, _c_i64, _c_i64, _c_vp, _c_int, _c_int, _c_vp, _c_i64, _c_vp,
                                      _c_vp, _c_i64, _c_vp]
        L.fasq_pq_gemm_ex.restype = _c_int
        L.fasq_pq_gemm_ex_workspace_bytes.argtypes = [_c_i64, _c_i64, _c_i64, _c_int, _c_int, _c_i64]
        L.fasq_pq_gemm_ex_workspace_bytes.restype = _c_i64
        L.fasq_pq_gemv_ex_noalloc.argtypes = [_c_vp, _c_i64, _c_i64, _c_i64, _c_vp, _c_int, _c_int, _c_vp, _c_i64,
                                              _c_i64, _c_vp, _c_vp]
        L.fasq_pq_gemv_ex_noalloc.restype = _c_int
        L.fasq_noalloc_scratch_bytes.argtypes = []
        L.fasq_noalloc_scratch_bytes.restype = _c_i64
        L.fasq_launch_list_create.argtypes = [ctypes.POINTER(_c_vp)]
        L.fasq_launch_list_create.restype = _c_int
        for name in ("fasq_launch_list_begin", "fasq_launch_list_end"):
            getattr(L, name).argtypes = [_c_vp]
            getattr(L, name).restype = _c_int
        L.fasq_launch_list_run.argtypes = [_c_vp, _c_vp]
        L.fasq_launch_list_run.restype = _c_int
        L.fasq_launch_list_size.argtypes = [_c_vp]
        L.fasq_launch_list_size.restype = _c_i64
        L.fasq_launch_list_destroy.argtypes = [_c_vp]
        L.fasq_launch_list_destroy.restype = None
        _lib = L
        return L


def library_loaded() -> bool:
    return _lib is not None


def abi_version() -> int:
    return lib().fasq_abi_version()


def idx_row_bytes(K: int, d: int, idx_bits: int) -> int:
    return lib().fasq_idx_row_bytes(K, d, idx_bits)


def plan(regime: str, M: int, K: int, N: int, idx_bits: int, d: int, C: int) -> str:
    """Kernel instantiation a call would launch: regime "gemv", "gemm", or
    "gemv_batched" (a grouped decode launch over several matrices of these
    sizes)."""
    code = {"gemv": 0, "gemm": 1, "gemv_batched": 2}[regime]
    return lib().fasq_pq_plan(code, M, K, N, idx_bits, d, C).decode()


def status_string(status: int) -> str:
    return lib().fasq_status_string(status).decode()


def last_error() -> str:
    return lib().fasq_last_error().decode()


def _check(status: int) -> None:
    if status != FASQ_OK:
        raise FasqError(status, f"{status_string(status)}: {last_error()}")


# ---------------------------------------------------------------------------
# Raw-pointer entry points (integers are device addresses; stream 0 = null)
# ---------------------------------------------------------------------------

def gemv_raw(x, M, K, N, idx, idx_bits, d, codebook, C, y, stream=0) -> int:
    return lib().fasq_pq_gemv(x, M, K, N, idx, idx_bits, d, codebook, C, y, stream)


def gemm_raw(x, M, K, N, idx, idx_bits, d, codebook, C, y, stream=0) -> int:
    return lib().fasq_pq_gemm(x, M, K, N, idx, idx_bits, d, codebook, C, y, stream)


def gemv_batched_raw(x, M, K, idx, N, codebook, C, y, idx_bits, d, stream=0) -> int:
    """``idx``, ``N``, ``codebook``, ``C`` and ``y`` are equal-length sequences of
    integers (device addresses, sizes); they are marshalled into host arrays."""
    n = len(idx)
    if not (len(N) == len(codebook) == len(C) == len(y) == n):
        raise ValueError("the matrix sequences must have equal lengths")
    arr_p = _c_vp * max(n, 1)
    arr_i = _c_i64 * max(n, 1)
    return lib().fasq_pq_gemv_batched(x, M, K, n, arr_p(*idx), arr_i(*N), arr_p(*codebook), arr_i(*C),
                                      arr_p(*y), idx_bits, d, stream)


def reconstruct_raw(idx, N, K, idx_bits, d, codebook, C, w, stream=0) -> int:
    return lib().fasq_pq_reconstruct(idx, N, K, idx_bits, d, codebook, C, w, stream)


# ---------------------------------------------------------------------------
# Torch-tensor entry points
# ---------------------------------------------------------------------------

def _torch():
    import torch

    return torch


def _stream_handle(tensor) -> int:
    torch = _torch()
    return torch.cuda.current_stream(tensor.device).cuda_stream


def _require(t, name, dtype, ndim):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.dim() != ndim:
        raise ValueError(f"{name} must be {ndim}-D")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _matmul(fn, x, idx, idx_bits, d, codebook, out=None):
    torch = _torch()
    _require(x, "x", torch.float16, 2)
    _require(idx, "idx", torch.uint8, 2)
    _require(codebook, "codebook", torch.float16, 2)
    M, K = x.shape
    N, R = idx.shape
    C, dd = codebook.shape
    if dd != d:
        raise ValueError(f"codebook is [C x {dd}] but d = {d}")
    want = idx_row_bytes(K, d, idx_bits)
    if want < 0:
        raise ValueError("invalid (K, d, idx_bits)")
    if R != want:
        raise ValueError(f"idx rows are {R} bytes, expected {want}")
    if out is None:
        out = torch.empty((M, N), dtype=torch.float16, device=x.device)
    else:
        _require(out, "out", torch.float16, 2)
        if tuple(out.shape) != (M, N):
            raise ValueError("out must be [M x N]")
    for t in (idx, codebook, out):
        if t.device != x.device:
            raise ValueError("all tensors must be on one device")
    with torch.cuda.device(x.device):
        _check(fn(x.data_ptr(), M, K, N, idx.data_ptr(), idx_bits, d, codebook.data_ptr(), C,
                  out.data_ptr(), _stream_handle(x)))
    return out


def pq_gemv(x, idx, idx_bits: int, d: int, codebook, out=None):
    """Decode-regime ``y = x . W_hat^T`` (fp16 [M x N]); see ``fasq_pq_gemv``."""
    return _matmul(lib().fasq_pq_gemv, x, idx, idx_bits, d, codebook, out)


def pq_gemm(x, idx, idx_bits: int, d: int, codebook, out=None):
    """Prefill-regime ``y = x . W_hat^T`` (MFMA path); see ``fasq_pq_gemm``."""
    return _matmul(lib().fasq_pq_gemm, x, idx, idx_bits, d, codebook, out)


def pq_gemm_lut(x, idx, idx_bits: int, d: int, codebook, out=None):
    """``y = x . W_hat^T`` with the paper's lookup-table GEMM design (for
    comparison); see ``fasq_pq_gemm_lut``."""
    return _matmul(lib().fasq_pq_gemm_lut, x, idx, idx_bits, d, codebook, out)


def gemm_lut_raw(x, M, K, N, idx, idx_bits, d, codebook, C, y, stream=0) -> int:
    return lib().fasq_pq_gemm_lut(x, M, K, N, idx, idx_bits, d, codebook, C, y, stream)


def pq_gemv_batched(x, idxs, idx_bits: int, d: int, codebooks, outs=None):
    """Decode-regime ``y_i = x . W_hat_i^T`` for several matrices sharing x;
    see ``fasq_pq_gemv_batched``.  Returns the list of outputs."""
    torch = _torch()
    _require(x, "x", torch.float16, 2)
    M, K = x.shape
    if len(idxs) != len(codebooks) or (outs is not None and len(outs) != len(idxs)):
        raise ValueError("idxs, codebooks and outs must have equal lengths")
    want = idx_row_bytes(K, d, idx_bits)
    if want < 0:
        raise ValueError("invalid (K, d, idx_bits)")
    ys = []
    for i, (idx, cb) in enumerate(zip(idxs, codebooks)):
        _require(idx, f"idx[{i}]", torch.uint8, 2)
        _require(cb, f"codebook[{i}]", torch.float16, 2)
        if cb.shape[1] != d:
            raise ValueError(f"codebook[{i}] is [C x {cb.shape[1]}] but d = {d}")
        if idx.shape[1] != want:
            raise ValueError(f"idx[{i}] rows are {idx.shape[1]} bytes, expected {want}")
        if outs is None:
            y = torch.empty((M, idx.shape[0]), dtype=torch.float16, device=x.device)
        else:
            y = outs[i]
            _require(y, f"out[{i}]", torch.float16, 2)
            if tuple(y.shape) != (M, idx.shape[0]):
                raise ValueError(f"out[{i}] must be [M x N]")
        for t in (idx, cb, y):
            if t.device != x.device:
                raise ValueError("all tensors must be on one device")
        ys.append(y)
    with torch.cuda.device(x.device):
        _check(gemv_batched_raw(x.data_ptr(), M, K, [t.data_ptr() for t in idxs], [t.shape[0] for t in idxs],
                                [t.data_ptr() for t in codebooks], [t.shape[0] for t in codebooks],
                                [t.data_ptr() for t in ys], idx_bits, d, _stream_handle(x)))
    return ys


def pq_reconstruct(idx, K: int, idx_bits: int, d: int, codebook, out=None):
    """Explicit ``W_hat`` (fp16 [N x K]), bit copies of codebook entries."""
    torch = _torch()
    _require(idx, "idx", torch.uint8, 2)
    _require(codebook, "codebook", torch.float16, 2)
    N, R = idx.shape
    C, dd = codebook.shape
    if dd != d:
        raise ValueError(f"codebook is [C x {dd}] but d = {d}")
    want = idx_row_bytes(K, d, idx_bits)
    if want < 0 or R != want:
        raise ValueError(f"idx rows are {R} bytes, expected {want}")
    if out is None:
        out = torch.empty((N, K), dtype=torch.float16, device=idx.device)
    else:
        _require(out, "out", torch.float16, 2)
        if tuple(out.shape) != (N, K):
            raise ValueError("out must be [N x K]")
    with torch.cuda.device(idx.device):
        _check(lib().fasq_pq_reconstruct(idx.data_ptr(), N, K, idx_bits, d, codebook.data_ptr(), C,
                                         out.data_ptr(), _stream_handle(idx)))
    return out


def encode_workspace_bytes(N: int, K: int, d: int, C: int) -> int:
    return lib().fasq_pq_encode_workspace_bytes(N, K, d, C)


def encode_raw(w, N, K, d, C, idx_bits, init_codebook, iters, codebook, idx, workspace, workspace_bytes,
               stream=0) -> int:
    return lib().fasq_pq_encode(w, N, K, d, C, idx_bits, init_codebook, iters, codebook, idx, workspace,
                                workspace_bytes, stream)


def pq_encode(w, d: int, idx_bits: int, init_codebook, iters: int, workspace=None):
    """k-means PQ encoding of dense fp16 weights ``w`` [N x K] with the
    starting codebook ``init_codebook`` (fp16 [C x d]); see ``fasq_pq_encode``.
    Returns ``(codebook, idx)``: fp16 [C x d] and uint8 [N x R] device tensors."""
    torch = _torch()
    _require(w, "w", torch.float16, 2)
    _require(init_codebook, "init_codebook", torch.float16, 2)
    N, K = w.shape
    C, dd = init_codebook.shape
    if dd != d:
        raise ValueError(f"init_codebook is [C x {dd}] but d = {d}")
    R = idx_row_bytes(K, d, idx_bits)
    if R < 0:
        raise ValueError("invalid (K, d, idx_bits)")
    need = encode_workspace_bytes(N, K, d, C)
    if need < 0:
        raise ValueError("invalid encoder sizes")
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=w.device)
    elif not (workspace.is_cuda and workspace.is_contiguous() and workspace.numel() * workspace.element_size() >= need):
        raise ValueError(f"workspace must be a contiguous device tensor of at least {need} bytes")
    if init_codebook.device != w.device or workspace.device != w.device:
        raise ValueError("all tensors must be on one device")
    codebook = torch.empty((C, d), dtype=torch.float16, device=w.device)
    idx = torch.empty((N, R), dtype=torch.uint8, device=w.device)
    with torch.cuda.device(w.device):
        _check(encode_raw(w.data_ptr(), N, K, d, C, idx_bits, init_codebook.data_ptr(), iters, codebook.data_ptr(),
                          idx.data_ptr(), workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                          _stream_handle(w)))
    return codebook, idx


def gemv_ex_workspace_bytes(M: int, K: int, N: int, idx_bits: int, d: int, C: int, cb_stride: int) -> int:
    return lib().fasq_pq_gemv_ex_workspace_bytes(M, K, N, idx_bits, d, C, cb_stride)


def gemv_ex_raw(x, M, K, N, idx, idx_bits, d, codebook, C, cb_stride, y, workspace, workspace_bytes, stream=0) -> int:
    return lib().fasq_pq_gemv_ex(x, M, K, N, idx, idx_bits, d, codebook, C, cb_stride, y, workspace,
                                 workspace_bytes, stream)


def gemv_ex_noalloc_raw(x, M, K, N, idx, idx_bits, d, codebook, C, cb_stride, y, stream=0) -> int:
    return lib().fasq_pq_gemv_ex_noalloc(x, M, K, N, idx, idx_bits, d, codebook, C, cb_stride, y, stream)


def noalloc_scratch_bytes() -> int:
    return lib().fasq_noalloc_scratch_bytes()


def pq_gemv_ex(x, idx, idx_bits: int, d: int, codebook, out=None, workspace=None):
    """Decode-regime ``y = x . W_hat^T`` with per-subspace codebooks
    (``codebook`` fp16 [S x C x d]) or one shared codebook ([C x d]); see
    ``fasq_pq_gemv_ex``."""
    torch = _torch()
    _require(x, "x", torch.float16, 2)
    _require(idx, "idx", torch.uint8, 2)
    if not isinstance(codebook, torch.Tensor) or codebook.dim() not in (2, 3):
        raise ValueError("codebook must be [C x d] or [S x C x d]")
    _require(codebook, "codebook", torch.float16, codebook.dim())
    M, K = x.shape
    N, R = idx.shape
    if codebook.shape[-1] != d:
        raise ValueError(f"codebook entries have {codebook.shape[-1]} values but d = {d}")
    C = codebook.shape[-2]
    if codebook.dim() == 3:
        if codebook.shape[0] != K // d:
            raise ValueError(f"per-subspace codebook has {codebook.shape[0]} books, expected K / d = {K // d}")
        stride = C * d
    else:
        stride = 0
    want = idx_row_bytes(K, d, idx_bits)
    if want < 0 or R != want:
        raise ValueError(f"idx rows are {R} bytes, expected {want}")
    if out is None:
        out = torch.empty((M, N), dtype=torch.float16, device=x.device)
    else:
        _require(out, "out", torch.float16, 2)
        if tuple(out.shape) != (M, N):
            raise ValueError("out must be [M x N]")
    need = gemv_ex_workspace_bytes(M, K, N, idx_bits, d, C, stride)
    if need < 0:
        raise ValueError("invalid sizes")
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=x.device)
    ws_ptr = workspace.data_ptr() if workspace is not None else 0
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    for t in (idx, codebook, out):
        if t.device != x.device:
            raise ValueError("all tensors must be on one device")
    with torch.cuda.device(x.device):
        _check(gemv_ex_raw(x.data_ptr(), M, K, N, idx.data_ptr(), idx_bits, d, codebook.data_ptr(), C, stride,
                           out.data_ptr(), ws_ptr, ws_bytes, _stream_handle(x)))
    return out


def gemm_ex_workspace_bytes(M: int, K: int, N: int, idx_bits: int, d: int, C: int) -> int:
    return lib().fasq_pq_gemm_ex_workspace_bytes(M, K, N, idx_bits, d, C)


def gemm_ex_raw(x, M, K, N, idx, idx_bits, d, codebook, C, y, workspace, workspace_bytes, stream=0) -> int:
    return lib().fasq_pq_gemm_ex(x, M, K, N, idx, idx_bits, d, codebook, C, y, workspace, workspace_bytes, stream)


def pq_gemm_ex(x, idx, idx_bits: int, d: int, codebook, out=None, workspace=None):
    """Prefill-regime ``y = x . W_hat^T`` that may also split K over
    workgroups, with a workspace for the partial sums (allocated here when
    not given); see ``fasq_pq_gemm_ex``."""
    torch = _torch()
    _require(x, "x", torch.float16, 2)
    M, K = x.shape
    N = idx.shape[0] if isinstance(idx, torch.Tensor) and idx.dim() == 2 else 0
    C = codebook.shape[0] if isinstance(codebook, torch.Tensor) and codebook.dim() == 2 else 0
    need = gemm_ex_workspace_bytes(M, K, N, idx_bits, d, C) if N and C else 0
    if need < 0:
        raise ValueError("invalid sizes")
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=x.device)
    ws_ptr = workspace.data_ptr() if workspace is not None else 0
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0

    def call(xp, M_, K_, N_, ip, bits, dd, cp, C_, yp, stream):
        return lib().fasq_pq_gemm_ex(xp, M_, K_, N_, ip, bits, dd, cp, C_, yp, ws_ptr, ws_bytes, stream)

    return _matmul(call, x, idx, idx_bits, d, codebook, out)


# ---------------------------------------------------------------------------
# Launch lists
# ---------------------------------------------------------------------------

class LaunchList:
    """The kernel launches of a sequence of fasq calls, recorded once and
    queued again with :meth:`run` (``fasq_launch_list_*``).

    Calls made on this thread inside ``with lst:`` (or between :meth:`begin`
    and :meth:`end`) are checked and planned as usual but only recorded; the
    buffers they name must stay alive while the list may run.
    """

    def __init__(self):
        h = _c_vp()
        _check(lib().fasq_launch_list_create(ctypes.byref(h)))
        self._h = h

    @property
    def handle(self) -> int:
        """The ``fasq_launch_list*`` (0 once closed)."""
        return (self._h.value or 0) if self._h is not None else 0

    def begin(self) -> None:
        _check(lib().fasq_launch_list_begin(self._live()))

    def end(self) -> None:
        _check(lib().fasq_launch_list_end(self._live()))

    def __enter__(self) -> "LaunchList":
        self.begin()
        return self

    def __exit__(self, *exc) -> bool:
        self.end()
        return False

    def run(self, stream=None) -> None:
        """Queue the recorded launches on ``stream`` (an integer HIP stream
        handle, a torch stream, or None for torch's current stream)."""
        if stream is None:
            stream = _torch().cuda.current_stream().cuda_stream
        elif not isinstance(stream, int):
            stream = stream.cuda_stream
        _check(lib().fasq_launch_list_run(self._live(), stream))

    def __len__(self) -> int:
        return int(lib().fasq_launch_list_size(self._live()))

    def close(self) -> None:
        if self._h is not None and self._h.value:
            lib().fasq_launch_list_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _live(self):
        if self._h is None or not self._h.value:
            raise ValueError("the launch list is closed")
        return self._h
