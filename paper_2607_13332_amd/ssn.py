"""Thin ctypes binding over libssn.so (the C ABI declared in include/ssn.h).

Argument marshalling only: dtype / shape / device checks on torch tensors,
device pointers and the current HIP stream go to the C entry points, and every
step of the computation runs in the library's HIP kernels.  There is no
fallback: if libssn.so is missing or a call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libssn.so")

SSN_F32, SSN_BF16 = 0, 1
OPS = {"compress": 0, "decompress": 1, "project_grad": 2, "project_weights": 3,
       "compress_projected": 4}
MAX_BATCH = 16
NOALLOC_SCRATCH_BYTES = 32 << 20
SPARTA_MAX_SENDERS = 64

_c_i64 = ctypes.c_int64
_c_p = ctypes.c_void_p


class SSNError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn} failed with status {status} ({msg})")
        self.status = status


def _declare(lib):
    lib.ssn_abi_version.restype = ctypes.c_int
    lib.ssn_abi_version.argtypes = []
    lib.ssn_status_string.restype = ctypes.c_char_p
    lib.ssn_status_string.argtypes = [ctypes.c_int]
    lib.ssn_kernel_family.restype = ctypes.c_char_p
    lib.ssn_kernel_family.argtypes = [ctypes.c_int, ctypes.c_int, _c_i64, _c_i64]
    lib.ssn_compress.restype = ctypes.c_int
    lib.ssn_compress.argtypes = [ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_i64,
                                 _c_p, _c_p, _c_p, _c_p, _c_p, _c_p]
    lib.ssn_decompress.restype = ctypes.c_int
    lib.ssn_decompress.argtypes = [ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_i64,
                                   _c_p, _c_p, _c_p, _c_p, _c_p, _c_p]
    lib.ssn_project_grad.restype = ctypes.c_int
    lib.ssn_project_grad.argtypes = [ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_p, _c_p]
    lib.ssn_compress_ex.restype = ctypes.c_int
    lib.ssn_compress_ex.argtypes = [ctypes.c_int, ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_i64,
                                    _c_p, _c_p, _c_p, _c_p, _c_i64, _c_p, _c_p]
    lib.ssn_decompress_ex.restype = ctypes.c_int
    lib.ssn_decompress_ex.argtypes = [ctypes.c_int, ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_i64,
                                      _c_p, _c_p, _c_p, _c_p, _c_i64, _c_p, _c_p]
    lib.ssn_project_grad_ex.restype = ctypes.c_int
    lib.ssn_project_grad_ex.argtypes = [ctypes.c_int, ctypes.c_int, _c_i64, _c_i64, _c_i64,
                                        _c_p, _c_p, _c_i64, _c_p, _c_p]
    lib.ssn_project_grad_workspace_bytes.restype = ctypes.c_size_t
    lib.ssn_project_grad_workspace_bytes.argtypes = [ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_i64]
    lib.ssn_project_grad_ws.restype = ctypes.c_int
    lib.ssn_project_grad_ws.argtypes = [ctypes.c_int, ctypes.c_int, _c_i64, _c_i64, _c_i64,
                                        _c_p, _c_p, _c_i64, _c_p, _c_p, ctypes.c_size_t, _c_p]
    lib.ssn_compress_projected_ex.restype = ctypes.c_int
    lib.ssn_compress_projected_ex.argtypes = [ctypes.c_int, ctypes.c_int, _c_i64, _c_i64, _c_i64,
                                              _c_i64, _c_p, _c_p, _c_p, _c_p, _c_i64, _c_p, _c_p]
    lib.ssn_check_ids.restype = ctypes.c_int
    lib.ssn_check_ids.argtypes = [_c_i64, _c_i64, _c_p, _c_p, _c_p]
    lib.ssn_pad_basis.restype = ctypes.c_int
    lib.ssn_pad_basis.argtypes = [ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_p]
    lib.ssn_project_table.restype = ctypes.c_int
    lib.ssn_project_table.argtypes = [ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_p, _c_p]
    lib.ssn_compress_projected.restype = ctypes.c_int
    lib.ssn_compress_projected.argtypes = [ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_i64,
                                           _c_p, _c_p, _c_p, _c_p, _c_p, _c_p]
    lib.ssn_reparam_forward.restype = ctypes.c_int
    lib.ssn_reparam_forward.argtypes = [ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_i64,
                                        _c_p, _c_p, _c_p, _c_p, _c_p, _c_p]
    lib.ssn_reparam_workspace_bytes.restype = ctypes.c_size_t
    lib.ssn_reparam_workspace_bytes.argtypes = [ctypes.c_int, _c_i64, _c_i64, _c_i64]
    lib.ssn_reparam_backward.restype = ctypes.c_int
    lib.ssn_reparam_backward.argtypes = [ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_i64,
                                         _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p,
                                         ctypes.c_size_t, _c_p]
    lib.ssn_reparam_backward_noalloc.restype = ctypes.c_int
    lib.ssn_reparam_backward_noalloc.argtypes = [ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_i64,
                                                 _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p]
    lib.ssn_factored_embedding.restype = ctypes.c_int
    lib.ssn_factored_embedding.argtypes = [ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_i64,
                                           _c_p, _c_p, _c_p, _c_p, _c_p]
    lib.ssn_project_weights_workspace_bytes.restype = ctypes.c_size_t
    lib.ssn_project_weights_workspace_bytes.argtypes = [_c_i64, _c_i64, _c_i64]
    lib.ssn_project_weights.restype = ctypes.c_int
    lib.ssn_project_weights.argtypes = [ctypes.c_int, _c_i64, _c_i64, _c_i64, _c_p, _c_p, _c_p,
                                        ctypes.c_size_t, _c_p]
    lib.ssn_sparta_segment.restype = ctypes.c_int
    lib.ssn_sparta_segment.argtypes = [_c_i64, _c_i64, _c_i64, ctypes.POINTER(_c_i64),
                                       ctypes.POINTER(_c_i64)]
    lib.ssn_sparta_snapshot.restype = ctypes.c_int
    lib.ssn_sparta_snapshot.argtypes = [_c_i64, _c_i64, _c_p, _c_i64, _c_p, _c_p, _c_p]
    lib.ssn_sparta_average.restype = ctypes.c_int
    lib.ssn_sparta_average.argtypes = [_c_i64, _c_i64, ctypes.POINTER(_c_p),
                                       ctypes.POINTER(ctypes.c_float), _c_p,
                                       ctypes.POINTER(_c_p), _c_p]
    lib.ssn_delta_rule.restype = ctypes.c_int
    lib.ssn_delta_rule.argtypes = [_c_i64, _c_i64, _c_p, _c_i64, _c_p, _c_p, _c_p,
                                   ctypes.c_float, _c_p]
    lib.ssn_project_weights_batched.restype = ctypes.c_int
    lib.ssn_project_weights_batched.argtypes = [ctypes.c_int, _c_i64, _c_i64,
                                                ctypes.POINTER(_c_i64), _c_i64,
                                                ctypes.POINTER(_c_p), _c_p, _c_p]
    return lib


_lib = None


def lib():
    """The loaded C library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2607_13332_amd.build`")
        _lib = _declare(ctypes.CDLL(LIB_PATH))
    return _lib


def status_string(status: int) -> str:
    return lib().ssn_status_string(status).decode()


def kernel_family(op: str, dtype, d: int, k: int) -> str:
    return lib().ssn_kernel_family(OPS[op], _dt_code(dtype), d, k).decode()


def _check(fn: str, status: int):
    if status != 0:
        raise SSNError(fn, status, status_string(status))


def _dt_code(dtype) -> int:
    if dtype in (torch.bfloat16, "bf16", SSN_BF16):
        return SSN_BF16
    if dtype in (torch.float32, "f32", SSN_F32):
        return SSN_F32
    raise TypeError(f"unsupported storage dtype {dtype}")


_raw_current_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)


def _stream(stream) -> int:
    """hipStream_t of `stream`, or of the current stream of the current device."""
    if stream is None:
        if _raw_current_stream is not None:
            # the raw handle directly (torch.cuda.current_stream() builds a
            # Stream object per call, a few microseconds)
            return int(_raw_current_stream(torch.cuda.current_device()))
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


def _dev(t: torch.Tensor, name: str, dtype=None, ndim=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor (the codec has no CPU path)")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims, got shape {tuple(t.shape)}")
    return t.data_ptr()


def _same_device(*ts):
    devs = {t.device for t in ts if t is not None}
    if len(devs) > 1:
        raise ValueError(f"tensors are on different devices: {devs}")


def compress(X: torch.Tensor, ids: torch.Tensor, E: torch.Tensor, U: torch.Tensor,
             out: Optional[torch.Tensor] = None, stream=None,
             z_dtype: torch.dtype = torch.float32, k: Optional[int] = None) -> torch.Tensor:
    """Z = (X - E[ids]) U  ([N, k] in z_dtype: float32, or bfloat16 rounded once).
    k < U.shape[1]: U is a zero-padded basis whose first k columns are used."""
    N, d = X.shape
    V, ldu = E.shape[0], U.shape[1]
    k = ldu if k is None else int(k)
    if E.shape[1] != d or U.shape[0] != d or ids.shape != (N,):
        raise ValueError(f"shape mismatch X{tuple(X.shape)} ids{tuple(ids.shape)} "
                         f"E{tuple(E.shape)} U{tuple(U.shape)}")
    if out is None:
        out = torch.empty((N, k), dtype=z_dtype, device=X.device)
    _same_device(X, ids, E, U, out)
    t = X.dtype
    _check("ssn_compress_ex", lib().ssn_compress_ex(
        _dt_code(t), _dt_code(z_dtype), N, d, k, V, _dev(X, "X", t, 2),
        _dev(ids, "ids", torch.int32, 1), _dev(E, "E", t, 2), _dev(U, "U", t, 2), ldu,
        _dev(out, "out", z_dtype, 2), _stream(stream)))
    return out


def decompress(Z: torch.Tensor, ids: Optional[torch.Tensor], E: Optional[torch.Tensor],
               U: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """X' = E[ids] + Z U^T (storage dtype of U); with ids = E = None, Z U^T.
    Z is float32 or bfloat16 (the coordinate dtype on the wire); U may be a
    zero-padded basis with more columns than Z."""
    N, k = Z.shape
    d, ldu = U.shape
    if ldu < k:
        raise ValueError(f"shape mismatch Z{tuple(Z.shape)} U{tuple(U.shape)}")
    if (E is None) != (ids is None):
        raise ValueError("pass both ids and E, or neither")
    t = U.dtype
    V = 0
    if E is not None:
        V = E.shape[0]
        if E.shape[1] != d or ids.shape != (N,):
            raise ValueError(f"shape mismatch E{tuple(E.shape)} ids{tuple(ids.shape)}")
    if out is None:
        out = torch.empty((N, d), dtype=t, device=Z.device)
    _same_device(Z, ids, E, U, out)
    _check("ssn_decompress_ex", lib().ssn_decompress_ex(
        _dt_code(t), _dt_code(Z.dtype), N, d, k, V, _dev(Z, "Z", Z.dtype, 2),
        None if ids is None else _dev(ids, "ids", torch.int32, 1),
        None if E is None else _dev(E, "E", t, 2), _dev(U, "U", t, 2), ldu,
        _dev(out, "out", t, 2), _stream(stream)))
    return out


def expand_grad(GZ: torch.Tensor, U: torch.Tensor, out: Optional[torch.Tensor] = None,
                stream=None) -> torch.Tensor:
    """Sender-side gradient G_Z U^T (decompress without the embedding)."""
    return decompress(GZ, None, None, U, out=out, stream=stream)


def project_grad(G: torch.Tensor, U: torch.Tensor, out: Optional[torch.Tensor] = None,
                 stream=None, z_dtype: torch.dtype = torch.float32,
                 k: Optional[int] = None, workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """G_Z = G U ([N, k] in z_dtype: float32, or bfloat16 rounded once).
    k < U.shape[1]: U is a zero-padded basis whose first k columns are used.
    workspace: a 1-D uint8 device tensor, e.g. from project_grad_workspace()
    (ssn_project_grad_ws: d split into ranges with few tokens)."""
    N, d = G.shape
    ldu = U.shape[1]
    k = ldu if k is None else int(k)
    if U.shape[0] != d:
        raise ValueError(f"shape mismatch G{tuple(G.shape)} U{tuple(U.shape)}")
    if out is None:
        out = torch.empty((N, k), dtype=z_dtype, device=G.device)
    _same_device(G, U, out)
    t = G.dtype
    if workspace is None:
        _check("ssn_project_grad_ex", lib().ssn_project_grad_ex(
            _dt_code(t), _dt_code(z_dtype), N, d, k, _dev(G, "G", t, 2), _dev(U, "U", t, 2), ldu,
            _dev(out, "out", z_dtype, 2), _stream(stream)))
        return out
    _same_device(G, workspace)
    _check("ssn_project_grad_ws", lib().ssn_project_grad_ws(
        _dt_code(t), _dt_code(z_dtype), N, d, k, _dev(G, "G", t, 2), _dev(U, "U", t, 2), ldu,
        _dev(out, "out", z_dtype, 2), _dev(workspace, "workspace", torch.uint8, 1),
        workspace.numel(), _stream(stream)))
    return out


def project_grad_workspace_bytes(N: int, d: int, k: int, ldu: Optional[int] = None,
                                 dtype: torch.dtype = torch.bfloat16) -> int:
    """Workspace size that lets ssn_project_grad_ws split d into every range
    count it may take for this shape (0: no split for this shape)."""
    ldu = k if ldu is None else int(ldu)
    return int(lib().ssn_project_grad_workspace_bytes(_dt_code(dtype), N, d, k, ldu))


def project_grad_workspace(N: int, d: int, k: int, device, ldu: Optional[int] = None,
                           dtype: torch.dtype = torch.bfloat16) -> Optional[torch.Tensor]:
    """A workspace for project_grad(..., workspace=...) at this shape (None
    when the shape takes no split); calls that share it must not overlap."""
    n = project_grad_workspace_bytes(N, d, k, ldu, dtype)
    return torch.empty(n, dtype=torch.uint8, device=device) if n > 0 else None


def check_ids(ids: torch.Tensor, V: int, out: Optional[torch.Tensor] = None,
              stream=None) -> torch.Tensor:
    """Number of ids outside [0, V), counted on the device into a one-element
    int64 tensor (read it after the stream has run)."""
    if ids.dim() != 1:
        raise ValueError(f"ids must be 1-D, got {tuple(ids.shape)}")
    if out is None:
        out = torch.empty((1,), dtype=torch.int64, device=ids.device)
    _same_device(ids, out)
    _check("ssn_check_ids", lib().ssn_check_ids(
        ids.shape[0], int(V), _dev(ids, "ids", torch.int32, 1), _dev(out, "out", torch.int64, 1),
        _stream(stream)))
    return out


def pad_basis(U: torch.Tensor, ldu: Optional[int] = None, out: Optional[torch.Tensor] = None,
              stream=None) -> torch.Tensor:
    """U [d, k] with zero columns appended up to ldu (default: the next
    multiple of 16), the layout the `_ex` entry points read with aligned
    16-byte pieces; pass it with k= to compress / project_grad."""
    d, k = U.shape
    ldu = 16 * ((k + 15) // 16) if ldu is None else int(ldu)
    if out is None:
        out = torch.empty((d, ldu), dtype=U.dtype, device=U.device)
    if out.shape != (d, ldu):
        raise ValueError(f"out has shape {tuple(out.shape)}, expected ({d}, {ldu})")
    _same_device(U, out)
    t = U.dtype
    _check("ssn_pad_basis", lib().ssn_pad_basis(_dt_code(t), d, k, ldu, _dev(U, "U", t, 2),
                                                _dev(out, "out", t, 2), _stream(stream)))
    return out


def project_table(E: torch.Tensor, U: torch.Tensor, out: Optional[torch.Tensor] = None,
                  stream=None) -> torch.Tensor:
    """P = E U (float32 [V, k]): the fixed embedding table, projected once."""
    V, d = E.shape
    k = U.shape[1]
    if U.shape[0] != d:
        raise ValueError(f"shape mismatch E{tuple(E.shape)} U{tuple(U.shape)}")
    if out is None:
        out = torch.empty((V, k), dtype=torch.float32, device=E.device)
    _same_device(E, U, out)
    t = E.dtype
    _check("ssn_project_table", lib().ssn_project_table(
        _dt_code(t), V, d, k, _dev(E, "E", t, 2), _dev(U, "U", t, 2),
        _dev(out, "out", torch.float32, 2), _stream(stream)))
    return out


def compress_projected(X: torch.Tensor, ids: torch.Tensor, P: torch.Tensor, U: torch.Tensor,
                       out: Optional[torch.Tensor] = None, stream=None,
                       z_dtype: torch.dtype = torch.float32) -> torch.Tensor:
    """Z = X U - P[ids] ([N, k] in z_dtype), with P from project_table(E, U)."""
    N, d = X.shape
    V, k = P.shape
    ldu = U.shape[1]
    if U.shape[0] != d or ldu < k or ids.shape != (N,):
        raise ValueError(f"shape mismatch X{tuple(X.shape)} ids{tuple(ids.shape)} "
                         f"P{tuple(P.shape)} U{tuple(U.shape)}")
    if out is None:
        out = torch.empty((N, k), dtype=z_dtype, device=X.device)
    _same_device(X, ids, P, U, out)
    t = X.dtype
    _check("ssn_compress_projected_ex", lib().ssn_compress_projected_ex(
        _dt_code(t), _dt_code(z_dtype), N, d, k, V, _dev(X, "X", t, 2),
        _dev(ids, "ids", torch.int32, 1), _dev(P, "P", torch.float32, 2), _dev(U, "U", t, 2),
        ldu, _dev(out, "out", z_dtype, 2), _stream(stream)))
    return out


def reparam_forward(H: torch.Tensor, Zp: torch.Tensor, U: torch.Tensor, T=None, Y=None,
                    stream=None):
    """Reparameterized projection: T = H Zp (float32 [N, k]), Y = T U^T
    (storage dtype [N, d]).  Returns (T, Y)."""
    N, din = H.shape
    d, k = U.shape
    if Zp.shape != (din, k):
        raise ValueError(f"shape mismatch H{tuple(H.shape)} Zp{tuple(Zp.shape)} U{tuple(U.shape)}")
    t = H.dtype
    if T is None:
        T = torch.empty((N, k), dtype=torch.float32, device=H.device)
    if Y is None:
        Y = torch.empty((N, d), dtype=t, device=H.device)
    _same_device(H, Zp, U, T, Y)
    _check("ssn_reparam_forward", lib().ssn_reparam_forward(
        _dt_code(t), N, din, d, k, _dev(H, "H", t, 2), _dev(Zp, "Zp", t, 2), _dev(U, "U", t, 2),
        _dev(T, "T", torch.float32, 2), _dev(Y, "Y", t, 2), _stream(stream)))
    return T, Y


def reparam_workspace_bytes(dtype, N: int, din: int, k: int) -> int:
    return int(lib().ssn_reparam_workspace_bytes(_dt_code(dtype), N, din, k))


def reparam_backward(H: torch.Tensor, Zp: torch.Tensor, U: torch.Tensor, G: torch.Tensor,
                     GT=None, GH=None, GZp=None, workspace=None, stream=None):
    """Gradients for G = dL/dY: GT = G U, GH = (G U) Zp^T, GZp = H^T (G U).
    Returns (GT, GH, GZp)."""
    N, din = H.shape
    d, k = U.shape
    if Zp.shape != (din, k) or G.shape != (N, d):
        raise ValueError(f"shape mismatch H{tuple(H.shape)} Zp{tuple(Zp.shape)} U{tuple(U.shape)} "
                         f"G{tuple(G.shape)}")
    t = H.dtype
    dev = H.device
    if GT is None:
        GT = torch.empty((N, k), dtype=torch.float32, device=dev)
    if GH is None:
        GH = torch.empty((N, din), dtype=t, device=dev)
    if GZp is None:
        GZp = torch.empty((din, k), dtype=torch.float32, device=dev)
    need = reparam_workspace_bytes(t, N, din, k)
    if workspace is None:
        workspace = torch.empty((max(need, 4) + 3) // 4, dtype=torch.float32, device=dev)
    _same_device(H, Zp, U, G, GT, GH, GZp, workspace)
    _check("ssn_reparam_backward", lib().ssn_reparam_backward(
        _dt_code(t), N, din, d, k, _dev(H, "H", t, 2), _dev(Zp, "Zp", t, 2), _dev(U, "U", t, 2),
        _dev(G, "G", t, 2), _dev(GT, "GT", torch.float32, 2), _dev(GH, "GH", t, 2),
        _dev(GZp, "GZp", torch.float32, 2), _dev(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), _stream(stream)))
    return GT, GH, GZp


def reparam_backward_noalloc(H: torch.Tensor, Zp: torch.Tensor, U: torch.Tensor, G: torch.Tensor,
                             GT: torch.Tensor, GH: torch.Tensor, GZp: torch.Tensor, stream=None):
    """reparam_backward with the library's own scratch memory: the caller
    passes every output, and the call allocates nothing on the device."""
    N, din = H.shape
    d, k = U.shape
    if Zp.shape != (din, k) or G.shape != (N, d) or GT.shape != (N, k) or GH.shape != (N, din) \
            or GZp.shape != (din, k):
        raise ValueError(f"shape mismatch H{tuple(H.shape)} Zp{tuple(Zp.shape)} U{tuple(U.shape)} "
                         f"G{tuple(G.shape)} GT{tuple(GT.shape)} GH{tuple(GH.shape)} "
                         f"GZp{tuple(GZp.shape)}")
    t = H.dtype
    _same_device(H, Zp, U, G, GT, GH, GZp)
    _check("ssn_reparam_backward_noalloc", lib().ssn_reparam_backward_noalloc(
        _dt_code(t), N, din, d, k, _dev(H, "H", t, 2), _dev(Zp, "Zp", t, 2), _dev(U, "U", t, 2),
        _dev(G, "G", t, 2), _dev(GT, "GT", torch.float32, 2), _dev(GH, "GH", t, 2),
        _dev(GZp, "GZp", torch.float32, 2), _stream(stream)))
    return GT, GH, GZp


def factored_embedding(ids: torch.Tensor, E: torch.Tensor, U: torch.Tensor,
                       out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """X0 = E[ids] U^T for the factored embedding E [V, k] (float32)."""
    (N,) = ids.shape
    V, k = E.shape
    d = U.shape[0]
    if U.shape[1] != k:
        raise ValueError(f"shape mismatch E{tuple(E.shape)} U{tuple(U.shape)}")
    t = U.dtype
    if out is None:
        out = torch.empty((N, d), dtype=t, device=U.device)
    _same_device(ids, E, U, out)
    _check("ssn_factored_embedding", lib().ssn_factored_embedding(
        _dt_code(t), N, d, k, V, _dev(ids, "ids", torch.int32, 1), _dev(E, "E", torch.float32, 2),
        _dev(U, "U", t, 2), _dev(out, "out", t, 2), _stream(stream)))
    return out


def project_weights_workspace_bytes(d: int, n: int, k: int) -> int:
    return int(lib().ssn_project_weights_workspace_bytes(d, n, k))


def project_weights(W: torch.Tensor, U: torch.Tensor, workspace: Optional[torch.Tensor] = None,
                    stream=None) -> torch.Tensor:
    """In place: W <- U (U^T W) for W [d, n].  `workspace` (device memory of at
    least project_weights_workspace_bytes(d, n, k) bytes) is allocated here
    when it is needed and not given."""
    d, n = W.shape
    k = U.shape[1]
    if U.shape[0] != d:
        raise ValueError(f"shape mismatch W{tuple(W.shape)} U{tuple(U.shape)}")
    need = project_weights_workspace_bytes(d, n, k)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=W.device)
    _same_device(W, U, workspace)
    t = W.dtype
    wptr = None if workspace is None else _dev(workspace, "workspace")
    wbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check("ssn_project_weights", lib().ssn_project_weights(
        _dt_code(t), d, n, k, _dev(W, "W", t, 2), _dev(U, "U", t, 2), wptr, wbytes,
        _stream(stream)))
    return W


def project_weights_batched(Ws: Sequence[torch.Tensor], U: torch.Tensor, stream=None):
    """In place, one launch: W <- U (U^T W) for every W [d, n_b] in Ws."""
    count = len(Ws)
    if not 1 <= count <= MAX_BATCH:
        raise ValueError(f"1 <= len(Ws) <= {MAX_BATCH}")
    d, k = U.shape
    t = U.dtype
    ns = (_c_i64 * count)()
    ps = (_c_p * count)()
    for b, W in enumerate(Ws):
        if W.dim() != 2 or W.shape[0] != d:
            raise ValueError(f"W[{b}] has shape {tuple(W.shape)}, expected ({d}, n)")
        ns[b] = W.shape[1]
        ps[b] = _dev(W, f"W[{b}]", t, 2)
    _same_device(U, *Ws)
    _check("ssn_project_weights_batched", lib().ssn_project_weights_batched(
        _dt_code(t), count, d, ns, k, ps, _dev(U, "U", t, 2), _stream(stream)))
    return Ws


# --------------------------------------------------------------------------
# Sparse weight averaging with the delta rule (section 4.2): float32 master
# weights theta [n]; a round's positions are an int64 list I or a segment.
# --------------------------------------------------------------------------
SPARTA_SEGMENTS = 20


def sparta_segment(n: int, r: int, segments: int = SPARTA_SEGMENTS):
    """(first, m) of the segment averaged in round r (ssn_sparta_segment)."""
    first, m = _c_i64(), _c_i64()
    _check("ssn_sparta_segment", lib().ssn_sparta_segment(n, r, segments, ctypes.byref(first),
                                                          ctypes.byref(m)))
    return first.value, m.value


def _positions(I, m, first):
    if I is None:
        if m is None:
            raise ValueError("give the index list I or the segment length m")
        return 0, int(m), int(first)
    return _dev(I, "I", torch.int64, 1), I.numel(), 0


def sparta_snapshot(theta: torch.Tensor, I: Optional[torch.Tensor] = None, first: int = 0,
                    m: Optional[int] = None, out: Optional[torch.Tensor] = None,
                    stream=None) -> torch.Tensor:
    """snap = theta[P] with P = I, or the segment [first, first + m)."""
    pI, m, first = _positions(I, m, first)
    if out is None:
        out = torch.empty(m, dtype=torch.float32, device=theta.device)
    _same_device(theta, I, out)
    _check("ssn_sparta_snapshot", lib().ssn_sparta_snapshot(
        theta.numel(), m, pI, first, _dev(theta, "theta", torch.float32, 1),
        _dev(out, "snap", torch.float32, 1), _stream(stream)))
    return out


def sparta_average(chunks: Sequence[torch.Tensor], weights: Optional[Sequence[float]] = None,
                   acc: Optional[torch.Tensor] = None, deltas=None, stream=None):
    """acc = sum_r w_r c_r / sum_r w_r and delta_r = acc - c_r for the R
    senders' chunks (float32 [m] each).  deltas: None allocates them, False
    skips them, a list (entries may be None) receives them."""
    R = len(chunks)
    if not 1 <= R <= SPARTA_MAX_SENDERS:
        raise ValueError(f"1 <= len(chunks) <= {SPARTA_MAX_SENDERS}")
    m = chunks[0].numel()
    dev = chunks[0].device
    if acc is None:
        acc = torch.empty(m, dtype=torch.float32, device=dev)
    if deltas is None:
        deltas = [torch.empty(m, dtype=torch.float32, device=dev) for _ in range(R)]
    cs = (_c_p * R)()
    for r, c in enumerate(chunks):
        if c.numel() != m:
            raise ValueError(f"chunk {r} has {c.numel()} values, expected {m}")
        cs[r] = _dev(c, f"chunks[{r}]", torch.float32, 1)
    ds = None
    if deltas is not False:
        if len(deltas) != R:
            raise ValueError(f"{len(deltas)} delta buffers for {R} senders")
        ds = (_c_p * R)()
        for r, dl in enumerate(deltas):
            if dl is not None:
                if dl.numel() != m:
                    raise ValueError(f"delta {r} has {dl.numel()} values, expected {m}")
                ds[r] = _dev(dl, f"deltas[{r}]", torch.float32, 1)
    ws = None
    if weights is not None:
        if len(weights) != R:
            raise ValueError(f"{len(weights)} weights for {R} senders")
        ws = (ctypes.c_float * R)(*[float(w) for w in weights])
    _same_device(acc, *chunks, *([dl for dl in deltas if dl is not None] if deltas else []))
    _check("ssn_sparta_average", lib().ssn_sparta_average(
        R, m, cs, ws, _dev(acc, "acc", torch.float32, 1), ds, _stream(stream)))
    return acc, (deltas if deltas is not False else None)


def delta_rule(theta: torch.Tensor, avg: torch.Tensor, snap: Optional[torch.Tensor] = None,
               I: Optional[torch.Tensor] = None, first: int = 0, lam: float = 1.0,
               stream=None) -> torch.Tensor:
    """In place: theta[P] += lam (avg - snap), or += lam avg without snap."""
    pI, m, first = _positions(I, avg.numel() if I is None else None, first)
    if avg.numel() != m or (snap is not None and snap.numel() != m):
        raise ValueError(f"avg/snap must hold {m} values")
    _same_device(theta, avg, snap, I)
    _check("ssn_delta_rule", lib().ssn_delta_rule(
        theta.numel(), m, pI, first, _dev(theta, "theta", torch.float32, 1),
        _dev(avg, "avg", torch.float32, 1),
        0 if snap is None else _dev(snap, "snap", torch.float32, 1), float(lam), _stream(stream)))
    return theta
