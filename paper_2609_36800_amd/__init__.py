"""Python binding of the MI355X binary-delta matmul library (``libbitdelta.so``).

Argument marshalling only: every step of the operator runs in the gfx950 HIP
kernels behind the C ABI of ``include/bitdelta.h``.  PyTorch provides device
memory and the current stream.  There is no fallback: if the library is not
built, importing works but every call raises.

    pack(signs)                          -> int32 [rows, K/32] packed sign words
    unpack(packed, K, dtype)             -> [rows, K] of +1 / -1
    matmul(x, w_base, packed_s, alpha, tenant_ids=None, out_dtype=bf16) -> y

The operator (the standard and batched BitDelta GEMMs, Section 4.4 of the
paper) is  y[m, n] = sum_k x[m, k] W[n, k] + alpha[t] sum_k x[m, k] s_t[n, k],
with s = 2b - 1 decoded from the packed bits (Appendix A.2).
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libbitdelta.so")

OK = 0
F32, BF16, I8, F16 = 0, 1, 2, 3
PATH_AUTO, PATH_SKINNY, PATH_PREFILL = 0, 1, 2

EXPORTED = (
    "bitdelta_pack",
    "bitdelta_unpack",
    "bitdelta_compress",
    "bitdelta_matmul",
    "bitdelta_matmul_with_path",
    "bitdelta_matmul_typed",
    "bitdelta_matmul_noalloc",
    "bitdelta_matmul_path",
    "bitdelta_status_string",
    "bitdelta_version",
)

_lib = None


class BitDeltaError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"bitdelta status {status}: {msg}")
        self.status = status


def load_library(path: str = LIB_PATH):
    """Load ``libbitdelta.so`` (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is missing: build the HIP library first "
            "(python -c 'import __graft_entry__ as g; g.build()')")
    # The library takes its HIP runtime from whatever libamdhip64 is already
    # in the process.  torch ships its own copy: load it first, or the process
    # ends up with two runtimes (torch's, owning the tensors and streams, and
    # the system one the library would pull in) and launches on torch's
    # memory fail.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(path)
    P, I64, I32, I = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int
    lib.bitdelta_pack.argtypes = [P, I, I64, I64, P, P]
    lib.bitdelta_pack.restype = I
    lib.bitdelta_unpack.argtypes = [P, I64, I64, P, I, P]
    lib.bitdelta_unpack.restype = I
    lib.bitdelta_compress.argtypes = [P, P, I64, I64, I, P, P, P, P]
    lib.bitdelta_compress.restype = I
    lib.bitdelta_matmul.argtypes = [P, I64, I64, P, I64, P, P, P, I32, P, I, P]
    lib.bitdelta_matmul.restype = I
    lib.bitdelta_matmul_with_path.argtypes = [P, I64, I64, P, I64, P, P, P, I32, P, I, I, P]
    lib.bitdelta_matmul_with_path.restype = I
    lib.bitdelta_matmul_typed.argtypes = [P, I64, I64, P, I64, P, P, P, I32, I, P, I, I, P]
    lib.bitdelta_matmul_typed.restype = I
    lib.bitdelta_matmul_noalloc.argtypes = [P, I64, I64, P, I64, P, P, P, I32, I, P, I, I, P]
    lib.bitdelta_matmul_noalloc.restype = I
    lib.bitdelta_matmul_path.argtypes = [I64, I64, I64, I32, I]
    lib.bitdelta_matmul_path.restype = I
    lib.bitdelta_status_string.argtypes = [I]
    lib.bitdelta_status_string.restype = ctypes.c_char_p
    lib.bitdelta_version.argtypes = []
    lib.bitdelta_version.restype = I
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load_library().bitdelta_status_string(status).decode()


def _check(status: int):
    if status != OK:
        raise BitDeltaError(status, status_string(status))


def _stream(t):
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _dtype_code(dt):
    import torch
    codes = {torch.float32: F32, torch.bfloat16: BF16, torch.int8: I8, torch.float16: F16}
    if dt not in codes:
        raise TypeError(f"unsupported dtype {dt}")
    return codes[dt]


def _dev(t, name, dtypes):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _shape(t, shape, name):
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


def pack(signs, out=None):
    """Pack signs [rows, K] (float32 / bfloat16 / float16 / int8) into int32 words [rows, K/32]."""
    import torch
    if signs.dim() != 2:
        raise ValueError(f"signs must be [rows, K], got shape {tuple(signs.shape)}")
    rows, K = signs.shape
    if K % 32:
        raise ValueError(f"K = {K} is not a multiple of 32")
    if out is not None:
        _shape(out, (rows, K // 32), "out")
    _dev(signs, "signs", (torch.float32, torch.bfloat16, torch.float16, torch.int8))
    if out is None:
        out = torch.empty((rows, K // 32), dtype=torch.int32, device=signs.device)
    _dev(out, "out", (torch.int32,))
    _check(load_library().bitdelta_pack(signs.data_ptr(), _dtype_code(signs.dtype), rows, K,
                                        out.data_ptr(), _stream(signs)))
    return out


def unpack(packed, K: int, dtype=None, out=None):
    """Decode int32 words [rows, K/32] into [rows, K] of +1 / -1 (float32 by default)."""
    import torch
    dtype = dtype or torch.float32
    if packed.dim() != 2:
        raise ValueError(f"packed must be [rows, K/32], got shape {tuple(packed.shape)}")
    rows = packed.shape[0]
    if K % 32 or packed.shape[1] * 32 != K:
        raise ValueError(f"packed has {packed.shape[1]} words per row; K = {K} needs K/32")
    if out is not None:
        _shape(out, (rows, K), "out")
    _dev(packed, "packed", (torch.int32,))
    if out is None:
        out = torch.empty((rows, K), dtype=dtype, device=packed.device)
    _dev(out, "out", (torch.float32, torch.bfloat16, torch.float16, torch.int8))
    _check(load_library().bitdelta_unpack(packed.data_ptr(), rows, K, out.data_ptr(),
                                          _dtype_code(out.dtype), _stream(packed)))
    return out


def compress(w_fine, w_base, with_alpha: bool = True):
    """Binary delta of w_fine against w_base (both bf16, or both float16, [rows, K]).

    Returns (packed int32 [rows, K/32], alpha fp32 [1] or None, row_abs_sum
    fp32 [rows]): the packed signs of w_fine - w_base, their least-squares
    scale mean|w_fine - w_base|, and the per-row sums of |w_fine - w_base|.
    """
    import torch
    if w_fine.shape != w_base.shape or w_fine.dim() != 2:
        raise ValueError("w_fine and w_base must be [rows, K] of the same shape")
    rows, K = w_fine.shape
    if K % 32:
        raise ValueError(f"K = {K} is not a multiple of 32")
    _dev(w_fine, "w_fine", (torch.bfloat16, torch.float16))
    _dev(w_base, "w_base", (w_fine.dtype,))
    packed = torch.empty((rows, K // 32), dtype=torch.int32, device=w_fine.device)
    row_abs = torch.empty((rows,), dtype=torch.float32, device=w_fine.device)
    alpha = torch.empty((1,), dtype=torch.float32, device=w_fine.device) if with_alpha else None
    _check(load_library().bitdelta_compress(
        w_fine.data_ptr(), w_base.data_ptr(), rows, K, _dtype_code(w_fine.dtype), packed.data_ptr(),
        row_abs.data_ptr(),
        None if alpha is None else alpha.data_ptr(), _stream(w_fine)))
    return packed, alpha, row_abs


def matmul(x, w_base, packed_s, alpha, tenant_ids=None, out_dtype=None, out=None,
           path: int = PATH_AUTO):
    """y = x W^T + alpha_t x S_t^T.

    x [M, K] and w_base [N, K] both bfloat16 or both float16, packed_s int32
    [T, N, K/32] (or [N, K/32]), alpha fp32 [T], tenant_ids int32 [M] or None,
    out_dtype float32 or the input type (the default); out, if given, [M, N].
    Every shape is checked before anything reaches the library, which sees
    only raw pointers.
    """
    import torch
    if x.dim() != 2 or w_base.dim() != 2 or alpha.dim() != 1 or packed_s.dim() not in (2, 3):
        raise ValueError("x and w_base must be 2-D, alpha 1-D, packed_s 2-D or 3-D")
    M, K = x.shape
    N = w_base.shape[0]
    T = alpha.numel()
    if packed_s.dim() == 2:
        packed_s = packed_s.unsqueeze(0)
    if K % 32 or tuple(packed_s.shape) != (T, N, K // 32) or w_base.shape[1] != K:
        raise ValueError(f"shape mismatch: x {tuple(x.shape)}, w {tuple(w_base.shape)}, "
                         f"packed {tuple(packed_s.shape)}, alpha {T}")
    if tenant_ids is not None and (tenant_ids.dim() != 1 or tenant_ids.numel() != M):
        raise ValueError("tenant_ids needs one entry per row")
    if out is not None:
        _shape(out, (M, N), "out")
    _dev(x, "x", (torch.bfloat16, torch.float16))
    _dev(w_base, "w_base", (x.dtype,))
    out_dtype = out_dtype or x.dtype
    _dev(packed_s, "packed_s", (torch.int32,))
    _dev(alpha, "alpha", (torch.float32,))
    tptr = None
    if tenant_ids is not None:
        _dev(tenant_ids, "tenant_ids", (torch.int32,))
        tptr = tenant_ids.data_ptr()
    if out is None:
        out = torch.empty((M, N), dtype=out_dtype, device=x.device)
    _dev(out, "out", (torch.float32, x.dtype))
    _check(load_library().bitdelta_matmul_typed(
        x.data_ptr(), M, K, w_base.data_ptr(), N, packed_s.data_ptr(), alpha.data_ptr(),
        tptr, T, _dtype_code(x.dtype), out.data_ptr(), _dtype_code(out.dtype), path, _stream(x)))
    return out


def matmul_path(M: int, N: int, K: int, T: int, multi_tenant: bool) -> int:
    return load_library().bitdelta_matmul_path(M, N, K, T, int(bool(multi_tenant)))
