"""Reference oracle for the binary-delta matmul -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library
(``paper_2609_36800_amd``) never imports it, and the two share no source: the
oracle is plain C (``oracle.c``, fp64, plain loops) plus an exact-rational
brute force (``brute.py``).

What it computes follows the definition of the BitDelta GEMM evaluated in the
paper (Section 4.4 standard and batched variants; the ``2b-1`` sign decode of
Appendix A.2, "BitDelta" paragraph):

    y[m, n] = sum_k x[m, k] W[n, k] + alpha[t(m)] * sum_k x[m, k] s_t(m)[n, k]

It also holds the compression of a fine-tuned weight into that form
(``compress``: the signs of W_fine - W_base and their least-squares scale).

Every function here is pinned by ``tests/test_oracle.py`` against facts that do
not come from the oracle itself (library packers, exact brute force, closed
forms, algebraic identities).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile ``oracle.c`` into ``liboracle.so`` with gcc + OpenMP.

    Generic x86-64 code (no ``-march=native``) so the library built here also
    runs on a host with a different CPU.
    """
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        cmd = ["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11",
               "-Wall", "-Wextra", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build(force=False)
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    I64 = ctypes.c_int64
    lib.oracle_num_threads.restype = ctypes.c_int
    for name in ("oracle_pack_f32", "oracle_pack_bf16", "oracle_pack_i8"):
        f = getattr(lib, name)
        f.argtypes = [P, I64, I64, P]
        f.restype = ctypes.c_int
    lib.oracle_unpack_f64.argtypes = [P, I64, I64, P]
    lib.oracle_unpack_f64.restype = ctypes.c_int
    lib.oracle_compress.argtypes = [P, P, I64, I64, ctypes.c_int, P, P, P]
    lib.oracle_compress.restype = ctypes.c_int
    lib.oracle_matmul_parts.argtypes = [P, I64, I64, P, I64, P, P, P, ctypes.c_int32,
                                        P, I64, ctypes.c_int, P, P, P]
    lib.oracle_matmul_parts.restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def num_threads() -> int:
    """OpenMP threads the oracle's parallel loop uses."""
    return int(_load().oracle_num_threads())


def pack(signs: np.ndarray) -> np.ndarray:
    """Pack a [rows, K] float32 / bfloat16-bits (uint16) / int8 array of signs.

    Bit i of word j of a row is set exactly when element 32*j+i has a clear
    sign bit.  Returns uint32 [rows, K/32].
    """
    lib = _load()
    signs = np.ascontiguousarray(signs)
    rows, K = signs.shape
    if K % 32:
        raise ValueError("K must be a multiple of 32")
    out = np.zeros((rows, K // 32), dtype=np.uint32)
    fn = {np.dtype(np.float32): lib.oracle_pack_f32,
          np.dtype(np.uint16): lib.oracle_pack_bf16,
          np.dtype(np.int8): lib.oracle_pack_i8}.get(signs.dtype)
    if fn is None:
        raise TypeError(f"unsupported sign dtype {signs.dtype}")
    rc = fn(_ptr(signs), rows, K, _ptr(out))
    if rc != 0:
        raise RuntimeError(f"oracle pack failed ({rc})")
    return out


def unpack(packed: np.ndarray, K: int) -> np.ndarray:
    """Decode uint32 [rows, K/32] into float64 [rows, K] of +1 / -1 (s = 2b - 1)."""
    lib = _load()
    packed = np.ascontiguousarray(packed, dtype=np.uint32)
    rows = packed.shape[0]
    if packed.shape[1] * 32 != K:
        raise ValueError("packed shape does not match K")
    out = np.empty((rows, K), dtype=np.float64)
    rc = lib.oracle_unpack_f64(_ptr(packed), rows, K, _ptr(out))
    if rc != 0:
        raise RuntimeError(f"oracle unpack failed ({rc})")
    return out


_DT = {"bf16": 1, "f16": 3}


def compress(fine_bits, base_bits, dtype: str = "bf16"):
    """Binary delta of a fine-tuned weight against its base, in fp64.

    fine_bits, base_bits  uint16 [rows, K] (bf16 or fp16 bit patterns, per dtype)
    Returns (packed uint32 [rows, K/32], row_abs float64 [rows], alpha float):
    the packed signs of delta = fine - base (bit set when delta's sign bit is
    clear), sum_k |delta| per row, and alpha = mean |delta|, the scale that
    minimises ||delta - alpha * s||_F for those signs.
    """
    lib = _load()
    fine_bits = np.ascontiguousarray(fine_bits, dtype=np.uint16)
    base_bits = np.ascontiguousarray(base_bits, dtype=np.uint16)
    if fine_bits.shape != base_bits.shape or fine_bits.ndim != 2:
        raise ValueError("fine and base must be [rows, K] of the same shape")
    rows, K = fine_bits.shape
    if K % 32:
        raise ValueError("K must be a multiple of 32")
    packed = np.zeros((rows, K // 32), dtype=np.uint32)
    row_abs = np.zeros(rows, dtype=np.float64)
    alpha = np.zeros(1, dtype=np.float64)
    rc = lib.oracle_compress(_ptr(fine_bits), _ptr(base_bits), rows, K, _DT[dtype], _ptr(packed),
                             _ptr(row_abs), _ptr(alpha))
    if rc != 0:
        raise RuntimeError(f"oracle compress failed ({rc})")
    return packed, row_abs, float(alpha[0])


def matmul_parts(x_bits, w_bits, packed, alpha, tenant_ids=None, n_idx=None, dtype="bf16"):
    """fp64 evaluation of the binary-delta matmul.

    x_bits  uint16 [M, K] (bf16 or fp16 bit patterns, per dtype)
    w_bits  uint16 [N, K] (same type)
    packed  uint32 [T, N, K/32] (or [N, K/32] for one tenant)
    alpha   float32 [T]
    tenant_ids  int32 [M] or None (all rows use tenant 0)
    n_idx   int64 list of output features to evaluate, or None for all N

    Returns (base, delta, y), each float64 [M, len(n_idx) or N], where
    base = x W^T, delta = x S_t^T (before alpha) and y = base + alpha_t * delta.
    Rows whose tenant id is outside [0, T) are NaN.
    """
    lib = _load()
    x_bits = np.ascontiguousarray(x_bits, dtype=np.uint16)
    w_bits = np.ascontiguousarray(w_bits, dtype=np.uint16)
    packed = np.ascontiguousarray(packed, dtype=np.uint32)
    if packed.ndim == 2:
        packed = packed[None]
    alpha = np.ascontiguousarray(np.atleast_1d(alpha), dtype=np.float32)
    M, K = x_bits.shape
    N = w_bits.shape[0]
    T = packed.shape[0]
    if w_bits.shape[1] != K or packed.shape[1] != N or packed.shape[2] * 32 != K:
        raise ValueError("inconsistent shapes")
    if alpha.shape[0] != T:
        raise ValueError("alpha must have one entry per tenant")
    tid = None
    if tenant_ids is not None:
        tid = np.ascontiguousarray(tenant_ids, dtype=np.int32)
        if tid.shape != (M,):
            raise ValueError("tenant_ids must have one entry per row")
    idx = None
    cnt = N
    if n_idx is not None:
        idx = np.ascontiguousarray(n_idx, dtype=np.int64)
        cnt = idx.shape[0]
    base = np.empty((M, cnt), dtype=np.float64)
    delta = np.empty((M, cnt), dtype=np.float64)
    y = np.empty((M, cnt), dtype=np.float64)
    rc = lib.oracle_matmul_parts(_ptr(x_bits), M, K, _ptr(w_bits), N, _ptr(packed),
                                 _ptr(alpha), _ptr(tid), T, _ptr(idx), cnt, _DT[dtype],
                                 _ptr(base), _ptr(delta), _ptr(y))
    if rc != 0:
        raise RuntimeError(f"oracle matmul failed ({rc})")
    return base, delta, y


def matmul(x_bits, w_bits, packed, alpha, tenant_ids=None, n_idx=None, dtype="bf16"):
    """y = x W^T + alpha_t x S_t^T in fp64 (see ``matmul_parts``)."""
    return matmul_parts(x_bits, w_bits, packed, alpha, tenant_ids, n_idx, dtype)[2]
