"""Helpers for the GPU tests: host arrays <-> device tensors, and one call of the
HIP path through the C ABI (via the thin binding)."""
from __future__ import annotations

import sys

import numpy as np


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def torch():
    import torch as _t
    return _t


def dev_bf16(bits: np.ndarray):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(t.bfloat16).cuda()


def dev_half(bits: np.ndarray, dtype: str):
    """bf16 or fp16 bit patterns -> device tensor of that type."""
    t = torch()
    tt = t.float16 if dtype == "f16" else t.bfloat16
    return t.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(tt).cuda()


def dev_words(words: np.ndarray):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(words).view(np.int32)).cuda()


def dev_f32(a: np.ndarray):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def dev_i32(a: np.ndarray):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()


def host_words(t_words) -> np.ndarray:
    return t_words.cpu().numpy().view(np.uint32)


def host_out(y) -> np.ndarray:
    """Device output (fp32, bf16 or fp16) -> float64 host array."""
    t = torch()
    if y.dtype == t.bfloat16:
        bits = y.view(t.int16).cpu().numpy().view(np.uint16)
        return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    if y.dtype == t.float16:
        return y.view(t.int16).cpu().numpy().view(np.float16).astype(np.float64)
    return y.cpu().numpy().astype(np.float64)


def run_matmul(p, packed=None, path=0, y_dtype=None):
    """Run the HIP path on Problem p (packed words override p.packed)."""
    import paper_2609_36800_amd as bd
    t = torch()
    packed = p.packed if packed is None else packed
    yd = y_dtype or p.y_dtype
    dt = getattr(p, "dtype", "bf16")
    out_dtype = t.float32 if yd == "f32" else (t.float16 if dt == "f16" else t.bfloat16)
    tid = None if p.tenant_ids is None else dev_i32(p.tenant_ids)
    y = bd.matmul(dev_half(p.x, dt), dev_half(p.w, dt), dev_words(packed), dev_f32(p.alpha),
                  tenant_ids=tid, out_dtype=out_dtype, path=path)
    t.cuda.synchronize()
    return y
